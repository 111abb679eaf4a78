"""fp64 CPU oracle for DeltaLog one-token decoding -- TEST INFRASTRUCTURE ONLY.

This package is the plain, slow, obviously correct reference that the HIP path is
checked against.  It is imported only by ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py``; the product path (``paper_2608_15533_amd``)
never imports, links or calls it, and it never imports the product path.

Contents
--------
``eager``          the dense eager recurrence (Eq. 3 with the Table 1 instantiations for
                   GDN, KDA, RWKV6, linear attention, RetNet and GLA) in float64 -- the
                   *definition* the GPU must match.
``deltalog_model`` the paper's base-plus-log state machine (Alg. 1, append Eq. 5,
                   merge Eq. 6, invariant Eq. 7) in float64, used to check log contents
                   and the equivalence argument of Sec. 3.2 ("Closure under the recurrence").

All arithmetic is float64; inputs are upcast from the exact bytes the GPU consumes.
Every public function is exercised by ``tests/test_oracle_pins.py`` against something
other than itself (closed forms, special cases, 2x2 brute force in exact rationals,
invariants, a plain GEMM), and ``tests/test_oracle_mutants.py`` shows that a planted
mistake in any term fails one of those pins.  The pinned functions are: ``eager.row_decay``,
``eager.gdn_kda_step``, ``eager.rwkv6_step``, ``eager.additive_step``, ``eager.eager_step``,
``eager.rel_fro`` and every method of ``deltalog_model.DeltaLogModel``.
"""

from . import eager, deltalog_model  # noqa: F401

__all__ = ["eager", "deltalog_model"]
