"""Seeded synthetic decode workloads (inputs only -- none of the method's arithmetic).

The paper measures its kernels on synthetic one-token decode inputs (Sec. 5.1,
Table 3: H/dk/dv = 32/128/128, bf16 activations, fp32 state); no dataset is
involved.  This module generates such inputs, reproducibly, for the workloads the
library is tested and benchmarked on.  It is the only code shared by the HIP path's
tests/bench and the CPU oracle's tests: it draws random numbers and rounds them to the
storage dtype, nothing else.

Recipe:

* Seeds: ``numpy.random.default_rng([20261202, cfg, layer, stream, idx])`` with
  stream 0 = initial state (idx = slot), 1 = step inputs (idx = step t; warm-up steps
  use 10_000 + w), 2 = RWKV6 bonus u, 3 = staggered log-fill offsets.
* Per step the draws are, in this order, full ``[B, H, ...]`` float64 standard
  normals for q (r for RWKV6), k, v, the gate and beta, then transformed:
  - GDN: q, k L2-normalised over dk; v ~ N(0,1); alpha = sigmoid(3 + 0.5 z) per head,
    stored as lambda = log(alpha); beta = sigmoid(z) per head.
  - KDA: as GDN but lambda = -softplus(z)/16 per key (so alpha = exp(lambda)).
  - RWKV6: r, k, v ~ N(0,1) unnormalised; lambda = log(w) = -exp(-0.5 + 0.5 z) per key;
    no beta; bonus u ~ N(0, 0.1) of shape [H, dk], drawn once.
  - Linear attention: q, k = phi(z) / |phi(z)| with the positive feature map
    phi = elu + 1; v ~ N(0,1); no gate (no decay) and no beta are drawn.
  - RetNet: q, k L2-normalised; v ~ N(0,1); the decay is the fixed per-head
    gamma_h = 1 - 2^(-5 - 5h/H) (lambda = log gamma_h, the same every step); no gate
    or beta drawn.
  - GLA: q, k L2-normalised; v ~ N(0,1); lambda = log sigmoid(z) / 16 per key; no beta.
  - Initial state S0 ~ N(0, 0.02) (standard deviation) for every workload.
* Rounding: float64 draw -> float32 (round to nearest even) -> bf16 (round to nearest
  even) for bf16 activations.  Gates (lambda) and beta stay float32.  Arrays are returned
  as float32 whose values are exactly representable in the storage dtype, so both sides
  read identical numbers.
"""

from dataclasses import dataclass, replace

import numpy as np

ROOT_SEED = 20261202
PER_KEY_OPS = ("kda", "rwkv6", "gla")
DELTA_OPS = ("gdn", "kda")
WARMUP_IDX0 = 10_000


@dataclass(frozen=True)
class Workload:
    name: str
    cfg: int            # seed component identifying the workload
    op: str             # "gdn" | "kda" | "rwkv6" | "linattn" | "retnet" | "gla"
    B: int              # sequences (state slots)
    H: int              # heads
    dk: int
    dv: int
    M: int              # merge interval (live-log capacity C = M - 1)
    steps: int          # decode steps of one rollout
    in_dtype: str = "bf16"   # activations q/r, k, v: "bf16" or "f32"
    layers: int = 1     # independent recurrent layers (the serving stack)
    staggered: bool = False  # per-slot log-fill offsets uniform in {0..M-1}

    @property
    def heads_total(self):
        return self.B * self.H

    @property
    def dl(self):
        """Width of the log-decay metadata: 1 (head-wise scalar, or none) or dk (per key)."""
        return self.dk if self.op in PER_KEY_OPS else 1

    def with_(self, **kw):
        return replace(self, **kw)


# The five workloads (Table 3 shapes, reshaped per operator).
GDN_SMALL = Workload("gdn_b1_h2_d64_m8", 1, "gdn", 1, 2, 64, 64, 8, 64, in_dtype="f32")
GDN_B64 = Workload("gdn_b64_h32_d128_m16", 2, "gdn", 64, 32, 128, 128, 16, 256)
KDA_B128 = Workload("kda_b128_h32_d128_m16", 3, "kda", 128, 32, 128, 128, 16, 256)
RWKV6_B128 = Workload("rwkv6_b128_h40_d64_m16", 4, "rwkv6", 128, 40, 64, 64, 16, 256)
GDN_STACK = Workload("gdn_stack24_b256_h32_d128_m16", 5, "gdn", 256, 32, 128, 128, 16, 128,
                     layers=24, staggered=True)

# The other operators of Table 1, at the GDN / KDA shapes (scalar / per-key decay).
LINATTN_B64 = Workload("linattn_b64_h32_d128_m16", 6, "linattn", 64, 32, 128, 128, 16, 256)
RETNET_B64 = Workload("retnet_b64_h32_d128_m16", 7, "retnet", 64, 32, 128, 128, 16, 256)
GLA_B128 = Workload("gla_b128_h32_d128_m16", 8, "gla", 128, 32, 128, 128, 16, 256)

WORKLOADS = {w.name: w for w in (GDN_SMALL, GDN_B64, KDA_B128, RWKV6_B128, GDN_STACK,
                                 LINATTN_B64, RETNET_B64, GLA_B128)}


def kda_with_merge_interval(M):
    """The KDA workload at merge interval M (swept over {8, 16, 32})."""
    return KDA_B128.with_(name=f"kda_b128_h32_d128_m{M}", M=M)


def _rng(w, layer, stream, idx):
    return np.random.default_rng([ROOT_SEED, w.cfg, layer, stream, idx])


def round_bf16(x):
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def _store(x64, dtype):
    x32 = np.asarray(x64, dtype=np.float32)
    if dtype == "bf16":
        return round_bf16(x32)
    if dtype == "f32":
        return x32
    raise ValueError(dtype)


def _l2norm(x):
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def _softplus(z):
    return np.logaddexp(0.0, z)


def initial_state(w, layer=0, slots=None):
    """S0 [len(slots), H, dk, dv] float32, drawn per slot (stream 0, idx = slot)."""
    slots = range(w.B) if slots is None else slots
    out = np.empty((len(slots), w.H, w.dk, w.dv), dtype=np.float32)
    for n, b in enumerate(slots):
        out[n] = _rng(w, layer, 0, int(b)).normal(0.0, 0.02, size=(w.H, w.dk, w.dv))
    return out


def _elu1(x):
    return np.where(x > 0, x + 1.0, np.exp(np.minimum(x, 0.0)))


def retnet_log_decay(H):
    """RetNet's fixed multi-scale decays, one per head: gamma_h = 1 - 2^(-5 - 5h/H)."""
    return np.log1p(-(2.0 ** (-5.0 - 5.0 * np.arange(H) / H)))


def step_inputs(w, t, layer=0, warmup=None):
    """Token inputs for decode step ``t`` (or warm-up step ``warmup``) of all B slots.

    Returns a dict of float32 arrays: q [B,H,dk] (r for RWKV6), k [B,H,dk], v [B,H,dv],
    lam [B,H] (GDN, RetNet) or [B,H,dk] (KDA, RWKV6, GLA) or None (linear attention),
    beta [B,H] (delta rule only, else None).
    """
    idx = t if warmup is None else WARMUP_IDX0 + warmup
    g = _rng(w, layer, 1, idx)
    B, H, dk, dv = w.B, w.H, w.dk, w.dv
    q = g.standard_normal((B, H, dk))
    k = g.standard_normal((B, H, dk))
    v = g.standard_normal((B, H, dv))
    beta = None
    if w.op in ("gdn", "kda", "rwkv6", "gla"):
        gate = g.standard_normal((B, H) if w.op == "gdn" else (B, H, dk))
    if w.op == "gdn":
        q, k = _l2norm(q), _l2norm(k)
        lam = np.log(_sigmoid(3.0 + 0.5 * gate))
        beta = _sigmoid(g.standard_normal((B, H)))
    elif w.op == "kda":
        q, k = _l2norm(q), _l2norm(k)
        lam = -_softplus(gate) / 16.0
        beta = _sigmoid(g.standard_normal((B, H)))
    elif w.op == "rwkv6":
        lam = -np.exp(-0.5 + 0.5 * gate)
    elif w.op == "linattn":
        q, k = _l2norm(_elu1(q)), _l2norm(_elu1(k))     # positive feature map phi
        lam = None
    elif w.op == "retnet":
        q, k = _l2norm(q), _l2norm(k)
        lam = np.broadcast_to(retnet_log_decay(H), (B, H))
    elif w.op == "gla":
        q, k = _l2norm(q), _l2norm(k)
        lam = -_softplus(-gate) / 16.0                  # log sigmoid(gate) / 16
    else:
        raise ValueError(w.op)
    return {
        "q": _store(q, w.in_dtype),
        "k": _store(k, w.in_dtype),
        "v": _store(v, w.in_dtype),
        "lam": None if lam is None else np.ascontiguousarray(lam, dtype=np.float32),
        "beta": None if beta is None else beta.astype(np.float32),
    }


def bonus(w, layer=0):
    """RWKV6 per-head bonus u [H, dk] float32 (stream 2); None for other operators."""
    if w.op != "rwkv6":
        return None
    return _rng(w, layer, 2, 0).normal(0.0, 0.1, size=(w.H, w.dk)).astype(np.float32)


def fill_offsets(w):
    """Per-slot log-fill offsets o_b uniform in {0..M-1} (stream 3); zeros if unstaggered."""
    if not w.staggered:
        return np.zeros(w.B, dtype=np.int64)
    return _rng(w, 0, 3, 0).integers(0, w.M, size=w.B)


def warmup_schedule(w):
    """Warm-up rounds that bring slot b to live length o_b before step 0.

    Round ``r`` (0 <= r < M-1) steps the slots with o_b >= M-1-r, so slot b takes
    exactly o_b warm-up steps (all appends) and all slots align at step 0.
    Returns a list of (round, slot index array) pairs, skipping empty rounds.
    """
    off = fill_offsets(w)
    sched = []
    for r in range(w.M - 1):
        sl = np.nonzero(off >= w.M - 1 - r)[0]
        if sl.size:
            sched.append((r, sl))
    return sched


def select_rows(inputs, rows):
    """The token rows ``rows`` of a step-input dict (a partial decode batch)."""
    return {k: (None if a is None else np.ascontiguousarray(a[rows])) for k, a in inputs.items()}
