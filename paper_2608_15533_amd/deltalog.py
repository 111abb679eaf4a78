"""ctypes binding of libdeltalog.so -- argument marshalling only.

The entry points keep the C names (``dl_eager_step``, ``dl_append_step``, ``dl_merge``,
``dl_readout``) and take torch CUDA tensors; each call checks layouts, builds the C
structs and calls the library, which launches the HIP kernels on the current (or the
given) stream.  No arithmetic of the method happens here.  PyTorch is used only to
own device memory and to name the stream.

Importing this module loads the library and raises ImportError when it has not been
built -- there is no fallback path.
"""

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# DELTALOG_LIB selects another build of the same library (e.g. a tuning variant).
LIB_PATH = os.environ.get("DELTALOG_LIB") or os.path.join(_HERE, "libdeltalog.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build it with `python -m paper_2608_15533_amd.build` "
        "(the DeltaLog path has no non-HIP fallback)")

_lib = ctypes.CDLL(LIB_PATH)

# ----------------------------------------------------------------- constants (deltalog.h)
DL_ABI_VERSION = 4
DL_MAX_MERGE_INTERVAL = 64
DL_OK, DL_E_NULL, DL_E_SHAPE, DL_E_DTYPE, DL_E_ALIGN, DL_E_UNSUPPORTED, DL_E_HIP, DL_E_VERSION = (
    0, -1, -2, -3, -4, -5, -6, -7)
DL_E_SCRATCH = -8
DL_NOALLOC_SCRATCH_BYTES = 4 << 20
DL_OP_GDN, DL_OP_KDA, DL_OP_RWKV6, DL_OP_LINATTN, DL_OP_RETNET, DL_OP_GLA = 0, 1, 2, 3, 4, 5
DL_F32, DL_BF16 = 0, 1
OP_IDS = {"gdn": DL_OP_GDN, "kda": DL_OP_KDA, "rwkv6": DL_OP_RWKV6, "linattn": DL_OP_LINATTN,
          "retnet": DL_OP_RETNET, "gla": DL_OP_GLA}
DELTA_OP_IDS = (DL_OP_GDN, DL_OP_KDA)                  # b = beta (v - correction); needs beta
PER_KEY_OP_IDS = (DL_OP_KDA, DL_OP_RWKV6, DL_OP_GLA)   # lambda is [.., dk]; else one per head
DTYPE_IDS = {"f32": DL_F32, "bf16": DL_BF16}
TORCH_DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16}

EXPORTED = ("dl_eager_step", "dl_append_step", "dl_merge", "dl_readout",
            "dl_append_step_tiled", "dl_tiled_workspace_bytes", "dl_status_str",
            "dl_abi_version", "dl_build_flags", "dl_append_step_tiled_noalloc")


class dl_desc(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_int32), ("op", ctypes.c_int32),
                ("num_slots", ctypes.c_int32), ("heads", ctypes.c_int32),
                ("dk", ctypes.c_int32), ("dv", ctypes.c_int32),
                ("merge_interval", ctypes.c_int32), ("in_dtype", ctypes.c_int32),
                ("u_log_dtype", ctypes.c_int32), ("state_dtype", ctypes.c_int32)]


class dl_state(ctypes.Structure):
    _fields_ = [("S", ctypes.c_void_p), ("k_log", ctypes.c_void_p),
                ("u_log", ctypes.c_void_p), ("lam_log", ctypes.c_void_p),
                ("len", ctypes.c_void_p), ("err", ctypes.c_void_p)]


class dl_token(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("beta", ctypes.c_void_p), ("lam", ctypes.c_void_p), ("u", ctypes.c_void_p)]


_P = ctypes.c_void_p
_lib.dl_eager_step.argtypes = [ctypes.POINTER(dl_desc), _P, ctypes.POINTER(dl_token), _P, _P,
                               ctypes.c_int32, _P]
_lib.dl_append_step.argtypes = [ctypes.POINTER(dl_desc), ctypes.POINTER(dl_state),
                                ctypes.POINTER(dl_token), _P, _P, ctypes.c_int32, _P]
_lib.dl_merge.argtypes = [ctypes.POINTER(dl_desc), ctypes.POINTER(dl_state),
                          ctypes.POINTER(dl_token), _P, _P, ctypes.c_int32, _P]
_lib.dl_readout.argtypes = [ctypes.POINTER(dl_desc), ctypes.POINTER(dl_state), _P, _P, _P,
                            ctypes.c_int32, _P]
_lib.dl_append_step_tiled.argtypes = [ctypes.POINTER(dl_desc), ctypes.POINTER(dl_state),
                                      ctypes.POINTER(dl_token), _P, _P, ctypes.c_int32,
                                      ctypes.c_int32, ctypes.c_int32, _P, ctypes.c_size_t, _P]
_lib.dl_tiled_workspace_bytes.argtypes = [ctypes.POINTER(dl_desc), ctypes.c_int32,
                                          ctypes.POINTER(ctypes.c_size_t)]
_lib.dl_append_step_tiled_noalloc.argtypes = [ctypes.POINTER(dl_desc), ctypes.POINTER(dl_state),
                                              ctypes.POINTER(dl_token), _P, _P, ctypes.c_int32,
                                              ctypes.c_int32, _P]
for _f in ("dl_eager_step", "dl_append_step", "dl_merge", "dl_readout", "dl_append_step_tiled",
           "dl_tiled_workspace_bytes", "dl_abi_version", "dl_append_step_tiled_noalloc"):
    getattr(_lib, _f).restype = ctypes.c_int
_lib.dl_status_str.argtypes = [ctypes.c_int]
_lib.dl_status_str.restype = ctypes.c_char_p
_lib.dl_build_flags.argtypes = []
_lib.dl_build_flags.restype = ctypes.c_char_p

lib = _lib


class DeltaLogError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {dl_status_str(status)} ({status})")


def dl_status_str(status):
    return _lib.dl_status_str(int(status)).decode()


def dl_abi_version():
    return _lib.dl_abi_version()


def dl_build_flags():
    return _lib.dl_build_flags().decode()


if dl_abi_version() != DL_ABI_VERSION:
    raise ImportError(f"libdeltalog ABI {dl_abi_version()} != binding ABI {DL_ABI_VERSION}")


# ----------------------------------------------------------------- descriptors
def make_desc(op, B, H, dk, dv, M, in_dtype="bf16", state_dtype="f32"):
    """dl_desc for operator ``op`` (a key of ``OP_IDS``) with merge interval M."""
    u_dtype = "f32" if OP_IDS[op] in DELTA_OP_IDS else in_dtype
    return dl_desc(DL_ABI_VERSION, OP_IDS[op], B, H, dk, dv, M, DTYPE_IDS[in_dtype],
                   DTYPE_IDS[u_dtype], DTYPE_IDS[state_dtype])


def state_torch_dtype(desc):
    return torch.bfloat16 if desc.state_dtype == DL_BF16 else torch.float32


def decay_width(desc):
    """Width of lambda, ell and the Lam_log snapshots: dk (per-key decay) or 1 (one value
    per head); 0 for linear attention, which has no decay."""
    if desc.op == DL_OP_LINATTN:
        return 0
    return desc.dk if desc.op in PER_KEY_OP_IDS else 1


def _ptr(t):
    return None if t is None else t.data_ptr()


def _need(t, name, dtype, shape, device=None):
    if t is None:
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


class DeltaLogState:
    """Device buffers of the physical state (Sec. 3.1), allocated with torch.

    S [B,H,dk,dv] state dtype, k_log [B,H,C,dk] in_dtype, u_log [B,H,C,dv], lam_log
    [B,H,C,dl] f32 ([B,C,H] for one log-decay per head), len [B,H] int32, err [1] int32.
    ``S`` starts as a copy of ``S0`` (the prefill state, converted to the state dtype);
    the log starts empty (Sec. 4 slot lifecycle).  The cumulative log-decay of Sec. 3.1
    is not a buffer: it is the newest snapshot (0 with an empty log), which the kernels
    read.  Linear attention has no decay, so ``lam_log`` is None (NULL to the library).
    """

    def __init__(self, desc, S0=None, device="cuda"):
        self.desc = desc
        B, H, dk, dv, M = desc.num_slots, desc.heads, desc.dk, desc.dv, desc.merge_interval
        C = M - 1
        dl = decay_width(desc)
        in_t = torch.bfloat16 if desc.in_dtype == DL_BF16 else torch.float32
        u_t = torch.bfloat16 if desc.u_log_dtype == DL_BF16 else torch.float32
        f32 = dict(dtype=torch.float32, device=device)
        st = state_torch_dtype(desc)
        self.S = (torch.zeros((B, H, dk, dv), dtype=st, device=device) if S0 is None else
                  S0.to(device=device, dtype=st).contiguous().clone())
        self.k_log = torch.zeros((B, H, max(C, 0), dk), dtype=in_t, device=device)
        self.u_log = torch.zeros((B, H, max(C, 0), dv), dtype=u_t, device=device)
        # scalar snapshots are entry-major [B, C, H] (the heads of a slot side by side)
        if dl == 1:
            self.lam_log = torch.zeros((B, max(C, 0), H), **f32)
        else:
            self.lam_log = torch.zeros((B, H, max(C, 0), dl), **f32) if dl else None
        self.len = torch.zeros((B, H), dtype=torch.int32, device=device)
        self.err = torch.zeros((1,), dtype=torch.int32, device=device)
        self.struct = dl_state(_ptr(self.S),
                               _ptr(self.k_log) if C > 0 else None,
                               _ptr(self.u_log) if C > 0 else None,
                               _ptr(self.lam_log) if C > 0 and dl else None,
                               _ptr(self.len), _ptr(self.err))

    def buffers(self):
        return dict(S=self.S, k_log=self.k_log, u_log=self.u_log,
                    lam_log=self.lam_log, len=self.len, err=self.err)


class Token:
    """Device tensors of one decode step's inputs plus the dl_token struct over them."""

    def __init__(self, desc, n, q, k, v, lam, beta=None, u=None):
        H, dk, dv = desc.heads, desc.dk, desc.dv
        dl = decay_width(desc)
        it = torch.bfloat16 if desc.in_dtype == DL_BF16 else torch.float32
        _need(q, "q", it, (n, H, dk))
        _need(k, "k", it, (n, H, dk))
        _need(v, "v", it, (n, H, dv))
        if dl:
            _need(lam, "lam", torch.float32, (n, H) if dl == 1 else (n, H, dl))
        else:
            lam = None                       # linear attention: no decay input
        if desc.op == DL_OP_RWKV6:
            _need(u, "u", torch.float32, (H, dk))
        else:
            u = None
        if desc.op in DELTA_OP_IDS:
            _need(beta, "beta", torch.float32, (n, H))
        else:
            beta = None
        self.n = n
        self.tensors = (q, k, v, lam, beta, u)
        self.struct = dl_token(_ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(lam), _ptr(u))


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _rows(desc, slots, n):
    """(device slot-list pointer or None, rows n of the launch).  Token row i drives slot
    slots[i] for i < n, so a token given with the call must hold at least n rows (extra
    rows are not read); without a slot list n is the token's row count or B."""
    rows = (desc.num_slots if n is None else n) if slots is None else slots.numel()
    if n is not None and n < rows:
        raise ValueError(f"the token holds {n} rows but the launch drives {rows}")
    if slots is None:
        return None, rows
    _need(slots, "slots", torch.int32, (rows,))
    return slots.data_ptr(), rows


def _check(rc, where):
    if rc != DL_OK:
        raise DeltaLogError(rc, where)


# ----------------------------------------------------------------- entry points
def dl_eager_step(desc, S, tok, o, slots=None, stream=None):
    """Eager dense step (Eq. 3) on S [B,H,dk,dv]; writes o [n,H,dv] f32."""
    sp, n = _rows(desc, slots, tok.n)
    _need(o, "o", torch.float32, (n, desc.heads, desc.dv))
    _need(S, "S", state_torch_dtype(desc), (desc.num_slots, desc.heads, desc.dk, desc.dv))
    _check(_lib.dl_eager_step(ctypes.byref(desc), _ptr(S), ctypes.byref(tok.struct), _ptr(o),
                              sp, n, _stream(stream)), "dl_eager_step")


def dl_append_step(desc, state, tok, o, slots=None, stream=None):
    """One DeltaLog step (Alg. 1): append if L < C else merge; writes o [n,H,dv] f32."""
    sp, n = _rows(desc, slots, tok.n)
    _need(o, "o", torch.float32, (n, desc.heads, desc.dv))
    _check(_lib.dl_append_step(ctypes.byref(desc), ctypes.byref(state.struct),
                               ctypes.byref(tok.struct), _ptr(o), sp, n, _stream(stream)),
           "dl_append_step")


def dl_merge(desc, state, tok=None, o=None, slots=None, stream=None):
    """Merge at the current L with the token (writes o), or flush when tok is None."""
    sp, n = _rows(desc, slots, None if tok is None else tok.n)
    if tok is not None:
        _need(o, "o", torch.float32, (n, desc.heads, desc.dv))
    _check(_lib.dl_merge(ctypes.byref(desc), ctypes.byref(state.struct),
                         None if tok is None else ctypes.byref(tok.struct),
                         _ptr(o) if tok is not None else None, sp, n, _stream(stream)),
           "dl_merge")


def dl_readout(desc, state, q, o, slots=None, stream=None):
    """o = q^T S_logical (Eq. 7) for q [n,H,dk]; mutates nothing."""
    n = q.shape[0]
    sp, n = _rows(desc, slots, n)
    it = torch.bfloat16 if desc.in_dtype == DL_BF16 else torch.float32
    _need(q, "q", it, (n, desc.heads, desc.dk))
    _need(o, "o", torch.float32, (n, desc.heads, desc.dv))
    _check(_lib.dl_readout(ctypes.byref(desc), ctypes.byref(state.struct), _ptr(q), _ptr(o),
                           sp, n, _stream(stream)), "dl_readout")


def dl_tiled_workspace_bytes(desc, n):
    """Bytes of scratch dl_append_step_tiled needs for n rows with split replay."""
    out = ctypes.c_size_t(0)
    _check(_lib.dl_tiled_workspace_bytes(ctypes.byref(desc), int(n), ctypes.byref(out)),
           "dl_tiled_workspace_bytes")
    return out.value


def tiled_workspace(desc, n, device="cuda"):
    """A device buffer of the split-replay scratch size for n rows (None if no log)."""
    nbytes = dl_tiled_workspace_bytes(desc, n)
    return torch.empty((nbytes,), dtype=torch.uint8, device=device) if nbytes else None


def dl_append_step_tiled(desc, state, tok, o, slots=None, value_tiles=4, split_replay=True,
                         workspace=None, stream=None):
    """Value-tiled DeltaLog step (Sec. 3.3): the same operation as dl_append_step with
    ``value_tiles`` workgroups per head; ``split_replay`` prepares the replay
    coefficients once per head into ``workspace`` (see ``tiled_workspace``)."""
    sp, n = _rows(desc, slots, tok.n)
    _need(o, "o", torch.float32, (n, desc.heads, desc.dv))
    wp, wn = (None, 0) if workspace is None else (workspace.data_ptr(), workspace.numel() *
                                                  workspace.element_size())
    _check(_lib.dl_append_step_tiled(ctypes.byref(desc), ctypes.byref(state.struct),
                                     ctypes.byref(tok.struct), _ptr(o), sp, n,
                                     int(value_tiles), int(bool(split_replay)), wp, wn,
                                     _stream(stream)), "dl_append_step_tiled")


def dl_append_step_tiled_noalloc(desc, state, tok, o, slots=None, value_tiles=4, stream=None):
    """dl_append_step_tiled with split replay whose coefficient scratch is the library's
    fixed per-GPU array (DL_NOALLOC_SCRATCH_BYTES): the call allocates nothing.  Calls
    that may overlap on one GPU race on that array."""
    sp, n = _rows(desc, slots, tok.n)
    _need(o, "o", torch.float32, (n, desc.heads, desc.dv))
    _check(_lib.dl_append_step_tiled_noalloc(ctypes.byref(desc), ctypes.byref(state.struct),
                                             ctypes.byref(tok.struct), _ptr(o), sp, n,
                                             int(value_tiles), _stream(stream)),
           "dl_append_step_tiled_noalloc")
