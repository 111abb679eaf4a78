/*
 * deltalog.h -- C ABI of libdeltalog.so: DeltaLog one-token decode state update for
 * linear-attention recurrences (the Table 1 operators: GDN, KDA, RWKV6, linear
 * attention, RetNet, GLA) on AMD Instinct MI355X (gfx950).
 *
 * The method (deferred materialisation of recurrent states, Sec. 3): the dense
 * recurrent state of each (slot, head) is kept as a dense base S plus a bounded log of
 * compact update factors.  Most decode steps read S once, replay the live log, emit
 * the output and append one entry (Eq. 5); every M-th step folds the log and the
 * current token back into S with a single dense write (Eq. 6).  The represented
 * state is always Eq. 7:
 *
 *     S_logical = D(ell) S + sum_{i<L} D(ell - Lam_i) K_i U_i^T,   D(l) = diag(exp l)
 *
 * and equals the eager recurrence of Eq. 3 (Table 1 instantiations) in exact
 * arithmetic.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every data pointer is a DEVICE pointer (hipMalloc'd or a torch CUDA tensor),
 *    owned by the caller.  The library never allocates, frees or synchronises; all
 *    work is enqueued on the caller's `stream`, and buffers must stay alive until the
 *    stream has executed it.  Calls on distinct buffers are re-entrant and thread-safe.
 *  - Arrays are dense, row-major, with the shapes given below.  B = desc->num_slots,
 *    H = desc->heads, C = desc->merge_interval - 1 (live-log capacity),
 *    dl = 1 for GDN and RetNet (one log-decay per head), dl = dk for KDA, RWKV6 and
 *    GLA (per key); linear attention has no decay (no lam_log or lam).
 *  - The state matrix of a head is dk x dv, rows indexed by the key dimension; the
 *    decay D(.) scales rows (Eq. 2); outputs are o = x^T S (length dv).
 *  - `slots` is a device int32 array of n distinct slot ids in [0, B): token row i
 *    drives slot slots[i].  slots == NULL means the identity and requires n == B,
 *    except that n == 0 is always a no-op: once the descriptor is valid and 0 <= n <= B
 *    it returns DL_OK without looking at any pointer.
 *    Duplicate ids in one call race (undefined).
 *  - Token arrays are packed by token row: [n, H, ...].  Outputs are written by token
 *    row, fp32, [n, H, dv].  `o` must not alias any input or state buffer.
 *  - Every argument check happens on the host BEFORE any HIP call; a failing check
 *    returns a negative dl_status and enqueues nothing (so the checks can be exercised
 *    without a GPU).  A failed launch returns DL_E_HIP.  Corruption that only the
 *    device can see (a slot id outside [0, B), a live length outside [0, C]) makes the
 *    affected (slot, head) skip its work and ORs a code into *state->err (if non-NULL):
 *    1 = bad slot id, 2 = live length out of range.
 *  - Alignment: S, k_log, u_log, q, k, v and o must be 16-byte aligned, and so must
 *    lam_log when dl == dk (KDA, RWKV6, GLA: its rows are read 16 bytes at a time);
 *    the other float/int32 arrays 4-byte aligned.
 *  - Supported shapes: dk, dv in {64, 128}; 1 <= M <= 64.
 */
#ifndef DELTALOG_H
#define DELTALOG_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DL_ABI_VERSION 4
#define DL_MAX_MERGE_INTERVAL 64

typedef enum {
  DL_OK = 0,
  DL_E_NULL = -1,        /* a required pointer is NULL                                  */
  DL_E_SHAPE = -2,       /* B, H, n or slot-list shape inconsistent                     */
  DL_E_DTYPE = -3,       /* dtype combination not allowed                               */
  DL_E_ALIGN = -4,       /* pointer not aligned as required                             */
  DL_E_UNSUPPORTED = -5, /* dk/dv/M/op outside the supported set                        */
  DL_E_HIP = -6,         /* the kernel launch failed                                    */
  DL_E_VERSION = -7,     /* desc->abi_version != DL_ABI_VERSION                         */
  DL_E_SCRATCH = -8      /* needs more than DL_NOALLOC_SCRATCH_BYTES of scratch          */
} dl_status;

typedef enum {
  DL_OP_GDN = 0,
  DL_OP_KDA = 1,
  DL_OP_RWKV6 = 2,
  DL_OP_LINATTN = 3,
  DL_OP_RETNET = 4,
  DL_OP_GLA = 5
} dl_op;
typedef enum { DL_F32 = 0, DL_BF16 = 1 } dl_dtype;

/* Problem description (host memory, read during the call only).
 * Operators (Table 1, Eq. 3):
 *   GDN     head-wise scalar decay, delta-rule pair (k, beta (v - k^T D(lambda) S)),
 *           post-update readout o = q^T S_t;
 *   KDA     per-key decay, the same pair and readout;
 *   RWKV6   per-key decay, pair (k, v), bonus readout o = r^T (S_{t-1} + diag(u) k v^T);
 *   LINATTN no decay, pair (phi(k), v) with phi applied by the caller, o = q^T S_t
 *           (Eq. 1);
 *   RETNET  head-wise scalar decay gamma_t = exp(lambda_t), pair (k, v), o = q^T S_t;
 *   GLA     per-key decay, pair (k, v), o = q^T S_t.
 * dl (the log-decay width) is dk for KDA, RWKV6 and GLA and 1 for GDN and RetNet;
 * linear attention has no log-decay and touches neither lam_log nor lam.
 * The cumulative log-decay ell of Sec. 3.1 is not a buffer here: Eq. 5 writes ell and
 * the new snapshot Lam_log[L] with the same value and Eq. 6 resets ell together with L,
 * so ell is always the newest snapshot Lam_log[L-1], or 0 when L = 0, and the library
 * reads it from there. */
typedef struct {
  int32_t abi_version;    /* must be DL_ABI_VERSION                                      */
  int32_t op;             /* dl_op                                                       */
  int32_t num_slots;      /* B >= 1: slots in the state buffers                          */
  int32_t heads;          /* H >= 1                                                      */
  int32_t dk, dv;         /* key / value head dims, each 64 or 128                       */
  int32_t merge_interval; /* M in [1, 64]: one merge every M steps (Sec. 3.1); C = M-1   */
  int32_t in_dtype;       /* dl_dtype of q/r, k, v; K_log stores exact copies of k       */
  int32_t u_log_dtype;    /* dl_dtype of U_log: DL_F32 for GDN/KDA (corrected values),   */
                          /* == in_dtype for the others (exact copies of v)              */
  int32_t state_dtype;    /* dl_dtype of the dense state S: DL_F32, or DL_BF16 (all       */
                          /* arithmetic in fp32, S rounded to bf16 -- nearest even -- on  */
                          /* every store; every other buffer keeps its dtype)            */
} dl_desc;

/* DeltaLog physical state (Sec. 3.1 list of buffers, less ell: see dl_desc), one entry
 * per (slot, head). */
typedef struct {
  void*    S;        /* [B,H,dk,dv] state_dtype dense base                               */
  void*    k_log;    /* [B,H,C,dk]  in_dtype   key-side factors   (may be NULL if C == 0) */
  void*    u_log;    /* [B,H,C,dv]  u_log_dtype value-side factors (may be NULL if C == 0)*/
  float*   lam_log;  /* [B,H,C,dl]  fp32 snapshot of ell per entry (may be NULL if C == 0)*/
                     /*             16-byte aligned when dl == dk, else 4-byte            */
                     /*             for dl == 1 stored entry-major, [B,C,H]               */
                     /*             (ignored, may be NULL, for LINATTN)                  */
  int32_t* len;      /* [B,H]       live-log length L in [0, C]                          */
  int32_t* err;      /* [1]         sticky device error word (see above); may be NULL    */
} dl_state;

/* Current-token inputs: the per-token interface of Eq. 3, one row per listed slot. */
typedef struct {
  const void*  q;    /* [n,H,dk] in_dtype: query (the receptance r for RWKV6)            */
  const void*  k;    /* [n,H,dk] in_dtype: key, the key-side factor a_t                  */
  const void*  v;    /* [n,H,dv] in_dtype: value                                         */
  const float* beta; /* [n,H]    fp32 delta-rule write strength (GDN/KDA); else ignored  */
  const float* lam;  /* [n,H,dl] fp32 per-step log-decay lambda_t = log(alpha_t) <= 0     */
                     /*          (ignored, may be NULL, for LINATTN)                     */
  const float* u;    /* [H,dk]   fp32 RWKV6 bonus (per-head parameter); NULL otherwise   */
} dl_token;

/* Eager dense step (Eq. 3): S <- D(lambda) S + a b^T with the readout of Table 1, for
 * the listed slots of a dense state S [B,H,dk,dv] of state_dtype (no log).  Writes
 * o [n,H,dv].
 * This is the baseline that reads and writes the whole state every token (Sec. 2.3).
 * desc->merge_interval is validated but otherwise ignored. */
int dl_eager_step(const dl_desc* desc, void* S, const dl_token* tok, float* o,
                  const int32_t* slots, int32_t n, hipStream_t stream);

/* One DeltaLog decode step (Alg. 1) for the listed slots: per (slot, head) read the
 * base once, replay the live log, write the output, then append the factors
 * (Eq. 5) if L < C, else merge log and token into the base (Eq. 6) and reset L (the
 * cumulative log-decay restarts at 0).  With M == 1 every step merges and the result
 * equals dl_eager_step. */
int dl_append_step(const dl_desc* desc, const dl_state* state, const dl_token* tok,
                   float* o, const int32_t* slots, int32_t n, hipStream_t stream);

/* Merge now, at any live length L in [0, C] (Eq. 6 is defined for general L).
 * tok != NULL: consume the token exactly like the merge branch of dl_append_step and
 *              write o (required).
 * tok == NULL: flush -- materialise Eq. 7 into the base and reset (slot reuse,
 *              eviction, checkpoint; Sec. 4 slot lifecycle); o is ignored. */
int dl_merge(const dl_desc* desc, const dl_state* state, const dl_token* tok, float* o,
             const int32_t* slots, int32_t n, hipStream_t stream);

/* Read-only readout of the represented state (Eq. 7): o = x^T S_logical for a query
 * x [n,H,dk] in in_dtype.  Mutates nothing.  (No RWKV6 bonus: there is no token.) */
int dl_readout(const dl_desc* desc, const dl_state* state, const void* q, float* o,
               const int32_t* slots, int32_t n, hipStream_t stream);

/* Value-tiled DeltaLog step (Sec. 3.3, the kernel ownership path): the same operation
 * as dl_append_step (results equal up to floating-point reassociation), with each
 * (slot, head) state split along the value dimension into value_tiles tiles of
 * dk x dv/value_tiles, one workgroup each.  Three launches on the stream:
 *   [ReplayPrep]  split_replay != 0 and C > 0 only: the key-side replay coefficients
 *                 q^T D(ell - Lam_i) K_i and k^T D(ell - Lam_i) K_i of every live entry,
 *                 once per (row, head), into the caller's workspace (fp32);
 *   AppendDecode  per value tile: stream the tile, replay the log on its columns (with
 *                 the prepared coefficients, or recomputing them per tile when
 *                 split_replay == 0), write the output slice, append the tile's U_log
 *                 shard (tile 0 also writes K_log[L] and Lam_log[L]) or merge the tile;
 *   Finalize      per (row, head): commit L exactly once.
 * value_tiles: 2 or 4.  Only state_dtype == DL_F32 (else DL_E_DTYPE).
 * workspace: device memory of at least dl_tiled_workspace_bytes(desc, n) bytes, 16-byte
 * aligned, owned by the caller; required when split_replay != 0 and C > 0, ignored
 * otherwise.  Its contents are scratch: overwritten, never read across calls.  Calls
 * that share a workspace must not overlap.  If a later launch fails, DL_E_HIP is
 * returned and the earlier launches of the call may already be enqueued. */
int dl_append_step_tiled(const dl_desc* desc, const dl_state* state, const dl_token* tok,
                         float* o, const int32_t* slots, int32_t n, int32_t value_tiles,
                         int32_t split_replay, void* workspace, size_t workspace_bytes,
                         hipStream_t stream);

/* Bytes of workspace dl_append_step_tiled needs for n rows with split replay:
 * n * H * 2 * (M - 1) * sizeof(float) (0 when M == 1).  Writes *bytes. */
int dl_tiled_workspace_bytes(const dl_desc* desc, int32_t n, size_t* bytes);

/* Size of the fixed scratch of dl_append_step_tiled_noalloc, per GPU. */
#define DL_NOALLOC_SCRATCH_BYTES (4u << 20)

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): dl_append_step_tiled with split
 * replay, its workspace taken from a scratch array of DL_NOALLOC_SCRATCH_BYTES that the
 * library holds in device memory, one per GPU, for the life of the process.  The caller
 * still passes the state, token and output buffers; the call allocates and frees
 * nothing and enqueues exactly the launches of dl_append_step_tiled(..., split_replay=1,
 * ...).
 * The scratch needed is dl_tiled_workspace_bytes(desc, n); a call that needs more than
 * DL_NOALLOC_SCRATCH_BYTES returns DL_E_SCRATCH (after the argument checks, before any
 * HIP call) and enqueues nothing.
 * Every call on a GPU shares that GPU's scratch: calls that may overlap on one GPU (on
 * different streams, or from different threads without ordering) race and must not be
 * issued; calls ordered on one stream are safe.  The scratch keeps the last call's
 * contents; a call reads only what it wrote itself.  On its first call on a device the
 * entry point looks up that device's scratch address (a HIP runtime query, no
 * allocation) and keeps it; a failed lookup returns DL_E_HIP. */
int dl_append_step_tiled_noalloc(const dl_desc* desc, const dl_state* state,
                                 const dl_token* tok, float* o, const int32_t* slots,
                                 int32_t n, int32_t value_tiles, hipStream_t stream);

/* Human-readable name of a dl_status value (static storage). */
const char* dl_status_str(int status);

/* DL_ABI_VERSION of the loaded library. */
int dl_abi_version(void);

/* The compiler flags the library's kernels were built with beyond the optimisation
 * level and target (static storage), so that measurements can be matched to the exact
 * build that produced them. */
const char* dl_build_flags(void);

#ifdef __cplusplus
}
#endif

#endif /* DELTALOG_H */
