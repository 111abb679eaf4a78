// C-ABI front end of libdeltalog.so: argument validation and dispatch.
//
// Every check runs on the host before the single HIP call of an entry point (the
// kernel launch), so a rejected call enqueues nothing.  See include/deltalog.h for
// the contract of each entry point.
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "deltalog.h"
#include "dl_internal.h"

namespace {

using dl::KParams;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool is_delta(int op) { return op == DL_OP_GDN || op == DL_OP_KDA; }
bool has_decay(int op) { return op != DL_OP_LINATTN; }
bool per_key(int op) { return op == DL_OP_KDA || op == DL_OP_RWKV6 || op == DL_OP_GLA; }

int check_desc(const dl_desc* d) {
  if (!d) return DL_E_NULL;
  if (d->abi_version != DL_ABI_VERSION) return DL_E_VERSION;
  if (d->op < DL_OP_GDN || d->op > DL_OP_GLA) return DL_E_UNSUPPORTED;
  if ((d->dk != 64 && d->dk != 128) || (d->dv != 64 && d->dv != 128)) return DL_E_UNSUPPORTED;
  if (d->merge_interval < 1 || d->merge_interval > DL_MAX_MERGE_INTERVAL) return DL_E_UNSUPPORTED;
  if (d->num_slots < 1 || d->heads < 1) return DL_E_SHAPE;
  // One workgroup per (token row, head): the grid must fit a 32-bit dimension.
  if (int64_t(d->num_slots) * d->heads > int64_t(0x7fffffff)) return DL_E_SHAPE;
  if (d->in_dtype != DL_F32 && d->in_dtype != DL_BF16) return DL_E_DTYPE;
  if (d->state_dtype != DL_F32 && d->state_dtype != DL_BF16) return DL_E_DTYPE;
  if (is_delta(d->op)) {
    if (d->u_log_dtype != DL_F32) return DL_E_DTYPE;        // U_log holds computed b
  } else {
    if (d->u_log_dtype != d->in_dtype) return DL_E_DTYPE;   // U_log holds copies of v
  }
  return DL_OK;
}

int check_rows(const dl_desc* d, const int32_t* slots, int32_t n) {
  if (n < 0 || n > d->num_slots) return DL_E_SHAPE;
  if (n == 0) return DL_OK;
  if (!slots && n != d->num_slots) return DL_E_SHAPE;
  if (slots && !aligned(slots, 4)) return DL_E_ALIGN;
  return DL_OK;
}

int check_token(const dl_desc* d, const dl_token* t) {
  if (!t || !t->q || !t->k || !t->v) return DL_E_NULL;
  if (has_decay(d->op)) {
    if (!t->lam) return DL_E_NULL;
    if (!aligned(t->lam, 4)) return DL_E_ALIGN;
  }
  if (d->op == DL_OP_RWKV6) {
    if (!t->u) return DL_E_NULL;
    if (!aligned(t->u, 4)) return DL_E_ALIGN;
  }
  if (is_delta(d->op)) {
    if (!t->beta) return DL_E_NULL;
    if (!aligned(t->beta, 4)) return DL_E_ALIGN;
  }
  if (!aligned(t->q, 16) || !aligned(t->k, 16) || !aligned(t->v, 16)) return DL_E_ALIGN;
  return DL_OK;
}

int check_state(const dl_desc* d, const dl_state* s) {
  const bool decay = has_decay(d->op);
  if (!s || !s->S || !s->len) return DL_E_NULL;
  if (d->merge_interval > 1 && (!s->k_log || !s->u_log)) return DL_E_NULL;
  if (d->merge_interval > 1 && decay && !s->lam_log) return DL_E_NULL;
  if (!aligned(s->S, 16) || !aligned(s->len, 4)) return DL_E_ALIGN;
  if (s->k_log && !aligned(s->k_log, 16)) return DL_E_ALIGN;
  if (s->u_log && !aligned(s->u_log, 16)) return DL_E_ALIGN;
  // Per-key snapshot rows are read with 16-byte loads.
  if (s->lam_log && !aligned(s->lam_log, per_key(d->op) ? 16 : 4)) return DL_E_ALIGN;
  if (s->err && !aligned(s->err, 4)) return DL_E_ALIGN;
  return DL_OK;
}

KParams base_params(const dl_desc* d, const int32_t* slots, int32_t n) {
  KParams p{};
  p.slots = slots;
  p.n = n;
  p.B = d->num_slots;
  p.H = d->heads;
  p.C = d->merge_interval - 1;
  return p;
}

void set_state(KParams& p, const dl_state* s) {
  p.S = s->S;
  p.k_log = s->k_log;
  p.u_log = s->u_log;
  p.lam_log = s->lam_log;
  p.len = s->len;
  p.err = s->err;
}

void set_token(KParams& p, const dl_token* t) {
  p.q = t->q;
  p.k = t->k;
  p.v = t->v;
  p.beta = t->beta;
  p.lam = t->lam;
  p.u = t->u;
}

int launch(const dl_desc* d, int mode, const KParams& p, hipStream_t stream) {
  if (p.n == 0) return DL_OK;
  const bool bf16 = d->in_dtype == DL_BF16;
  const bool sbf16 = d->state_dtype == DL_BF16;
  hipError_t e = hipErrorInvalidValue;
  switch (d->op) {
    case DL_OP_GDN: e = dl::launch_gdn(mode, d->dk, d->dv, bf16, sbf16, p, stream); break;
    case DL_OP_KDA: e = dl::launch_kda(mode, d->dk, d->dv, bf16, sbf16, p, stream); break;
    case DL_OP_RWKV6: e = dl::launch_rwkv6(mode, d->dk, d->dv, bf16, sbf16, p, stream); break;
    case DL_OP_LINATTN: e = dl::launch_linattn(mode, d->dk, d->dv, bf16, sbf16, p, stream); break;
    case DL_OP_RETNET: e = dl::launch_retnet(mode, d->dk, d->dv, bf16, sbf16, p, stream); break;
    case DL_OP_GLA: e = dl::launch_gla(mode, d->dk, d->dv, bf16, sbf16, p, stream); break;
  }
  return e == hipSuccess ? DL_OK : DL_E_HIP;
}

#define DL_TRY(x)            \
  do {                       \
    const int rc_ = (x);     \
    if (rc_ != DL_OK) return rc_; \
  } while (0)

}  // namespace

namespace dl {

int tiled_check(const dl_desc* desc, const dl_state* state, const dl_token* tok, float* o,
                const int32_t* slots, int32_t n, int32_t value_tiles) {
  DL_TRY(check_desc(desc));
  DL_TRY(check_rows(desc, slots, n));
  if (value_tiles != 2 && value_tiles != 4) return DL_E_UNSUPPORTED;
  if (desc->state_dtype != DL_F32) return DL_E_DTYPE;
  if (n == 0) return DL_OK;               // nothing to do, whatever the other pointers are
  if (int64_t(n) * desc->heads * value_tiles > int64_t(0x7fffffff)) return DL_E_SHAPE;
  DL_TRY(check_state(desc, state));
  DL_TRY(check_token(desc, tok));
  if (!o) return DL_E_NULL;
  if (!aligned(o, 16)) return DL_E_ALIGN;
  return DL_OK;
}

int tiled_launch(const dl_desc* desc, const dl_state* state, const dl_token* tok, float* o,
                 const int32_t* slots, int32_t n, int32_t value_tiles, bool split, float* coef,
                 hipStream_t stream) {
  KParams p = base_params(desc, slots, n);
  set_state(p, state);
  set_token(p, tok);
  p.o = o;
  const bool bf16 = desc->in_dtype == DL_BF16;
  if (!split) coef = nullptr;
  hipError_t e = hipErrorInvalidValue;
  switch (desc->op) {
    case DL_OP_GDN: e = launch_tiled_gdn(desc->dk, desc->dv, bf16, value_tiles, split, p, coef, stream); break;
    case DL_OP_KDA: e = launch_tiled_kda(desc->dk, desc->dv, bf16, value_tiles, split, p, coef, stream); break;
    case DL_OP_RWKV6: e = launch_tiled_rwkv6(desc->dk, desc->dv, bf16, value_tiles, split, p, coef, stream); break;
    case DL_OP_LINATTN: e = launch_tiled_linattn(desc->dk, desc->dv, bf16, value_tiles, split, p, coef, stream); break;
    case DL_OP_RETNET: e = launch_tiled_retnet(desc->dk, desc->dv, bf16, value_tiles, split, p, coef, stream); break;
    case DL_OP_GLA: e = launch_tiled_gla(desc->dk, desc->dv, bf16, value_tiles, split, p, coef, stream); break;
  }
  return e == hipSuccess ? DL_OK : DL_E_HIP;
}

}  // namespace dl

extern "C" {

int dl_abi_version(void) { return DL_ABI_VERSION; }

#ifndef DL_BUILD_FLAGS
#define DL_BUILD_FLAGS ""
#endif
const char* dl_build_flags(void) { return DL_BUILD_FLAGS; }

const char* dl_status_str(int status) {
  switch (status) {
    case DL_OK: return "DL_OK";
    case DL_E_NULL: return "DL_E_NULL: a required pointer is NULL";
    case DL_E_SHAPE: return "DL_E_SHAPE: inconsistent batch, head or slot-list shape";
    case DL_E_DTYPE: return "DL_E_DTYPE: dtype combination not allowed";
    case DL_E_ALIGN: return "DL_E_ALIGN: pointer not aligned as required";
    case DL_E_UNSUPPORTED: return "DL_E_UNSUPPORTED: dk, dv, merge interval or operator not supported";
    case DL_E_HIP: return "DL_E_HIP: kernel launch failed";
    case DL_E_VERSION: return "DL_E_VERSION: descriptor ABI version mismatch";
    case DL_E_SCRATCH: return "DL_E_SCRATCH: the call needs more than the allocation-free entry point's fixed scratch";
  }
  return "unknown dl_status";
}

int dl_eager_step(const dl_desc* desc, void* S, const dl_token* tok, float* o,
                  const int32_t* slots, int32_t n, hipStream_t stream) {
  DL_TRY(check_desc(desc));
  DL_TRY(check_rows(desc, slots, n));
  if (n == 0) return DL_OK;               // nothing to do, whatever the other pointers are
  if (!S || !o) return DL_E_NULL;
  if (!aligned(S, 16) || !aligned(o, 16)) return DL_E_ALIGN;
  DL_TRY(check_token(desc, tok));
  KParams p = base_params(desc, slots, n);
  p.S = S;
  p.o = o;
  set_token(p, tok);
  return launch(desc, dl::M_EAGER, p, stream);
}

int dl_append_step(const dl_desc* desc, const dl_state* state, const dl_token* tok, float* o,
                   const int32_t* slots, int32_t n, hipStream_t stream) {
  DL_TRY(check_desc(desc));
  DL_TRY(check_rows(desc, slots, n));
  if (n == 0) return DL_OK;               // nothing to do, whatever the other pointers are
  DL_TRY(check_state(desc, state));
  DL_TRY(check_token(desc, tok));
  if (!o) return DL_E_NULL;
  if (!aligned(o, 16)) return DL_E_ALIGN;
  KParams p = base_params(desc, slots, n);
  set_state(p, state);
  set_token(p, tok);
  p.o = o;
  return launch(desc, dl::M_STEP, p, stream);
}

int dl_merge(const dl_desc* desc, const dl_state* state, const dl_token* tok, float* o,
             const int32_t* slots, int32_t n, hipStream_t stream) {
  DL_TRY(check_desc(desc));
  DL_TRY(check_rows(desc, slots, n));
  if (n == 0) return DL_OK;               // nothing to do, whatever the other pointers are
  DL_TRY(check_state(desc, state));
  KParams p = base_params(desc, slots, n);
  set_state(p, state);
  if (tok) {
    DL_TRY(check_token(desc, tok));
    if (!o) return DL_E_NULL;
    if (!aligned(o, 16)) return DL_E_ALIGN;
    set_token(p, tok);
    p.o = o;
    return launch(desc, dl::M_MERGE, p, stream);
  }
  return launch(desc, dl::M_FLUSH, p, stream);
}

int dl_readout(const dl_desc* desc, const dl_state* state, const void* q, float* o,
               const int32_t* slots, int32_t n, hipStream_t stream) {
  DL_TRY(check_desc(desc));
  DL_TRY(check_rows(desc, slots, n));
  if (n == 0) return DL_OK;               // nothing to do, whatever the other pointers are
  DL_TRY(check_state(desc, state));
  if (!q || !o) return DL_E_NULL;
  if (!aligned(q, 16) || !aligned(o, 16)) return DL_E_ALIGN;
  KParams p = base_params(desc, slots, n);
  set_state(p, state);
  p.q = q;
  p.o = o;
  return launch(desc, dl::M_READOUT, p, stream);
}

int dl_tiled_workspace_bytes(const dl_desc* desc, int32_t n, size_t* bytes) {
  DL_TRY(check_desc(desc));
  if (!bytes) return DL_E_NULL;
  if (n < 0 || n > desc->num_slots) return DL_E_SHAPE;
  *bytes = size_t(n) * size_t(desc->heads) * 2 * size_t(desc->merge_interval - 1) * sizeof(float);
  return DL_OK;
}

int dl_append_step_tiled(const dl_desc* desc, const dl_state* state, const dl_token* tok,
                         float* o, const int32_t* slots, int32_t n, int32_t value_tiles,
                         int32_t split_replay, void* workspace, size_t workspace_bytes,
                         hipStream_t stream) {
  DL_TRY(dl::tiled_check(desc, state, tok, o, slots, n, value_tiles));
  if (n == 0) return DL_OK;               // nothing to do, whatever the other pointers are
  const bool split = split_replay != 0;
  if (split && desc->merge_interval > 1) {
    size_t need = 0;
    DL_TRY(dl_tiled_workspace_bytes(desc, n, &need));
    if (!workspace) return DL_E_NULL;
    if (!aligned(workspace, 16)) return DL_E_ALIGN;
    if (workspace_bytes < need) return DL_E_SHAPE;
  }
  return dl::tiled_launch(desc, state, tok, o, slots, n, value_tiles, split,
                          static_cast<float*>(workspace), stream);
}

}  // extern "C"
