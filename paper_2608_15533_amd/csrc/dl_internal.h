// Internal interface between the C-ABI front end (abi.cpp) and the kernel translation
// units (one per operator).  Plain C++ types only.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#include "deltalog.h"

namespace dl {

enum OpId {
  OP_GDN = DL_OP_GDN,
  OP_KDA = DL_OP_KDA,
  OP_RWKV6 = DL_OP_RWKV6,
  OP_LINATTN = DL_OP_LINATTN,
  OP_RETNET = DL_OP_RETNET,
  OP_GLA = DL_OP_GLA
};
enum ModeId { M_EAGER = 0, M_STEP = 1, M_MERGE = 2, M_FLUSH = 3, M_READOUT = 4 };

// Everything a kernel needs, passed by value (all pointers are device pointers).
struct KParams {
  void* S;               // [B,H,dk,dv] dense base (or the eager dense state), fp32 or bf16
  void* k_log;           // [B,H,C,dk]
  void* u_log;           // [B,H,C,dv]
  float* lam_log;        // [B,H,C,dl]
  int32_t* len;          // [B,H]
  int32_t* err;          // [1] or null
  const void* q;         // [n,H,dk] (also the readout query)
  const void* k;         // [n,H,dk]
  const void* v;         // [n,H,dv]
  const float* beta;     // [n,H]
  const float* lam;      // [n,H,dl]
  const float* u;        // [H,dk]
  float* o;              // [n,H,dv]
  const int32_t* slots;  // [n] or null (identity)
  int32_t n, B, H, C;
};

// Launch the kernel for (op, mode, dk, dv, input dtype, state dtype) with one
// workgroup per (token row, head).  Returns the hipError_t of the launch.
hipError_t launch_gdn(int mode, int dk, int dv, bool bf16, bool state_bf16, const KParams& p,
                      hipStream_t s);
hipError_t launch_kda(int mode, int dk, int dv, bool bf16, bool state_bf16, const KParams& p,
                      hipStream_t s);
hipError_t launch_rwkv6(int mode, int dk, int dv, bool bf16, bool state_bf16, const KParams& p,
                        hipStream_t s);
hipError_t launch_linattn(int mode, int dk, int dv, bool bf16, bool state_bf16, const KParams& p,
                          hipStream_t s);
hipError_t launch_retnet(int mode, int dk, int dv, bool bf16, bool state_bf16, const KParams& p,
                         hipStream_t s);
hipError_t launch_gla(int mode, int dk, int dv, bool bf16, bool state_bf16, const KParams& p,
                      hipStream_t s);

// Value-tiled step (fp32 state): [ReplayPrep into coef when split] -> tiles -> Finalize.
#define DL_DECLARE_TILED(name)                                                          \
  hipError_t launch_tiled_##name(int dk, int dv, bool bf16, int nv, bool split,          \
                                 const KParams& p, float* coef, hipStream_t s)
DL_DECLARE_TILED(gdn);
DL_DECLARE_TILED(kda);
DL_DECLARE_TILED(rwkv6);
DL_DECLARE_TILED(linattn);
DL_DECLARE_TILED(retnet);
DL_DECLARE_TILED(gla);
#undef DL_DECLARE_TILED

// The argument checks of the value-tiled step other than its workspace (host only; no
// HIP call), and its launches with `coef` as the split-replay scratch.
int tiled_check(const dl_desc* desc, const dl_state* state, const dl_token* tok, float* o,
                const int32_t* slots, int32_t n, int32_t value_tiles);
int tiled_launch(const dl_desc* desc, const dl_state* state, const dl_token* tok, float* o,
                 const int32_t* slots, int32_t n, int32_t value_tiles, bool split, float* coef,
                 hipStream_t stream);

}  // namespace dl
