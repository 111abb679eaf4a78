// DeltaLog decode kernels for gfx950 (CDNA4, wave64).
//
// One workgroup owns one (slot, head) state: a dk x dv matrix (64 KiB at 128x128 fp32).
// Thread layout: NCG = dv/4 column groups (one float4 column slice each) times
// NRG = dk/RPT row groups; every thread keeps RPT rows x 4 columns of the state in
// registers (rows rg, rg+NRG, ..., so one wave-wide float4 load covers whole
// consecutive rows, 1 KiB contiguous).  RPT = 16, or 4 for 64 x 64 heads.  The state
// is read from HBM exactly once per step and, when the step materialises (merge /
// eager / flush), written back exactly once from the same registers -- the read, the
// key-dimension reductions and the write never leave the workgroup.  Because one
// workgroup owns all of a head's value columns, the replay coefficients are computed
// once per (slot, head) and the shared log metadata (K_log[L], Lam_log[L], L) has a
// single writer without any cross-workgroup finalisation (the ownership problem of
// Sec. 3.3).  The cumulative log-decay ell is not stored: it equals the newest snapshot
// Lam_log[L-1], or 0 with an empty log.
//
// Modes (one template per mode; the per-slot append/merge branch of Alg. 1 is taken
// on the device from that slot's live length):
//   EAGER   Eq. 3 on a dense state (no log).
//   STEP    Alg. 1: readout + replay, then append (Eq. 5) if L < C, else merge (Eq. 6).
//   MERGE   the merge branch at the current L (a forced merge, any 0 <= L <= C).
//   FLUSH   materialise Eq. 7 into the base and reset (no token).
//   READOUT o = x^T (Eq. 7 state), no writes to the state.
//
// Per (slot, head) and step the arithmetic is (l' = ell + lambda):
//   replay coefficient of entry i for a vector x:  g_i(x) = sum_r e^(l_r - Lam_i,r) x_r K_i,r
//   base readout:   sum_r e^(l_r) x_r S_r,:      (l = ell for RWKV6, l' otherwise)
//   correction c = base(k) + sum_i g_i(k) U_i ;  b = beta (v - c)             (GDN/KDA)
//              b = v                             (RWKV6, linear attention, RetNet, GLA)
//   output     o = base(q) + sum_i g_i(q) U_i + (q.k) b    (post-update: all but RWKV6)
//              o = base(r) + sum_i g_i(r) U_i + (r.(u*k)) v                   (RWKV6)
//   merge      S <- diag(e^l') S + sum_i diag(e^(l'-Lam_i)) K_i U_i^T + k b^T  (Eq. 6)
// Linear attention has no decay: every e^(.) above is 1 and ell, Lam_log and lambda are
// never touched.
// Every decay factor is evaluated as exp of a log-decay *difference* (<= 0 in normal
// use), never as a product of exp(l') and exp(-Lam_i).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "dl_internal.h"

namespace dl {

// ------------------------------------------------------------------ loads/stores
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float ld1(const float* p) { return *p; }
__device__ __forceinline__ float ld1(const uint16_t* p) { return __uint_as_float(uint32_t(*p) << 16); }

__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 ld4(const uint16_t* p) {
  const uint2 w = *reinterpret_cast<const uint2*>(p);
  return make_float4(bf_lo(w.x), bf_hi(w.x), bf_lo(w.y), bf_hi(w.y));
}

// Copy four elements verbatim (bit-exact log entries).
__device__ __forceinline__ void cp4(float* d, const float* s) {
  *reinterpret_cast<float4*>(d) = *reinterpret_cast<const float4*>(s);
}
__device__ __forceinline__ void cp4(uint16_t* d, const uint16_t* s) {
  *reinterpret_cast<uint2*>(d) = *reinterpret_cast<const uint2*>(s);
}

__device__ __forceinline__ void st4(float* d, float4 v) { *reinterpret_cast<float4*>(d) = v; }

__device__ __forceinline__ float4 f4(float a) { return make_float4(a, a, a, a); }
__device__ __forceinline__ float4 operator+(float4 a, float4 b) {
  return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}
__device__ __forceinline__ float4 operator-(float4 a, float4 b) {
  return make_float4(a.x - b.x, a.y - b.y, a.z - b.z, a.w - b.w);
}
__device__ __forceinline__ float4 operator*(float s, float4 a) {
  return make_float4(s * a.x, s * a.y, s * a.z, s * a.w);
}
// a + s * b, written as separate fused multiply-adds per lane element.
__device__ __forceinline__ float4 fma4(float s, float4 b, float4 a) {
  return make_float4(fmaf(s, b.x, a.x), fmaf(s, b.y, a.y), fmaf(s, b.z, a.z), fmaf(s, b.w, a.w));
}

__device__ __forceinline__ float shfl_xor(float v, int m) { return __shfl_xor(v, m, 64); }

// Sum over aligned groups of N lanes (N = 4, 8 or 16), every lane of a group ending with
// the group's sum.  With DL_DPP_REDUCE the lane exchanges are DPP moves inside a 16-lane
// row (mirror over 16 lanes, mirror over 8, then swaps of lane pairs of pairs and of lane
// pairs), and the exchanges across rows below are the gfx950 row-swap instructions:
// none needs an LDS round trip.  Otherwise all are xor shuffles.  Callers reduce only
// where every lane of the wave is active.
#ifndef DL_DPP_REDUCE
#define DL_DPP_REDUCE 1
#endif
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int N>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(N == 4 || N == 8 || N == 16, "DPP rows hold 16 lanes");
  if constexpr (DL_DPP_REDUCE) {
    if constexpr (N == 16) v += dpp_move<0x140>(v);   // row_mirror: lane i <- 15 - i
    if constexpr (N >= 8) v += dpp_move<0x141>(v);    // row_half_mirror: lane i <- 7 - i
    v += dpp_move<0x4E>(v);                           // quad_perm [2,3,0,1]
    v += dpp_move<0xB1>(v);                           // quad_perm [1,0,3,2]
  } else {
#pragma unroll
    for (int m = N / 2; m >= 1; m >>= 1) v += shfl_xor(v, m);
  }
  return v;
}
// v(lane) + v(lane ^ 16): v_permlane16_swap with both operands v hands each lane the two
// values of its row pair.
__device__ __forceinline__ float xor16_sum(float v) {
  if constexpr (DL_DPP_REDUCE) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
  } else {
    return v + shfl_xor(v, 16);
  }
}
// v(lane) + v(lane ^ 32), with v_permlane32_swap likewise.
__device__ __forceinline__ float xor32_sum(float v) {
  if constexpr (DL_DPP_REDUCE) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
  } else {
    return v + shfl_xor(v, 32);
  }
}
__device__ __forceinline__ float4 xor16_sum(float4 v) {
  return make_float4(xor16_sum(v.x), xor16_sum(v.y), xor16_sum(v.z), xor16_sum(v.w));
}
__device__ __forceinline__ float4 xor32_sum(float4 v) {
  return make_float4(xor32_sum(v.x), xor32_sum(v.y), xor32_sum(v.z), xor32_sum(v.w));
}

// Decay factors exp(x) for log-decay differences x <= 0: the hardware base-2
// exponential of x * log2(e) (two instructions instead of the 13 of a correctly
// rounded expf).  Its relative error is about 2^-24 * |x| * log2(e) plus one ulp
// (below 2e-6 for |x| <= 40); exp(0) is exactly 1.
__device__ __forceinline__ float dl_exp(float x) { return __expf(x); }

// State-tile traffic.  The base is streamed once per step and not reused by this
// workgroup, so by default its loads and stores carry the non-temporal hint.
#ifndef DL_NT_STATE
#define DL_NT_STATE 1
#endif
// Cache policy of the state-tile stores alone (the merged base): -1 = as the loads;
// by default non-temporal with device scope (nt sc1), so that the base is written
// through the XCD's L2 rather than held there as dirty lines while the other
// workgroups of the launch stream their tiles in.
#ifndef DL_STATE_STORE_POLICY
#define DL_STATE_STORE_POLICY (DL_NT_STATE ? 18 : -1)
#endif
// Log keys of the first coefficient pass / the first replay values of each row group
// are loaded before the first barrier (1) or where they are used (0).
#ifndef DL_PREFETCH_KEYS
#define DL_PREFETCH_KEYS 1
#endif
#ifndef DL_PREFETCH_U
#define DL_PREFETCH_U 1
#endif
// Per-key log snapshots of the first coefficient pass are loaded before the first
// barrier (1) or right after it (0, fewer live registers).
#ifndef DL_PREFETCH_PER_KEY
#define DL_PREFETCH_PER_KEY 0
#endif
#ifndef DL_PREFETCH_PER_KEY_SMALL
#define DL_PREFETCH_PER_KEY_SMALL 1
#endif
// ... and for a bf16 state, whose tile holds half the registers of an fp32 one.
#ifndef DL_PREFETCH_PER_KEY_BF16_STATE
#define DL_PREFETCH_PER_KEY_BF16_STATE 1
#endif
// Row order of the staged K~ chunk in LDS: key row r = c * RPL + x (run c of the
// coefficient pass, element x of the run) is kept at row x * LPE + c (1), or at r (0).
// The coefficient pass writes one entry of RPL consecutive rows per lane; in key order
// the lanes of a wave would meet in a few LDS banks, in this order their rows differ by
// the run index instead.  The contraction's reads of row rg + NRG j stay at offsets
// that are constant per j.
#ifndef DL_KT_ROW_ORDER
#define DL_KT_ROW_ORDER 1
#endif
// Order of the per-row token vectors the coefficient pass reads (k, q and the per-key
// log-decays) in LDS: row r = c * RPL + x (run c, element x) at position x * LPE + c (1),
// or at r (0).  A coefficient pass reads element x of every run at once, RPL rows
// apart: in row order the 16 lanes of an entry meet in a few banks, in this order they
// read consecutive words.
#ifndef DL_COEF_LDS_ORDER
#define DL_COEF_LDS_ORDER 1
#endif
// Long logs.  The STEP and MERGE kernels come in two builds: one for a capacity of at
// most one coefficient pass (C <= 16), and one for longer logs, chosen by the host from
// the descriptor's merge interval.  Only the long build carries the machinery below, so
// the registers and LDS of the short build stay as they are.
//   DL_STAGE_CHUNKS        merge chunks of decayed log keys staged in LDS by the
//                          coefficient passes themselves (same loads and exps); later
//                          chunks are staged from global memory.
//   DL_PREFETCH_NEXT_PASS  load the next coefficient pass's log keys (1: and snapshots;
//                          2: keys only) while the current pass computes.
//   DL_PREFETCH_NEXT_PASS_PER_KEY  the same for 128-row per-key heads with bf16
//                          activations, where it fits in the 4-wave long build (off:
//                          the second pass's loads already leave right behind the
//                          first pass's, and it measured no gain).
//   DL_U_EARLY             load the log values of the next merge chunk before
//                          contracting the current one.
#ifndef DL_STAGE_CHUNKS
#define DL_STAGE_CHUNKS 2
#endif
#ifndef DL_PREFETCH_NEXT_PASS
#define DL_PREFETCH_NEXT_PASS 1
#endif
#ifndef DL_PREFETCH_NEXT_PASS_PER_KEY
#define DL_PREFETCH_NEXT_PASS_PER_KEY 0
#endif
//   DL_PREFETCH_U_LATER    load the first pair of the replay's later log values
//                          (entries rg + 2 NRG and rg + 3 NRG) with the first two, before
//                          the first barrier, instead of after the coefficient passes.
//                          Long builds with per-key decay, bf16 activations, an fp32 state
//                          and 8 row groups only (128-row heads, whose later values start
//                          with the second pass); the other builds would spill or lose a
//                          wave.
#ifndef DL_PREFETCH_U_LATER
#define DL_PREFETCH_U_LATER 1
#endif
#ifndef DL_U_EARLY
#define DL_U_EARLY 1
#endif
//   DL_REPLAY_PAIRS        replay the log values past the first two per row group two
//                          at a time, with both loads issued before either is used.
#ifndef DL_REPLAY_PAIRS
#define DL_REPLAY_PAIRS 1
#endif
// The merge's rank-(L+1) contraction (Eq. 6) on the matrix cores (1: fp32 MFMA, twice
// the rate of plain fp32 FMAs) or on the vector ALUs (0).  See MfmaMerge below.
// DL_MFMA_MERGE_64COL = 0 keeps 64-column heads, DL_MFMA_MERGE_BF16_STATE = 0 a bf16
// state, on the VALU path.
#ifndef DL_MFMA_MERGE
#define DL_MFMA_MERGE 1
#endif
#ifndef DL_MFMA_MERGE_64COL
#define DL_MFMA_MERGE_64COL 1
#endif
#ifndef DL_MFMA_MERGE_BF16_STATE
#define DL_MFMA_MERGE_BF16_STATE 1
#endif
#ifndef DL_MFMA_DRAIN
#define DL_MFMA_DRAIN 1
#endif
// LDS layout of the staged K~ chunk where the merge contracts on MFMA: row R starts at
// R * S + (R / 16) * P floats (1, S and P per head shape), or at R * 20 (0; the VALU
// contraction's float4 reads need it).  An LDS access by a wave is served 32 lanes at a
// time over 32 banks.  The MFMA operand read has those 32 lanes on 16 or 32 different rows
// at one entry; the staging write has them on 16 consecutive rows at two entries.  With
// the padded layout both land in 32 different banks (with R * 20, the read met in 4 or 8).
#ifndef DL_KT_PAD
#define DL_KT_PAD 1
#endif
// Issue order of the log entries relative to the state tile (see the kernel).
#ifndef DL_LOG_FIRST
#define DL_LOG_FIRST 0
#endif
// Occupancy target (waves per SIMD) handed to the register allocator; 0 = compiler's choice.
#ifndef DL_WAVES_PER_EU
#define DL_WAVES_PER_EU 0
#endif

// The state tile of one (slot, head) is addressed through a buffer resource: the
// head's base address lives in scalar registers, each lane keeps one 32-bit offset and
// the row blocks differ by a scalar offset, so no per-row 64-bit addresses occupy
// vector registers between the load and the store.  The resource covers exactly the
// head's dk x dv state elements; the hardware drops accesses outside it.
constexpr int kStateCachePolicy = DL_NT_STATE ? 2 : 0;   // 2 = non-temporal (nt)
constexpr int kStateStorePolicy =            // 18 = nt (2) + device scope (sc1, 16)
    DL_STATE_STORE_POLICY >= 0 ? DL_STATE_STORE_POLICY : kStateCachePolicy;
constexpr int kRawBufferFlags = 0x00020000;                // 32-bit data format, raw access

__device__ __forceinline__ __amdgpu_buffer_rsrc_t state_rsrc(void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, int(bytes), kRawBufferFlags);
}

// Round fp32 to bf16, nearest even (finite values).
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// Four consecutive state elements of one row, as held by one lane between the load and
// the store.  fp32 state: one 16-byte access; bf16 state: one 8-byte access, widened to
// fp32 on use and rounded (nearest even) on store.
template <typename TS> struct StateQuad;
template <> struct StateQuad<float> {
  float4 w;
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kStateCachePolicy);
    w = make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]),
                    __uint_as_float(v[3]));
  }
  __device__ __forceinline__ float4 get() const { return w; }
  static __device__ __forceinline__ void store(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                               uint32_t soff, float4 v) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 x = {__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z),
                     __float_as_uint(v.w)};
    __builtin_amdgcn_raw_buffer_store_b128(x, r, voff, soff, kStateStorePolicy);
  }
  // The materialised rows at the end of a kernel: the row registers are the store data
  // and nothing writes them afterwards.
  template <int N>
  static __device__ __forceinline__ void store_rows(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                                    uint32_t row_block, const float4 (&m)[N]) {
#pragma unroll
    for (int j = 0; j < N; ++j) store(r, voff, j * row_block, m[j]);
  }
};
template <> struct StateQuad<uint16_t> {
  uint2 w;
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, kStateCachePolicy);
    w = make_uint2(v[0], v[1]);
  }
  __device__ __forceinline__ float4 get() const {
    return make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u),
                       __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xffff0000u));
  }
  static __device__ __forceinline__ void store(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                               uint32_t soff, float4 v) {
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 x = {bf16_rne(v.x) | (bf16_rne(v.y) << 16), bf16_rne(v.z) | (bf16_rne(v.w) << 16)};
    __builtin_amdgcn_raw_buffer_store_b64(x, r, voff, soff, kStateStorePolicy);
  }
  // The materialised rows at the end of a kernel.
  template <int N>
  static __device__ __forceinline__ void store_rows(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                                    uint32_t row_block, const float4 (&m)[N]) {
#pragma unroll
    for (int j = 0; j < N; ++j) store(r, voff, j * row_block, m[j]);
  }
};

// N consecutive elements (N a multiple of 4) widened to fp32, loaded with 16-byte accesses
// (8-byte accesses for bf16 runs whose length is not a multiple of 8).
template <int N>
__device__ __forceinline__ void ld_run(const float* p, float (&o)[N]) {
#pragma unroll
  for (int x = 0; x < N; x += 4) {
    const float4 v = ld4(p + x);
    o[x] = v.x; o[x + 1] = v.y; o[x + 2] = v.z; o[x + 3] = v.w;
  }
}
template <int N>
__device__ __forceinline__ void ld_run(const uint16_t* p, float (&o)[N]) {
  static_assert(N % 4 == 0, "run length");
  if constexpr (N % 8 != 0) {
#pragma unroll
    for (int x = 0; x < N; x += 4) {
      const uint2 w = *reinterpret_cast<const uint2*>(p + x);
      o[x + 0] = bf_lo(w.x); o[x + 1] = bf_hi(w.x); o[x + 2] = bf_lo(w.y); o[x + 3] = bf_hi(w.y);
    }
    return;
  }
#pragma unroll
  for (int x = 0; x < N; x += 8) {
    const uint4 w = *reinterpret_cast<const uint4*>(p + x);
    o[x + 0] = bf_lo(w.x); o[x + 1] = bf_hi(w.x); o[x + 2] = bf_lo(w.y); o[x + 3] = bf_hi(w.y);
    o[x + 4] = bf_lo(w.z); o[x + 5] = bf_hi(w.z); o[x + 6] = bf_lo(w.w); o[x + 7] = bf_hi(w.w);
  }
}

constexpr uint32_t kXcds = 8;   // accelerator complex dies of an MI355X
// (row, head) pairs per XCD chunk: 32 heads' 4-byte metadata is one 128-byte line.
// 0 gives each XCD a single contiguous range instead.
#ifndef DL_XCD_CHUNK
#define DL_XCD_CHUNK 32
#endif
constexpr uint32_t kXcdChunk = DL_XCD_CHUNK;

// Raw register images of loads whose conversion to fp32 is deferred: converting right
// after a load makes the wave wait for it, and (loads completing in issue order) for
// every load issued before it -- the state tile included.
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(uint16_t x) { return __uint_as_float(uint32_t(x) << 16); }

template <typename T> struct Raw4;                 // four consecutive elements
template <> struct Raw4<float> {
  float4 w;
  __device__ __forceinline__ void load(const float* p) { w = *reinterpret_cast<const float4*>(p); }
  __device__ __forceinline__ float4 get() const { return w; }
};
template <> struct Raw4<uint16_t> {
  uint2 w;
  __device__ __forceinline__ void load(const uint16_t* p) { w = *reinterpret_cast<const uint2*>(p); }
  __device__ __forceinline__ float4 get() const {
    return make_float4(bf_lo(w.x), bf_hi(w.x), bf_lo(w.y), bf_hi(w.y));
  }
};

template <typename T, int N> struct RawRun;         // N consecutive elements, N % 4 == 0
template <int N> struct RawRun<float, N> {
  float4 w[N / 4];
  __device__ __forceinline__ void load(const float* p) {
#pragma unroll
    for (int i = 0; i < N / 4; ++i) w[i] = reinterpret_cast<const float4*>(p)[i];
  }
  __device__ __forceinline__ void get(float (&o)[N]) const {
#pragma unroll
    for (int i = 0; i < N / 4; ++i) {
      o[4 * i] = w[i].x; o[4 * i + 1] = w[i].y; o[4 * i + 2] = w[i].z; o[4 * i + 3] = w[i].w;
    }
  }
};
template <int N> struct RawRun<uint16_t, N> {
  static_assert(N % 4 == 0, "run length");
  static constexpr bool W16 = N % 8 == 0;           // 16-byte words, else 8-byte words
  using Word = std::conditional_t<W16, uint4, uint2>;
  Word w[W16 ? N / 8 : N / 4];
  __device__ __forceinline__ void load(const uint16_t* p) {
#pragma unroll
    for (int i = 0; i < (W16 ? N / 8 : N / 4); ++i) w[i] = reinterpret_cast<const Word*>(p)[i];
  }
  __device__ __forceinline__ void get(float (&o)[N]) const {
    if constexpr (W16) {
#pragma unroll
      for (int i = 0; i < N / 8; ++i) {
        o[8 * i + 0] = bf_lo(w[i].x); o[8 * i + 1] = bf_hi(w[i].x);
        o[8 * i + 2] = bf_lo(w[i].y); o[8 * i + 3] = bf_hi(w[i].y);
        o[8 * i + 4] = bf_lo(w[i].z); o[8 * i + 5] = bf_hi(w[i].z);
        o[8 * i + 6] = bf_lo(w[i].w); o[8 * i + 7] = bf_hi(w[i].w);
      }
    } else {
#pragma unroll
      for (int i = 0; i < N / 4; ++i) {
        o[4 * i + 0] = bf_lo(w[i].x); o[4 * i + 1] = bf_hi(w[i].x);
        o[4 * i + 2] = bf_lo(w[i].y); o[4 * i + 3] = bf_hi(w[i].y);
      }
    }
  }
};

// Lam_log addressing.  Per-key snapshots of a (slot, head) are contiguous rows of dk
// values, [B,H,C,dk].  Scalar snapshots are stored entry-major, [B,C,H]: the H heads of a
// slot append entry L side by side (one 128-byte line for 32 heads) instead of each
// writing 4 bytes into a sector of its own.  Entry i of a (slot, head) is at
// base[i * stride].
template <int DL>
__device__ __forceinline__ float* lam_log_base(const KParams& p, int slot, int h) {
  if constexpr (DL == 1) return p.lam_log + size_t(slot) * size_t(p.C) * p.H + h;
  else return p.lam_log + (size_t(slot) * p.H + h) * size_t(p.C) * DL;
}
template <int DL>
__device__ __forceinline__ size_t lam_log_stride(const KParams& p) {
  return DL == 1 ? size_t(p.H) : size_t(DL);
}

// Read one float at a workgroup-uniform address through the scalar path (the constant
// address space): the read waits on its own counter instead of queueing behind the
// vector loads in flight.  Only for data that no workgroup of the launch writes (the
// scalar cache is invalidated at every kernel launch).
__device__ __forceinline__ float scalar_ld(const float* ptr) {
  typedef const float __attribute__((address_space(4))) const_float;
  return *(const_float*)ptr;
}

// Nothing may be scheduled across this point (loads keep their issue order).
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// ------------------------------------------------------------------ configuration
// Threads per workgroup for a dk x dv head: dv/4 column groups x dk/rows-per-thread
// row groups.  Small (64 x 64) heads keep 4 rows per thread (four waves per head: short
// per-thread chains for a 16 KiB state), the others 16 rows per thread.
#ifndef DL_SMALL_HEAD_RPT
#define DL_SMALL_HEAD_RPT 4
#endif
constexpr int rows_per_thread(int dk, int dv) {
  return (dk == 64 && dv == 64) ? DL_SMALL_HEAD_RPT : 16;
}
constexpr int threads_per_head(int dk, int dv) { return (dv / 4) * (dk / rows_per_thread(dk, dv)); }

// What distinguishes the operators of Table 1 inside the kernel.
template <int OP>
struct OpTraits {
  static constexpr bool DELTA = OP == OP_GDN || OP == OP_KDA;   // b = beta (v - correction)
  static constexpr bool PER_KEY = OP == OP_KDA || OP == OP_RWKV6 || OP == OP_GLA;
  static constexpr bool DECAY = OP != OP_LINATTN;               // linear attention: none
  static constexpr bool BONUS = OP == OP_RWKV6;   // pre-update readout plus r^T diag(u) k v^T
};

template <int OP, int DK, int DV, int MODE, bool LONG = false>
struct Cfg {
  static constexpr int RPT = rows_per_thread(DK, DV);   // state rows held per thread
  static constexpr int NCG = DV / 4;             // float4 column groups
  static constexpr int NRG = DK / RPT;           // row groups
  static constexpr int NT = NCG * NRG;           // threads per workgroup
  static constexpr int NW = NT / 64;             // waves per workgroup
  static constexpr int DL = OpTraits<OP>::PER_KEY ? DK : 1;   // log-decay width
  static constexpr int EPP = 16;                 // log entries per coefficient pass
  static constexpr int LPE = NT / EPP;           // lanes per log entry (coefficient pass)
  static constexpr int RPL = DK / LPE;           // key rows per lane (coefficient pass)
  static constexpr int CH = 16;                  // log entries staged per merge chunk
  static constexpr int KTS = CH + 4;             // LDS row stride, VALU layout
  // Padded layout (row R at R * KT_S + (R / 16) * KT_P) for the MFMA contraction; the
  // per-shape constants are the bank-conflict-free ones for its reads and the staging
  // writes (a 64 x 128 or 128 x 64 head keeps a 2-way conflict on the read).
  static constexpr bool KT_PADDED = DL_KT_PAD && DL_MFMA_MERGE &&
                                    (DV / 4 == 32 || DL_MFMA_MERGE_64COL) && DL_MFMA_MERGE_BF16_STATE;
  static constexpr int KT_S = !KT_PADDED ? KTS : DK == DV ? 18 : 20;
  static constexpr int KT_P = !KT_PADDED ? 0 : DV / 4 == 32 ? 1 : 2;
  static constexpr int kt_base_c(int r) { return r * KT_S + (r / 16) * KT_P; }
  static constexpr int KT_CHUNK = (kt_base_c(DK) + 3) / 4 * 4;   // floats per staged chunk
  // K~ chunks staged by the coefficient passes.  With per-key decay the long build keeps
  // one: the second chunk's staging slows every append (measured), and the merge stages
  // the later chunks itself, one chunk ahead.
  static constexpr int NSTAGE = (LONG && !OpTraits<OP>::PER_KEY) ? DL_STAGE_CHUNKS : 1;
  static constexpr bool U_EARLY = LONG && DL_U_EARLY;      // (fp32 state only: see kernel)
  // The short build of STEP and MERGE only runs with a capacity of at most one pass
  // (C <= CH); the other modes run with any capacity.
  static constexpr bool CAP_ONE_PASS = (MODE == M_STEP || MODE == M_MERGE) && !LONG;
  // A row group sees a second live entry (row group rg replays rg, rg + NRG, ...).
  static constexpr bool TWO_PER_GROUP = !(CAP_ONE_PASS && NRG >= CH);
  static constexpr int UPT = CH * NCG / NT;     // log-value quads per thread and merge chunk
  static constexpr bool DELTA = OpTraits<OP>::DELTA;
  static constexpr bool DECAY = OpTraits<OP>::DECAY;
  static constexpr bool BONUS = OpTraits<OP>::BONUS;
  static constexpr bool HAS_LOG = MODE != M_EAGER;
  static constexpr bool HAS_TOKEN = MODE == M_EAGER || MODE == M_STEP || MODE == M_MERGE;
  static constexpr bool READS_OUT = MODE != M_FLUSH;
  static constexpr bool NEEDS_C = DELTA && HAS_TOKEN;
  static constexpr bool CAN_MERGE = MODE != M_READOUT;
  static constexpr bool MERGES_LOG = CAN_MERGE && HAS_LOG;
  static constexpr bool REPLAYS = HAS_LOG && READS_OUT;   // readout of the live log
  static_assert(NT % 64 == 0 && NT <= 256, "workgroup must be whole waves");
  static_assert(64 % NCG == 0, "a wave must hold whole rows");
  static_assert(NT % LPE == 0 && DK % LPE == 0, "coefficient pass layout");
  static_assert(NT >= DK, "one thread per key row in the prologue");
  static_assert(RPL == 4 || RPL == 8 || RPL == 16, "coefficient pass run length");
  static_assert(NRG % RPL == 0 || RPL % NRG == 0, "row groups and coefficient runs nest");
  static_assert(CH == EPP, "merge chunk c is staged by coefficient pass c");
  static_assert(CH * NCG % NT == 0 && UPT >= 1, "whole log-value quads per thread");
  static_assert(NSTAGE >= 1 && NSTAGE <= 4, "staged merge chunks");
  // LDS row of key row r in the staged K~ chunk (a permutation of [0, DK)), and the
  // same for the two ways the kernel names a row: element x of coefficient run c, and
  // row j of row group rg (rg + NRG j), written so that the part that depends on x or j
  // is a compile-time constant.
  static __device__ __forceinline__ int kt_row(int r) {
    return DL_KT_ROW_ORDER ? (r % RPL) * LPE + r / RPL : r;
  }
  static __device__ __forceinline__ int kt_row_run(int c, int x) {
    return DL_KT_ROW_ORDER ? x * LPE + c : c * RPL + x;
  }
  // LDS offset of row r of the staged chunk, and of element x of coefficient run c (with
  // the row order above, c < LPE and LPE dividing 16 keep (x LPE + c) / 16 = x LPE / 16,
  // so the part that depends on x is a compile-time constant).
  static __device__ __forceinline__ int kt_base(int r) { return r * KT_S + (r >> 4) * KT_P; }
  static __device__ __forceinline__ int kt_off_run(int c, int x) {
    if constexpr (DL_KT_ROW_ORDER) return c * KT_S + (x * LPE * KT_S + ((x * LPE) >> 4) * KT_P);
    else return kt_base(c * RPL + x);
  }
  // LDS position of token row r in the vectors the coefficient pass reads (the same
  // permutation as the K~ rows).
  static __device__ __forceinline__ int cp_pos(int r) {
    return DL_COEF_LDS_ORDER ? (r % RPL) * LPE + r / RPL : r;
  }
  static __device__ __forceinline__ int cp_pos_run(int c, int x) {
    return DL_COEF_LDS_ORDER ? x * LPE + c : c * RPL + x;
  }
  static __device__ __forceinline__ int cp_pos_group(int rg, int j) {
    if constexpr (!DL_COEF_LDS_ORDER) return rg + NRG * j;
    else return kt_row_group_order(rg, j);
  }
  static __device__ __forceinline__ int kt_row_group(int rg, int j) {
    if constexpr (!DL_KT_ROW_ORDER) return rg + NRG * j;
    else return kt_row_group_order(rg, j);
  }
  // (rg + NRG j) % RPL * LPE + (rg + NRG j) / RPL, with the part that depends on j a
  // compile-time constant.
  static __device__ __forceinline__ int kt_row_group_order(int rg, int j) {
    if constexpr (NRG % RPL == 0) {
      return (rg % RPL) * LPE + rg / RPL + (NRG / RPL) * j;
    } else {
      constexpr int q = RPL / NRG;                  // RPL is a multiple of NRG
      return (rg + NRG * (j % q)) * LPE + j / q;
    }
  }
  static_assert(LPE <= 16 && 16 % LPE == 0, "an entry's lanes share one 16-lane row");
  static_assert(NT == threads_per_head(DK, DV), "launch bound must match the layout");
  static_assert(!(BONUS && DL == 1), "the bonus readout is only defined with per-key decay");
};

// ------------------------------------------------------------ MFMA merge contraction
// The merge adds sum_i K~_i U_i^T to the decayed tile (Eq. 6), a product of a dk x n and
// an n x dv matrix for a chunk of n log entries.  The tile is held row-streamed: thread
// (rg, cg) owns rows rg + NRG j (j < RPT) and columns 4 cg .. 4 cg + 3, one 16-byte load
// or store per row.  An fp32 MFMA leaves each lane one output column and a fixed set of
// output rows.  Both index maps of the product are free, so they are chosen to make the
// MFMA's output fragment the thread's own tile registers, with no data movement:
//   * output column n of block b (b < 4) is state column 4 n + b, so the four blocks of
//     a lane hold the four columns of its quad;
//   * output row m is the state row that the lane holding m owns, so a lane's output
//     rows are its own rows rg + NRG j.
// With 128 columns (NCG = 32) a wave owns two row groups, 32 rows, and the product is
// v_mfma_f32_32x32x2f32: lane l = 32 h + n holds output rows 8 (k / 4) + 4 h + k % 4
// (k < 16), i.e. row group 2 w + h, row j = k.  The A operand (K~) of lane (h, n) is entry
// h of the K-step at the row whose output lane n owns; the B operand (U) is entry h at
// column 4 n + b, i.e. component b of the U quad of column group n = cg.  With 64
// columns (NCG = 16) a wave owns four row groups and the product is
// v_mfma_f32_16x16x4f32 over RPT / 4 blocks of 16 rows: lane l = 16 g + n holds rows
// 4 g + k of a block, i.e. row group 4 w + g, row j = 4 mb + k.  The accumulators must be
// ordinary VGPRs (the build's -amdgpu-mfma-vgpr-form): AGPR accumulators would add the
// tile's registers again.
template <int NCG, int RPT>
struct MfmaMerge {                                // unused: VALU contraction
  static constexpr int KS = 2, NMB = 1;
  static __device__ __forceinline__ int row_of(int, int, int, int) { return 0; }
  __device__ __forceinline__ void from_rows(const float4*) {}
  __device__ __forceinline__ void to_rows(float4*) const {}
  __device__ __forceinline__ void step(const float*, float4) {}
  __device__ __forceinline__ void drain() {}
  __device__ __forceinline__ void store_rows(__amdgpu_buffer_rsrc_t, uint32_t, uint32_t) const {}
};

template <int RPT>
struct MfmaMerge<32, RPT> {                       // v_mfma_f32_32x32x2f32
  static_assert(RPT == 16, "a 32-row block is the two row groups of a wave");
  using V = float __attribute__((ext_vector_type(16)));
  static constexpr int KS = 2;                    // log entries per MFMA
  static constexpr int NMB = 1;                   // row blocks per wave
  V acc[4];
  // State row of output row m of the wave's block (row group 2w + (m / 4) % 2, row
  // 4 (m / 8) + m % 4 of it).
  static __device__ __forceinline__ int row_of(int w, int /*mb*/, int m, int NRG) {
    return 2 * w + (m / 4) % 2 + NRG * (4 * (m / 8) + m % 4);
  }
  __device__ __forceinline__ void from_rows(const float4* t) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      acc[0][j] = t[j].x; acc[1][j] = t[j].y; acc[2][j] = t[j].z; acc[3][j] = t[j].w;
    }
  }
  __device__ __forceinline__ void to_rows(float4* t) const {
#pragma unroll
    for (int j = 0; j < 16; ++j) t[j] = make_float4(acc[0][j], acc[1][j], acc[2][j], acc[3][j]);
  }
  __device__ __forceinline__ void step(const float* a, float4 b) {
    acc[0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b.x, acc[0], 0, 0, 0);
    acc[1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b.y, acc[1], 0, 0, 0);
    acc[2] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b.z, acc[2], 0, 0, 0);
    acc[3] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b.w, acc[3], 0, 0, 0);
  }
  // The tile's rows from the accumulators (component b of row j of the lane's quad is
  // register j of block b), one 16-byte store per row.  Every row is gathered into
  // registers of its own, and all of them stay allocated until the last store has issued:
  // gathered into one reused set of four registers, each row's registers were rewritten
  // right behind its store, and on the GPU that store then wrote the next row's value in
  // lanes 12-15 of each 16-lane row now and then.
  __device__ __forceinline__ void store_rows(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                             uint32_t row_block) const {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    u32x4 x[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      x[j] = u32x4{__float_as_uint(acc[0][j]), __float_as_uint(acc[1][j]),
                   __float_as_uint(acc[2][j]), __float_as_uint(acc[3][j])};
      asm volatile("" : "+v"(x[j]));
    }
#pragma unroll
    for (int j = 0; j < 16; ++j)
      __builtin_amdgcn_raw_buffer_store_b128(x[j], r, voff, j * row_block, kStateStorePolicy);
#pragma unroll
    for (int j = 0; j < 16; ++j) asm volatile("" ::"v"(x[j]));
  }
  // Wait states between the last MFMA and the first VALU read of its results, on top
  // of those the compiler inserts.
  __device__ __forceinline__ void drain() {
#if DL_MFMA_DRAIN
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]));
#endif
  }
};

template <int RPT>
struct MfmaMerge<16, RPT> {                       // v_mfma_f32_16x16x4f32 (64 columns)
  static_assert(RPT % 4 == 0, "16-row blocks, four rows per lane");
  using V = float __attribute__((ext_vector_type(4)));
  static constexpr int KS = 4;                    // log entries per MFMA
  static constexpr int NMB = RPT / 4;             // row blocks per wave
  V acc[NMB][4];
  // State row of output row m of block mb: a wave owns four row groups (4 w + m / 4),
  // and lane (g, n) holds rows 4 g + k of the block, row j = 4 mb + k of its group.
  static __device__ __forceinline__ int row_of(int w, int mb, int m, int NRG) {
    return 4 * w + m / 4 + NRG * (4 * mb + m % 4);
  }
  __device__ __forceinline__ void from_rows(const float4* t) {
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float4 r = t[4 * mb + k];
        acc[mb][0][k] = r.x; acc[mb][1][k] = r.y; acc[mb][2][k] = r.z; acc[mb][3][k] = r.w;
      }
  }
  __device__ __forceinline__ void to_rows(float4* t) const {
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
      for (int k = 0; k < 4; ++k)
        t[4 * mb + k] = make_float4(acc[mb][0][k], acc[mb][1][k], acc[mb][2][k], acc[mb][3][k]);
  }
  __device__ __forceinline__ void step(const float* a, float4 b) {
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
      acc[mb][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mb], b.x, acc[mb][0], 0, 0, 0);
      acc[mb][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mb], b.y, acc[mb][1], 0, 0, 0);
      acc[mb][2] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mb], b.z, acc[mb][2], 0, 0, 0);
      acc[mb][3] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mb], b.w, acc[mb][3], 0, 0, 0);
    }
  }
  // As for 128 columns: every row in registers of its own, held until the last store.
  __device__ __forceinline__ void store_rows(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                             uint32_t row_block) const {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    u32x4 x[RPT];
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int j = 4 * mb + k;
        x[j] = u32x4{__float_as_uint(acc[mb][0][k]), __float_as_uint(acc[mb][1][k]),
                     __float_as_uint(acc[mb][2][k]), __float_as_uint(acc[mb][3][k])};
        asm volatile("" : "+v"(x[j]));
      }
#pragma unroll
    for (int j = 0; j < RPT; ++j)
      __builtin_amdgcn_raw_buffer_store_b128(x[j], r, voff, j * row_block, kStateStorePolicy);
#pragma unroll
    for (int j = 0; j < RPT; ++j) asm volatile("" ::"v"(x[j]));
  }
  __device__ __forceinline__ void drain() {
#if DL_MFMA_DRAIN
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb)
      asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
                   : "+v"(acc[mb][0]), "+v"(acc[mb][1]), "+v"(acc[mb][2]), "+v"(acc[mb][3]));
#endif
  }
};

// U_log holds the delta rule's corrected values in fp32, and exact copies of v (in the
// activation dtype) for every other operator.
template <int OP, typename TIN>
struct UType { using type = std::conditional_t<OpTraits<OP>::DELTA, float, TIN>; };

// Occupancy target (waves per SIMD) for the register allocator: DL_WAVES_PER_EU for every
// kernel if set, else DL_SMALL_HEAD_WAVES for 64 x 64 heads (1 = no target).
#ifndef DL_SMALL_HEAD_WAVES
#define DL_SMALL_HEAD_WAVES 6
#endif
// The long build of 128^2 heads with bf16 activations is held to 4 waves per SIMD (128
// registers), the occupancy its short build has.
#ifndef DL_LONG_WAVES
#define DL_LONG_WAVES 4
#endif
constexpr int waves_target(int dk, int dv, bool long_build, int in_bytes) {
  return DL_WAVES_PER_EU > 0 ? DL_WAVES_PER_EU
         : (dk == 64 && dv == 64) ? DL_SMALL_HEAD_WAVES
         : (long_build && dk == 128 && dv == 128 && in_bytes == 2) ? DL_LONG_WAVES
                                                                    : 1;
}
#define DL_OCCUPANCY \
  __attribute__((amdgpu_waves_per_eu(waves_target(DK, DV, LONG, int(sizeof(TIN))))))

// ------------------------------------------------------------------ the kernel
// Every global load a workgroup needs is issued before its first barrier: the token
// rows, the state tile, the first pass of log keys/snapshots and the first log values
// of the replay; only the live length (and the slot id, for slot lists) precede them.
template <int OP, int DK, int DV, int MODE, typename TIN, typename TS, bool LONG>
__global__ __launch_bounds__(threads_per_head(DK, DV)) DL_OCCUPANCY
void deltalog_kernel(KParams p) {
  using CF = Cfg<OP, DK, DV, MODE, LONG>;
  using TU = typename UType<OP, TIN>::type;
  constexpr int NT = CF::NT, NCG = CF::NCG, NRG = CF::NRG, RPT = CF::RPT, DL = CF::DL;
  constexpr int RPL = CF::RPL;

  __shared__ float s_kf[DK];      // k (raw)
  __shared__ float s_qf[DK];      // q or r (raw)
  __shared__ float s_xk[DK];      // e^(l_r) k_r       (base correction vector)
  __shared__ float s_xq[DK];      // e^(l_r) q_r       (base readout vector)
  __shared__ float s_em[DK];      // e^(l'_r)          (materialisation row scale)
  __shared__ float s_lr[DL];      // readout log-decay l
  __shared__ float s_lm[DL];      // materialisation log-decay l'
  __shared__ float s_gk[DL_MAX_MERGE_INTERVAL];
  __shared__ float s_gq[DL_MAX_MERGE_INTERVAL];
  __shared__ float s_red[CF::NW][2][DV];
  __shared__ float s_dotw[CF::NW];
  // K~ chunks [NSTAGE][KT_CHUNK]: staged by the coefficient passes where the kernel
  // replays the log, else (flush) one chunk at a time from global memory
  constexpr int kKtChunks = CF::REPLAYS ? CF::NSTAGE : 1;
  __shared__ float s_kt[CF::MERGES_LOG ? kKtChunks * CF::KT_CHUNK : 1];
  __shared__ float4 s_u[CF::MERGES_LOG ? CF::CH * NCG : 1];          // U chunk  [CH][NCG]

  const int tid = threadIdx.x;
  const int H = p.H;
  // Workgroups are dispatched round-robin over the 8 XCDs (each with its own L2).  Map
  // them so that each XCD owns whole chunks of DL_XCD_CHUNK consecutive (row, head)
  // pairs: the 4-byte per-head metadata (L and the head-wise log-decay snapshots) and token
  // scalars of a chunk then fill whole 128-byte lines in one L2 instead of being
  // written back partially by eight different caches.  Chunks are dealt to the XCDs
  // in turn, so a run of consecutive slots that merge in the same step (slots admitted
  // together) is spread over all eight XCDs instead of loading one of them.  Rows past
  // the last whole round of chunks keep the hardware order.
  uint32_t lin = blockIdx.x;
  const uint32_t nblk = gridDim.x;
  if constexpr (kXcdChunk > 0) {
    const uint32_t full = nblk - nblk % (kXcds * kXcdChunk);
    if (lin < full) {
      const uint32_t x = lin % kXcds, j = lin / kXcds;
      lin = ((j / kXcdChunk) * kXcds + x) * kXcdChunk + j % kXcdChunk;
    }
  } else if (nblk % kXcds == 0) {
    lin = (lin % kXcds) * (nblk / kXcds) + lin / kXcds;   // one contiguous range per XCD
  }
  const int row = int(lin) / H;                   // token row
  const int h = int(lin) - row * H;               // head
  const int slot = p.slots ? p.slots[row] : row;
  if (slot < 0 || slot >= p.B) {                  // uniform per workgroup
    if (tid == 0 && p.err) atomicOr(p.err, 1);
    return;
  }
  const size_t sh = size_t(slot) * H + h;         // state (slot, head) index
  const size_t th = size_t(row) * H + h;          // token (row, head) index
  const int C = p.C;
  // The live length is read through the scalar path (its own wait counter); it is
  // first used only after the tile loads below have been issued.
  int L_raw = 0;
  if constexpr (CF::HAS_LOG) L_raw = p.len[sh];

  // Vector loads return in issue order, so a wait for one load is a wait for every
  // load issued before it.  The issue order is therefore: the small token rows (needed
  // first, by the prologue), then the 64 KiB state tile, then the log entries (needed
  // after the first barrier, once the live length is known).  Compiler barriers keep
  // that order.

  // ---- 1. token row values (the prologue's inputs) ---------------------------------
  const TIN* kin = static_cast<const TIN*>(p.k) + th * DK;
  const TIN* qin = static_cast<const TIN*>(p.q) + th * DK;
  const int cg = tid % NCG;
  const int rg = tid / NCG;
  const int r0 = tid;                              // this thread's key row in the prologue
  // Every thread loads (threads past dk re-read the last row and ignore it): a load
  // under a branch would need its value at the branch join, i.e. an early wait.
  const int rl = r0 < DK ? r0 : DK - 1;
  const int rd = (DL == 1) ? 0 : rl;
  TIN k_raw = TIN(0), q_raw = TIN(0);
  float lam = 0.f, ell = 0.f, uf = 0.f;
  if constexpr (CF::HAS_TOKEN) {
    k_raw = kin[rl];
    if constexpr (CF::DECAY) lam = p.lam[th * DL + rd];
    if constexpr (CF::BONUS) uf = p.u[size_t(h) * DK + rl];
  }
  if constexpr (CF::READS_OUT) q_raw = qin[rl];
  Raw4<TIN> v_raw{};
  float beta = 0.f;
  if constexpr (CF::HAS_TOKEN) {
    v_raw.load(static_cast<const TIN*>(p.v) + th * DV + 4 * cg);
    if constexpr (CF::DELTA) beta = p.beta[th];
  }
  asm volatile("" ::: "memory");
  sched_fence();

  // ---- 2. the state tile and the log entries of the first pass ---------------------
  // Default order: tile, then (once the live length is back) the log entries, so the
  // tile never waits for the length.  DL_LOG_FIRST = 1 waits for the length first and
  // issues the log entries ahead of the tile, so the coefficient pass does not wait
  // for the tile.
  TS* const Sh = static_cast<TS*>(p.S) + sh * size_t(DK) * DV;
  const auto srs = state_rsrc(Sh, DK * DV * sizeof(TS));
  const uint32_t toff = uint32_t(rg * DV + 4 * cg) * sizeof(TS);   // lane's byte offset in a row block
  constexpr uint32_t kRowBlock = NRG * DV * sizeof(TS);             // bytes from row j to row j+1 of a lane
  StateQuad<TS> t[RPT];
  if constexpr (!DL_LOG_FIRST) {
#pragma unroll
    for (int j = 0; j < RPT; ++j) t[j].load(srs, toff, j * kRowBlock);
    asm volatile("" ::: "memory");
    sched_fence();
  }

  int L = __builtin_amdgcn_readfirstlane(L_raw);
  const bool bad_len = L < 0 || L > C;
  if (bad_len) L = 0;                             // keeps every address below in bounds
  if (bad_len) {
    if (tid == 0 && p.err) atomicOr(p.err, 2);
    return;
  }

  const TIN* Kb = static_cast<const TIN*>(p.k_log) + sh * size_t(C) * DK;
  float* const Lw = CF::DECAY ? lam_log_base<DL>(p, slot, h) : nullptr;
  const float* Lb = Lw;
  const size_t LS = lam_log_stride<DL>(p);
  const TU* Ub = static_cast<const TU*>(p.u_log) + sh * size_t(C) * DV;
  // The cumulative log-decay is not stored: after an append it equals the newest
  // snapshot (Eq. 5 writes both with the same value), after a merge it is 0 (Eq. 6
  // resets it with L).  Entry L-1 is not written by this launch (an append writes entry
  // L), so one value per head is read through the scalar path, without waiting for the
  // tile in flight; per-key values are one vector load per row.
  if constexpr (CF::HAS_LOG && CF::DECAY) {
    if constexpr (DL == 1) ell = L > 0 ? scalar_ld(Lb + size_t(L - 1) * LS) : 0.f;
    else ell = L > 0 ? Lb[size_t(L - 1) * LS + rd] : 0.f;
  }
  const int e_ = tid / CF::LPE;                   // coefficient pass: entry within the pass
  const int c_ = tid % CF::LPE;                   //                   key-row run
  // Per-key snapshots are prefetched only where the registers allow it (small heads, or
  // a bf16 state).
  constexpr bool kPrefetchPerKey = DL_PREFETCH_PER_KEY || (DL_PREFETCH_PER_KEY_SMALL && RPT <= 8) ||
                                   (DL_PREFETCH_PER_KEY_BF16_STATE && sizeof(TS) == 2 && RPL <= 8);
  float kr[RPL], lr_[(DL == 1) ? 1 : RPL];
  RawRun<TIN, RPL> kr_raw{};
  RawRun<float, (DL == 1) ? 8 : RPL> lr_raw{};      // per-key snapshots (unused for DL == 1)
  float lr0 = 0.f;                                   // scalar snapshot (DL == 1)
  // The prefetch loads are unconditional (a load under a per-lane condition makes the
  // wait counters conservative, i.e. waits for the tile): lanes past the live length
  // re-read entry L-1 (same cache lines), an empty log reads entry 0, and a log of
  // capacity 0 reads the head's own state tile instead; such values are never used.
  const int Lm1 = L > 0 ? L - 1 : 0;
  const TIN* Kp = C > 0 ? Kb : reinterpret_cast<const TIN*>(Sh);
  const float* Lp = C > 0 ? Lb : reinterpret_cast<const float*>(Sh);
  const TU* Up = C > 0 ? Ub : reinterpret_cast<const TU*>(Sh);
  if constexpr (CF::REPLAYS && DL_PREFETCH_KEYS && (DL == 1 || kPrefetchPerKey)) {
    const int ek = min(e_, Lm1);
    kr_raw.load(Kp + size_t(ek) * DK + c_ * RPL);
    if constexpr (DL == 1) {
      if constexpr (CF::DECAY) lr0 = Lp[size_t(ek) * LS];
    } else {
      lr_raw.load(Lp + size_t(ek) * DK + c_ * RPL);
    }
  }
  Raw4<TU> up0_raw{}, up1_raw{};                     // first two replay values of this row group
  // ... and, in the long build, the next two (re-reads of entry L-1 where they are past
  // the live length; the replay gives those a zero coefficient).
  constexpr bool kLaterEarly = LONG && DL > 1 && sizeof(TIN) == 2 && sizeof(TS) == 4 &&
                               CF::REPLAYS && DL_PREFETCH_U && DL_PREFETCH_U_LATER &&
                               DL_REPLAY_PAIRS && 2 * NRG == CF::CH;
  Raw4<TU> up2_raw{}, up3_raw{};
  if constexpr (CF::REPLAYS && DL_PREFETCH_U) {
    up0_raw.load(Up + size_t(min(rg, Lm1)) * DV + 4 * cg);
    if constexpr (CF::TWO_PER_GROUP) up1_raw.load(Up + size_t(min(rg + NRG, Lm1)) * DV + 4 * cg);
    if constexpr (kLaterEarly) {
      up2_raw.load(Up + size_t(min(rg + 2 * NRG, Lm1)) * DV + 4 * cg);
      up3_raw.load(Up + size_t(min(rg + 3 * NRG, Lm1)) * DV + 4 * cg);
    }
  }
  if constexpr (DL_LOG_FIRST) {
    sched_fence();
#pragma unroll
    for (int j = 0; j < RPT; ++j) t[j].load(srs, toff, j * kRowBlock);
  }
  sched_fence();
  const float kf = to_f32(k_raw), qf = to_f32(q_raw);

  // Does this (slot, head) materialise in this launch?  (Uniform per workgroup.)
  const bool merging = MODE == M_MERGE || MODE == M_FLUSH || MODE == M_EAGER ||
                       (MODE == M_STEP && L == C);
  if constexpr (CF::MERGES_LOG) {
    // The first chunk of log values is staged by the replay below; entries at or past L
    // in that chunk must read as zero in the merge contraction.
    if (merging)
      for (int x = tid; x < CF::CH * NCG; x += NT)
        if (x / NCG >= L) s_u[x] = f4(0.f);
  }

  // ---- 4. per-row decay factors (LDS) and the token dot product ---------------------
  if (r0 < DK) {
    float lr, lm;
    // Readouts of the decayed state (the delta-rule correction, and the post-update
    // output's base part), except RWKV6, which reads the old state.
    if constexpr (MODE == M_EAGER) {
      lr = CF::BONUS ? 0.f : lam;
      lm = lam;
    } else if constexpr (MODE == M_STEP || MODE == M_MERGE) {
      lm = ell + lam;
      lr = CF::BONUS ? ell : lm;
    } else {                        // FLUSH, READOUT: the represented state as it stands
      lr = ell;
      lm = ell;
    }
    const float er = dl_exp(lr);
    const int pr = CF::cp_pos(r0);                // coefficient-pass order
    s_kf[pr] = kf;
    s_qf[pr] = qf;
    s_xk[r0] = er * kf;
    s_xq[r0] = er * qf;
    s_em[r0] = dl_exp(lm);
    if (r0 < DL) {                                // DL == 1: r0 == 0 == pr
      s_lr[pr] = lr;
      s_lm[pr] = lm;
    }
  }
  if constexpr (CF::HAS_TOKEN) {
    // q.k (post-update readout of the new term) or r.(u*k) (RWKV6 bonus)
    float d = CF::BONUS ? qf * uf * kf : qf * kf;
    if (r0 >= DK) d = 0.f;                        // threads past dk hold a repeated row
    d = xor32_sum(xor16_sum(group_sum<16>(d)));
    if ((tid & 63) == 0) s_dotw[tid >> 6] = d;
  }
  __syncthreads();

  // ---- 5. replay coefficients g_i(k), g_i(q) of the live entries --------------------
  // A merging workgroup also writes the decayed keys K~_i[r] = e^(l'_r - Lam_i,r) K_i[r]
  // of the first NSTAGE chunks to LDS here, from the same loads and exps (the merge
  // decay l' equals the readout decay, except for RWKV6, which reads at ell).  With
  // DL_PREFETCH_NEXT_PASS the next pass's keys and snapshots are loaded before the
  // current pass computes.
  if constexpr (CF::REPLAYS) {
    constexpr bool kFirstPrefetched = DL_PREFETCH_KEYS && (DL == 1 || kPrefetchPerKey);
    // The next pass is prefetched where the registers allow it at the build's occupancy:
    // one log-decay per head (a scalar snapshot) or small heads; optionally 128² per-key
    // heads with bf16 activations (the 4-wave long build; the bonus readout's extra
    // registers leave room for the keys only).  With fp32 activations or other shapes a
    // 128-row per-key head would need 12 more registers across the pass (one wave less).
    constexpr int kNextPerKey =
        (sizeof(TIN) == 2 && DK == 128 && DV == 128 && DL_PREFETCH_NEXT_PASS_PER_KEY)
            ? (CF::BONUS ? 2 : DL_PREFETCH_NEXT_PASS) : 0;
    constexpr int kNext = !LONG ? 0 : (DL == 1 || RPT <= 8) ? DL_PREFETCH_NEXT_PASS : kNextPerKey;
    RawRun<TIN, RPL> kn_raw{};
    RawRun<float, (DL == 1) ? 8 : RPL> ln_raw{};
    float ln0 = 0.f;
    bool next_ready = false;                      // uniform
    // The short STEP/MERGE build runs with C <= EPP: at most one pass, compiled as such.
    const int passes_end = CF::CAP_ONE_PASS ? min(L, 1) : L;
    for (int i0 = 0; i0 < passes_end; i0 += CF::EPP) {   // uniform trip count
      const int i = i0 + e_;
      const int chunk = i0 / CF::CH;
      const bool stage = CF::MERGES_LOG && merging && chunk < kKtChunks;
      float* const kt = s_kt + (stage ? chunk : 0) * CF::KT_CHUNK;
      float ak = 0.f, aq = 0.f;
      const bool from_next = next_ready;
      const bool from_first = kFirstPrefetched && i0 == 0;
      constexpr bool kNextSnap = kNext == 1;      // snapshots prefetched too
      // This pass's own loads, issued together and unconditionally (lanes past the live
      // length re-read entry L-1, unused): a load under a per-lane condition is waited
      // for at the condition's end, which would serialise the key and snapshot round
      // trips.
      const bool keys_here = !from_next && !from_first;                   // uniform
      const bool snaps_here = !from_first && !(from_next && kNextSnap);
      const int ic = min(i, L - 1);
      RawRun<TIN, RPL> kc_raw{};
      RawRun<float, (DL == 1) ? 8 : RPL> lc_raw{};
      float lc0 = 0.f;
      if (keys_here) kc_raw.load(Kb + size_t(ic) * DK + c_ * RPL);
      if (snaps_here) {
        if constexpr (DL == 1) {
          if constexpr (CF::DECAY) lc0 = Lb[size_t(ic) * LS];
        } else {
          lc_raw.load(Lb + size_t(ic) * DK + c_ * RPL);
        }
      }
      if (keys_here) kc_raw.get(kr);
      if (snaps_here) {
        if constexpr (DL == 1) lr_[0] = lc0;
        else lc_raw.get(lr_);
      }
      if (from_next) {
        kn_raw.get(kr);
        if constexpr (kNextSnap) {
          if constexpr (DL == 1) lr_[0] = ln0;
          else ln_raw.get(lr_);
        }
      } else if (from_first) {
        kr_raw.get(kr);
        if constexpr (DL == 1) lr_[0] = lr0;
        else lr_raw.get(lr_);
      }
      next_ready = false;
      if constexpr (kNext > 0) {
        if (i0 + CF::EPP < L) {                   // uniform
          const int en = min(i + CF::EPP, L - 1);
          kn_raw.load(Kb + size_t(en) * DK + c_ * RPL);
          if constexpr (kNextSnap) {
            if constexpr (DL == 1) {
              if constexpr (CF::DECAY) ln0 = Lb[size_t(en) * LS];
            } else {
              ln_raw.load(Lb + size_t(en) * DK + c_ * RPL);
            }
          }
          next_ready = true;
        }
      }
      if (i < L) {
        if constexpr (DL == 1) {
#pragma unroll
          for (int x = 0; x < RPL; ++x) {
            const int pr = CF::cp_pos_run(c_, x);
            if constexpr (CF::NEEDS_C) ak = fmaf(kr[x], s_kf[pr], ak);
            aq = fmaf(kr[x], s_qf[pr], aq);
          }
          const float w = CF::DECAY ? dl_exp(s_lr[0] - lr_[0]) : 1.f;
          if constexpr (CF::NEEDS_C) ak *= w;
          aq *= w;
          if (stage) {
#pragma unroll
            for (int x = 0; x < RPL; ++x) {
              kt[CF::kt_off_run(c_, x) + e_] = w * kr[x];
            }
          }
        } else {
#pragma unroll 2
          for (int x = 0; x < RPL; ++x) {
            const int pr = CF::cp_pos_run(c_, x);
            const float wk = dl_exp(s_lr[pr] - lr_[x]) * kr[x];
            if constexpr (CF::NEEDS_C) ak = fmaf(wk, s_kf[pr], ak);
            aq = fmaf(wk, s_qf[pr], aq);
            if (stage)
              kt[CF::kt_off_run(c_, x) + e_] =
                  CF::BONUS ? dl_exp(s_lm[pr] - lr_[x]) * kr[x] : wk;
          }
        }
      } else if (stage) {
#pragma unroll
        for (int x = 0; x < RPL; ++x) {
          kt[CF::kt_off_run(c_, x) + e_] = 0.f;
        }
      }
      if constexpr (CF::NEEDS_C) ak = group_sum<CF::LPE>(ak);   // the delta-rule correction only
      aq = group_sum<CF::LPE>(aq);
      if (c_ == 0 && i < L) {
        if constexpr (CF::NEEDS_C) s_gk[i] = ak;
        s_gq[i] = aq;
      }
    }
    __syncthreads();
  }

  // ---- 6. base readouts from the registers + log replay, reduced over rows -------
  float4 cv = f4(0.f), ov = f4(0.f);
  if constexpr (CF::READS_OUT) {
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
      const int r = rg + NRG * j;
      const float4 sj = t[j].get();
      if constexpr (CF::NEEDS_C) cv = fma4(s_xk[r], sj, cv);
      ov = fma4(s_xq[r], sj, ov);
    }
    if constexpr (CF::HAS_LOG) {
      // Each log value row is read by exactly one row group; a merging workgroup keeps
      // the first chunk of them in LDS for the merge contraction.
      const bool stage_u = CF::MERGES_LOG && merging;
      const float4 up0 = up0_raw.get(), up1 = up1_raw.get();
      if (DL_PREFETCH_U && rg < L) {
        if constexpr (CF::NEEDS_C) cv = fma4(s_gk[rg], up0, cv);
        ov = fma4(s_gq[rg], up0, ov);
        if (stage_u && rg < CF::CH) s_u[rg * NCG + cg] = up0;
      }
      if (CF::TWO_PER_GROUP && DL_PREFETCH_U && rg + NRG < L) {
        if constexpr (CF::NEEDS_C) cv = fma4(s_gk[rg + NRG], up1, cv);
        ov = fma4(s_gq[rg + NRG], up1, ov);
        if (stage_u && rg + NRG < CF::CH) s_u[(rg + NRG) * NCG + cg] = up1;
      }
      constexpr int kFirstLater = DL_PREFETCH_U ? 2 * NRG : 0;   // first entry replayed here
      if constexpr (LONG && DL_REPLAY_PAIRS && kFirstLater >= CF::CH) {
        // The later values two rows of entries at a time, on a loop bound that is uniform
        // over the workgroup: both loads are issued before either is used.  Lanes past
        // the live length re-read entry L-1 (a finite value) with a zero coefficient, so
        // no load waits at the end of a per-lane condition.
        if constexpr (kLaterEarly) {              // the pair loaded before the first barrier
          if (kFirstLater < L) {
            const int i0 = kFirstLater + rg, i1 = kFirstLater + NRG + rg;
            const int j0 = min(i0, L - 1), j1 = min(i1, L - 1);
            const float4 u0 = up2_raw.get();
            if constexpr (CF::NEEDS_C) cv = fma4(i0 < L ? s_gk[j0] : 0.f, u0, cv);
            ov = fma4(i0 < L ? s_gq[j0] : 0.f, u0, ov);
            const float4 u1 = up3_raw.get();
            if constexpr (CF::NEEDS_C) cv = fma4(i1 < L ? s_gk[j1] : 0.f, u1, cv);
            ov = fma4(i1 < L ? s_gq[j1] : 0.f, u1, ov);
          }
        }
        for (int base = kFirstLater + (kLaterEarly ? 2 * NRG : 0); base < L; base += 2 * NRG) {
          const int i0 = base + rg, i1 = base + NRG + rg;
          const int j0 = min(i0, L - 1), j1 = min(i1, L - 1);
          Raw4<TU> r0, r1;                        // (bf16 values widened one at a time)
          r0.load(Ub + size_t(j0) * DV + 4 * cg);
          r1.load(Ub + size_t(j1) * DV + 4 * cg);
          const float4 u0 = r0.get();
          if constexpr (CF::NEEDS_C) cv = fma4(i0 < L ? s_gk[j0] : 0.f, u0, cv);
          ov = fma4(i0 < L ? s_gq[j0] : 0.f, u0, ov);
          const float4 u1 = r1.get();
          if constexpr (CF::NEEDS_C) cv = fma4(i1 < L ? s_gk[j1] : 0.f, u1, cv);
          ov = fma4(i1 < L ? s_gq[j1] : 0.f, u1, ov);
        }
      } else if constexpr (!(CF::CAP_ONE_PASS && DL_PREFETCH_U && 2 * NRG >= CF::CH)) {
        for (int i = rg + kFirstLater; i < L; i += NRG) {
          const float4 uv = ld4(Ub + size_t(i) * DV + 4 * cg);
          if constexpr (CF::NEEDS_C) cv = fma4(s_gk[i], uv, cv);
          ov = fma4(s_gq[i], uv, ov);
          if (stage_u && i < CF::CH) s_u[i * NCG + cg] = uv;
        }
      }
    }
    // Rows of one column group live in lanes NCG apart inside a wave, then across waves.
    static_assert(NCG == 16 || NCG == 32, "column groups fill one or two 16-lane rows");
    if constexpr (NCG == 16) {
      if constexpr (CF::NEEDS_C) cv = xor16_sum(cv);
      ov = xor16_sum(ov);
    }
    if constexpr (CF::NEEDS_C) cv = xor32_sum(cv);
    ov = xor32_sum(ov);
    if constexpr (CF::NW > 1) {
      const int w = tid / 64, lane = tid % 64;
      if (lane < NCG) {
        if constexpr (CF::NEEDS_C) st4(&s_red[w][0][4 * cg], cv);
        st4(&s_red[w][1][4 * cg], ov);
      }
      __syncthreads();
      cv = f4(0.f);
      ov = f4(0.f);
#pragma unroll
      for (int w2 = 0; w2 < CF::NW; ++w2) {
        if constexpr (CF::NEEDS_C) cv = cv + *reinterpret_cast<const float4*>(&s_red[w2][0][4 * cg]);
        ov = ov + *reinterpret_cast<const float4*>(&s_red[w2][1][4 * cg]);
      }
    }
  }

  // ---- 7. update factors and output ------------------------------------------------
  float4 bv = f4(0.f);
  if constexpr (CF::HAS_TOKEN) {
    const float4 vv = v_raw.get();
    float dot = 0.f;
#pragma unroll
    for (int w2 = 0; w2 < CF::NW; ++w2) dot += s_dotw[w2];
    if constexpr (CF::DELTA) {
      bv = beta * (vv - cv);                // b = beta (v - c)
      ov = fma4(dot, bv, ov);               // + (q.k) b : post-update readout
    } else {
      bv = vv;                              // b = v
      ov = fma4(dot, vv, ov);               // + (q.k) v, or the RWKV6 bonus (r.(u*k)) v
    }
  }
  if constexpr (CF::READS_OUT) {
    if (rg == 0) st4(p.o + th * DV + 4 * cg, ov);
  }
  if constexpr (MODE == M_READOUT) return;

  // ---- 8a. append (Eq. 5): L < C in STEP mode --------------------------------------
  if constexpr (MODE == M_STEP) {
    if (L < C) {
      const size_t ent = sh * size_t(C) + L;
      TU* Ud = static_cast<TU*>(p.u_log) + ent * DV + 4 * cg;
      if (rg == 0) {
        if constexpr (CF::DELTA) st4(reinterpret_cast<float*>(Ud), bv);
        else cp4(Ud, static_cast<const TIN*>(p.v) + th * DV + 4 * cg);
      }
      TIN* Kd = static_cast<TIN*>(p.k_log) + ent * DK;
      constexpr int KCH = DK * int(sizeof(TIN)) / 16;   // 16-byte chunks of one key row
      for (int x = tid; x < KCH; x += NT)
        reinterpret_cast<uint4*>(Kd)[x] = reinterpret_cast<const uint4*>(kin)[x];
      if constexpr (CF::DECAY) {
        for (int x = tid; x < DL; x += NT) {
          Lw[size_t(L) * LS + x] = s_lm[CF::cp_pos(x)];
        }
      }
      if (tid == 0) p.len[sh] = L + 1;
      return;
    }
  }

  // ---- 8b. materialise (Eq. 6 / Eq. 7 / Eq. 3) ---------------------------------------
  if constexpr (CF::CAN_MERGE) {
    float4 m[RPT];                                  // the materialised rows, fp32
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
      const int r = rg + NRG * j;
      m[j] = s_em[r] * t[j].get();
      if constexpr (CF::HAS_TOKEN) m[j] = fma4(s_kf[CF::cp_pos_group(rg, j)], bv, m[j]);
    }
    // The contraction on MFMA.  An fp32 state is stored straight from the
    // accumulators; a bf16 state is rounded from them.
    using MM = MfmaMerge<NCG, RPT>;
    constexpr bool kMfma = DL_MFMA_MERGE && (NCG == 32 || DL_MFMA_MERGE_64COL) &&
                           CF::MERGES_LOG && (sizeof(TS) == 4 || DL_MFMA_MERGE_BF16_STATE);
    static_assert(kMfma || !CF::KT_PADDED || !CF::MERGES_LOG,
                  "the VALU contraction reads K~ rows as float4: unpadded layout only");
    MM mm;
    if constexpr (CF::MERGES_LOG) {
      // Log values of chunk c >= 1 (chunk 0 was staged by the replay): UPT quads per
      // thread, loaded before the previous chunk's contraction where DL_U_EARLY.
      constexpr int UPT = CF::UPT;
      float4 ur[UPT];
      // Loaded unconditionally (entries past the live length re-read entry L-1) and
      // zeroed when staged: a load under a per-lane condition would be waited for at
      // once.
      Raw4<TU> ur_raw[UPT];
      int u_c0 = 0;
      auto load_u = [&](int c0) {
        u_c0 = c0;
#pragma unroll
        for (int k = 0; k < UPT; ++k) {
          const int x = tid + k * NT, ii = x / NCG, c4 = x % NCG;
          ur_raw[k].load(Ub + size_t(min(c0 + ii, L - 1)) * DV + 4 * c4);
        }
      };
      auto widen_u = [&]() {
#pragma unroll
        for (int k = 0; k < UPT; ++k) {
          const int ii = (tid + k * NT) / NCG;
          ur[k] = (u_c0 + ii < L) ? ur_raw[k].get() : f4(0.f);
        }
      };
      const int first_global = CF::REPLAYS ? CF::CH : 0;   // first chunk whose U is loaded here
      // A bf16 state leaves no registers for holding the next chunk's values.
      constexpr bool kUEarly = CF::U_EARLY && sizeof(TS) == 4;
      if (kUEarly && first_global < L) load_u(first_global);
      // Decayed keys of the chunks the coefficient passes did not stage: the same run
      // layout as the passes (entry e_ of the chunk, rows c_ RPL .. c_ RPL + RPL - 1, one
      // 16-byte key load and the snapshots of the run), loaded one chunk ahead where
      // kUEarly, and written to LDS chunk slot 0 (free once chunk 0 is contracted).
      RawRun<TIN, RPL> kg_raw{};
      RawRun<float, (DL == 1) ? 8 : RPL> lg_raw{};
      float lg0 = 0.f;
      auto load_kt = [&](int c0) {
        const int ig = min(c0 + e_, L - 1);       // lanes past L re-read entry L-1 (unused)
        kg_raw.load(Kb + size_t(ig) * DK + c_ * RPL);
        if constexpr (CF::DECAY) {
          if constexpr (DL == 1) lg0 = Lb[size_t(ig) * LS];
          else lg_raw.load(Lb + size_t(ig) * DK + c_ * RPL);
        }
      };
      auto store_kt = [&](int c0) {
        float kv[RPL];
        kg_raw.get(kv);
        // Entries past the live length (re-reads of entry L-1, finite) get a factor of
        // 0 rather than a branch, so that neither load is moved under a per-lane
        // condition and waited for there.
        const float live = c0 + e_ < L ? 1.f : 0.f;
        if constexpr (DL == 1) {
          const float w = live * (CF::DECAY ? dl_exp(s_lm[0] - lg0) : 1.f);
#pragma unroll
          for (int x = 0; x < RPL; ++x) s_kt[CF::kt_off_run(c_, x) + e_] = w * kv[x];
        } else {
          float lv[RPL];
          lg_raw.get(lv);
#pragma unroll
          for (int x = 0; x < RPL; ++x) {
            const float w = live * dl_exp(s_lm[CF::cp_pos_run(c_, x)] - lv[x]);
            s_kt[CF::kt_off_run(c_, x) + e_] = w * kv[x];
          }
        }
      };
      const int first_kt = CF::REPLAYS ? CF::NSTAGE * CF::CH : 0;   // first chunk staged here
      // Keys and snapshots one chunk ahead only where they fit beside the contraction's
      // registers at full occupancy (one log-decay per head, or small heads); a 128-row
      // per-key head loads them after the barrier (recently read: L2 hits).
      constexpr bool kKtEarly = kUEarly && CF::NSTAGE == 1 && (DL == 1 || RPT <= 8);
      if (kKtEarly && first_kt < L) load_kt(first_kt);
      // One chunk in the short STEP build (the MERGE kernel keeps the general loop: its
      // registers come out lower that way, 112 against 140 for a 128² per-key head).
      const int chunks_end = (CF::CAP_ONE_PASS && MODE == M_STEP) ? min(L, 1) : L;
      int a_off[MM::NMB];                           // LDS offset of this lane's A row, per block
      const int kq = (tid % 64) / NCG;              // the lane's entry within a K-step
      if constexpr (kMfma) {
#pragma unroll
        for (int mb = 0; mb < MM::NMB; ++mb)
          a_off[mb] = CF::kt_base(CF::kt_row(MM::row_of(tid / 64, mb, cg, NRG))) + kq;
        mm.from_rows(m);
      }
      for (int i0 = 0; i0 < chunks_end; i0 += CF::CH) {         // uniform trip count
        const int chunk = i0 / CF::CH;
        const int n = min(CF::CH, L - i0);
        const bool kt_staged = CF::REPLAYS && chunk < CF::NSTAGE;
        const float* const kt = s_kt + (kt_staged ? chunk : 0) * CF::KT_CHUNK;
        __syncthreads();                            // previous chunk consumed / chunk 0 visible
        if (!(CF::REPLAYS && chunk == 0)) {
          if (!kt_staged) {                         // K~_i[r] = e^(l'_r - Lam_i,r) K_i[r]
            if (!kKtEarly) load_kt(i0);
            store_kt(i0);
          }
          if (!kUEarly) load_u(i0);
          widen_u();
#pragma unroll
          for (int k = 0; k < UPT; ++k) s_u[tid + k * NT] = ur[k];
          if (kUEarly && i0 + CF::CH < L) {         // the next chunk, in flight meanwhile
            load_u(i0 + CF::CH);
            if (kKtEarly && i0 + CF::CH >= first_kt) load_kt(i0 + CF::CH);
          }
          __syncthreads();
        }
        if constexpr (kMfma) {
          // The operands of the whole chunk are read from LDS up front (the compiler
          // spreads the reads over the first MFMAs).  The chunk is zero-padded to CH
          // entries (both K~ and U); the second half is skipped when the chunk holds at
          // most CH / 2 entries.
          constexpr int NKS = CF::CH / MM::KS;
          float a[NKS][MM::NMB];
          float4 b[NKS];
#pragma unroll
          for (int k = 0; k < NKS; ++k) {
#pragma unroll
            for (int mb = 0; mb < MM::NMB; ++mb) a[k][mb] = kt[a_off[mb] + k * MM::KS];
            b[k] = s_u[(k * MM::KS + kq) * NCG + cg];
          }
#pragma unroll
          for (int k = 0; k < NKS / 2; ++k) mm.step(a[k], b[k]);
          if (n > CF::CH / 2) {
#pragma unroll
            for (int k = NKS / 2; k < NKS; ++k) mm.step(a[k], b[k]);
          }
          continue;
        }
#pragma unroll 1
        for (int ii = 0; ii < n; ii += 4) {          // zero-padded to a multiple of 4
          const float4 u0 = s_u[(ii + 0) * NCG + cg];
          const float4 u1 = s_u[(ii + 1) * NCG + cg];
          const float4 u2 = s_u[(ii + 2) * NCG + cg];
          const float4 u3 = s_u[(ii + 3) * NCG + cg];
#pragma unroll
          for (int j = 0; j < RPT; ++j) {
            const float4 k4 =
                *reinterpret_cast<const float4*>(&kt[CF::kt_base(CF::kt_row_group(rg, j)) + ii]);
            m[j] = fma4(k4.x, u0, m[j]);
            m[j] = fma4(k4.y, u1, m[j]);
            m[j] = fma4(k4.z, u2, m[j]);
            m[j] = fma4(k4.w, u3, m[j]);
          }
        }
      }
      if constexpr (kMfma) mm.drain();
    }
    // The live length is written before the rows, so that no register is written
    // behind the state stores.
    if constexpr (CF::HAS_LOG) {
      if (tid == 0) p.len[sh] = 0;                 // the cumulative log-decay restarts at 0
    }
    if constexpr (kMfma && sizeof(TS) == 4) {
      mm.store_rows(srs, toff, kRowBlock);
    } else if constexpr (kMfma) {
      mm.to_rows(m);
      StateQuad<TS>::store_rows(srs, toff, kRowBlock, m);
    } else {
      StateQuad<TS>::store_rows(srs, toff, kRowBlock, m);
    }
  }
}

}  // namespace dl
