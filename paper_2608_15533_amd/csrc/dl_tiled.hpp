// Value-tiled DeltaLog decode step (Sec. 3.3, the kernel ownership path): the state of
// one (slot, head) is split along the value dimension into NV tiles of dk x dv/NV, one
// workgroup per (token row, head, tile), in three stages:
//
//   replay_prep_kernel  (split replay only) once per (row, head): the key-side replay
//                       coefficients g_i(k), g_i(q) of every live entry, into an fp32
//                       scratch buffer [n, H, 2, C] owned by the caller;
//   tile_step_kernel    per value tile: stream the dense-base tile, replay the live log
//                       on the tile's columns (coefficients from the scratch buffer, or
//                       recomputed by every tile in the fused variant), write the
//                       output slice, then either append the tile's U_log[L] shard --
//                       tile 0 being the designated writer of the shared K_log[L] and
//                       Lam_log[L] -- or merge the tile's columns of the base;
//   finalize_kernel     once per (row, head): commit L (append: L + 1; merge: 0) after
//                       every tile has read it.
//
// The arithmetic per element is that of dl_kernel.hpp; the coefficient routine is shared
// by the prepare kernel and the fused tile kernel, so the split and fused variants give
// bit-identical results.  Only fp32 dense state is supported on this path.
#pragma once

#include "dl_kernel.hpp"

namespace dl {

constexpr int tile_threads(int dk, int dv, int nv) {
  return dk * (dv / nv) / 16 > 256 ? 256 : dk * (dv / nv) / 16;   // 4 rows x 4 columns per thread
}

template <int DK, int DV, int NV>
struct TileCfg {
  static constexpr int DVT = DV / NV;              // value columns per tile
  static constexpr int NCG = DVT / 4;              // float4 column groups
  static constexpr int NT = tile_threads(DK, DV, NV);
  static constexpr int NRG = NT / NCG;             // row groups
  static constexpr int RPT = DK / NRG;             // rows per thread
  static constexpr int NW = NT / 64;               // waves
  static constexpr int CH = 16;                    // log entries staged per merge chunk
  static constexpr int KTS = CH + 4;               // LDS row stride of a staged K~ chunk
  static_assert(DV % NV == 0 && DVT % 4 == 0, "value tiles of whole column quads");
  static_assert(NT % 64 == 0 && NT >= DK, "whole waves; one thread per key row in the prologue");
  static_assert(64 % NCG == 0 && NT == NCG * NRG && DK == NRG * RPT, "thread layout");
};

// Replay coefficients of the live entries for the readout vectors k and q (LDS s_kf,
// s_qf) at readout log-decay s_lr:  g_i(x) = sum_r e^(s_lr[r] - Lam_i,r) x_r K_i,r.
// Every entry is reduced by 16 lanes of dk/16 rows each, whatever the workgroup size, so
// every caller produces the same bits.  Results go to gk[i], gq[i] (i < L).
template <int OP, int DK, int NT, typename TIN, typename Sink>
__device__ __forceinline__ void replay_coefficients(const TIN* Kb, const float* Lb, size_t LS,
                                                    int L, const float* s_kf, const float* s_qf,
                                                    const float* s_lr, Sink sink) {
  using TR = OpTraits<OP>;
  constexpr int DL = TR::PER_KEY ? DK : 1;
  constexpr int LPE = 16, EPP = NT / LPE, RPL = DK / LPE;
  const int tid = threadIdx.x;
  const int e_ = tid / LPE, c_ = tid % LPE;
  for (int i0 = 0; i0 < L; i0 += EPP) {           // uniform trip count
    const int i = i0 + e_;
    float ak = 0.f, aq = 0.f;
    if (i < L) {
#pragma unroll
      for (int x = 0; x < RPL; ++x) {
        const int r = c_ * RPL + x;
        float kr = ld1(Kb + size_t(i) * DK + r);
        if constexpr (TR::DECAY && DL != 1) kr *= dl_exp(s_lr[r] - Lb[size_t(i) * LS + r]);
        ak = fmaf(kr, s_kf[r], ak);
        aq = fmaf(kr, s_qf[r], aq);
      }
      if constexpr (TR::DECAY && DL == 1) {
        const float w = dl_exp(s_lr[0] - Lb[size_t(i) * LS]);
        ak *= w;
        aq *= w;
      }
    }
#pragma unroll
    for (int m = LPE / 2; m >= 1; m >>= 1) {
      ak += shfl_xor(ak, m);
      aq += shfl_xor(aq, m);
    }
    if (c_ == 0 && i < L) sink(i, ak, aq);
  }
}

// Cumulative log-decay of a (slot, head) at live length L, element x: the newest
// snapshot, 0 with an empty log (it is not stored; see the step kernel).
template <int OP, int DK>
__device__ __forceinline__ float cumulative_decay(const KParams& p, size_t sh, int L, int x) {
  using TR = OpTraits<OP>;
  if constexpr (!TR::DECAY) {
    return 0.f;
  } else if constexpr (!TR::PER_KEY) {
    const int slot = int(sh / size_t(p.H)), h = int(sh % size_t(p.H));
    return L > 0 ? scalar_ld(lam_log_base<1>(p, slot, h) + size_t(L - 1) * lam_log_stride<1>(p))
                 : 0.f;
  } else {
    const int slot = int(sh / size_t(p.H)), h = int(sh % size_t(p.H));
    return L > 0 ? lam_log_base<DK>(p, slot, h)[size_t(L - 1) * DK + x] : 0.f;
  }
}

// Live length of a (slot, head) if the row's slot and the length are valid, else -1.
__device__ __forceinline__ int tiled_row(const KParams& p, int row, int h, size_t& sh) {
  const int slot = p.slots ? p.slots[row] : row;
  if (slot < 0 || slot >= p.B) return -1;
  sh = size_t(slot) * p.H + h;
  const int L = p.len[sh];
  return (L < 0 || L > p.C) ? -1 : L;
}

// ------------------------------------------------------------------ ReplayPrep
template <int OP, int DK, typename TIN>
__global__ __launch_bounds__(256) void replay_prep_kernel(KParams p, float* coef) {
  using TR = OpTraits<OP>;
  constexpr int DL = TR::PER_KEY ? DK : 1;
  __shared__ float s_kf[DK], s_qf[DK], s_lr[DL];
  const int tid = threadIdx.x;
  const int row = int(blockIdx.x) / p.H, h = int(blockIdx.x) - row * p.H;
  size_t sh = 0;
  const int L = tiled_row(p, row, h, sh);          // uniform per workgroup
  if (L <= 0) return;                              // nothing live (or invalid: reported by the tiles)
  const size_t th = size_t(row) * p.H + h;
  if (tid < DK) {
    s_kf[tid] = to_f32(static_cast<const TIN*>(p.k)[th * DK + tid]);
    s_qf[tid] = to_f32(static_cast<const TIN*>(p.q)[th * DK + tid]);
  }
  if (tid < DL) {
    float lr = 0.f;
    if constexpr (TR::DECAY) {
      const float ell = cumulative_decay<OP, DK>(p, sh, L, tid);
      lr = TR::BONUS ? ell : ell + p.lam[th * DL + tid];   // readout decay, as in the step
    }
    s_lr[tid] = lr;
  }
  __syncthreads();
  const int C = p.C;
  float* out = coef + th * 2 * size_t(C);
  const int slot = int(sh / size_t(p.H));
  replay_coefficients<OP, DK, 256>(static_cast<const TIN*>(p.k_log) + sh * size_t(C) * DK,
                                   TR::DECAY ? lam_log_base<DL>(p, slot, h) : nullptr,
                                   lam_log_stride<DL>(p), L,
                                   s_kf, s_qf, s_lr, [&](int i, float gk, float gq) {
                                     out[i] = gk;
                                     out[C + i] = gq;
                                   });
}

// ------------------------------------------------------------------ tile step
template <int OP, int DK, int DV, int NV, bool SPLIT, typename TIN>
__global__ __launch_bounds__(tile_threads(DK, DV, NV))
void tile_step_kernel(KParams p, const float* __restrict__ coef) {
  using TC = TileCfg<DK, DV, NV>;
  using TR = OpTraits<OP>;
  using TU = typename UType<OP, TIN>::type;
  constexpr int NT = TC::NT, NCG = TC::NCG, NRG = TC::NRG, RPT = TC::RPT, DVT = TC::DVT;
  constexpr int CH = TC::CH, KTS = TC::KTS;
  constexpr int DL = TR::PER_KEY ? DK : 1;
  constexpr bool NEEDS_C = TR::DELTA;

  __shared__ float s_kf[DK], s_qf[DK], s_xk[DK], s_xq[DK], s_em[DK];
  __shared__ float s_lr[DL], s_lm[DL];
  __shared__ float s_gk[DL_MAX_MERGE_INTERVAL], s_gq[DL_MAX_MERGE_INTERVAL];
  __shared__ __align__(16) float s_red[TC::NW][2][DVT];
  __shared__ float s_dotw[TC::NW];
  __shared__ __align__(16) float s_kt[DK * KTS];   // K~ chunk [DK][KTS] (merge)
  __shared__ float4 s_u[CH * NCG];                 // U chunk  [CH][NCG] (merge)

  const int tid = threadIdx.x;
  const int H = p.H;
  // Chunks of consecutive (row, head, tile) triples are dealt to the XCDs in turn (as in
  // the untiled kernel); a head's tiles sit in one chunk and share one L2.
  uint32_t lin = blockIdx.x;
  const uint32_t nblk = gridDim.x;
  if constexpr (kXcdChunk > 0) {
    const uint32_t full = nblk - nblk % (kXcds * kXcdChunk);
    if (lin < full) {
      const uint32_t x = lin % kXcds, jj = lin / kXcds;
      lin = ((jj / kXcdChunk) * kXcds + x) * kXcdChunk + jj % kXcdChunk;
    }
  }
  const int j = int(lin % NV);                     // value tile
  const int rh = int(lin / NV);
  const int row = rh / H, h = rh - row * H;
  const int slot = p.slots ? p.slots[row] : row;
  if (slot < 0 || slot >= p.B) {
    if (tid == 0 && p.err) atomicOr(p.err, 1);
    return;
  }
  const size_t sh = size_t(slot) * H + h;
  const size_t th = size_t(row) * H + h;
  const int C = p.C;
  const int L = p.len[sh];
  if (L < 0 || L > C) {
    if (tid == 0 && p.err) atomicOr(p.err, 2);
    return;
  }

  const int cg = tid % NCG, rg = tid / NCG;
  const int c0 = j * DVT + 4 * cg;                 // this thread's first value column
  const TIN* kin = static_cast<const TIN*>(p.k) + th * DK;
  const TIN* qin = static_cast<const TIN*>(p.q) + th * DK;

  // ---- tile slice (rows rg + NRG * i, columns c0 .. c0 + 3) --------------------------
  float* const Sh = static_cast<float*>(p.S) + sh * size_t(DK) * DV;
  const auto srs = state_rsrc(Sh, DK * DV * sizeof(float));
  const uint32_t toff = uint32_t(rg * DV + c0) * sizeof(float);
  constexpr uint32_t kRowBlock = NRG * DV * sizeof(float);
  StateQuad<float> t[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) t[i].load(srs, toff, i * kRowBlock);

  // ---- prologue: per-row decay factors, token vectors, the token dot product --------
  float kf = 0.f, qf = 0.f, uf = 0.f;
  if (tid < DK) {
    kf = to_f32(kin[tid]);
    qf = to_f32(qin[tid]);
    if constexpr (TR::BONUS) uf = p.u[size_t(h) * DK + tid];
    float ell = 0.f, lam = 0.f;
    if constexpr (TR::DECAY) {
      ell = cumulative_decay<OP, DK>(p, sh, L, DL == 1 ? 0 : tid);
      lam = p.lam[th * DL + (DL == 1 ? 0 : tid)];
    }
    const float lm = ell + lam;
    const float lr = TR::BONUS ? ell : lm;
    const float er = dl_exp(lr);
    s_kf[tid] = kf;
    s_qf[tid] = qf;
    s_xk[tid] = er * kf;
    s_xq[tid] = er * qf;
    s_em[tid] = dl_exp(lm);
    if (tid < DL) {
      s_lr[tid] = lr;
      s_lm[tid] = lm;
    }
  }
  {
    float d = tid < DK ? (TR::BONUS ? qf * uf * kf : qf * kf) : 0.f;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) d += shfl_xor(d, m);
    if ((tid & 63) == 0) s_dotw[tid >> 6] = d;
  }
  const float4 vv = ld4(static_cast<const TIN*>(p.v) + th * DV + c0);
  float beta = 0.f;
  if constexpr (TR::DELTA) beta = p.beta[th];
  const TIN* Kb = static_cast<const TIN*>(p.k_log) + sh * size_t(C) * DK;
  float* const Lw = TR::DECAY ? lam_log_base<DL>(p, slot, h) : nullptr;
  const float* Lb = Lw;
  const size_t LS = lam_log_stride<DL>(p);
  const TU* Ub = static_cast<const TU*>(p.u_log) + sh * size_t(C) * DV;
  __syncthreads();

  // ---- replay coefficients ------------------------------------------------------------
  if constexpr (SPLIT) {
    const float* cp = coef + th * 2 * size_t(C);
    for (int i = tid; i < L; i += NT) {
      s_gk[i] = cp[i];
      s_gq[i] = cp[C + i];
    }
  } else {
    replay_coefficients<OP, DK, NT>(Kb, Lb, LS, L, s_kf, s_qf, s_lr, [&](int i, float gk, float gq) {
      s_gk[i] = gk;
      s_gq[i] = gq;
    });
  }
  __syncthreads();

  // ---- base readouts of the tile's columns plus log replay, reduced over rows -------
  float4 cv = f4(0.f), ov = f4(0.f);
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int r = rg + NRG * i;
    const float4 sj = t[i].get();
    if constexpr (NEEDS_C) cv = fma4(s_xk[r], sj, cv);
    ov = fma4(s_xq[r], sj, ov);
  }
  for (int i = rg; i < L; i += NRG) {
    const float4 uv = ld4(Ub + size_t(i) * DV + c0);
    if constexpr (NEEDS_C) cv = fma4(s_gk[i], uv, cv);
    ov = fma4(s_gq[i], uv, ov);
  }
#pragma unroll
  for (int m = NCG; m < 64; m <<= 1) {
    if constexpr (NEEDS_C) {
      cv.x += shfl_xor(cv.x, m); cv.y += shfl_xor(cv.y, m);
      cv.z += shfl_xor(cv.z, m); cv.w += shfl_xor(cv.w, m);
    }
    ov.x += shfl_xor(ov.x, m); ov.y += shfl_xor(ov.y, m);
    ov.z += shfl_xor(ov.z, m); ov.w += shfl_xor(ov.w, m);
  }
  if constexpr (TC::NW > 1) {
    const int w = tid / 64, lane = tid % 64;
    if (lane < NCG) {
      if constexpr (NEEDS_C) st4(&s_red[w][0][4 * cg], cv);
      st4(&s_red[w][1][4 * cg], ov);
    }
    __syncthreads();
    cv = f4(0.f);
    ov = f4(0.f);
#pragma unroll
    for (int w2 = 0; w2 < TC::NW; ++w2) {
      if constexpr (NEEDS_C) cv = cv + *reinterpret_cast<const float4*>(&s_red[w2][0][4 * cg]);
      ov = ov + *reinterpret_cast<const float4*>(&s_red[w2][1][4 * cg]);
    }
  }

  // ---- update factors and the output slice --------------------------------------------
  float dot = 0.f;
#pragma unroll
  for (int w2 = 0; w2 < TC::NW; ++w2) dot += s_dotw[w2];
  const float4 bv = TR::DELTA ? beta * (vv - cv) : vv;
  ov = fma4(dot, bv, ov);
  if (rg == 0) st4(p.o + th * DV + c0, ov);

  // ---- append (Eq. 5): the tile's U_log shard; tile 0 writes the shared entries ------
  if (L < C) {
    const size_t ent = sh * size_t(C) + L;
    if (rg == 0) {
      TU* Ud = static_cast<TU*>(p.u_log) + ent * DV + c0;
      if constexpr (TR::DELTA) st4(reinterpret_cast<float*>(Ud), bv);
      else cp4(Ud, static_cast<const TIN*>(p.v) + th * DV + c0);
    }
    if (j == 0) {
      TIN* Kd = static_cast<TIN*>(p.k_log) + ent * DK;
      constexpr int KCH = DK * int(sizeof(TIN)) / 16;
      for (int x = tid; x < KCH; x += NT)
        reinterpret_cast<uint4*>(Kd)[x] = reinterpret_cast<const uint4*>(kin)[x];
      if constexpr (TR::DECAY)
        for (int x = tid; x < DL; x += NT) Lw[size_t(L) * LS + x] = s_lm[x];
    }
    return;                                        // L: finalize_kernel
  }

  // ---- merge (Eq. 6) of the tile's columns -------------------------------------------
  float4 m[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int r = rg + NRG * i;
    m[i] = fma4(s_kf[r], bv, s_em[r] * t[i].get());
  }
  for (int i0 = 0; i0 < L; i0 += CH) {              // uniform trip count
    const int n = min(CH, L - i0);
    __syncthreads();                                // the previous chunk is consumed
    for (int x = tid; x < DK * CH; x += NT) {
      const int r = x % DK, ii = x / DK;
      float val = 0.f;
      if (ii < n) {
        const int i = i0 + ii;
        val = ld1(Kb + size_t(i) * DK + r);
        if constexpr (TR::DECAY)
          val *= dl_exp(s_lm[DL == 1 ? 0 : r] - Lb[size_t(i) * LS + (DL == 1 ? 0 : r)]);
      }
      s_kt[r * KTS + ii] = val;                     // K~_i[r] = e^(l'_r - Lam_i,r) K_i[r]
    }
    for (int x = tid; x < CH * NCG; x += NT) {
      const int ii = x / NCG, c4 = x % NCG;
      s_u[x] = ii < n ? ld4(Ub + size_t(i0 + ii) * DV + j * DVT + 4 * c4) : f4(0.f);
    }
    __syncthreads();
    for (int ii = 0; ii < n; ii += 4) {             // zero-padded to a multiple of 4
      const float4 u0 = s_u[(ii + 0) * NCG + cg];
      const float4 u1 = s_u[(ii + 1) * NCG + cg];
      const float4 u2 = s_u[(ii + 2) * NCG + cg];
      const float4 u3 = s_u[(ii + 3) * NCG + cg];
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        const int r = rg + NRG * i;
        const float4 kt = *reinterpret_cast<const float4*>(&s_kt[r * KTS + ii]);
        m[i] = fma4(kt.x, u0, m[i]);
        m[i] = fma4(kt.y, u1, m[i]);
        m[i] = fma4(kt.z, u2, m[i]);
        m[i] = fma4(kt.w, u3, m[i]);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i) StateQuad<float>::store(srs, toff, i * kRowBlock, m[i]);
}

// ------------------------------------------------------------------ Finalize
// One wave per (row, head): append -> L + 1; merge -> L = 0.  The cumulative log-decay
// follows from Lam_log[L] (written by tile 0) and L, so L is all there is to commit.
template <int OP, int DK>
__global__ __launch_bounds__(64) void finalize_kernel(KParams p) {
  const int tid = threadIdx.x;
  const int row = int(blockIdx.x) / p.H, h = int(blockIdx.x) - row * p.H;
  size_t sh = 0;
  const int L = tiled_row(p, row, h, sh);           // every lane reads L before lane 0 writes it
  if (L < 0) return;                                // invalid: reported by the tiles
  if (L < p.C) {
    if (tid == 0) p.len[sh] = L + 1;
  } else {
    if (tid == 0) p.len[sh] = 0;
  }
}

// ------------------------------------------------------------------ dispatch
template <int OP, int DK, int DV, int NV, bool SPLIT, typename TIN>
hipError_t launch_tiled_one(const KParams& p, const float* coef, hipStream_t s) {
  using TC = TileCfg<DK, DV, NV>;
  KParams arg = p;
  const float* carg = coef;
  void* args[] = {&arg, &carg};
  return hipLaunchKernel(reinterpret_cast<const void*>(&tile_step_kernel<OP, DK, DV, NV, SPLIT, TIN>),
                         dim3(unsigned(p.n) * unsigned(p.H) * NV), dim3(TC::NT), args, 0, s);
}

template <int OP, int DK, typename TIN>
hipError_t launch_prep(const KParams& p, float* coef, hipStream_t s) {
  KParams arg = p;
  float* carg = coef;
  void* args[] = {&arg, &carg};
  return hipLaunchKernel(reinterpret_cast<const void*>(&replay_prep_kernel<OP, DK, TIN>),
                         dim3(unsigned(p.n) * unsigned(p.H)), dim3(256), args, 0, s);
}

template <int OP, int DK>
hipError_t launch_finalize(const KParams& p, hipStream_t s) {
  KParams arg = p;
  void* args[] = {&arg};
  return hipLaunchKernel(reinterpret_cast<const void*>(&finalize_kernel<OP, DK>),
                         dim3(unsigned(p.n) * unsigned(p.H)), dim3(64), args, 0, s);
}

template <int OP, int DK, int DV, typename TIN>
hipError_t launch_tiled_shape(int nv, bool split, const KParams& p, float* coef, hipStream_t s) {
  hipError_t e = hipSuccess;
  if (split && p.C > 0) e = launch_prep<OP, DK, TIN>(p, coef, s);
  if (e != hipSuccess) return e;
  if (nv == 2) e = split ? launch_tiled_one<OP, DK, DV, 2, true, TIN>(p, coef, s)
                         : launch_tiled_one<OP, DK, DV, 2, false, TIN>(p, coef, s);
  else if (nv == 4) e = split ? launch_tiled_one<OP, DK, DV, 4, true, TIN>(p, coef, s)
                              : launch_tiled_one<OP, DK, DV, 4, false, TIN>(p, coef, s);
  else return hipErrorInvalidValue;
  if (e != hipSuccess) return e;
  return launch_finalize<OP, DK>(p, s);
}

template <int OP, typename TIN>
hipError_t launch_tiled_in(int dk, int dv, int nv, bool split, const KParams& p, float* coef,
                           hipStream_t s) {
  if (dk == 128 && dv == 128) return launch_tiled_shape<OP, 128, 128, TIN>(nv, split, p, coef, s);
  if (dk == 64 && dv == 64) return launch_tiled_shape<OP, 64, 64, TIN>(nv, split, p, coef, s);
  if (dk == 64 && dv == 128) return launch_tiled_shape<OP, 64, 128, TIN>(nv, split, p, coef, s);
  if (dk == 128 && dv == 64) return launch_tiled_shape<OP, 128, 64, TIN>(nv, split, p, coef, s);
  return hipErrorInvalidValue;
}

template <int OP>
hipError_t launch_tiled_op(int dk, int dv, bool bf16, int nv, bool split, const KParams& p,
                           float* coef, hipStream_t s) {
  return bf16 ? launch_tiled_in<OP, uint16_t>(dk, dv, nv, split, p, coef, s)
              : launch_tiled_in<OP, float>(dk, dv, nv, split, p, coef, s);
}

}  // namespace dl
