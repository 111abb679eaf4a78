// Template dispatch from runtime (mode, dk, dv, dtype) to a kernel instantiation.
#pragma once

#include "dl_kernel.hpp"

namespace dl {

template <int OP, int DK, int DV, int MODE, typename TIN, typename TS, bool LONG>
hipError_t launch_build(const KParams& p, hipStream_t s) {
  using CF = Cfg<OP, DK, DV, MODE, LONG>;
  const dim3 grid(unsigned(p.n) * unsigned(p.H));
  const dim3 block(CF::NT);
  KParams arg = p;
  void* args[] = {&arg};
  return hipLaunchKernel(
      reinterpret_cast<const void*>(&deltalog_kernel<OP, DK, DV, MODE, TIN, TS, LONG>), grid,
      block, args, 0, s);
}

// The STEP and MERGE kernels have a second build for logs longer than one coefficient
// pass (capacity C > 16), picked from the descriptor's merge interval.
template <int OP, int DK, int DV, int MODE, typename TIN, typename TS>
hipError_t launch_one(const KParams& p, hipStream_t s) {
  constexpr bool kHasLong = MODE == M_STEP || MODE == M_MERGE;
  if (kHasLong && p.C > Cfg<OP, DK, DV, MODE>::CH)
    return launch_build<OP, DK, DV, MODE, TIN, TS, kHasLong>(p, s);
  return launch_build<OP, DK, DV, MODE, TIN, TS, false>(p, s);
}

template <int OP, int DK, int DV, typename TIN, typename TS>
hipError_t launch_mode(int mode, const KParams& p, hipStream_t s) {
  switch (mode) {
    case M_EAGER: return launch_one<OP, DK, DV, M_EAGER, TIN, TS>(p, s);
    case M_STEP: return launch_one<OP, DK, DV, M_STEP, TIN, TS>(p, s);
    case M_MERGE: return launch_one<OP, DK, DV, M_MERGE, TIN, TS>(p, s);
    case M_FLUSH: return launch_one<OP, DK, DV, M_FLUSH, TIN, TS>(p, s);
    case M_READOUT: return launch_one<OP, DK, DV, M_READOUT, TIN, TS>(p, s);
  }
  return hipErrorInvalidValue;
}

template <int OP, typename TIN, typename TS>
hipError_t launch_shape(int mode, int dk, int dv, const KParams& p, hipStream_t s) {
  if (dk == 128 && dv == 128) return launch_mode<OP, 128, 128, TIN, TS>(mode, p, s);
  if (dk == 64 && dv == 64) return launch_mode<OP, 64, 64, TIN, TS>(mode, p, s);
  if (dk == 64 && dv == 128) return launch_mode<OP, 64, 128, TIN, TS>(mode, p, s);
  if (dk == 128 && dv == 64) return launch_mode<OP, 128, 64, TIN, TS>(mode, p, s);
  return hipErrorInvalidValue;
}

template <int OP, typename TS>
hipError_t launch_in(int mode, int dk, int dv, bool bf16, const KParams& p, hipStream_t s) {
  return bf16 ? launch_shape<OP, uint16_t, TS>(mode, dk, dv, p, s)
              : launch_shape<OP, float, TS>(mode, dk, dv, p, s);
}

template <int OP>
hipError_t launch_op(int mode, int dk, int dv, bool bf16, bool state_bf16, const KParams& p,
                     hipStream_t s) {
  return state_bf16 ? launch_in<OP, uint16_t>(mode, dk, dv, bf16, p, s)
                    : launch_in<OP, float>(mode, dk, dv, bf16, p, s);
}

}  // namespace dl
