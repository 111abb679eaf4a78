/*
 * Pure-C use of the DeltaLog C ABI: no torch, no C++, only include/deltalog.h and the
 * HIP runtime API.  Built into a small shared library next to this file (the tests load
 * it with ctypes and call dl_example_run), it allocates every buffer with hipMalloc,
 * steps a GDN layer through three merge cycles with dl_append_step, steps a dense copy
 * of the same state with dl_eager_step, and compares the two on every output row and,
 * after a flush (dl_merge without a token), on the state itself.
 *
 * In exact arithmetic the two paths give the same outputs and state (the invariant of
 * Eq. 7); in fp32 they differ by rounding only, so the relative Frobenius error of each
 * step's outputs and of the flushed state must stay below 1e-4.
 *
 * Return value: 0 on success; a negative dl_status from the library; 100 + the HIP
 * error code for a failed runtime call; 1 for an error word set on the device; 2 for a
 * mismatch above the bar.  *max_rel_err receives the largest error seen.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "deltalog.h"

enum { B = 4, H = 2, DK = 64, DV = 64, M = 4, STEPS = 3 * M + 1 };

/* 32-bit linear congruential generator (Numerical Recipes constants), uniform in [-1, 1) */
static uint32_t lcg_state = 12345u;
static float urand(void) {
  lcg_state = lcg_state * 1664525u + 1013904223u;
  return (float)((double)(lcg_state >> 8) / 8388608.0 - 1.0);
}

static void fill_unit_rows(float* x, int rows, int d) {
  for (int r = 0; r < rows; ++r) {
    double n = 0.0;
    for (int i = 0; i < d; ++i) {
      x[r * d + i] = urand();
      n += (double)x[r * d + i] * x[r * d + i];
    }
    const float s = (float)(1.0 / sqrt(n));
    for (int i = 0; i < d; ++i) x[r * d + i] *= s;
  }
}

static double rel_err(const float* a, const float* b, size_t n) {
  double num = 0.0, den = 0.0;
  for (size_t i = 0; i < n; ++i) {
    const double d = (double)a[i] - (double)b[i];
    num += d * d;
    den += (double)b[i] * b[i];
  }
  return sqrt(num / (den > 0.0 ? den : 1.0));
}

#define HIP_TRY(call)                                  \
  do {                                                 \
    hipError_t e_ = (call);                            \
    if (e_ != hipSuccess) { rc = 100 + (int)e_; goto done; } \
  } while (0)
#define DL_TRY(call)                                   \
  do {                                                 \
    int s_ = (call);                                   \
    if (s_ != DL_OK) { rc = s_; goto done; }           \
  } while (0)

int dl_example_run(double* max_rel_err) {
  const int C = M - 1;
  const size_t nS = (size_t)B * H * DK * DV, nq = (size_t)B * H * DK, nv = (size_t)B * H * DV;
  const size_t nbh = (size_t)B * H;
  int rc = 0;
  double worst = 0.0;
  float *hS = NULL, *hq = NULL, *hk = NULL, *hv = NULL, *hlam = NULL, *hbeta = NULL;
  float *ho = NULL, *hoe = NULL, *hS2 = NULL;
  float *S = NULL, *Se = NULL, *u_log = NULL, *lam_log = NULL;
  float *q = NULL, *k = NULL, *v = NULL, *lam = NULL, *beta = NULL, *o = NULL, *oe = NULL;
  float *k_log = NULL;
  int32_t *len = NULL, *err = NULL, herr = 0;

  hS = malloc(nS * 4); hS2 = malloc(nS * 4);
  hq = malloc(nq * 4); hk = malloc(nq * 4); hv = malloc(nv * 4);
  hlam = malloc(nbh * 4); hbeta = malloc(nbh * 4); ho = malloc(nv * 4); hoe = malloc(nv * 4);
  if (!hS || !hS2 || !hq || !hk || !hv || !hlam || !hbeta || !ho || !hoe) { rc = 3; goto done; }
  for (size_t i = 0; i < nS; ++i) hS[i] = 0.02f * urand();

  HIP_TRY(hipMalloc((void**)&S, nS * 4));
  HIP_TRY(hipMalloc((void**)&Se, nS * 4));
  HIP_TRY(hipMalloc((void**)&k_log, nbh * C * DK * 4));
  HIP_TRY(hipMalloc((void**)&u_log, nbh * C * DV * 4));
  HIP_TRY(hipMalloc((void**)&lam_log, nbh * C * 4));          /* dl = 1: [B, C, H] */
  HIP_TRY(hipMalloc((void**)&len, nbh * 4));
  HIP_TRY(hipMalloc((void**)&err, 4));
  HIP_TRY(hipMalloc((void**)&q, nq * 4));
  HIP_TRY(hipMalloc((void**)&k, nq * 4));
  HIP_TRY(hipMalloc((void**)&v, nv * 4));
  HIP_TRY(hipMalloc((void**)&lam, nbh * 4));
  HIP_TRY(hipMalloc((void**)&beta, nbh * 4));
  HIP_TRY(hipMalloc((void**)&o, nv * 4));
  HIP_TRY(hipMalloc((void**)&oe, nv * 4));
  HIP_TRY(hipMemcpy(S, hS, nS * 4, hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(Se, hS, nS * 4, hipMemcpyHostToDevice));
  HIP_TRY(hipMemset(len, 0, nbh * 4));                        /* empty log: L = 0 */
  HIP_TRY(hipMemset(err, 0, 4));

  {
    dl_desc d;
    memset(&d, 0, sizeof d);
    d.abi_version = DL_ABI_VERSION;
    d.op = DL_OP_GDN;
    d.num_slots = B;
    d.heads = H;
    d.dk = DK;
    d.dv = DV;
    d.merge_interval = M;
    d.in_dtype = DL_F32;
    d.u_log_dtype = DL_F32;
    d.state_dtype = DL_F32;
    dl_state st = {S, k_log, u_log, lam_log, len, err};
    dl_token tok = {q, k, v, beta, lam, NULL};

    for (int t = 0; t < STEPS; ++t) {
      fill_unit_rows(hq, B * H, DK);
      fill_unit_rows(hk, B * H, DK);
      for (size_t i = 0; i < nv; ++i) hv[i] = urand();
      for (size_t i = 0; i < nbh; ++i) {
        const float g = 3.0f + 0.5f * urand();                 /* log sigmoid(g) < 0 */
        hlam[i] = -(float)log1p(exp(-(double)g));
        hbeta[i] = (float)(1.0 / (1.0 + exp(-(double)urand())));
      }
      HIP_TRY(hipMemcpy(q, hq, nq * 4, hipMemcpyHostToDevice));
      HIP_TRY(hipMemcpy(k, hk, nq * 4, hipMemcpyHostToDevice));
      HIP_TRY(hipMemcpy(v, hv, nv * 4, hipMemcpyHostToDevice));
      HIP_TRY(hipMemcpy(lam, hlam, nbh * 4, hipMemcpyHostToDevice));
      HIP_TRY(hipMemcpy(beta, hbeta, nbh * 4, hipMemcpyHostToDevice));
      DL_TRY(dl_append_step(&d, &st, &tok, o, NULL, B, NULL));
      DL_TRY(dl_eager_step(&d, Se, &tok, oe, NULL, B, NULL));
      HIP_TRY(hipDeviceSynchronize());
      HIP_TRY(hipMemcpy(ho, o, nv * 4, hipMemcpyDeviceToHost));
      HIP_TRY(hipMemcpy(hoe, oe, nv * 4, hipMemcpyDeviceToHost));
      const double e = rel_err(ho, hoe, nv);
      if (e > worst) worst = e;
    }
    DL_TRY(dl_merge(&d, &st, NULL, NULL, NULL, B, NULL));     /* flush: S becomes Eq. 7 */
    HIP_TRY(hipDeviceSynchronize());
    HIP_TRY(hipMemcpy(hS, S, nS * 4, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(hS2, Se, nS * 4, hipMemcpyDeviceToHost));
    {
      const double e = rel_err(hS, hS2, nS);
      if (e > worst) worst = e;
    }
    HIP_TRY(hipMemcpy(&herr, err, 4, hipMemcpyDeviceToHost));
    if (herr != 0) rc = 1;
    else if (!(worst <= 1e-4)) rc = 2;
  }

done:
  if (max_rel_err) *max_rel_err = worst;
  hipFree(S); hipFree(Se); hipFree(k_log); hipFree(u_log); hipFree(lam_log);
  hipFree(len); hipFree(err); hipFree(q); hipFree(k); hipFree(v); hipFree(lam);
  hipFree(beta); hipFree(o); hipFree(oe);
  free(hS); free(hS2); free(hq); free(hk); free(hv); free(hlam); free(hbeta); free(ho);
  free(hoe);
  return rc;
}
