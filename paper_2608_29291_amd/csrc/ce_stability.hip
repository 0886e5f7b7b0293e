// Drop-set stability signals of the routing decisions (paper section 3.4, UCS
// operators (3) diffusion-head cache reuse and (4) denoising-step early exit).
//
// For each sequence, the drop set D_t of a timestep is its routable tokens
// (not always-kept) with token_pos < 0. Between two timesteps:
//   J    = |D_t n D_ref| / |D_t u D_ref|          (Eq. 10; 1 for an empty union)
//   J_rd = E[J] for two independent uniformly random subsets of the routable
//          tokens with the same sizes (hypergeometric overlap)
//   RDA  = (J - J_rd) / (1 - J_rd)                 (Eq. 11; 1 when J_rd = 1)
//
// One workgroup per sequence: the four counts (routable, dropped at t, dropped
// at t_ref, dropped at both) are reduced over the block, J is formed from the
// integers and J_rd in fp64 by the whole block. The overlap X of the two random
// sets is hypergeometric with mean E = a b / n; by Hoeffding's inequality for
// sampling without replacement, P(|X - E| >= s) <= 2 exp(-2 s^2 / m) with
// m = min(a, b), so the window E +- sqrt(48 m) misses less than 1e-41 of the
// mass. Each thread takes a contiguous run of that window: the probability at
// the run's point nearest the mode comes from lgamma, the others from the
// exact ratio of consecutive terms walking away from it (so the terms only
// shrink and an underflow to zero is harmless). The per-thread sums are then
// added in a fixed order.
#include "ce_device.hpp"
#include "ce_launch.hpp"
#include "ce_router.h"

namespace ce {

namespace {

__device__ double log_choose(double n, double k) {
  return lgamma(n + 1.0) - lgamma(k + 1.0) - lgamma(n - k + 1.0);
}

__device__ double jaccard_of(int64_t x, int64_t a, int64_t b) {
  const int64_t u = a + b - x;
  return u == 0 ? 1.0 : (double)x / (double)u;
}

// this thread's share of E[J] over the window (see above); every thread calls it
__device__ double expected_random_jaccard_part(int64_t n, int64_t a, int64_t b, int tid) {
  int64_t xlo = a + b - n > 0 ? a + b - n : 0;
  int64_t xhi = a < b ? a : b;
  const double mean = (double)a * (double)b / (double)(n > 0 ? n : 1);
  const double half = sqrt(48.0 * (double)xhi) + 2.0;
  const int64_t wlo = (int64_t)floor(mean - half), whi = (int64_t)ceil(mean + half);
  xlo = wlo > xlo ? wlo : xlo;
  xhi = whi < xhi ? whi : xhi;
  const int64_t per = (xhi - xlo + 256) / 256;
  const int64_t c0 = xlo + (int64_t)tid * per;
  const int64_t c1 = c0 + per - 1 < xhi ? c0 + per - 1 : xhi;
  if (c0 > c1) return 0.0;
  int64_t xm = (int64_t)(((double)(a + 1) * (double)(b + 1)) / (double)(n + 2));
  const int64_t x0 = xm < c0 ? c0 : (xm > c1 ? c1 : xm);
  const double p0 = exp(log_choose((double)a, (double)x0) + log_choose((double)(n - a), (double)(b - x0)) -
                        log_choose((double)n, (double)b));
  if (p0 == 0.0) return 0.0;
  double sum = p0 * jaccard_of(x0, a, b);
  const double c = (double)(n - a - b);
  double q = p0;
  for (int64_t x = x0; x < c1; ++x) {  // P(x + 1) / P(x) = (a - x)(b - x) / ((x + 1)(n - a - b + x + 1))
    q *= ((double)(a - x) * (double)(b - x)) / ((double)(x + 1) * (c + (double)(x + 1)));
    sum += q * jaccard_of(x + 1, a, b);
  }
  q = p0;
  for (int64_t x = x0; x > c0; --x) {  // P(x - 1) / P(x) = x (n - a - b + x) / ((a - x + 1)(b - x + 1))
    q *= ((double)x * (c + (double)x)) / ((double)(a - x + 1) * (double)(b - x + 1));
    sum += q * jaccard_of(x - 1, a, b);
  }
  return sum;
}

__global__ __launch_bounds__(256) void stability_kernel(const int32_t* __restrict__ offs,
                                                        const uint8_t* __restrict__ flags, int T,
                                                        const int32_t* __restrict__ tp_t,
                                                        const int32_t* __restrict__ tp_r,
                                                        float* __restrict__ jac,
                                                        float* __restrict__ jrand,
                                                        float* __restrict__ rda) {
  __shared__ int cnt[4][4];
  __shared__ double part[4];
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  int o0 = offs[b], o1 = offs[b + 1];
  const int lo = o0 < 0 ? 0 : (o0 > T ? T : o0);
  const int hi = o1 < lo ? lo : (o1 > T ? T : o1);
  int n = 0, na = 0, nb = 0, nx = 0;
  for (int i = lo + tid; i < hi; i += 256) {
    if (flags[i] & CE_TOK_KEEP) continue;
    const bool dt = tp_t[i] < 0, dr = tp_r[i] < 0;
    n += 1;
    na += dt;
    nb += dr;
    nx += dt && dr;
  }
  for (int o = 32; o > 0; o >>= 1) {
    n += __shfl_xor(n, o);
    na += __shfl_xor(na, o);
    nb += __shfl_xor(nb, o);
    nx += __shfl_xor(nx, o);
  }
  if ((tid & 63) == 0) {
    cnt[tid >> 6][0] = n;
    cnt[tid >> 6][1] = na;
    cnt[tid >> 6][2] = nb;
    cnt[tid >> 6][3] = nx;
  }
  __syncthreads();
  int64_t c[4];
  for (int k = 0; k < 4; ++k) c[k] = (int64_t)cnt[0][k] + cnt[1][k] + cnt[2][k] + cnt[3][k];
  // c[0] = routable tokens, c[1] / c[2] = dropped at t / t_ref, c[3] = dropped at both
  double jr;
  const int64_t xlo = c[1] + c[2] - c[0] > 0 ? c[1] + c[2] - c[0] : 0;
  const int64_t xhi = c[1] < c[2] ? c[1] : c[2];
  if (xlo >= xhi) {
    jr = jaccard_of(xlo, c[1], c[2]);  // a single possible overlap
  } else {
    double v = expected_random_jaccard_part(c[0], c[1], c[2], tid);
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    if ((tid & 63) == 0) part[tid >> 6] = v;
    __syncthreads();
    jr = (part[0] + part[1]) + (part[2] + part[3]);
  }
  if (tid != 0) return;
  const double j = jaccard_of(c[3], c[1], c[2]);
  jac[b] = (float)j;
  if (jrand) jrand[b] = (float)jr;
  if (rda) rda[b] = (float)(jr >= 1.0 ? 1.0 : (j - jr) / (1.0 - jr));
}

}  // namespace

hipError_t launch_stability(const int32_t* seq_offsets, const uint8_t* flags, int B, int T,
                            const int32_t* tp_t, const int32_t* tp_ref, float* jaccard, float* j_rand,
                            float* rda, hipStream_t stream) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(stability_kernel, dim3(B), dim3(256), 0, stream, seq_offsets, flags, T, tp_t, tp_ref,
                     jaccard, j_rand, rda);
  return hipGetLastError();
}

}  // namespace ce
