// Layer-skipping redundancy gap (paper section 3.4, UCS operator (1), Eq. 7).
//
//   cos[i]      = <x_in[i], x_out[i]> / (||x_in[i]|| ||x_out[i]||)   per token
//                 (1 when both rows are zero, 0 when exactly one is)
//   rho_all[b]  = mean of cos over the tokens of sequence b            (1 if empty)
//   rho_ret[b]  = mean of cos over its retained tokens (token_pos >= 0),
//                 rho_all[b] when there are none
//   gap[b]      = rho_all[b] - rho_ret[b]                               (Eq. 7)
//   skip[b]     = gap[b] <= delta_LS
//
// The fused routed block (ce_routed_block_gap) gets the per-token sums from
// its down GEMM's epilogue instead (token_cos_parts_kernel), so it reads
// neither matrix again. The standalone entry point takes
// two launches, both bandwidth-bound on the two [T x d] reads: a wave per
// token accumulates the three sums in fp64 from 16-byte loads (bf16 and fp32
// products are exact in fp64, so only the summation order rounds) and writes
// the token's cosine; then a workgroup per sequence adds the cosines in fp64
// in a fixed order. Results are deterministic.
#include "ce_device.hpp"
#include "ce_launch.hpp"

namespace ce {

namespace {

template <bool kBF16>
__global__ __launch_bounds__(256) void token_cos_kernel(const char* __restrict__ x_in, const char* __restrict__ x_out,
                                                        int T, int d, float* __restrict__ cos_out) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= T) return;
  constexpr int kPer = kBF16 ? 8 : 4;
  const int chunks = d / kPer;
  const int64_t row = (int64_t)i * d * (kBF16 ? 2 : 4);
  const u32x4_t* a = reinterpret_cast<const u32x4_t*>(x_in + row);
  const u32x4_t* b = reinterpret_cast<const u32x4_t*>(x_out + row);
  double dot = 0.0, na = 0.0, nb = 0.0;
  auto add = [&](const u32x4_t& va, const u32x4_t& vb) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      float fa, fb;
      if constexpr (kBF16) {
        fa = bf16_to_f32((va[k >> 1] >> (16 * (k & 1))) & 0xffffu);
        fb = bf16_to_f32((vb[k >> 1] >> (16 * (k & 1))) & 0xffffu);
      } else {
        fa = __uint_as_float(va[k]);
        fb = __uint_as_float(vb[k]);
      }
      const double xa = fa, xb = fb;
      dot = fma(xa, xb, dot);
      na = fma(xa, xa, na);
      nb = fma(xb, xb, nb);
    }
  };
  int c = lane;
  for (; c + 128 < chunks; c += 192) {
    const u32x4_t a0 = a[c], a1 = a[c + 64], a2 = a[c + 128];
    const u32x4_t b0 = b[c], b1 = b[c + 64], b2 = b[c + 128];
    add(a0, b0);
    add(a1, b1);
    add(a2, b2);
  }
  for (; c < chunks; c += 64) add(a[c], b[c]);
  for (int o = 32; o > 0; o >>= 1) {
    dot += __shfl_xor(dot, o);
    na += __shfl_xor(na, o);
    nb += __shfl_xor(nb, o);
  }
  if (lane == 0) {
    const double both = sqrt(na) * sqrt(nb);
    cos_out[i] = (float)(both > 0.0 ? dot / both : (na == 0.0 && nb == 0.0 ? 1.0 : 0.0));
  }
}

// Per-token cosine of a routed block from the down GEMM's per-row partial
// sums (a wave per token): dropped tokens bypass the layer (output = input),
// so their cosine is 1 (also for a zero row); for a retained token the lanes
// load the gap_np slots of its packed row together (lane q, q + 64, ...) and
// add them in fp64, then across the wave in a fixed tree order.
__global__ __launch_bounds__(256) void token_cos_parts_kernel(const double* __restrict__ gap_part, int gap_np, int T,
                                                              int cap, const int32_t* __restrict__ token_pos,
                                                              float* __restrict__ cos_out) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= T) return;
  const int p = token_pos[i];
  if (p < 0) {
    if (lane == 0) cos_out[i] = 1.0f;
    return;
  }
  if (p >= cap) {  // more retained rows than the capacity (reported in the status word)
    if (lane == 0) cos_out[i] = __builtin_nanf("");
    return;
  }
  const double* g = gap_part + (int64_t)p * gap_np * 4;
  double dot = 0.0, na = 0.0, nb = 0.0;
  for (int q = lane; q < gap_np; q += 64) {
    dot += g[4 * q + 0];
    na += g[4 * q + 1];
    nb += g[4 * q + 2];
  }
  for (int o = 32; o > 0; o >>= 1) {
    dot += __shfl_xor(dot, o);
    na += __shfl_xor(na, o);
    nb += __shfl_xor(nb, o);
  }
  if (lane == 0) {
    const double both = sqrt(na) * sqrt(nb);
    cos_out[i] = (float)(both > 0.0 ? dot / both : (na == 0.0 && nb == 0.0 ? 1.0 : 0.0));
  }
}

__global__ __launch_bounds__(256) void gap_kernel(const int32_t* __restrict__ offs, int T,
                                                  const int32_t* __restrict__ token_pos,
                                                  const float* __restrict__ cos_tok, float delta,
                                                  float* __restrict__ rho_all, float* __restrict__ rho_ret,
                                                  float* __restrict__ gap, uint8_t* __restrict__ skip) {
  __shared__ double red[2][4];
  __shared__ int cnt[4];
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int o0 = offs[b], o1 = offs[b + 1];
  const int lo = o0 < 0 ? 0 : (o0 > T ? T : o0);
  const int hi = o1 < lo ? lo : (o1 > T ? T : o1);
  double sa = 0.0, sr = 0.0;
  int nr = 0;
  for (int i = lo + tid; i < hi; i += 256) {
    const double c = cos_tok[i];
    sa += c;
    if (token_pos[i] >= 0) {
      sr += c;
      nr += 1;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    sa += __shfl_xor(sa, o);
    sr += __shfl_xor(sr, o);
    nr += __shfl_xor(nr, o);
  }
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = sa;
    red[1][tid >> 6] = sr;
    cnt[tid >> 6] = nr;
  }
  __syncthreads();
  if (tid != 0) return;
  const int n = hi - lo;
  const int n_ret = cnt[0] + cnt[1] + cnt[2] + cnt[3];
  const double all = n > 0 ? ((red[0][0] + red[0][1]) + (red[0][2] + red[0][3])) / n : 1.0;
  const double ret = n_ret > 0 ? ((red[1][0] + red[1][1]) + (red[1][2] + red[1][3])) / n_ret : all;
  const double g = all - ret;
  rho_all[b] = (float)all;
  rho_ret[b] = (float)ret;
  gap[b] = (float)g;
  if (skip) skip[b] = g <= (double)delta ? 1 : 0;
}

}  // namespace

hipError_t launch_gap_from_parts(const double* gap_part, int gap_np, int cap, const int32_t* seq_offsets, int B,
                                 int T, const int32_t* token_pos, float delta, float* cos_tok, float* rho_all,
                                 float* rho_ret, float* gap, uint8_t* skip, hipStream_t stream) {
  if (T > 0) {
    hipLaunchKernelGGL(token_cos_parts_kernel, dim3((T + 3) / 4), dim3(256), 0, stream, gap_part, gap_np, T, cap,
                       token_pos, cos_tok);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(gap_kernel, dim3(B), dim3(256), 0, stream, seq_offsets, T, token_pos,
                     (const float*)cos_tok, delta, rho_all, rho_ret, gap, skip);
  return hipGetLastError();
}

hipError_t launch_layer_gap(const char* x_in, const char* x_out, const int32_t* seq_offsets, int B, int T, int d,
                            bool bf16, const int32_t* token_pos, float delta, float* cos_tok, float* rho_all,
                            float* rho_ret, float* gap, uint8_t* skip, hipStream_t stream) {
  if (T > 0) {
    const dim3 grid((T + 3) / 4);
    if (bf16) hipLaunchKernelGGL(token_cos_kernel<true>, grid, dim3(256), 0, stream, x_in, x_out, T, d, cos_tok);
    else hipLaunchKernelGGL(token_cos_kernel<false>, grid, dim3(256), 0, stream, x_in, x_out, T, d, cos_tok);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(gap_kernel, dim3(B), dim3(256), 0, stream, seq_offsets, T, token_pos,
                     (const float*)cos_tok, delta, rho_all, rho_ret, gap, skip);
  return hipGetLastError();
}

}  // namespace ce
