// Residual merge of the packed FFN output back into the full sequence
// (paper section 3.4: retained tokens are updated, dropped tokens follow the
// bypass path):
//   out[kept_idx[j]] = in[kept_idx[j]] + ffn[j]   (fp32 add, one rounding to dtype)
// plus a row copy used when the output is a separate buffer.
#include "ce_device.hpp"
#include "ce_launch.hpp"

namespace ce {

namespace {

// One wave per packed row; each lane handles 8 bf16 or 4 fp32 values per step.
template <bool kBF16>
__global__ __launch_bounds__(256) void scatter_kernel(const char* __restrict__ ffn,
                                                      const int32_t* __restrict__ kept_idx,
                                                      const int32_t* __restrict__ kept_offsets,
                                                      int B, int cap, int T, int d,
                                                      const char* h_in, char* h_out) {
  constexpr int kElem = kBF16 ? 2 : 4;
  int kt = kept_offsets[B];
  kt = kt < 0 ? 0 : (kt > cap ? cap : kt);
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= kt) return;
  const int tok = kept_idx[j];
  if (tok < 0 || tok >= T) return;  // invalid caller index: row skipped
  const int64_t row_bytes = (int64_t)d * kElem;
  const char* f = ffn + (int64_t)j * row_bytes;
  const char* src = h_in + (int64_t)tok * row_bytes;
  char* dst = h_out + (int64_t)tok * row_bytes;
  for (int64_t o = (threadIdx.x & 63) * 16; o < row_bytes; o += 64 * 16) {
    const u32x4_t x = *reinterpret_cast<const u32x4_t*>(src + o);
    const u32x4_t y = *reinterpret_cast<const u32x4_t*>(f + o);
    u32x4_t r;
    if constexpr (kBF16) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float lo = bf16_to_f32(x[q] & 0xffffu) + bf16_to_f32(y[q] & 0xffffu);
        const float hi = bf16_to_f32(x[q] >> 16) + bf16_to_f32(y[q] >> 16);
        r[q] = pack_bf16(lo, hi);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) r[q] = __float_as_uint(__uint_as_float(x[q]) + __uint_as_float(y[q]));
    }
    *reinterpret_cast<u32x4_t*>(dst + o) = r;
  }
}

__global__ __launch_bounds__(256) void copy_rows_kernel(const char* __restrict__ src,
                                                        char* __restrict__ dst, int64_t row_bytes,
                                                        int T, const int32_t* __restrict__ token_pos) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= T) return;
  if (token_pos && token_pos[i] >= 0) return;
  const char* s = src + (int64_t)i * row_bytes;
  char* d = dst + (int64_t)i * row_bytes;
  for (int64_t o = (threadIdx.x & 63) * 16; o < row_bytes; o += 64 * 16)
    *reinterpret_cast<u32x4_t*>(d + o) = *reinterpret_cast<const u32x4_t*>(s + o);
}

}  // namespace

hipError_t launch_scatter(const char* ffn_out, const int32_t* kept_idx, const int32_t* kept_offsets,
                          int B, int cap, int T, int d, bool bf16, const char* h_in, char* h_out,
                          hipStream_t stream) {
  if (cap <= 0) return hipSuccess;
  const dim3 grid((cap + 3) / 4);
  if (bf16)
    hipLaunchKernelGGL(scatter_kernel<true>, grid, dim3(256), 0, stream, ffn_out, kept_idx,
                       kept_offsets, B, cap, T, d, h_in, h_out);
  else
    hipLaunchKernelGGL(scatter_kernel<false>, grid, dim3(256), 0, stream, ffn_out, kept_idx,
                       kept_offsets, B, cap, T, d, h_in, h_out);
  return hipGetLastError();
}

hipError_t launch_copy_rows(const char* h_in, char* h_out, int64_t row_bytes, int T,
                            const int32_t* token_pos, hipStream_t stream) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy_rows_kernel, dim3((T + 3) / 4), dim3(256), 0, stream, h_in, h_out,
                     row_bytes, T, token_pos);
  return hipGetLastError();
}

}  // namespace ce
