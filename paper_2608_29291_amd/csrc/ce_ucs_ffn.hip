// FFN-pruning signal on the retained rows (paper section 3.4, UCS operator (2),
// Eq. 8-9) and the channel mask that turns the full FFN into the pruned one.
//
//   norms[set][c]  = ||W_down[set][:, c]||_2                        (per weight set)
//   s[b][c]        = mean over the packed rows j of sequence b of
//                    |act[j][c]| * norms[set(j)][c]                   (Eq. 8)
//   lambda[b]      = sum_{c in P} s[b][c] / sum_c s[b][c]             (Eq. 9; 0 if the sum is 0)
//   use_pruned[b]  = lambda[b] <= delta
//   masking: act[j][c] = 0 for c in P on the rows of sequences with use_pruned,
//            so the down projection then computes the pruned FFN exactly.
//
// act is the SwiGLU activation matrix [cap x d_ff] in packed-row order (the
// output of the gate/up step); set(j) is the MoT weight set of the row's token
// (its GEN bit when there are two sets). Every sum runs in fp32 in a fixed
// order, so the results are deterministic. All kernels are bandwidth-bound:
// the saliency reads the activations once (16-byte loads, each sequence's
// rows split over several workgroups whose partial sums sit in the FFN
// workspace), a channel-parallel pass combines the splits and totals each
// 256-channel chunk, and one thread per sequence adds the chunk totals; the
// norms read W_down once.
#include "ce_device.hpp"
#include "ce_launch.hpp"
#include "ce_router.h"
#include "ce_host.hpp"

namespace ce {

namespace {

// Column norms of W_down ([d x d_ff] row-major) of weight set blockIdx.y.
// Workgroup: 8 groups of kPer consecutive channels (one 16-byte load per row
// each) x 32 row lanes; lane l sums rows l, l + 32, ... and the 32 lane sums
// of a channel are then added in lane order.
template <bool kBF16>
__global__ __launch_bounds__(256) void colnorm_kernel(const char* __restrict__ w0, const char* __restrict__ w1,
                                                      int d, int d_ff, float* __restrict__ norms) {
  constexpr int kPer = kBF16 ? 8 : 4;
  constexpr int kCh = 8 * kPer;
  __shared__ float red[32][kCh + 1];
  const int g = threadIdx.x & 7, lane = threadIdx.x >> 3;
  const int c0 = blockIdx.x * kCh + g * kPer;
  const char* w = blockIdx.y == 0 ? w0 : w1;
  float acc[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) acc[k] = 0.0f;
  auto row = [&](int r) __attribute__((always_inline)) {
    const u32x4_t v = *reinterpret_cast<const u32x4_t*>(w + ((int64_t)r * d_ff + c0) * (kBF16 ? 2 : 4));
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      float x;
      if constexpr (kBF16) x = bf16_to_f32((v[k >> 1] >> (16 * (k & 1))) & 0xffffu);
      else x = __uint_as_float(v[k]);
      acc[k] = fmaf(x, x, acc[k]);
    }
  };
  int r = lane;
  for (; r + 96 < d; r += 128) {
    row(r);
    row(r + 32);
    row(r + 64);
    row(r + 96);
  }
  for (; r < d; r += 32) row(r);
#pragma unroll
  for (int k = 0; k < kPer; ++k) red[lane][g * kPer + k] = acc[k];
  __syncthreads();
  if (threadIdx.x < kCh) {
    float t = 0.0f;
    for (int l = 0; l < 32; ++l) t += red[l][threadIdx.x];
    norms[(int64_t)blockIdx.y * d_ff + blockIdx.x * kCh + threadIdx.x] = sqrtf(t);
  }
}

struct SalArgs {
  const char* act;
  const int32_t* kept_idx;
  const int32_t* kept_offsets;
  const uint8_t* flags;
  const float* norms;
  int B, T, cap, d_ff, n_sets, splits;
  float* part;  // [splits x B x d_ff]
};

// Workgroup (channel chunk x, sequence y, row split z): thread t owns kPer
// consecutive channels (one 16-byte load per row) and sums |act| * norm over
// its share of the sequence's packed rows, four rows in flight.
template <bool kBF16>
__global__ __launch_bounds__(256) void saliency_part_kernel(SalArgs a) {
  constexpr int kPer = kBF16 ? 8 : 4;
  const int c0 = (blockIdx.x * 256 + threadIdx.x) * kPer;
  const int b = blockIdx.y;
  const int r = blockIdx.z;
  if (c0 >= a.d_ff) return;
  int j0 = a.kept_offsets[b], j1 = a.kept_offsets[b + 1];
  j0 = j0 < 0 ? 0 : (j0 > a.cap ? a.cap : j0);
  j1 = j1 < j0 ? j0 : (j1 > a.cap ? a.cap : j1);
  const int per = (j1 - j0 + a.splits - 1) / a.splits;
  const int s0 = j0 + r * per;
  const int s1 = min(j1, s0 + per);
  float n0[kPer], n1[kPer], acc[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    n0[k] = a.norms[c0 + k];
    n1[k] = a.n_sets == 2 ? a.norms[(int64_t)a.d_ff + c0 + k] : n0[k];
    acc[k] = 0.0f;
  }
  auto row = [&](int j) __attribute__((always_inline)) {
    bool set1 = false;
    if (a.n_sets == 2) {
      const int tok = a.kept_idx[j];
      set1 = tok >= 0 && tok < a.T && (a.flags[tok] & CE_TOK_GEN);
    }
    const u32x4_t v = *reinterpret_cast<const u32x4_t*>(a.act + ((int64_t)j * a.d_ff + c0) * (kBF16 ? 2 : 4));
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      float x;
      if constexpr (kBF16) x = bf16_to_f32((v[k >> 1] >> (16 * (k & 1))) & 0xffffu);
      else x = __uint_as_float(v[k]);
      acc[k] = fmaf(fabsf(x), set1 ? n1[k] : n0[k], acc[k]);
    }
  };
  int j = s0;
  for (; j + 4 <= s1; j += 4) {
    row(j);
    row(j + 1);
    row(j + 2);
    row(j + 3);
  }
  for (; j < s1; ++j) row(j);
  float* out = a.part + ((int64_t)r * a.B + b) * a.d_ff + c0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) out[k] = acc[k];
}

// workgroup (channel chunk x, sequence y), thread per channel: saliency = (sum
// of the row-split partials, in split order) / rows; the chunk's totals over
// all channels and over the mask go to chunk_tot[y][x][0..1]
__global__ __launch_bounds__(256) void saliency_combine_kernel(const float* __restrict__ part, int splits, int B,
                                                               const int32_t* __restrict__ kept_offsets, int cap,
                                                               const uint8_t* __restrict__ mask, int d_ff,
                                                               float* __restrict__ saliency,
                                                               float* __restrict__ chunk_tot) {
  __shared__ float red[2][4];
  const int b = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  int j0 = kept_offsets[b], j1 = kept_offsets[b + 1];
  j0 = j0 < 0 ? 0 : (j0 > cap ? cap : j0);
  j1 = j1 < j0 ? j0 : (j1 > cap ? cap : j1);
  const float inv = j1 > j0 ? 1.0f / (float)(j1 - j0) : 0.0f;
  float tot = 0.0f, pm = 0.0f;
  if (c < d_ff) {
    float v = 0.0f;
    for (int r = 0; r < splits; ++r) v += part[((int64_t)r * B + b) * d_ff + c];
    v *= inv;
    saliency[(int64_t)b * d_ff + c] = v;
    tot = v;
    pm = mask[c] ? v : 0.0f;
  }
  for (int o = 32; o > 0; o >>= 1) {
    tot += __shfl_xor(tot, o);
    pm += __shfl_xor(pm, o);
  }
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = tot;
    red[1][threadIdx.x >> 6] = pm;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float* o = chunk_tot + ((int64_t)b * gridDim.x + blockIdx.x) * 2;
    o[0] = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
    o[1] = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
  }
}

// thread per sequence: leakage = masked total / total over the channel chunks, in chunk order
__global__ __launch_bounds__(256) void leakage_kernel(const float* __restrict__ chunk_tot, int chunks, int B,
                                                      float delta, float* __restrict__ lambda,
                                                      uint8_t* __restrict__ use_pruned,
                                                      const int32_t* __restrict__ kept_offsets, int cap,
                                                      uint8_t* __restrict__ row_flag) {
  // one wave per sequence: lane l adds chunks l, l + 64, ..., then the lanes
  // are added in a fixed tree
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (b >= B) return;
  float t = 0.0f, p = 0.0f;
  for (int k = lane; k < chunks; k += 64) {
    t += chunk_tot[((int64_t)b * chunks + k) * 2];
    p += chunk_tot[((int64_t)b * chunks + k) * 2 + 1];
  }
  for (int o = 32; o > 0; o >>= 1) {
    t += __shfl_xor(t, o);
    p += __shfl_xor(p, o);
  }
  // lane 0's totals (a butterfly may round differently in other lanes)
  t = __shfl(t, 0);
  p = __shfl(p, 0);
  const float lam = t > 0.0f ? p / t : 0.0f;
  const uint8_t use = lam <= delta ? 1 : 0;
  if (lane == 0) {
    lambda[b] = lam;
    if (use_pruned) use_pruned[b] = use;
  }
  if (row_flag) {
    // the choice for each packed row of the sequence (the pruned down GEMM
    // reads one byte per row instead of row -> sequence -> choice)
    int j0 = kept_offsets[b], j1 = kept_offsets[b + 1];
    j0 = j0 < 0 ? 0 : (j0 > cap ? cap : j0);
    j1 = j1 < j0 ? j0 : (j1 > cap ? cap : j1);
    for (int j = j0 + lane; j < j1; j += 64) row_flag[j] = use;
  }
}

// one workgroup per packed row: zero the masked channels of rows whose sequence runs pruned
template <bool kBF16>
__global__ __launch_bounds__(256) void mask_kernel(char* __restrict__ act, const int32_t* __restrict__ kept_offsets,
                                                   int B, int cap, int d_ff, const uint8_t* __restrict__ mask,
                                                   const uint8_t* __restrict__ use_pruned) {
  const int j = blockIdx.x;
  // sequence of row j: the last b with kept_offsets[b] <= j (offsets are non-decreasing)
  int lo = 0, hi = B;  // invariant: answer in [lo, hi)
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (kept_offsets[mid] <= j) lo = mid;
    else hi = mid;
  }
  int end = kept_offsets[B];
  end = end < 0 ? 0 : (end > cap ? cap : end);
  if (j >= end || !use_pruned[lo]) return;
  for (int c = threadIdx.x; c < d_ff; c += 256) {
    if (!mask[c]) continue;
    if constexpr (kBF16) reinterpret_cast<uint16_t*>(act)[(int64_t)j * d_ff + c] = 0;
    else reinterpret_cast<float*>(act)[(int64_t)j * d_ff + c] = 0.0f;
  }
}

// row_seq[p] = b for the packed rows p of sequence b (workgroup per sequence)
__global__ __launch_bounds__(256) void row_seq_kernel(const int32_t* __restrict__ kept_offsets, int cap,
                                                      int32_t* __restrict__ row_seq, int32_t* __restrict__ seq_cnt) {
  const int b = blockIdx.x;
  if (threadIdx.x == 0) seq_cnt[b] = 0;  // the saliency kernel's arrival counter of sequence b
  int j0 = kept_offsets[b], j1 = kept_offsets[b + 1];
  j0 = j0 < 0 ? 0 : (j0 > cap ? cap : j0);
  j1 = j1 < j0 ? j0 : (j1 > cap ? cap : j1);
  for (int j = j0 + threadIdx.x; j < j1; j += 256) row_seq[j] = b;
}

// Saliency from the gate/up epilogue's segment sums (workgroup: channel chunk
// x, sequence y; thread per channel). The token tiles are enumerated as the
// GEMM does (set 0 rows, then set 1 rows, 256 per tile); each tile's segments
// of sequence b add their |z| sums in tile order, per weight set; a tile with
// more segments than the epilogue kept adds the rows of b from act instead.
// saliency = (sum_set0 * norm0 + sum_set1 * norm1) / rows of b; the chunk's
// totals over all channels and over the tail [n_keep, d_ff) go to chunk_tot,
// and the sequence's last workgroup turns them into its leakage.
struct SegSalArgs {
  const float* sal_part;
  const int32_t* sal_meta;
  const char* act;  // bf16 [cap x d_ff], GEMM row order
  const int32_t* grp;  // GEMM row -> packed row (two weight sets) or NULL
  const int32_t* row_seq;
  const int32_t* kept_offsets;
  const int32_t* kt_ptr;
  const int32_t* n0_ptr;
  const float* norms;
  int B, cap, d_ff, n_sets, n_keep;
  float* saliency;
  float* chunk_tot;
  // leakage (Eq. 9) and the choice, by the last workgroup of each sequence
  int32_t* seq_cnt;  // [B] arrival counters, zero on entry
  float delta;
  float* lambda;
  uint8_t* use_pruned;
  uint8_t* row_flag;
};

constexpr int kMetaTiles = 64;  // token tiles whose segment lists are staged in LDS at a time

__global__ __launch_bounds__(256) void saliency_seg_kernel(SegSalArgs a) {
  __shared__ int32_t meta_s[kMetaTiles * (kSalSegs + 1)];
  __shared__ int match_s[kMetaTiles];
  __shared__ float red[2][4];
  __shared__ int last_s;
  __shared__ float lam_s;
  const int b = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  int kt = *a.kt_ptr;
  kt = kt < 0 ? 0 : (kt > a.cap ? a.cap : kt);
  int n0 = kt;
  if (a.n_sets == 2 && a.n0_ptr) {
    n0 = *a.n0_ptr;
    n0 = n0 < 0 ? 0 : (n0 > kt ? kt : n0);
  }
  const int tiles0 = (n0 + 255) / 256;
  const int tiles = tiles0 + (kt - n0 + 255) / 256;
  int j0 = a.kept_offsets[b], j1 = a.kept_offsets[b + 1];
  j0 = j0 < 0 ? 0 : (j0 > kt ? kt : j0);
  j1 = j1 < j0 ? j0 : (j1 > kt ? kt : j1);
  // one FFN set: GEMM rows are packed rows, so only the tiles over [j0, j1)
  // hold rows of sequence b; two sets: its rows may sit in any tile
  const int t_lo = a.n_sets == 2 ? 0 : j0 / 256;
  const int t_hi = a.n_sets == 2 ? tiles : (j1 > j0 ? (j1 - 1) / 256 + 1 : t_lo);
  float tot = 0.0f, pm = 0.0f;
  float acc[2] = {0.0f, 0.0f};
  for (int tb = t_lo; tb < t_hi; tb += kMetaTiles) {
    const int nt = min(kMetaTiles, t_hi - tb);
    // the segment lists of tiles tb .. tb + nt - 1 in one round of loads,
    // then the segment of sequence b in each (-1: none; -2: the tile has more
    // segments than the epilogue kept, or b in more than one)
    __syncthreads();
    for (int i = threadIdx.x; i < nt * (kSalSegs + 1); i += 256)
      meta_s[i] = a.sal_meta[(int64_t)tb * (kSalSegs + 1) + i];
    __syncthreads();
    if ((int)threadIdx.x < nt) {
      const int* m = meta_s + threadIdx.x * (kSalSegs + 1);
      const int cnt = m[0];
      int km = -1, hits = 0;
      for (int k = 0; k < (cnt <= kSalSegs ? cnt : 0); ++k)
        if (m[1 + k] == b) {
          km = k;
          ++hits;
        }
      match_s[threadIdx.x] = (cnt > kSalSegs || hits > 1) ? -2 : km;
    }
    __syncthreads();
    if (c >= a.d_ff) continue;
    // four tiles' sums loaded together (a tile without a segment of b reads
    // its slot 0 and drops it), added in tile order
#pragma unroll 1
    for (int t0 = 0; t0 < nt; t0 += 4) {
      float v[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int t = min(t0 + j, nt - 1);
        const int km = match_s[t];
        v[j] = a.sal_part[((int64_t)(tb + t) * kSalSegs + (km > 0 ? km : 0)) * a.d_ff + c];
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (t0 + j >= nt) break;
        const int tt = tb + t0 + j;
        const int set = tt < tiles0 ? 0 : 1;
        const int km = match_s[t0 + j];
        if (km >= 0) {
          acc[set] += v[j];
        } else if (km == -2) {
          // the rows of b in this tile, from act
          const int lo = set == 0 ? tt * 256 : n0 + (tt - tiles0) * 256;
          const int hi = min(lo + 256, set == 0 ? n0 : kt);
          for (int jr = lo; jr < hi; ++jr) {
            const int p = a.grp ? a.grp[jr] : jr;
            if (p >= 0 && p < a.cap && a.row_seq[p] == b)
              acc[set] += fabsf(bf16_to_f32(reinterpret_cast<const uint16_t*>(a.act)[(int64_t)jr * a.d_ff + c]));
          }
        }
      }
    }
  }
  if (c < a.d_ff) {
    const float n1c = a.n_sets == 2 ? a.norms[(int64_t)a.d_ff + c] : 0.0f;
    const float v = j1 > j0 ? (acc[0] * a.norms[c] + acc[1] * n1c) / (float)(j1 - j0) : 0.0f;
    a.saliency[(int64_t)b * a.d_ff + c] = v;
    tot = v;
    pm = c >= a.n_keep ? v : 0.0f;
  }
  for (int o = 32; o > 0; o >>= 1) {
    tot += __shfl_xor(tot, o);
    pm += __shfl_xor(pm, o);
  }
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = tot;
    red[1][threadIdx.x >> 6] = pm;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float* o = a.chunk_tot + ((int64_t)b * gridDim.x + blockIdx.x) * 2;
    o[0] = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
    o[1] = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
    // the totals are visible device-wide before the arrival is counted
    __threadfence();
    last_s = atomicAdd(a.seq_cnt + b, 1) == (int)gridDim.x - 1;
  }
  __syncthreads();
  if (!last_s) return;
  // the last of sequence b's workgroups: its leakage from the per-chunk
  // totals (wave 0: lane l adds chunks l, l + 64, ..., then the lanes in a
  // fixed tree; coherent loads, the other workgroups wrote them), the choice,
  // and a flag byte for each of its packed rows
  __threadfence();
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const float* tp = a.chunk_tot + (int64_t)b * gridDim.x * 2;
    float t = 0.0f, p = 0.0f;
    for (int k = lane; k < (int)gridDim.x; k += 64) {
      t += __hip_atomic_load(tp + 2 * k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      p += __hip_atomic_load(tp + 2 * k + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    for (int o = 32; o > 0; o >>= 1) {
      t += __shfl_xor(t, o);
      p += __shfl_xor(p, o);
    }
    if (lane == 0) {
      const float lam = t > 0.0f ? p / t : 0.0f;
      lam_s = lam;
      a.lambda[b] = lam;
      a.use_pruned[b] = lam <= a.delta ? 1 : 0;
    }
  }
  __syncthreads();
  const uint8_t use = lam_s <= a.delta ? 1 : 0;
  for (int j = j0 + (int)threadIdx.x; j < j1; j += 256) a.row_flag[j] = use;
}

}  // namespace

hipError_t launch_row_seq(const int32_t* kept_offsets, int B, int cap, int32_t* row_seq, int32_t* seq_cnt,
                          hipStream_t stream) {
  hipLaunchKernelGGL(row_seq_kernel, dim3(B), dim3(256), 0, stream, kept_offsets, cap, row_seq, seq_cnt);
  return hipGetLastError();
}

hipError_t launch_saliency_segments(const FfnGemmArgs& g, const int32_t* kept_offsets, const float* norms, int B,
                                    int n_keep, float delta, float* chunk_tot, float* saliency, float* lambda,
                                    uint8_t* use_pruned, uint8_t* row_flag, int32_t* seq_cnt,
                                    hipStream_t stream) {
  // gate/up: GEMM row j is packed row map1[j] (the MoT grouping) or j; act is in GEMM row order
  SegSalArgs s{g.sal_part, g.sal_meta, g.out, g.map1, g.row_seq, kept_offsets, g.kt_ptr, g.n0_ptr, norms,
               B, g.cap, g.n_feat, g.n_sets, n_keep, saliency, chunk_tot, seq_cnt, delta, lambda, use_pruned,
               row_flag};
  const int chunks = (g.n_feat + 255) / 256;
  hipLaunchKernelGGL(saliency_seg_kernel, dim3(chunks, B), dim3(256), 0, stream, s);
  return hipGetLastError();
}

hipError_t launch_colnorms(const char* w0, const char* w1, int n_sets, int d, int d_ff, bool bf16,
                           float* norms, hipStream_t stream) {
  const dim3 grid(d_ff / (bf16 ? 64 : 32), n_sets);  // d_ff is a multiple of 64
  if (bf16) hipLaunchKernelGGL(colnorm_kernel<true>, grid, dim3(256), 0, stream, w0, w1, d, d_ff, norms);
  else hipLaunchKernelGGL(colnorm_kernel<false>, grid, dim3(256), 0, stream, w0, w1, d, d_ff, norms);
  return hipGetLastError();
}

hipError_t launch_saliency(const char* act, const int32_t* kept_idx, const int32_t* kept_offsets,
                           const uint8_t* flags, const float* norms, int B, int T, int cap, int d_ff,
                           int n_sets, bool bf16, const uint8_t* mask, float delta, float* part,
                           float* saliency, float* lambda, uint8_t* use_pruned, hipStream_t stream) {
  const int per_wg = 256 * (bf16 ? 8 : 4);
  const int chunks = (d_ff + per_wg - 1) / per_wg;
  // enough workgroups to keep the memory system busy: about 1024 in all
  int splits = (1024 + chunks * B - 1) / (chunks * B);
  splits = splits < 1 ? 1 : (splits > kSalSplits ? kSalSplits : splits);
  SalArgs a{act, kept_idx, kept_offsets, flags, norms, B, T, cap, d_ff, n_sets, splits, part};
  const dim3 grid(chunks, B, splits);
  if (bf16) hipLaunchKernelGGL(saliency_part_kernel<true>, grid, dim3(256), 0, stream, a);
  else hipLaunchKernelGGL(saliency_part_kernel<false>, grid, dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  float* chunk_tot = part + (size_t)kSalSplits * B * d_ff;
  const int cchunks = (d_ff + 255) / 256;
  hipLaunchKernelGGL(saliency_combine_kernel, dim3(cchunks, B), dim3(256), 0, stream, (const float*)part, splits,
                     B, kept_offsets, cap, mask, d_ff, saliency, chunk_tot);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(leakage_kernel, dim3((B + 3) / 4), dim3(256), 0, stream, (const float*)chunk_tot, cchunks,
                     B, delta, lambda, use_pruned, kept_offsets, cap, (uint8_t*)nullptr);
  return hipGetLastError();
}

hipError_t launch_mask_channels(char* act, const int32_t* kept_offsets, int B, int cap, int d_ff, bool bf16,
                                const uint8_t* mask, const uint8_t* use_pruned, hipStream_t stream) {
  if (cap <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(mask_kernel<true>, dim3(cap), dim3(256), 0, stream, act, kept_offsets, B, cap, d_ff, mask,
                       use_pruned);
  else
    hipLaunchKernelGGL(mask_kernel<false>, dim3(cap), dim3(256), 0, stream, act, kept_offsets, B, cap, d_ff, mask,
                       use_pruned);
  return hipGetLastError();
}

}  // namespace ce
