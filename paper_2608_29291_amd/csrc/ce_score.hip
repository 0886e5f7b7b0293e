// Core + expansion routing logits (paper section 3.2, Eq. 4) and sigmoid
// scores (section 3.4, Eq. 6).
//
//   understanding token:  l = c(h)            c(h) = w2c . SiLU(W1c h + b1c) + b2c
//   generation token:     l = c(h) + e_m(h)   e_m(h) = w2e[m] . SiLU(W1e[m] h + b1e[m]) + b2e[m]
//   m = min(floor(n_seg * t_b), n_seg - 1), t_b the timestep of the token's sequence.
//
// One workgroup scores a tile of up to 64 consecutive tokens of one sequence
// (tiles never straddle sequences, so the segment m is uniform per tile). The
// first layer is an MFMA GEMM of the stacked [core ; expansion m] rank rows
// (A operand) against the token rows (B operand), double-buffered through
// LDS. Tiles holding no generation token skip the expansion rows; tiles of
// only always-kept tokens read nothing and write +inf. The SiLU, the w2 dot
// and the biases run in fp32 on the accumulators; the sum over ranks is done
// in registers, then across the two lane halves, then across the two rank
// waves in a fixed order (deterministic).
#include "ce_device.hpp"
#include "ce_launch.hpp"

namespace ce {

namespace {

constexpr int kTR = 64;        // tokens per tile
constexpr int kMaxBlk = 16;    // rank blocks of 32 (r_core + r_exp <= 512)
constexpr int kMWmax = kMaxBlk / 2;

template <bool kBF16>
__global__ __launch_bounds__(256) void score_kernel(ScoreArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ float red_core[2][kTR];
  __shared__ float red_exp[2][kTR];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int ww = wave & 1;   // rank-block parity handled by this wave
  const int wt = wave >> 1;  // 32-token half handled by this wave

  // ---- locate the tile: sequence b, tokens [lo, hi) ----
  int tile = blockIdx.x;
  int b = -1, lo = 0, hi = 0;
  for (int s = 0; s < a.B; ++s) {
    int s0 = a.seq_offsets[s], s1 = a.seq_offsets[s + 1];
    s0 = s0 < 0 ? 0 : (s0 > a.T ? a.T : s0);
    s1 = s1 < s0 ? s0 : (s1 > a.T ? a.T : s1);
    const int nt = (s1 - s0 + kTR - 1) / kTR;
    if (tile < nt) {
      b = s;
      lo = s0 + tile * kTR;
      hi = min(lo + kTR, s1);
      break;
    }
    tile -= nt;
  }
  if (b < 0) return;

  // ---- token kinds in the tile ----
  const uint8_t fl = (tid < hi - lo) ? a.flags[lo + tid] : (uint8_t)2;
  const bool is_keep = (fl & 2) != 0;
  const bool is_gen = ((fl & 1) != 0) && !is_keep;
  const int any_scored = __syncthreads_or(!is_keep);
  const int any_gen = __syncthreads_or(is_gen);
  if (!any_scored) {
    if (tid < hi - lo) {
      a.logits[lo + tid] = __builtin_inff();
      if (a.probs) a.probs[lo + tid] = 1.0f;
    }
    return;
  }
  int m = 0;
  if (any_gen && a.r_exp > 0) {
    // exact product in double: floor(n_seg * t) never rounds across a bin edge
    const double mf = floor((double)a.n_seg * (double)a.t[b]);
    m = (mf >= 0.0) ? (int)fmin(mf, (double)(a.n_seg - 1)) : 0;  // NaN -> 0
  }
  const int nc = a.r_core / 32;
  const int nblk = nc + ((any_gen && a.r_exp > 0) ? a.r_exp / 32 : 0);
  const int stage = (nblk * 32 + kTR) * kKB;

  // ---- per-thread load pointers ----
  const int cchunk = tid & 7;
  const int rsub = tid >> 3;  // 0..31: row inside a 32-row block
  const char* wexp_base = a.w1e + ((int64_t)m * a.r_exp) * a.h_ld;
  auto wrow = [&](int blk) -> const char* {
    if (blk < nc) return a.w1c + (int64_t)(32 * blk + rsub) * a.h_ld + cchunk * 16;
    return wexp_base + (int64_t)(32 * (blk - nc) + rsub) * a.h_ld + cchunk * 16;
  };
  const char* tsrc[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = i * 32 + rsub;
    // always-kept rows are never scored: their hidden states are not read
    const bool live = (lo + r < hi) && !(a.flags[lo + r] & 2);
    tsrc[i] = live ? a.hidden + (int64_t)(lo + r) * a.h_ld + cchunk * 16 : nullptr;
  }

  u32x4_t wreg[kMaxBlk], treg[2];
  auto gload = [&](int kb) {
    const int koff = kb * kKB;
#pragma unroll
    for (int i = 0; i < kMaxBlk; ++i)
      if (i < nblk) wreg[i] = gload16_cached(wrow(i) + koff);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (tsrc[i]) treg[i] = gload16_cached(tsrc[i] + koff);
      else treg[i] = u32x4_t{0u, 0u, 0u, 0u};
    }
  };
  auto lstore = [&](int buf) {
    char* s = smem + buf * stage;
#pragma unroll
    for (int i = 0; i < kMaxBlk; ++i)
      if (i < nblk) lds_write16(s, lds_chunk_off(i * 32 + rsub, cchunk), wreg[i]);
#pragma unroll
    for (int i = 0; i < 2; ++i)
      lds_write16(s + nblk * 32 * kKB, lds_chunk_off(i * 32 + rsub, cchunk), treg[i]);
  };

  f32x16_t acc[kMWmax];
#pragma unroll
  for (int i = 0; i < kMWmax; ++i) acc[i] = f32x16_t{};

  const int nk = a.k_bytes / kKB;
  const int lrow = lane & 31;
  const int lhalf = lane >> 5;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kb = 0; kb < nk; ++kb) {
    if (kb + 1 < nk) gload(kb + 1);
    const char* s = smem + (kb & 1) * stage;
    const char* st = s + nblk * 32 * kKB;
#pragma unroll
    for (int step = 0; step < 4; ++step) {
      const int c = 2 * step + lhalf;
      const u32x4_t fb = lds_read16(st, lds_chunk_off(wt * 32 + lrow, c));
#pragma unroll
      for (int i = 0; i < kMWmax; ++i) {
        const int blk = 2 * i + ww;
        if (blk < nblk) {
          const u32x4_t fa = lds_read16(s, lds_chunk_off(blk * 32 + lrow, c));
          mfma_step<kBF16>(acc[i], fa, fb);
        }
      }
    }
    if (kb + 1 < nk) lstore((kb + 1) & 1);
    __syncthreads();
  }

  // ---- epilogue: SiLU, w2 dot, sum over ranks ----
  float pc = 0.0f, pe = 0.0f;
#pragma unroll
  for (int i = 0; i < kMWmax; ++i) {
    const int blk = 2 * i + ww;
    if (blk >= nblk) continue;
    const bool core = blk < nc;
    const int rb = core ? 32 * blk : 32 * (blk - nc);
    const float* b1 = core ? a.b1c : (a.b1e ? a.b1e + m * a.r_exp : nullptr);
    const float* w2 = core ? a.w2c : a.w2e + m * a.r_exp;
    float part = 0.0f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int r = rb + 8 * (v >> 2) + 4 * lhalf + (v & 3);
      float z = acc[i][v];
      if (b1) z += b1[r];
      part += w2[r] * silu_f32(z);
    }
    if (core) pc += part;
    else pe += part;
  }
  pc += __shfl_xor(pc, 32);
  pe += __shfl_xor(pe, 32);
  if (lhalf == 0) {
    red_core[ww][wt * 32 + lrow] = pc;
    red_exp[ww][wt * 32 + lrow] = pe;
  }
  __syncthreads();
  if (tid < hi - lo) {
    float l;
    if (is_keep) {
      l = __builtin_inff();
    } else {
      l = (red_core[0][tid] + red_core[1][tid]) + a.b2c;
      if (is_gen && a.r_exp > 0) {
        float e = red_exp[0][tid] + red_exp[1][tid];
        if (a.b2e) e += a.b2e[m];
        l += e;
      }
    }
    a.logits[lo + tid] = l;
    if (a.probs) a.probs[lo + tid] = is_keep ? 1.0f : 1.0f / (1.0f + expf(-l));
  }
}

template <bool kBF16>
hipError_t launch_t(const ScoreArgs& a, hipStream_t stream) {
  const int tiles = (a.T + kTR - 1) / kTR + a.B;
  const int rows = a.r_core + a.r_exp;
  const size_t lds = (size_t)2 * (rows + kTR) * kKB;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)score_kernel<kBF16>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(score_kernel<kBF16>, dim3(tiles), dim3(256), lds, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score(const ScoreArgs& a, bool bf16, hipStream_t stream) {
  if (a.T == 0) return hipSuccess;
  return bf16 ? launch_t<true>(a, stream) : launch_t<false>(a, stream);
}

}  // namespace ce
