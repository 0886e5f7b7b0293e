// Core + expansion routing logits (paper section 3.2, Eq. 4) and sigmoid
// scores (section 3.4, Eq. 6).
//
//   understanding token:  l = c(h)            c(h) = w2c . SiLU(W1c h + b1c) + b2c
//   generation token:     l = c(h) + e_m(h)   e_m(h) = w2e[m] . SiLU(W1e[m] h + b1e[m]) + b2e[m]
//   m = min(floor(n_seg * t_b), n_seg - 1), t_b the timestep of the token's sequence.
//
// Two launches:
//   score_tile_kernel   grid = token tiles x rank groups. A token tile holds
//                       kTR consecutive tokens of one sequence (tiles never
//                       straddle sequences, so the segment m is uniform); a
//                       rank group holds kRG ranks of the core scorer or of the
//                       active expansion. The first layer is an MFMA GEMM of the
//                       group's W1 rows (A operand) against the token rows (B
//                       operand); its epilogue applies b1, SiLU and the w2 dot
//                       over the group's ranks in fp32 and writes one partial
//                       logit per (group, token). Group 0 of the core adds b2c,
//                       group 0 of the expansion adds b2e[m].
//   score_finish_kernel sums a token's partials in a fixed order (core groups,
//                       then expansion groups for generation tokens), writes
//                       +inf for always-kept tokens, and the sigmoid score.
// Everything is deterministic (no atomics).
//
// K is streamed in 64-byte slabs fetched straight into a ring of LDS buffers
// by buffer loads with the LDS bit (one 1 KB wave instruction = 16 rows of 64
// bytes), so kStages - 1 slabs are in flight: the kernel is bound by memory
// latency and bandwidth, not by math. Rows are stored at chunk c ^ skey(r).
// Always-kept and out-of-tile token rows are fetched from past the end of the
// buffer resource, which returns zeros without touching memory, so their
// hidden states are never read.
#include "ce_device.hpp"
#include "ce_launch.hpp"

namespace ce {

namespace {

constexpr int kRowB = 64;  // bytes of K per staged row

__device__ __forceinline__ uint32_t skey(uint32_t r) { return ((r >> 1) ^ (r >> 3)) & 3u; }

// wait until at most `ahead` slabs of kPer instructions each remain in flight
template <int kPer, int kMaxAhead>
__device__ __forceinline__ void wait_slabs(int ahead) {
  if (ahead >= 6 && kMaxAhead >= 6) wait_vmcnt<6 * kPer>();
  else if (ahead == 5 && kMaxAhead >= 5) wait_vmcnt<5 * kPer>();
  else if (ahead == 4 && kMaxAhead >= 4) wait_vmcnt<4 * kPer>();
  else if (ahead == 3 && kMaxAhead >= 3) wait_vmcnt<3 * kPer>();
  else if (ahead == 2 && kMaxAhead >= 2) wait_vmcnt<2 * kPer>();
  else if (ahead == 1 && kMaxAhead >= 1) wait_vmcnt<1 * kPer>();
  else wait_vmcnt<0>();
}

template <bool kBF16, int kRG, int kTR, int kStages>
__global__ __launch_bounds__(256) void score_tile_kernel(ScoreArgs a, int ncg, float* __restrict__ part) {
  constexpr int kMW = kRG / 64;  // rank blocks per wave (2 x 2 waves)
  constexpr int kMT = kTR / 64;  // token blocks per wave
  constexpr int kStage = (kRG + kTR) * kRowB;
  constexpr int kWPer = kRG / 32;  // DMA instructions per slab, weight waves (0-1)
  constexpr int kTPer = kTR / 32;  // DMA instructions per slab, token waves (2-3)
  __shared__ __attribute__((aligned(1024))) char smem[kStages * kStage];
  __shared__ float red[2][kTR];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ww = wave & 1;
  const int wt = wave >> 1;

  // ---- locate the token tile: sequence b, tokens [lo, hi) ----
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
  const int n = hi - lo;

  // ---- token kinds in the tile, rank group ----
  bool kp = true, gen = false;
  if (tid < n) {
    const uint8_t f = a.flags[lo + tid];
    kp = (f & 2) != 0;
    gen = ((f & 1) != 0) && !kp;
  }
  const int any_scored = __syncthreads_or(!kp);
  const int any_gen = __syncthreads_or(gen);
  const int g = blockIdx.y;
  const bool core = g < ncg;
  if (!any_scored || (!core && !any_gen)) return;
  int m = 0;
  if (!core) {
    // exact product in double: floor(n_seg * t) never rounds across a bin edge
    const double mf = floor((double)a.n_seg * (double)a.t[b]);
    m = (mf >= 0.0) ? (int)fmin(mf, (double)(a.n_seg - 1)) : 0;  // NaN -> 0
  }
  const int r_tot = core ? a.r_core : a.r_exp;
  const int rank_lo = (core ? g : g - ncg) * kRG;
  const int nr = min(kRG, r_tot - rank_lo);
  const char* wbase = core ? a.w1c + (int64_t)rank_lo * a.h_ld
                           : a.w1e + ((int64_t)m * a.r_exp + rank_lo) * a.h_ld;

  // ---- DMA plan: waves 0-1 fetch the group's weight rows, waves 2-3 the token rows ----
  const bool is_w = wave < 2;
  const int r16 = lane >> 2;
  const int pch = lane & 3;
  const __amdgpu_buffer_rsrc_t wrs = make_rsrc(wbase, (uint32_t)(nr * a.h_ld));
  const __amdgpu_buffer_rsrc_t trs = make_rsrc(a.hidden + (int64_t)lo * a.h_ld, (uint32_t)(n * a.h_ld));
  constexpr int kPerMax = kWPer > kTPer ? kWPer : kTPer;
  uint32_t voff[kPerMax];
#pragma unroll
  for (int q = 0; q < kPerMax; ++q) {
    if (is_w) {
      const int r = (wave & 1) * (kRG / 2) + 16 * q + r16;
      voff[q] = (uint32_t)(r * a.h_ld) + ((uint32_t)(pch ^ (int)skey((uint32_t)r)) << 4);
    } else {
      const int r = (wave & 1) * (kTR / 2) + 16 * q + r16;
      const bool live = r < n && !(a.flags[lo + (r < n ? r : 0)] & 2);
      // rows that are never scored read past the resource end: zeros, no traffic
      voff[q] = live ? (uint32_t)(r * a.h_ld) + ((uint32_t)(pch ^ (int)skey((uint32_t)r)) << 4)
                     : 0x7ffffff0u;
    }
  }
  auto dma = [&](int kb, int buf) __attribute__((always_inline)) {
    const int soff = kb * kRowB;
    if (is_w) {
      char* region = smem + buf * kStage + (wave & 1) * (kRG / 2) * kRowB;
#pragma unroll
      for (int q = 0; q < kWPer; ++q)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            wrs, (__attribute__((address_space(3))) void*)(region + 16 * q * kRowB), 16, (int)voff[q],
            soff, 0, 0);
    } else {
      char* region = smem + buf * kStage + kRG * kRowB + (wave & 1) * (kTR / 2) * kRowB;
#pragma unroll
      for (int q = 0; q < kTPer; ++q)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            trs, (__attribute__((address_space(3))) void*)(region + 16 * q * kRowB), 16, (int)voff[q],
            soff, 0, 0);
    }
  };

  f32x16_t acc[kMW][kMT];
#pragma unroll
  for (int i = 0; i < kMW; ++i)
#pragma unroll
    for (int j = 0; j < kMT; ++j) acc[i][j] = f32x16_t{};
  const int lrow = lane & 31;
  const int lhalf = lane >> 5;
  const uint32_t rkey = skey((uint32_t)lrow);
  const uint32_t rowa = (uint32_t)((ww * (kRG / 2) + lrow) * kRowB);
  const uint32_t rowb = (uint32_t)(kRG * kRowB + (wt * (kTR / 2) + lrow) * kRowB);

  const int nk = a.k_bytes / kRowB;
  const int pre = min(nk, kStages - 1);
  for (int s = 0; s < pre; ++s) dma(s, s);
  int buf = 0;
  for (int kb = 0; kb < nk; ++kb) {
    const int ahead = min(nk - 1 - kb, kStages - 2);
    if (is_w) wait_slabs<kWPer, kStages - 2>(ahead);
    else wait_slabs<kTPer, kStages - 2>(ahead);
    lds_barrier();
    if (kb + kStages - 1 < nk) {
      int nb = buf + kStages - 1;
      nb = nb >= kStages ? nb - kStages : nb;
      dma(kb + kStages - 1, nb);
    }
    const char* sw = smem + buf * kStage;
#pragma unroll
    for (int step = 0; step < 2; ++step) {
      const uint32_t off = (((uint32_t)(2 * step + lhalf)) ^ rkey) << 4;
      u32x4_t fa[kMW], fb[kMT];
#pragma unroll
      for (int i = 0; i < kMW; ++i) fa[i] = *reinterpret_cast<const u32x4_t*>(sw + rowa + off + 32 * i * kRowB);
#pragma unroll
      for (int j = 0; j < kMT; ++j) fb[j] = *reinterpret_cast<const u32x4_t*>(sw + rowb + off + 32 * j * kRowB);
#pragma unroll
      for (int i = 0; i < kMW; ++i)
#pragma unroll
        for (int j = 0; j < kMT; ++j) mfma_step<kBF16>(acc[i][j], fa[i], fb[j]);
    }
    buf = buf + 1 == kStages ? 0 : buf + 1;
  }

  // ---- epilogue: b1, SiLU, w2 dot over this wave's ranks ----
  const float* b1 = core ? a.b1c : (a.b1e ? a.b1e + m * a.r_exp : nullptr);
  const float* w2 = core ? a.w2c : a.w2e + m * a.r_exp;
#pragma unroll
  for (int j = 0; j < kMT; ++j) {
    float pj = 0.0f;
#pragma unroll
    for (int i = 0; i < kMW; ++i) {
      const int rb = ww * (kRG / 2) + 32 * i;  // rank block offset inside the group
      if (rb >= nr) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = rank_lo + rb + 8 * (v >> 2) + 4 * lhalf + (v & 3);
        float z = acc[i][j][v];
        if (b1) z += b1[r];
        pj += w2[r] * silu_f32(z);
      }
    }
    pj += __shfl_xor(pj, 32);
    if (lhalf == 0) red[ww][wt * (kTR / 2) + 32 * j + lrow] = pj;
  }
  __syncthreads();
  if (tid < n) {
    float p = red[0][tid] + red[1][tid];
    if (rank_lo == 0) {
      if (core) p += a.b2c;
      else if (a.b2e) p += a.b2e[m];
    }
    part[(int64_t)g * a.T + lo + tid] = p;
  }
}

__global__ __launch_bounds__(256) void score_finish_kernel(ScoreArgs a, int ncg, int neg,
                                                           const float* __restrict__ part) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= a.T) return;
  const uint8_t f = a.flags[i];
  float l;
  if (f & 2) {
    l = __builtin_inff();
  } else {
    l = 0.0f;
    for (int g = 0; g < ncg; ++g) l += part[(int64_t)g * a.T + i];
    if ((f & 1) && a.r_exp > 0) {
      float e = 0.0f;
      for (int g = 0; g < neg; ++g) e += part[(int64_t)(ncg + g) * a.T + i];
      l += e;
    }
  }
  a.logits[i] = l;
  if (a.probs) a.probs[i] = (f & 2) ? 1.0f : 1.0f / (1.0f + expf(-l));
}

template <bool kBF16, int kRG, int kTR, int kStages>
hipError_t launch_tiles(const ScoreArgs& a, float* part, hipStream_t stream) {
  const int ncg = (a.r_core + kRG - 1) / kRG;
  const int neg = (a.r_exp + kRG - 1) / kRG;
  const int tiles = (a.T + kTR - 1) / kTR + a.B;
  hipLaunchKernelGGL((score_tile_kernel<kBF16, kRG, kTR, kStages>), dim3(tiles, ncg + neg), dim3(256), 0,
                     stream, a, ncg, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(score_finish_kernel, dim3((a.T + 255) / 256), dim3(256), 0, stream, a, ncg, neg,
                     (const float*)part);
  return hipGetLastError();
}

}  // namespace

// Tile choice: 64 ranks x 64 tokens keeps ~270+ workgroups busy on the
// narrow (d <= 2048) workloads; 128 x 128 halves the weight and token re-reads
// for wide ones (re-read traffic = T*d*(R/kRG) + R*d*(T/kTR)).
hipError_t launch_score(const ScoreArgs& a, bool bf16, float* part, hipStream_t stream) {
  if (a.T == 0) return hipSuccess;
  const bool wide = a.k_bytes >= 4096;
  if (bf16) {
    if (wide) return launch_tiles<true, 128, 128, 6>(a, part, stream);
    return launch_tiles<true, 64, 64, 8>(a, part, stream);
  }
  return launch_tiles<false, 64, 64, 8>(a, part, stream);
}

}  // namespace ce
