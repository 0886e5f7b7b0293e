// SwiGLU FFN over the packed (retained) rows: the gate/up GEMM with the SwiGLU
// epilogue, and the down GEMM with an optional residual-scatter epilogue.
//
// Both are "weights x tokens" GEMMs on MFMA (bf16 32x32x16 with fp32
// accumulation, or fp32 32x32x2 for fp32 data). A workgroup of kWW x kWT waves
// owns a kWR x kTR tile (weight rows x token rows); each wave owns a
// (kWR/kWW) x (kTR/kWT) sub-tile of 32x32 MFMA blocks. K is streamed in
// 128-byte steps through an XOR-swizzled LDS tile, double-buffered (one
// barrier per step) or single-buffered with a register prefetch (two barriers
// per step). With 8 waves, two waves share each SIMD, so one wave's MFMAs run
// while the other waits on LDS.
//
// Row mapping: GEMM row j (packed order, grouped by FFN set for MoT) maps to a
// source row through up to two index arrays: r = map2[map1[j]] (each level is
// skipped when its pointer is NULL). This lets the same kernel read rows
// straight out of the full hidden-state matrix (the gather fused into the
// token loads) or out of a packed buffer, and write results straight back to
// the token rows (the scatter fused into the epilogue).
//
// Tile order is XCD-aware: the hardware hands workgroup L to XCD L % 8, so the
// linear id is remapped to give each XCD a contiguous range of tiles, ordered
// feature-tile major; the weight tile a CU loads is then mostly shared with
// the other CUs of its XCD through that XCD's L2.
//
// The number of packed rows Kt and the size n0 of the first MoT group live in
// device memory; the grid is sized from the host-known capacity and tiles past
// Kt exit at once.
#include "ce_device.hpp"
#include "ce_launch.hpp"

namespace ce {

namespace {

__device__ __forceinline__ int map_row(int j, const int32_t* m1, const int32_t* m2) {
  int r = m1 ? m1[j] : j;
  return m2 ? m2[r] : r;
}

constexpr int kXcds = 8;

// kMode 0: gate/up + SwiGLU -> out[orow(j)][f]
// kMode 1: down (+ residual) -> out[orow(j)][f]
// kWW x kWT waves; each wave owns (kWR/kWW) x (kTR/kWT).
template <bool kBF16, int kMode, int kWR, int kTR, int kWW, int kWT, int kStages>
__global__ __launch_bounds__(64 * kWW * kWT) void ffn_gemm_kernel(FfnGemmArgs a, int n_tt, int n_ft) {
  constexpr int kThreads = 64 * kWW * kWT;
  constexpr int kElem = kBF16 ? 2 : 4;
  constexpr int kWRw = kWR / kWW;  // weight rows per wave
  constexpr int kTRw = kTR / kWT;  // token rows per wave
  constexpr int kMW = kWRw / 32;
  constexpr int kMT = kTRw / 32;
  static_assert(kMode == 1 || (kMW % 2) == 0, "gate/up blocks come in pairs");
  constexpr int kRowsPerPass = kThreads / kChunks;  // tile rows loaded per pass
  constexpr int kWLoads = kWR / kRowsPerPass;
  constexpr int kTLoads = kTR / kRowsPerPass;
  static_assert(kWLoads * kRowsPerPass == kWR && kTLoads * kRowsPerPass == kTR, "tile / threads");
  static_assert(kMode == 1 || (kRowsPerPass % 32) == 0 || (32 % kRowsPerPass) == 0, "pass rows");
  constexpr int kStage = (kWR + kTR) * kKB;

  __shared__ __attribute__((aligned(16))) char smem[kStages * kStage];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int ww = wave % kWW;
  const int wt = wave / kWW;

  // ---- XCD-aware tile order ----
  const int total = n_tt * n_ft;
  const int per = (total + kXcds - 1) / kXcds;
  const int w = (int)(blockIdx.x % kXcds) * per + (int)(blockIdx.x / kXcds);
  if (w >= total) return;
  const int ft = w / n_tt;
  const int tt = w - ft * n_tt;

  // ---- which packed rows this tile covers (grouped by weight set) ----
  int kt = *a.kt_ptr;
  kt = kt < 0 ? 0 : (kt > a.cap ? a.cap : kt);
  int n0 = kt;
  if (a.n_sets == 2 && a.n0_ptr) {
    n0 = *a.n0_ptr;
    n0 = n0 < 0 ? 0 : (n0 > kt ? kt : n0);
  }
  const int tiles0 = (n0 + kTR - 1) / kTR;
  int set, row_lo, row_hi;
  if (tt < tiles0) {
    set = 0;
    row_lo = tt * kTR;
    row_hi = min(row_lo + kTR, n0);
  } else {
    set = 1;
    row_lo = n0 + (tt - tiles0) * kTR;
    row_hi = min(row_lo + kTR, kt);
  }
  if (row_lo >= row_hi) return;

  const int n_feat = a.n_feat;
  constexpr int kFTile = (kMode == 0) ? kWR / 2 : kWR;
  const int f0 = ft * kFTile;

  // ---- per-thread source rows (fixed over the K loop) ----
  // Rows outside the tile (features >= n_feat, packed rows >= row_hi) are read
  // from a clamped, valid row instead of being predicated: their products only
  // reach outputs the epilogue never stores, and the loads stay branch-free.
  const int cchunk = tid & 7;
  const int rsub = tid >> 3;  // 0 .. kRowsPerPass-1
  const char* wsrc[kWLoads];
#pragma unroll
  for (int i = 0; i < kWLoads; ++i) {
    const int r = i * kRowsPerPass + rsub;  // tile row
    int feat;
    const char* base;
    if constexpr (kMode == 0) {
      const int blk = r >> 5;  // even blocks: gate rows, odd blocks: up rows
      feat = f0 + 32 * (blk >> 1) + (r & 31);
      base = (blk & 1) ? a.w1[set] : a.w0[set];
    } else {
      feat = f0 + r;
      base = a.w0[set];
    }
    feat = feat < n_feat ? feat : n_feat - 1;
    wsrc[i] = base + (int64_t)feat * a.w_ld + cchunk * 16;
  }
  const char* tsrc[kTLoads];
#pragma unroll
  for (int i = 0; i < kTLoads; ++i) {
    int j = row_lo + i * kRowsPerPass + rsub;
    j = j < row_hi ? j : row_hi - 1;
    tsrc[i] = a.tok + (int64_t)map_row(j, a.map1, a.map2) * a.tok_ld + cchunk * 16;
  }

  u32x4_t wreg[kWLoads], treg[kTLoads];
  auto gload = [&](int kb) {
    const int koff = kb * kKB;
#pragma unroll
    for (int i = 0; i < kWLoads; ++i) wreg[i] = gload16_cached(wsrc[i] + koff);
#pragma unroll
    for (int i = 0; i < kTLoads; ++i) treg[i] = gload16_cached(tsrc[i] + koff);
  };
  auto lstore = [&](int buf) {
    char* s = smem + buf * kStage;
#pragma unroll
    for (int i = 0; i < kWLoads; ++i)
      lds_write16(s, lds_chunk_off(i * kRowsPerPass + rsub, cchunk), wreg[i]);
#pragma unroll
    for (int i = 0; i < kTLoads; ++i)
      lds_write16(s + kWR * kKB, lds_chunk_off(i * kRowsPerPass + rsub, cchunk), treg[i]);
  };

  f32x16_t acc[kMW][kMT];
#pragma unroll
  for (int i = 0; i < kMW; ++i)
#pragma unroll
    for (int j = 0; j < kMT; ++j) acc[i][j] = f32x16_t{};

  const int lrow = lane & 31;
  const int lhalf = lane >> 5;
  auto compute = [&](int buf) {
    const char* sw = smem + buf * kStage;
    const char* st = sw + kWR * kKB;
#pragma unroll
    for (int step = 0; step < 4; ++step) {
      const int c = 2 * step + lhalf;
      u32x4_t fa[kMW], fb[kMT];
#pragma unroll
      for (int i = 0; i < kMW; ++i) fa[i] = lds_read16(sw, lds_chunk_off(ww * kWRw + 32 * i + lrow, c));
#pragma unroll
      for (int j = 0; j < kMT; ++j) fb[j] = lds_read16(st, lds_chunk_off(wt * kTRw + 32 * j + lrow, c));
#pragma unroll
      for (int i = 0; i < kMW; ++i)
#pragma unroll
        for (int j = 0; j < kMT; ++j) mfma_step<kBF16>(acc[i][j], fa[i], fb[j]);
    }
  };

  const int nk = a.k_bytes / kKB;
  gload(0);
  lstore(0);
  __syncthreads();
  if constexpr (kStages == 2) {
    for (int kb = 0; kb < nk; ++kb) {
      if (kb + 1 < nk) gload(kb + 1);
      compute(kb & 1);
      if (kb + 1 < nk) lstore((kb + 1) & 1);
      __syncthreads();
    }
  } else {
    for (int kb = 0; kb < nk; ++kb) {
      if (kb + 1 < nk) gload(kb + 1);
      compute(0);
      __syncthreads();
      if (kb + 1 < nk) {
        lstore(0);
        __syncthreads();
      }
    }
  }

  // ---- epilogue ----
#pragma unroll
  for (int j = 0; j < kMT; ++j) {
    const int jr = row_lo + wt * kTRw + 32 * j + lrow;
    if (jr >= row_hi) continue;
    const int orow_idx = map_row(jr, a.omap1, a.omap2);
    char* orow = a.out + (int64_t)orow_idx * a.out_ld;
    if constexpr (kMode == 0) {
#pragma unroll
      for (int p = 0; p < kMW / 2; ++p) {
        const int fb = f0 + 32 * (ww * (kMW / 2) + p) + 4 * lhalf;
        if (fb >= n_feat) continue;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x16_t& ag = acc[2 * p][j];
          const f32x16_t& au = acc[2 * p + 1][j];
          float v0 = silu_f32(ag[4 * g + 0]) * au[4 * g + 0];
          float v1 = silu_f32(ag[4 * g + 1]) * au[4 * g + 1];
          float v2 = silu_f32(ag[4 * g + 2]) * au[4 * g + 2];
          float v3 = silu_f32(ag[4 * g + 3]) * au[4 * g + 3];
          store4<kBF16>(orow + (int64_t)(fb + 8 * g) * kElem, v0, v1, v2, v3);
        }
      }
    } else {
      const char* rrow = a.res ? a.res + (int64_t)orow_idx * a.res_ld : nullptr;
#pragma unroll
      for (int i = 0; i < kMW; ++i) {
        const int fb = f0 + ww * kWRw + 32 * i + 4 * lhalf;
        if (fb >= n_feat) continue;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int f = fb + 8 * g;
          float v0 = acc[i][j][4 * g + 0], v1 = acc[i][j][4 * g + 1];
          float v2 = acc[i][j][4 * g + 2], v3 = acc[i][j][4 * g + 3];
          if (rrow) {
            f32x4_t r = load4<kBF16>(rrow + (int64_t)f * kElem);
            v0 += r.x; v1 += r.y; v2 += r.z; v3 += r.w;
          }
          store4<kBF16>(orow + (int64_t)f * kElem, v0, v1, v2, v3);
        }
      }
    }
  }
}

template <bool kBF16, int kMode, int kWR, int kTR, int kWW, int kWT, int kStages>
hipError_t launch_cfg(const FfnGemmArgs& a, hipStream_t stream) {
  constexpr int kFTile = (kMode == 0) ? kWR / 2 : kWR;
  const int n_tt = (a.cap + kTR - 1) / kTR + (a.n_sets - 1);
  const int n_ft = (a.n_feat + kFTile - 1) / kFTile;
  if (n_tt <= 0 || n_ft <= 0) return hipSuccess;
  const int total = n_tt * n_ft;
  const int grid = ((total + kXcds - 1) / kXcds) * kXcds;
  hipLaunchKernelGGL((ffn_gemm_kernel<kBF16, kMode, kWR, kTR, kWW, kWT, kStages>), dim3(grid),
                     dim3(64 * kWW * kWT), 0, stream, a, n_tt, n_ft);
  return hipGetLastError();
}

}  // namespace

// Tile shapes (weight rows x token rows, wave grid, LDS stages), from a sweep
// on the five named workloads:
//   gate/up: 256 x 256, 4 x 2 waves, 2 stages (128 output features x 256 tokens)
//   down:    256 x 128, 4 x 2 waves, 2 stages when d < 3072 (few output tiles);
//            128 x 128, 2 x 2 waves, 2 stages for the 7B width
// fp32 data (tiny workloads) uses 128 x 128 tiles.
hipError_t launch_ffn_gateup(const FfnGemmArgs& a, bool bf16, hipStream_t stream) {
  if (bf16) return launch_cfg<true, 0, 256, 256, 4, 2, 2>(a, stream);
  return launch_cfg<false, 0, 128, 128, 2, 2, 2>(a, stream);
}

hipError_t launch_ffn_down(const FfnGemmArgs& a, bool bf16, hipStream_t stream) {
  if (bf16) {
    if (a.n_feat < 3072) return launch_cfg<true, 1, 256, 128, 4, 2, 2>(a, stream);
    return launch_cfg<true, 1, 128, 128, 2, 2, 2>(a, stream);
  }
  return launch_cfg<false, 1, 128, 128, 2, 2, 2>(a, stream);
}

}  // namespace ce
