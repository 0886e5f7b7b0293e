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
#include <type_traits>

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
// kPf: how many K slabs ahead the global loads run (1, or 2 with two register
// sets); kGroup: feature tiles per group in the tile order.
template <bool kBF16, int kMode, int kWR, int kTR, int kWW, int kWT, int kStages, int kPf = 1,
          int kGroup = 1>
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

  // ---- XCD-aware, grouped tile order ----
  // Work item w runs on XCD w / per (contiguous ranges); items are ordered in
  // groups of kGroup feature tiles, token-tile major inside a group, so the
  // ~32 workgroups an XCD runs at once share kGroup weight tiles and
  // 32 / kGroup token tiles through its L2.
  const int total = n_tt * n_ft;
  const int per = (total + kXcds - 1) / kXcds;
  const int w = (int)(blockIdx.x % kXcds) * per + (int)(blockIdx.x / kXcds);
  if (w >= total) return;
  const int grp = w / (kGroup * n_tt);
  const int rem = w - grp * (kGroup * n_tt);
  const int gsz = min(kGroup, n_ft - grp * kGroup);
  const int tt = rem / gsz;
  const int ft = grp * kGroup + (rem - tt * gsz);

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

  struct Regs {
    u32x4_t w[kWLoads];
    u32x4_t t[kTLoads];
  };
  auto gload = [&](Regs& r, int kb) {
    const int koff = kb * kKB;
#pragma unroll
    for (int i = 0; i < kWLoads; ++i) r.w[i] = gload16_cached(wsrc[i] + koff);
#pragma unroll
    for (int i = 0; i < kTLoads; ++i) r.t[i] = gload16_cached(tsrc[i] + koff);
  };
  auto lstore = [&](const Regs& r, int buf) {
    char* s = smem + buf * kStage;
#pragma unroll
    for (int i = 0; i < kWLoads; ++i)
      lds_write16(s, lds_chunk_off(i * kRowsPerPass + rsub, cchunk), r.w[i]);
#pragma unroll
    for (int i = 0; i < kTLoads; ++i)
      lds_write16(s + kWR * kKB, lds_chunk_off(i * kRowsPerPass + rsub, cchunk), r.t[i]);
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
  if constexpr (kPf == 2) {
    static_assert(kStages == 2, "two-ahead prefetch uses two LDS buffers");
    // r0 / r1 alternate as the register sets of even / odd K slabs: the loads
    // of slab kb+2 are issued while slab kb is multiplied and written to LDS
    // one iteration later, so each load has two compute phases to land.
    Regs r0, r1;
    gload(r0, 0);
    if (nk > 1) gload(r1, 1);
    lstore(r0, 0);
    __syncthreads();
    for (int kb = 0; kb < nk; kb += 2) {
      if (kb + 2 < nk) gload(r0, kb + 2);
      compute(0);
      if (kb + 1 < nk) lstore(r1, 1);
      __syncthreads();
      if (kb + 1 >= nk) break;
      if (kb + 3 < nk) gload(r1, kb + 3);
      compute(1);
      if (kb + 2 < nk) lstore(r0, 0);
      __syncthreads();
    }
  } else if constexpr (kStages == 2) {
    Regs r;
    gload(r, 0);
    lstore(r, 0);
    __syncthreads();
    for (int kb = 0; kb < nk; ++kb) {
      if (kb + 1 < nk) gload(r, kb + 1);
      compute(kb & 1);
      if (kb + 1 < nk) lstore(r, (kb + 1) & 1);
      __syncthreads();
    }
  } else {
    Regs r;
    gload(r, 0);
    lstore(r, 0);
    __syncthreads();
    for (int kb = 0; kb < nk; ++kb) {
      if (kb + 1 < nk) gload(r, kb + 1);
      compute(0);
      __syncthreads();
      if (kb + 1 < nk) {
        lstore(r, 0);
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

// Large-tile bf16 variant: 4 waves (2 x 2), each owning a 128 x 128 sub-tile
// (4 x 4 MFMA blocks, 256 fp32 accumulators kept in AGPRs), one wave per SIMD.
// LDS fragment reads are software-pipelined: the fragments of K step s+1 are
// read into the second register set while the 16 MFMAs of step s run, so the
// single wave on each SIMD never waits on LDS between MFMA groups. Per 128-byte
// K slab a wave reads 32 fragments for 64 MFMAs (half the LDS traffic per
// MFMA of a 64 x 128 wave tile).
template <int kMode, int kGroup>
__global__ __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1))) void ffn_gemm_big_kernel(FfnGemmArgs a, int n_tt, int n_ft) {
  constexpr int kWR = 256, kTR = 256;
  constexpr int kMW = 4, kMT = 4;
  constexpr int kLoads = 8;  // per operand per thread per slab
  constexpr int kStage = (kWR + kTR) * kKB;
  __shared__ __attribute__((aligned(16))) char smem[2 * kStage];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int ww = wave & 1;
  const int wt = wave >> 1;

  const int total = n_tt * n_ft;
  const int per = (total + kXcds - 1) / kXcds;
  const int w = (int)(blockIdx.x % kXcds) * per + (int)(blockIdx.x / kXcds);
  if (w >= total) return;
  const int grp = w / (kGroup * n_tt);
  const int rem = w - grp * (kGroup * n_tt);
  const int gsz = min(kGroup, n_ft - grp * kGroup);
  const int tt = rem / gsz;
  const int ft = grp * kGroup + (rem - tt * gsz);

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
  const int cchunk = tid & 7;
  const int rsub = tid >> 3;  // 0..31

  // Buffer loads: one per-lane offset for all weight rows of this thread
  // (row blocks differ by a wave-uniform offset); rows past n_feat lie past
  // the resource's range and read as zero. Token rows are gathered, one
  // 32-bit offset each; rows past row_hi read a clamped valid row (their
  // results are never stored).
  __amdgpu_buffer_rsrc_t wr0, wr1;
  if constexpr (kMode == 0) {
    wr0 = make_rsrc(a.w0[set], (uint32_t)(n_feat * a.w_ld));
    wr1 = make_rsrc(a.w1[set], (uint32_t)(n_feat * a.w_ld));
  } else {
    wr0 = make_rsrc(a.w0[set], (uint32_t)(n_feat * a.w_ld));
    wr1 = wr0;
  }
  const __amdgpu_buffer_rsrc_t trs = make_rsrc(a.tok, 0xffffffffu);
  const uint32_t wvoff = (uint32_t)((int64_t)(f0 + rsub) * a.w_ld + cchunk * 16);
  uint32_t tvoff[kLoads];
#pragma unroll
  for (int i = 0; i < kLoads; ++i) {
    int j = row_lo + 32 * i + rsub;
    j = j < row_hi ? j : row_hi - 1;
    tvoff[i] = (uint32_t)((int64_t)map_row(j, a.map1, a.map2) * a.tok_ld + cchunk * 16);
  }

  // two register sets of in-flight global loads: the loads of slab kb+2 are
  // issued at the start of iteration kb and written to LDS at the end of
  // iteration kb+1, so each has almost two iterations of MFMA time to land
  u32x4_t rw0[kLoads], rt0[kLoads], rw1[kLoads], rt1[kLoads];
  auto gload = [&](u32x4_t (&rw)[kLoads], u32x4_t (&rt)[kLoads], int kb) __attribute__((always_inline)) {
    const uint32_t koff = (uint32_t)(kb * kKB);
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      // weight tile row block i: gate/up alternate in mode 0
      const uint32_t blk_off = (uint32_t)((kMode == 0 ? 32 * (i >> 1) : 32 * i) * a.w_ld);
      rw[i] = bload16((kMode == 0 && (i & 1)) ? wr1 : wr0, wvoff, blk_off + koff);
      rt[i] = bload16(trs, tvoff[i], koff);
    }
  };
  // LDS addresses are formed from two per-lane values plus immediates. The
  // swizzle key of tile row r = 32*i + x is (x ^ x>>3 ^ 4*i) & 7, so only the
  // parity of the row block i changes it. `opaque` hides the per-lane values
  // from loop-invariant hoisting, which would otherwise keep one address
  // register per fragment and per buffer alive across the K loop.
  auto opaque = [](uint32_t v) __attribute__((always_inline)) {
    asm volatile("" : "+v"(v));
    return v;
  };
  const uint32_t wkey = (uint32_t)((rsub ^ (rsub >> 3)) & 7);
  auto lstore = [&](const u32x4_t (&rw)[kLoads], const u32x4_t (&rt)[kLoads], int buf) __attribute__((always_inline)) {
    const uint32_t k = opaque(wkey);
    const uint32_t base = (uint32_t)(buf * kStage) + (uint32_t)rsub * kKB;
    const uint32_t even = base + ((cchunk ^ k) << 4);
    const uint32_t odd = base + ((cchunk ^ k ^ 4u) << 4);
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      const uint32_t o = ((i & 1) ? odd : even) + (uint32_t)(32 * i * kKB);
      *reinterpret_cast<u32x4_t*>(smem + o) = rw[i];
      *reinterpret_cast<u32x4_t*>(smem + o + kWR * kKB) = rt[i];
    }
  };

  f32x16_t acc[kMW][kMT];
#pragma unroll
  for (int i = 0; i < kMW; ++i)
#pragma unroll
    for (int j = 0; j < kMT; ++j) acc[i][j] = f32x16_t{};

  const int lrow = lane & 31;
  const int lhalf = lane >> 5;
  u32x4_t fa0[kMW], fb0[kMT], fa1[kMW], fb1[kMT];
  const uint32_t rkey = (uint32_t)((lrow ^ (lrow >> 3)) & 7);
  const uint32_t rowa = (uint32_t)((ww * 128 + lrow) * kKB);
  const uint32_t rowb = (uint32_t)(kWR * kKB + (wt * 128 + lrow) * kKB);
  auto read_frags = [&](u32x4_t (&fa)[kMW], u32x4_t (&fb)[kMT], const char* sw, int step) __attribute__((always_inline)) {
    const uint32_t k = opaque(rkey);
    const uint32_t c = (uint32_t)(2 * step + lhalf);
    const uint32_t se = (c ^ k) << 4;        // even row blocks
    const uint32_t so = (c ^ k ^ 4u) << 4;   // odd row blocks
    const char* pa = sw + rowa;
    const char* pb = sw + rowb;
#pragma unroll
    for (int i = 0; i < kMW; ++i)
      fa[i] = *reinterpret_cast<const u32x4_t*>(pa + ((i & 1) ? so : se) + 32 * i * kKB);
#pragma unroll
    for (int j = 0; j < kMT; ++j)
      fb[j] = *reinterpret_cast<const u32x4_t*>(pb + ((j & 1) ? so : se) + 32 * j * kKB);
  };
  auto mfmas = [&](const u32x4_t (&fa)[kMW], const u32x4_t (&fb)[kMT]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < kMW; ++i)
#pragma unroll
      for (int j = 0; j < kMT; ++j) mfma_step<true>(acc[i][j], fa[i], fb[j]);
  };

  // One K slab: fragments of step s+1 are read while the 16 MFMAs of step s
  // run; the next slab's LDS tile is written during the last step. The
  // scheduling groups pin that interleave (mask 0x008 MFMA, 0x100 LDS read,
  // 0x200 LDS write, 0x020 global read).
  auto slab = [&](auto load_tag, auto write_tag, const char* sw, int next_buf,
                  u32x4_t (&lw)[kLoads], u32x4_t (&lt)[kLoads], const u32x4_t (&sw_w)[kLoads],
                  const u32x4_t (&sw_t)[kLoads], int load_kb) __attribute__((always_inline)) {
    constexpr bool kLoad = decltype(load_tag)::value;
    constexpr bool kWrite = decltype(write_tag)::value;
    if constexpr (kLoad) gload(lw, lt, load_kb);
    read_frags(fa0, fb0, sw, 0);
    read_frags(fa1, fb1, sw, 1);
    mfmas(fa0, fb0);
    read_frags(fa0, fb0, sw, 2);
    mfmas(fa1, fb1);
    read_frags(fa1, fb1, sw, 3);
    mfmas(fa0, fb0);
    if constexpr (kWrite) lstore(sw_w, sw_t, next_buf);
    mfmas(fa1, fb1);
    if constexpr (kLoad) __builtin_amdgcn_sched_group_barrier(0x020, 2 * kLoads, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
    for (int st = 0; st < 3; ++st) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    }
    if constexpr (kWrite) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
      }
    } else {
      __builtin_amdgcn_sched_group_barrier(0x008, 16, 0);
    }
    __syncthreads();
  };
  using T = std::true_type;
  using F = std::false_type;

  const int nk = a.k_bytes / kKB;  // >= 2 (checked by the launcher)
  gload(rw0, rt0, 0);
  gload(rw1, rt1, 1);
  lstore(rw0, rt0, 0);
  __syncthreads();
  // Pairs of slabs (even slab in buffer 0, odd slab in buffer 1). The loads
  // two slabs ahead clamp the slab index to the last one: near the end they
  // re-read a slab from L2 and write it to a buffer that is never read again,
  // which keeps one branch-free loop body.
  int kb = 0;
  for (; kb + 1 < nk; kb += 2) {
    slab(T{}, T{}, smem, 1, rw0, rt0, rw1, rt1, min(kb + 2, nk - 1));
    slab(T{}, T{}, smem + kStage, 0, rw1, rt1, rw0, rt0, min(kb + 3, nk - 1));
  }
  if (kb < nk) slab(F{}, F{}, smem, 1, rw0, rt0, rw1, rt1, 0);  // odd slab count: last slab

#pragma unroll
  for (int j = 0; j < kMT; ++j) {
    const int jr = row_lo + wt * 128 + 32 * j + lrow;
    if (jr >= row_hi) continue;
    const int orow_idx = map_row(jr, a.omap1, a.omap2);
    char* orow = a.out + (int64_t)orow_idx * a.out_ld;
    if constexpr (kMode == 0) {
#pragma unroll
      for (int p = 0; p < kMW / 2; ++p) {
        const int fb0 = f0 + 32 * (ww * (kMW / 2) + p) + 4 * lhalf;
        if (fb0 >= n_feat) continue;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x16_t& ag = acc[2 * p][j];
          const f32x16_t& au = acc[2 * p + 1][j];
          float v0 = silu_f32(ag[4 * g + 0]) * au[4 * g + 0];
          float v1 = silu_f32(ag[4 * g + 1]) * au[4 * g + 1];
          float v2 = silu_f32(ag[4 * g + 2]) * au[4 * g + 2];
          float v3 = silu_f32(ag[4 * g + 3]) * au[4 * g + 3];
          store4<true>(orow + (int64_t)(fb0 + 8 * g) * 2, v0, v1, v2, v3);
        }
      }
    } else {
      const char* rrow = a.res ? a.res + (int64_t)orow_idx * a.res_ld : nullptr;
#pragma unroll
      for (int i = 0; i < kMW; ++i) {
        const int fb0 = f0 + ww * 128 + 32 * i + 4 * lhalf;
        if (fb0 >= n_feat) continue;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int f = fb0 + 8 * g;
          float v0 = acc[i][j][4 * g + 0], v1 = acc[i][j][4 * g + 1];
          float v2 = acc[i][j][4 * g + 2], v3 = acc[i][j][4 * g + 3];
          if (rrow) {
            f32x4_t r = load4<true>(rrow + (int64_t)f * 2);
            v0 += r.x; v1 += r.y; v2 += r.z; v3 += r.w;
          }
          store4<true>(orow + (int64_t)f * 2, v0, v1, v2, v3);
        }
      }
    }
  }
}

// DMA-staged large-tile bf16 kernel (the gate/up workhorse). 4 waves (2 x 2),
// each owning a 128 x 128 sub-tile (4 x 4 MFMA blocks, 256 fp32 accumulators
// in AGPRs). K is streamed in 64-byte slabs (32 bf16) fetched straight into a
// ring of kStages LDS buffers of 32 KB by buffer loads with the LDS bit: each
// wave instruction fills 1 KB of LDS (16 tile rows), lane i writing bytes
// [16 i, 16 i + 16), so lane i fetches the logical chunk that the swizzle puts
// at physical chunk i % 4 of row i / 4. No VGPRs hold slab data, no ds_write
// is issued, and up to kStages - 1 slabs are in flight (a CU at full MFMA
// rate consumes a 32 KB slab every ~1000 cycles; a load takes a few thousand
// to land). Waves 0-1 fetch the weight rows, waves 2-3 the token rows.
// The slab hand-off uses lds_barrier (no memory fence), so the compiler does
// not drain the in-flight slabs at every barrier.
// Rows are 64 bytes = 4 chunks, stored at chunk c ^ key64(r) with
// key64(r) = ((r >> 1) ^ (r >> 3)) & 3: conflict-free for 8 or 16 consecutive
// rows, and the same for every 32-row block, so a K step needs one address
// register per operand. Fragment reads of step s+1 are interleaved with the
// MFMAs of step s (scheduling groups).
constexpr int kRB = 64;  // bytes of K per staged row

__device__ __forceinline__ uint32_t key64(uint32_t r) { return ((r >> 1) ^ (r >> 3)) & 3u; }

template <int kMode, int kGroup, int kStages>
__global__ __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1))) void ffn_gemm_ring_kernel(
    FfnGemmArgs a, int n_tt, int n_ft) {
  constexpr int kWR = 256, kTR = 256;
  constexpr int kMW = 4, kMT = 4;
  constexpr int kStage = (kWR + kTR) * kRB;  // 32 KB
  __shared__ __attribute__((aligned(1024))) char smem[kStages * kStage];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ww = wave & 1;
  const int wt = wave >> 1;

  const int total = n_tt * n_ft;
  const int per = (total + kXcds - 1) / kXcds;
  const int w = (int)(blockIdx.x % kXcds) * per + (int)(blockIdx.x / kXcds);
  if (w >= total) return;
  const int grp = w / (kGroup * n_tt);
  const int rem = w - grp * (kGroup * n_tt);
  const int gsz = min(kGroup, n_ft - grp * kGroup);
  const int tt = rem / gsz;
  const int ft = grp * kGroup + (rem - tt * gsz);

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

  // ---- DMA plan: waves 0-1 fetch weight rows, waves 2-3 token rows; each
  //      wave instruction q fills 16 rows x 64 B = 1 KB ----
  const bool is_w = wave < 2;
  const int rbase = 128 * (wave & 1);
  const int r16 = lane >> 2;
  const int pch = lane & 3;
  const __amdgpu_buffer_rsrc_t wr0 = make_rsrc(a.w0[set], (uint32_t)(n_feat * a.w_ld));
  const __amdgpu_buffer_rsrc_t wr1 =
      (kMode == 0) ? make_rsrc(a.w1[set], (uint32_t)(n_feat * a.w_ld)) : wr0;
  const __amdgpu_buffer_rsrc_t trs = make_rsrc(a.tok, 0xffffffffu);
  uint32_t voff[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const int r = rbase + 16 * q + r16;
    const int c = pch ^ (int)key64((uint32_t)r);
    if (is_w) {
      int feat;
      if constexpr (kMode == 0) feat = f0 + 32 * ((r >> 5) >> 1) + (r & 31);
      else feat = f0 + r;
      voff[q] = (uint32_t)((int64_t)feat * a.w_ld + c * 16);
    } else {
      int j = row_lo + r;
      j = j < row_hi ? j : row_hi - 1;
      voff[q] = (uint32_t)((int64_t)map_row(j, a.map1, a.map2) * a.tok_ld + c * 16);
    }
  }
  // row block (rbase + 16q) / 32 has the parity of q / 2: the gate / up choice
  // is fixed per instruction at compile time
  auto dma = [&](int kb, int buf) __attribute__((always_inline)) {
    const int soff = kb * kRB;
    if (is_w) {
      char* region = smem + buf * kStage;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        __attribute__((address_space(3))) void* dst =
            (__attribute__((address_space(3))) void*)(region + (rbase + 16 * q) * kRB);
        __builtin_amdgcn_raw_ptr_buffer_load_lds((kMode == 0 && ((q >> 1) & 1)) ? wr1 : wr0, dst, 16,
                                                 (int)voff[q], soff, 0, 0);
      }
    } else {
      char* region = smem + buf * kStage + kWR * kRB;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        __attribute__((address_space(3))) void* dst =
            (__attribute__((address_space(3))) void*)(region + (rbase + 16 * q) * kRB);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(trs, dst, 16, (int)voff[q], soff, 0, 0);
      }
    }
  };

  f32x16_t acc[kMW][kMT];
#pragma unroll
  for (int i = 0; i < kMW; ++i)
#pragma unroll
    for (int j = 0; j < kMT; ++j) acc[i][j] = f32x16_t{};

  const int lrow = lane & 31;
  const int lhalf = lane >> 5;
  auto opaque = [](uint32_t v) __attribute__((always_inline)) {
    asm volatile("" : "+v"(v));
    return v;
  };
  const uint32_t rkey = key64((uint32_t)lrow);
  const uint32_t rowa = (uint32_t)((ww * 128 + lrow) * kRB);
  const uint32_t rowb = (uint32_t)(kWR * kRB + (wt * 128 + lrow) * kRB);
  u32x4_t fa0[kMW], fb0[kMT], fa1[kMW], fb1[kMT];
  auto read_frags = [&](u32x4_t (&fa)[kMW], u32x4_t (&fb)[kMT], const char* sw, int step) __attribute__((always_inline)) {
    const uint32_t off = (((uint32_t)(2 * step + lhalf)) ^ opaque(rkey)) << 4;
    const char* pa = sw + rowa + off;
    const char* pb = sw + rowb + off;
#pragma unroll
    for (int i = 0; i < kMW; ++i) fa[i] = *reinterpret_cast<const u32x4_t*>(pa + 32 * i * kRB);
#pragma unroll
    for (int j = 0; j < kMT; ++j) fb[j] = *reinterpret_cast<const u32x4_t*>(pb + 32 * j * kRB);
  };
  auto mfmas = [&](const u32x4_t (&fa)[kMW], const u32x4_t (&fb)[kMT]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < kMW; ++i)
#pragma unroll
      for (int j = 0; j < kMT; ++j) mfma_step<true>(acc[i][j], fa[i], fb[j]);
  };

  const int nk = a.k_bytes / kRB;  // >= kStages (checked by the launcher)
#pragma unroll
  for (int s = 0; s < kStages - 1; ++s) dma(s, s);
  int buf = 0;
  for (int kb = 0; kb < nk; ++kb) {
    // wait for slab kb: the loads of the (up to kStages - 2) later slabs may stay in flight
    const int ahead = min(nk - 1 - kb, kStages - 2);
    if (ahead >= 3) asm volatile("s_waitcnt vmcnt(24)" ::: "memory");
    else if (ahead == 2) asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
    else if (ahead == 1) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lds_barrier();
    // every wave is past slab kb-1: its buffer now receives slab kb + kStages - 1
    if (kb + kStages - 1 < nk) {
      int nb = buf + kStages - 1;
      nb = nb >= kStages ? nb - kStages : nb;
      dma(kb + kStages - 1, nb);
    }
    const char* sw = smem + buf * kStage;
    read_frags(fa0, fb0, sw, 0);
    read_frags(fa1, fb1, sw, 1);
    mfmas(fa0, fb0);
    mfmas(fa1, fb1);
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 24, 0);
    buf = buf + 1 == kStages ? 0 : buf + 1;
  }

#pragma unroll
  for (int j = 0; j < kMT; ++j) {
    const int jr = row_lo + wt * 128 + 32 * j + lrow;
    if (jr >= row_hi) continue;
    const int orow_idx = map_row(jr, a.omap1, a.omap2);
    char* orow = a.out + (int64_t)orow_idx * a.out_ld;
    if constexpr (kMode == 0) {
#pragma unroll
      for (int p = 0; p < kMW / 2; ++p) {
        const int fb0_ = f0 + 32 * (ww * (kMW / 2) + p) + 4 * lhalf;
        if (fb0_ >= n_feat) continue;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x16_t& ag = acc[2 * p][j];
          const f32x16_t& au = acc[2 * p + 1][j];
          float v0 = silu_f32(ag[4 * g + 0]) * au[4 * g + 0];
          float v1 = silu_f32(ag[4 * g + 1]) * au[4 * g + 1];
          float v2 = silu_f32(ag[4 * g + 2]) * au[4 * g + 2];
          float v3 = silu_f32(ag[4 * g + 3]) * au[4 * g + 3];
          store4<true>(orow + (int64_t)(fb0_ + 8 * g) * 2, v0, v1, v2, v3);
        }
      }
    } else {
      const char* rrow = a.res ? a.res + (int64_t)orow_idx * a.res_ld : nullptr;
#pragma unroll
      for (int i = 0; i < kMW; ++i) {
        const int fb0_ = f0 + ww * 128 + 32 * i + 4 * lhalf;
        if (fb0_ >= n_feat) continue;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int f = fb0_ + 8 * g;
          float v0 = acc[i][j][4 * g + 0], v1 = acc[i][j][4 * g + 1];
          float v2 = acc[i][j][4 * g + 2], v3 = acc[i][j][4 * g + 3];
          if (rrow) {
            f32x4_t rr = load4<true>(rrow + (int64_t)f * 2);
            v0 += rr.x; v1 += rr.y; v2 += rr.z; v3 += rr.w;
          }
          store4<true>(orow + (int64_t)f * 2, v0, v1, v2, v3);
        }
      }
    }
  }
}

template <int kMode, int kGroup, int kStages>
hipError_t launch_ring(const FfnGemmArgs& a, hipStream_t stream) {
  constexpr int kFTile = (kMode == 0) ? 128 : 256;
  const int n_tt = (a.cap + 255) / 256 + (a.n_sets - 1);
  const int n_ft = (a.n_feat + kFTile - 1) / kFTile;
  if (n_tt <= 0 || n_ft <= 0) return hipSuccess;
  const int total = n_tt * n_ft;
  const int grid = ((total + kXcds - 1) / kXcds) * kXcds;
  hipLaunchKernelGGL((ffn_gemm_ring_kernel<kMode, kGroup, kStages>), dim3(grid), dim3(256), 0, stream,
                     a, n_tt, n_ft);
  return hipGetLastError();
}

// The large-tile kernels address every operand with 32-bit buffer offsets and
// need at least a few K slabs; callers fall back to ffn_gemm_kernel otherwise.
inline bool big_ok(const FfnGemmArgs& a) {
  const int64_t lim = (int64_t)1 << 31;
  return a.k_bytes >= 2 * kKB && (int64_t)a.tok_rows * a.tok_ld < lim &&
         (int64_t)a.n_feat * a.w_ld < lim;
}
inline bool ring_ok(const FfnGemmArgs& a, int stages) { return big_ok(a) && a.k_bytes >= stages * kRB; }

template <int kMode, int kGroup>
hipError_t launch_big(const FfnGemmArgs& a, hipStream_t stream) {
  constexpr int kFTile = (kMode == 0) ? 128 : 256;
  const int n_tt = (a.cap + 255) / 256 + (a.n_sets - 1);
  const int n_ft = (a.n_feat + kFTile - 1) / kFTile;
  if (n_tt <= 0 || n_ft <= 0) return hipSuccess;
  const int total = n_tt * n_ft;
  const int grid = ((total + kXcds - 1) / kXcds) * kXcds;
  hipLaunchKernelGGL((ffn_gemm_big_kernel<kMode, kGroup>), dim3(grid), dim3(256), 0, stream, a, n_tt,
                     n_ft);
  return hipGetLastError();
}

template <bool kBF16, int kMode, int kWR, int kTR, int kWW, int kWT, int kStages, int kPf = 1,
          int kGroup = 1>
hipError_t launch_cfg(const FfnGemmArgs& a, hipStream_t stream) {
  constexpr int kFTile = (kMode == 0) ? kWR / 2 : kWR;
  const int n_tt = (a.cap + kTR - 1) / kTR + (a.n_sets - 1);
  const int n_ft = (a.n_feat + kFTile - 1) / kFTile;
  if (n_tt <= 0 || n_ft <= 0) return hipSuccess;
  const int total = n_tt * n_ft;
  const int grid = ((total + kXcds - 1) / kXcds) * kXcds;
  hipLaunchKernelGGL((ffn_gemm_kernel<kBF16, kMode, kWR, kTR, kWW, kWT, kStages, kPf, kGroup>), dim3(grid),
                     dim3(64 * kWW * kWT), 0, stream, a, n_tt, n_ft);
  return hipGetLastError();
}

}  // namespace

// Kernel and tile choice, from timing every variant on the five named workloads:
//   gate/up: the DMA ring kernel, 4 stages (128 output features x 256 tokens,
//            groups of 4 feature tiles); fallback 8-wave 256 x 256 register-staged;
//   down:    the 4-wave 256 x 256 kernel when it yields >= 200 tiles (enough
//            to fill the chip), else 256 x 128 (4 x 2 waves) for d < 3072 and
//            128 x 128 (2 x 2 waves) for the 7B width, token-tile-major order
//            (every weight tile of a token tile stays in one XCD's L2).
// fp32 data (tiny workloads) uses 128 x 128 tiles.
hipError_t launch_ffn_gateup(const FfnGemmArgs& a, bool bf16, hipStream_t stream) {
  if (bf16) {
    if (ring_ok(a, 4)) return launch_ring<0, 4, 4>(a, stream);
    return launch_cfg<true, 0, 256, 256, 4, 2, 1, 1, 4>(a, stream);
  }
  return launch_cfg<false, 0, 128, 128, 2, 2, 2>(a, stream);
}

hipError_t launch_ffn_down(const FfnGemmArgs& a, bool bf16, hipStream_t stream) {
  if (bf16) {
    const int64_t big_tiles = (int64_t)((a.cap + 255) / 256 + a.n_sets - 1) * ((a.n_feat + 255) / 256);
    if (a.n_feat < 3072 && big_tiles >= 200 && big_ok(a)) return launch_big<1, 64>(a, stream);
    if (a.n_feat < 3072) return launch_cfg<true, 1, 256, 128, 4, 2, 2, 1, 64>(a, stream);
    return launch_cfg<true, 1, 128, 128, 2, 2, 2, 1, 64>(a, stream);
  }
  return launch_cfg<false, 1, 128, 128, 2, 2, 2>(a, stream);
}

}  // namespace ce
