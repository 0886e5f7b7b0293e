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
#include "ce_host.hpp"

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
  if (a.clear_cnt && blockIdx.x == 0)
    for (int i = threadIdx.x; i < a.clear_n; i += kThreads) a.clear_cnt[i] = 0;
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
      double gdot = 0.0, gin = 0.0, gout = 0.0;  // layer-gap sums over this lane's features
#pragma unroll
      for (int i = 0; i < kMW; ++i) {
        const int fb = f0 + ww * kWRw + 32 * i + 4 * lhalf;
        if (fb >= n_feat) continue;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int f = fb + 8 * g;
          float v0 = acc[i][j][4 * g + 0], v1 = acc[i][j][4 * g + 1];
          float v2 = acc[i][j][4 * g + 2], v3 = acc[i][j][4 * g + 3];
          f32x4_t r = {0.0f, 0.0f, 0.0f, 0.0f};
          if (rrow) {
            r = load4<kBF16>(rrow + (int64_t)f * kElem);
            v0 += r.x; v1 += r.y; v2 += r.z; v3 += r.w;
          }
          store4<kBF16>(orow + (int64_t)f * kElem, v0, v1, v2, v3);
          if (a.gap_part) {
            // the values as stored (bf16: after the one rounding)
            const f32x4_t y = load4<kBF16>(orow + (int64_t)f * kElem);
            const float ri[4] = {r.x, r.y, r.z, r.w}, yo[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              gdot = fma((double)ri[e], (double)yo[e], gdot);
              gin = fma((double)ri[e], (double)ri[e], gin);
              gout = fma((double)yo[e], (double)yo[e], gout);
            }
          }
        }
      }
      if (a.gap_part) {
        // lanes l and l ^ 32 hold the same token's other features
        gdot += __shfl_xor(gdot, 32);
        gin += __shfl_xor(gin, 32);
        gout += __shfl_xor(gout, 32);
        // a wave whose features all lie past the last one has no slot
        if (lhalf == 0 && f0 + ww * kWRw < n_feat) {
          const int prow = a.omap1 ? a.omap1[jr] : jr;
          double* gp = a.gap_part + ((int64_t)prow * a.gap_np + (f0 + ww * kWRw) / kWRw) * 4;
          gp[0] = gdot;
          gp[1] = gin;
          gp[2] = gout;
        }
      }
    }
  }
}

// Token tiles of a gate/up launch over n packed rows: 256 rows each, except
// that with `absorb` a last tile of at most 32 rows joins the tile before it
// (which then holds 257 to 288 rows). A tile of a few rows would stream a
// whole weight tile through LDS for them; the joined tile reads those rows'
// fragments straight into registers while the weight superslabs it holds
// anyway are in LDS (one more 32 x 32 block per wave). Non-decreasing in n,
// and tiles(n0) + tiles(n1) <= tiles(n0 + n1) + 1, so a grid sized for the
// capacity covers any packed count below it, split over two weight sets too.
__host__ __device__ inline int gateup_token_tiles(int n, bool absorb) {
  if (n <= 0) return 0;
  int t = (n + 255) / 256;
  if (absorb && t >= 2 && n - 256 * (t - 1) <= 32) --t;
  return t;
}

// Ping-pong bf16 kernel (the gate/up workhorse, and the down GEMM on large
// grids): 8 waves, two per SIMD, over a 256 x 256 tile. Wave w owns weight
// rows 128 (w & 1) .. +128 and token rows 64 (w >> 1) .. +64 (4 x 2 MFMA
// blocks, 128 fp32 accumulators). Waves 0-3 (group A) and 4-7 (group B) share
// the four SIMDs (wave w on SIMD w % 4) and run half a phase apart: while one
// group issues its 16 MFMAs for 64 bytes of K, the other reads its fragments
// of the next 64 bytes from LDS and issues DMA. Every phase ends at a
// workgroup barrier; group B starts one barrier late and group A ends with one
// extra barrier, so both execute the same number.
//
// Operands reach LDS through buffer loads with the LDS bit, each wave
// instruction fetching 8 rows x 128 bytes: whole cache lines (16 rows x 64
// bytes, i.e. half lines, move about half as many bytes per clock from L2).
// A "superslab" is 128 bytes of K: 32 KB per operand. LDS holds 3 token
// superslabs and 2 weight superslabs (160 KB); tokens, which mostly miss L2,
// are fetched two superslabs ahead, weights one ahead. Waves 0-3 fetch weight
// rows, waves 4-7 token rows, half of their rows in each of the two memory
// phases of a superslab so the DMA writes into LDS do not bunch up. Rows are
// 128 bytes, chunk c of row r stored at chunk c ^ ((r >> 1) & 7). The LDS
// (64 banks of 4 bytes) serves a 16-byte read for 16 lanes per clock, here 16
// consecutive rows; consecutive rows start in alternate halves of the 256-byte
// bank line, so the 8 rows of each parity need 8 distinct keys for the 16
// lanes to cover all 64 banks (a key of r & 7 repeats every 8 rows: 2-way
// conflicts, measured as half of the LDS busy time).
// kSplit: 1 = whole tiles only; 2 = tail tiles in two K pieces; 0 = tail
// tiles in sp.pieces > 2 K pieces (separate instances keep the whole-tile and
// two-piece code free of the general merge).
// kPrune (down only): rows of sequences that run the pruned FFN read zeros
// for the channels of P (the K tail from superslab a.ns_keep on), and a whole
// tile of such rows stops its K loop there.
template <int kMode, int kGroup, bool kPrio, int kSplit, int kWBufs = 2, bool kSpreadW = true,
          bool kSpreadT = true, bool kPrune = false>
__global__ __launch_bounds__(512, 1) __attribute__((amdgpu_waves_per_eu(2, 2))) void ffn_gemm_pp2_kernel(
    FfnGemmArgs a, int n_tt, int n_ft, GemmSplit sp) {
  constexpr int kWR = 256, kTR = 256;
  constexpr int kMW = 4, kMT = 2;
  constexpr int kRow = 128;                  // bytes of K per staged row
  constexpr int kSlab = 256 * kRow;          // one operand's superslab: 32 KB
  constexpr int kTBufs = 5 - kWBufs;         // 160 KB of LDS in all
  static_assert(kWBufs >= 2 && kTBufs >= 2, "each ring holds two superslabs at least");
  __shared__ __attribute__((aligned(1024))) char smem[(kWBufs + kTBufs) * kSlab];
  char* const wsm = smem;                    // weight ring
  char* const tsm = smem + kWBufs * kSlab;   // token ring

  const int tid = threadIdx.x;
  if (a.clear_cnt && blockIdx.x == 0)
    for (int i = tid; i < a.clear_n; i += 512) a.clear_cnt[i] = 0;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ww = wave & 1;
  const int wt = wave >> 1;
  const bool late = wave >= 4;  // group B

  // ---- work item of this workgroup (see GemmSplit): the first whole_x
  //      workgroups of XCD x = blockIdx % 8 take whole tiles of its range
  //      [x per_x, (x + 1) per_x); the other workgroups of all XCDs take the
  //      K pieces of the tail tiles, numbered piece-major, so that each XCD
  //      streams one or two K ranges of many tail tiles (fewer distinct
  //      operand bytes through its L2 than every range of a few tiles) ----
  const int total = n_tt * n_ft;
  const int xcd = (int)(blockIdx.x % kXcds);
  const int loc = (int)(blockIdx.x / kXcds);
  int w, piece = 0, pieces = 1, slot = 0;
  if (kSplit == 1 || loc < sp.whole_x) {
    w = xcd * sp.per_x + loc;
  } else {
    const int n_tail = kXcds * sp.tail_x;  // tail tiles of the launch
    pieces = kSplit == 2 ? 2 : sp.pieces;
    const int g = xcd * (sp.tail_x * pieces) + (loc - sp.whole_x);
    piece = g / n_tail;
    slot = g - piece * n_tail;  // partial-sum tiles [slot x pieces, + pieces), counter [slot]
    const int sx = slot / sp.tail_x;
    w = sx * sp.per_x + sp.whole_x + (slot - sx * sp.tail_x);
  }
  if (w >= total) return;
  const int grp = w / (kGroup * n_tt);
  const int rem = w - grp * (kGroup * n_tt);
  const int gsz = min(kGroup, n_ft - grp * kGroup);
  const int tt = rem / gsz;
  const int ft = grp * kGroup + (rem - tt * gsz);

  // both sizes loaded back to back (one latency, not two)
  const bool two_sets = a.n_sets == 2 && a.n0_ptr;
  int kt = *a.kt_ptr;
  int n0 = *(two_sets ? a.n0_ptr : a.kt_ptr);
  kt = kt < 0 ? 0 : (kt > a.cap ? a.cap : kt);
  n0 = two_sets ? (n0 < 0 ? 0 : (n0 > kt ? kt : n0)) : kt;
  const bool absorb = kMode == 0 && kSplit == 1 && sp.absorb != 0;
  const int tiles0 = gateup_token_tiles(n0, absorb);
  int set, row_lo, row_hi;
  if (tt < tiles0) {
    set = 0;
    row_lo = tt * kTR;
    row_hi = tt == tiles0 - 1 ? n0 : row_lo + kTR;
  } else {
    set = 1;
    const int t1 = tt - tiles0, tiles1 = gateup_token_tiles(kt - n0, absorb);
    if (t1 >= tiles1) return;
    row_lo = n0 + t1 * kTR;
    row_hi = t1 == tiles1 - 1 ? kt : row_lo + kTR;
  }
  if (row_lo >= row_hi) return;
  // a tile holding the absorbed last rows [row_lo + 256, row_hi) of its set
  const bool ext = absorb && row_hi - row_lo > kTR;

  const int n_feat = a.n_feat;
  constexpr int kFTile = (kMode == 0) ? kWR / 2 : kWR;
  const int f0 = ft * kFTile;
  // gate/up with the FFN-pruning sums: the sequence of tile row tid - 256
  // (token waves), loaded here so that its latency hides behind the K loop
  // (in the epilogue instead where the two-piece merge leaves no register)
  int sal_key = -1;
  auto load_sal_key = [&]() __attribute__((always_inline)) {
    if (a.sal_part && tid >= 256) {
      const int jr = row_lo + tid - 256;
      if (jr < row_hi) sal_key = a.row_seq[a.map1 ? a.map1[jr] : jr];
    }
  };
  if constexpr (kMode == 0 && kSplit != 2) load_sal_key();

  // ---- DMA plan: waves 0-3 fetch weight rows 64 (w & 3) .. +63, waves 4-7
  //      the same token rows; instruction q covers 8 rows x 128 B ----
  const bool is_w = wave < 4;
  const int r8 = lane >> 3;
  const int pch = lane & 7;
  // (the set picked by a select: an index into the argument's arrays would
  // put them on the stack)
  const __amdgpu_buffer_rsrc_t wr0 = make_rsrc(set ? a.w0[1] : a.w0[0], (uint32_t)(n_feat * a.w_ld));
  const __amdgpu_buffer_rsrc_t wr1 =
      (kMode == 0) ? make_rsrc(set ? a.w1[1] : a.w1[0], (uint32_t)(n_feat * a.w_ld)) : wr0;
  // Token rows past the tile's last packed row (the final token tile is
  // partial) are fetched from past the resource's end: zeros and no memory
  // traffic. Their MFMAs then multiply zeros, which draws less power than
  // real data.
  const __amdgpu_buffer_rsrc_t trs = make_rsrc(a.tok, (uint32_t)(a.tok_rows * a.tok_ld));
  uint32_t voff[8];
  uint32_t voff2[kPrune ? 8 : 1];
  if (is_w) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int r = 64 * (wave & 3) + 8 * q + r8;
      const int c = pch ^ ((r >> 1) & 7);
      int feat;
      if constexpr (kMode == 0) feat = f0 + 32 * ((r >> 5) >> 1) + (r & 31);
      else feat = f0 + r;
      voff[q] = (uint32_t)((int64_t)feat * a.w_ld + c * 16);
    }
  } else {
    // source rows through the index maps: clamped, branch-free loads, so the
    // eight of a level are in flight together (per-row branches made the
    // compiler wait after each one)
    int src[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int j = row_lo + 64 * (wave & 3) + 8 * q + r8;
      src[q] = j < row_hi ? j : -1;
    }
    if (a.map1) {
      int v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = a.map1[src[q] < 0 ? 0 : src[q]];
#pragma unroll
      for (int q = 0; q < 8; ++q) src[q] = src[q] < 0 ? -1 : v[q];
    }
    if (a.map2) {
      int v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = a.map2[src[q] < 0 ? 0 : src[q]];
#pragma unroll
      for (int q = 0; q < 8; ++q) src[q] = src[q] < 0 ? -1 : v[q];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int r = 64 * (wave & 3) + 8 * q + r8;
      const int c = pch ^ ((r >> 1) & 7);
      voff[q] = src[q] < 0 ? 0x80000000u : (uint32_t)((int64_t)src[q] * a.tok_ld + c * 16);
    }
  }
  // Pruned FFN: lane l reads the flags of rows l, l + 64, l + 128, l + 192 of
  // the tile (through the packed-row map with two weight sets). Every wave
  // does, so each knows whether all rows of the tile run pruned without an
  // exchange; the token waves move the flags of their DMA rows over with
  // shuffles. The loads go out before the first DMAs and are used after them.
  [[maybe_unused]] int fl4[kPrune ? 4 : 1];
  [[maybe_unused]] bool ok4[kPrune ? 4 : 1];
  if constexpr (kPrune) {
    int jc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = row_lo + lane + 64 * i;
      ok4[i] = j < row_hi;
      jc[i] = ok4[i] ? j : row_lo;  // a valid row either way: branch-free loads
    }
    if (a.omap1) {
#pragma unroll
      for (int i = 0; i < 4; ++i) jc[i] = a.omap1[jc[i]];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) fl4[i] = a.row_flag[jc[i]];
  }
  bool tile_pruned = false;
  auto resolve_pruned = [&]() __attribute__((always_inline)) {
    if constexpr (kPrune) {
      bool pr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) pr[i] = ok4[i] && fl4[i] != 0;
      const bool lane_all = (!ok4[0] || pr[0]) && (!ok4[1] || pr[1]) && (!ok4[2] || pr[2]) && (!ok4[3] || pr[3]);
      tile_pruned = __ballot(!lane_all) == 0ull;
      if (!is_w) {
        // DMA row 64 (wave & 3) + 8 q + r8 is row lane 8 q + r8, slot wave & 3
        const int slot = wave & 3;
        const int mine = (int)(slot == 0 ? pr[0] : slot == 1 ? pr[1] : slot == 2 ? pr[2] : pr[3]);
#pragma unroll
        for (int q = 0; q < 8; ++q) voff2[q] = __shfl(mine, 8 * q + r8) ? 0x80000000u : voff[q];
      }
    }
  };
  // weight row block (64 w + 8 q) / 32 has the parity of q / 4: the gate / up
  // choice is fixed per instruction at compile time. kPart 0 issues all 8
  // instructions, 1 the first four (rows 0-31 of the wave's 64), 2 the rest.
  // tmode (pruned FFN, token rows): 0 = not a superslab of P, 1 = one, 2 =
  // decided here from s (the K loop runs as two loops, so only the prologue
  // selects per instruction)
  auto dma = [&](int s, int buf, auto part, auto tmode) __attribute__((always_inline)) {
    constexpr int kPart = decltype(part)::value;
    constexpr int kTail = decltype(tmode)::value;
    const int soff = s * kRow;
    char* region = (is_w ? wsm : tsm) + buf * kSlab + 64 * (wave & 3) * kRow;
    if (is_w) {
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (kPart == 0 || (kPart == 1) == (q < 4))
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              (kMode == 0 && ((q >> 2) & 1)) ? wr1 : wr0,
              (__attribute__((address_space(3))) void*)(region + 8 * q * kRow), 16, (int)voff[q], soff, 0, 0);
    } else {
      const bool tail = kPrune && (kTail == 1 || (kTail == 2 && s >= a.ns_keep));  // a superslab of P
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (kPart == 0 || (kPart == 1) == (q < 4))
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              trs, (__attribute__((address_space(3))) void*)(region + 8 * q * kRow), 16,
              (int)(tail ? voff2[kPrune ? q : 0] : voff[q]), soff, 0, 0);
    }
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;

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
  const uint32_t rkey = (uint32_t)((lrow >> 1) & 7);  // fragment rows start at multiples of 32
  // A wave whose 64 token rows all lie past the tile's last packed row (the
  // final token tile is partial) reads no fragments and issues no MFMAs: its
  // accumulators stay zero, and the epilogue stores none of its rows.
  const bool mfma_on = __builtin_amdgcn_readfirstlane((int)(row_lo + wt * 64 < row_hi)) != 0;
  const uint32_t rowa = (uint32_t)((ww * 128 + lrow) * kRow);
  const uint32_t rowb = (uint32_t)((wt * 64 + lrow) * kRow);
  u32x4_t fa[2][kMW], fb[2][kMT];
  // Absorbed rows (a tile with rows past row_lo + 256): lane l reads 16-byte
  // chunks of row row_lo + 256 + (l & 31) straight into registers, fx[H]
  // holding K half H of the next superslab, in the chunk order of the B
  // fragments; wave (ww, wt) multiplies them with its weight block wt (rows
  // 128 ww + 32 wt ..), so the 8 waves cover the tile's 256 weight rows once.
  constexpr bool kExt = kMode == 0 && kSplit == 1;
  f32x16_t accx = f32x16_t{};
  u32x4_t fx[2][2];
  uint32_t xoff = 0x80000000u;  // past the token resource: zeros
  if (kExt && ext) {
    const int j = row_lo + kTR + lrow;
    int src = j < row_hi ? j : -1;
    if (src >= 0 && a.map1) src = a.map1[src];
    if (src >= 0 && a.map2) src = a.map2[src];
    if (src >= 0) xoff = (uint32_t)((int64_t)src * a.tok_ld + 16 * lhalf);
  }
  auto fxload = [&](int s, auto hc) __attribute__((always_inline)) {
    constexpr int H = decltype(hc)::value;
    fx[H][0] = bload16(trs, xoff + 64 * H, (uint32_t)(s * kRow));
    fx[H][1] = bload16(trs, xoff + 64 * H + 32, (uint32_t)(s * kRow));
  };

  // superslabs [s0, ns) of K: all of them, or this piece's range when the
  // tile is split (>= 3 per range, checked by the launcher)
  const int ns_all = a.k_bytes / kRow;
  int s0 = ns_all * piece / pieces;
  int ns = ns_all * (piece + 1) / pieces;
  // each ring starts with all but one of its slots in flight; the first
  // superslab must have landed
  constexpr int kBufs0 = kWBufs;  // waves 0-3 (weights)
  constexpr int kBufs1 = kTBufs;  // waves 4-7 (tokens)
  // the pruning choice is needed before the first DMAs when they reach the
  // superslabs of P, or when the tile is split (its K pieces may move);
  // otherwise its loads overlap theirs
  const bool resolve_first = kPrune && (pieces > 1 || s0 + kBufs1 - 1 > a.ns_keep);
  if (resolve_first) resolve_pruned();
  // a split tile of pruned rows: its K pieces share the superslabs before P
  // (at least 3 each), so every piece does less work, not only the last
  if (kPrune && pieces > 1 && tile_pruned && a.ns_keep < ns_all && a.ns_keep >= 3 * pieces) {
    s0 = a.ns_keep * piece / pieces;
    ns = a.ns_keep * (piece + 1) / pieces;
  }
  using T2 = std::integral_constant<int, kPrune ? 2 : 0>;
  using I2 = std::integral_constant<int, 2>;
  if (kExt && ext) {
    // the absorbed rows' first fragments go out between the two halves of
    // the last prologue DMA, so the K loop starts with the loads in flight
    // of its steady state (the compiler's waits for fx count on that)
    static_assert(!kExt || (kBufs0 == 2 && kBufs1 == 3), "the ext waits assume rings of 2 and 3");
    if (is_w) {
      dma(s0, 0, I1{}, I0{});
      fxload(s0, I0{});
      dma(s0, 0, I2{}, I0{});
    } else {
      dma(s0, 0, I0{}, I0{});
      dma(s0 + 1, 1, I1{}, I0{});
      fxload(s0, I0{});
      dma(s0 + 1, 1, I2{}, I0{});
    }
    fxload(s0, I1{});
  } else if (is_w) {
#pragma unroll
    for (int q = 0; q < kBufs0 - 1; ++q) dma(s0 + q, q, I0{}, I0{});
  } else {
#pragma unroll
    for (int q = 0; q < kBufs1 - 1; ++q) dma(s0 + q, q, I0{}, T2{});
  }
  if (kPrune && !resolve_first) resolve_pruned();
  // a tile of pruned rows skips the superslabs of P (they would only
  // multiply zeros): a whole tile or a K piece stops at ns_keep (keeping at
  // least 3 superslabs, else it reads zeros there), and a K piece wholly in P
  // runs no superslab and hands in zero partial sums
  if (kPrune && tile_pruned && a.ns_keep < ns) {
    if (pieces > 1 && a.ns_keep <= s0) ns = s0;
    else if (a.ns_keep - s0 >= 3) ns = a.ns_keep;
  }
  if (kExt && ext) {
    // after superslab s0's DMA: fx (weights); superslab s0 + 1 and fx (tokens)
    if (is_w) wait_vmcnt<2>();
    else wait_vmcnt<12>();
  } else if (is_w) {
    wait_vmcnt<8 * (kBufs0 - 2)>();
  } else {
    wait_vmcnt<8 * (kBufs1 - 2)>();
  }
  lds_barrier();  // superslab 0 is in LDS
  if (late) lds_barrier();
  int wb = 0, tb = 0;  // ring slots of superslab s
  // one memory phase and one compute phase over K half H of superslab s.
  // xc: 0 = a tile without absorbed rows; with them: 1 = a superslab whose
  // DMAs and fragment loads all have a superslab to fetch (s < ns - 2),
  // 2 = superslab ns - 2 (weight DMAs and fragment loads only), 3 = the last
  // (neither)
  auto half = [&](int s, auto hc, auto on, auto tmode, auto xc) __attribute__((always_inline)) {
    constexpr int H = decltype(hc)::value;
    constexpr bool kOn = decltype(on)::value;
    constexpr int X = decltype(xc)::value;
    // ---- memory phase: fragments of K half H of superslab s ----
    const char* sa = wsm + wb * kSlab;
    const char* sb = tsm + tb * kSlab;
    if constexpr (kOn) {
#pragma unroll
      for (int step = 0; step < 2; ++step) {
        const uint32_t off = (((uint32_t)(4 * H + 2 * step + lhalf)) ^ opaque(rkey)) << 4;
#pragma unroll
        for (int i = 0; i < kMW; ++i) fa[step][i] = *reinterpret_cast<const u32x4_t*>(sa + rowa + off + 32 * i * kRow);
#pragma unroll
        for (int j = 0; j < kMT; ++j) fb[step][j] = *reinterpret_cast<const u32x4_t*>(sb + rowb + off + 32 * j * kRow);
      }
    }
    // superslab s - 1 is consumed by both groups: its slot receives superslab
    // s + kBufs - 1, either half of this wave's rows in each phase (spread) or
    // all of them in the first
    const int nb = is_w ? kBufs0 : kBufs1;
    const int slot = is_w ? wb : tb;
    const int fill = s + nb - 1;
    const int fslot = slot == 0 ? nb - 1 : slot - 1;
    if (X == 1 || (X != 3 && fill < ns)) {
      if (is_w) {
        if constexpr (kSpreadW) dma(fill, fslot, std::integral_constant<int, H + 1>{}, I0{});
        else if constexpr (H == 0) dma(fill, fslot, I0{}, I0{});
      } else {
        if constexpr (kSpreadT) dma(fill, fslot, std::integral_constant<int, H + 1>{}, tmode);
        else if constexpr (H == 0) dma(fill, fslot, I0{}, tmode);
      }
    }
    // superslab s + 1 is read right after the barrier that ends group A's
    // second compute phase and group B's second memory phase: each wave
    // waits for its part of it there, leaving the later superslabs in flight
    const bool more = H == 1 && s + 1 < ns && (min(ns - 1, fill) - (s + 1)) >= 1;
    // With absorbed rows each half also loads the fragments of superslab
    // s + 1 (2 loads, after the compute phase): 12 loads follow the last DMA
    // of superslab s + 1 here in the steady state, 4 in superslab ns - 2
    // (no DMA of s + 2).
    if (H == 1 && late && s + 1 < ns) {
      if constexpr (X == 1) {
        wait_vmcnt<12>();
      } else if constexpr (X == 2) {
        wait_vmcnt<4>();
      } else if constexpr (X == 0) {
        if (more) wait_vmcnt<8>();
        else wait_vmcnt<0>();
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    lds_barrier();
    __builtin_amdgcn_sched_barrier(0);
    // ---- compute phase ----
    if constexpr (kPrio) __builtin_amdgcn_s_setprio(1);
    if constexpr (kOn) {
#pragma unroll
      for (int step = 0; step < 2; ++step)
#pragma unroll
        for (int i = 0; i < kMW; ++i)
#pragma unroll
          for (int j = 0; j < kMT; ++j) mfma_step<true>(acc[i][j], fa[step][i], fb[step][j]);
    }
    if constexpr (X != 0) {
      // the absorbed rows against weight block wt (a wave-uniform choice)
#pragma unroll
      for (int i = 0; i < kMW; ++i)
        if (i == wt) {
          mfma_step<true>(accx, fa[0][i], fx[H][0]);
          mfma_step<true>(accx, fa[1][i], fx[H][1]);
        }
      if constexpr (X != 3) fxload(s + 1, hc);
    }
    if constexpr (kPrio) __builtin_amdgcn_s_setprio(0);
    __builtin_amdgcn_sched_barrier(0);
    if (H == 1 && !late && s + 1 < ns) {
      if constexpr (X == 1 || X == 2) {
        wait_vmcnt<2>();  // only the fragment loads just issued stay in flight
      } else if constexpr (X == 0) {
        if (more) wait_vmcnt<8>();
        else wait_vmcnt<0>();
      }
    }
    lds_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };
  // two instances of the K loop, picked once per tile: with MFMAs, and
  // without them for a wave whose rows are all past the tile's end (same DMA
  // and barriers); a branch inside the loop cost 1-1.5% on full tiles
  // The pruned FFN's K loop runs in two parts: the token DMAs of the first
  // fill superslabs before P, those of the second superslabs of P (token
  // waves fill superslab s + kBufs1 - 1 in iteration s).
  auto kloop = [&](auto on) __attribute__((always_inline)) {
    auto run = [&](int lo, int hi, auto tmode) __attribute__((always_inline)) {
      for (int s = lo; s < hi; ++s) {
        half(s, I0{}, on, tmode, I0{});
        half(s, I1{}, on, tmode, I0{});
        wb = wb + 1 == kBufs0 ? 0 : wb + 1;
        tb = tb + 1 == kBufs1 ? 0 : tb + 1;
      }
    };
    if constexpr (kPrune) {
      const int s_sw = min(max(a.ns_keep - (kBufs1 - 1), s0), ns);
      run(s0, s_sw, I0{});
      run(s_sw, ns, I1{});
    } else {
      run(s0, ns, I0{});
    }
  };
  // tiles with absorbed rows: a steady loop whose every half issues the same
  // loads (so the compiler's waits for fx are exact), then the last two
  // superslabs written out (a loop over them gets the most conservative
  // waits of both)
  auto kloop_x = [&]() __attribute__((always_inline)) {
    auto superslab = [&](int s, auto xc) __attribute__((always_inline)) {
      half(s, I0{}, std::true_type{}, I0{}, xc);
      half(s, I1{}, std::true_type{}, I0{}, xc);
      wb = wb + 1 == kBufs0 ? 0 : wb + 1;
      tb = tb + 1 == kBufs1 ? 0 : tb + 1;
    };
    for (int s = s0; s < ns - 2; ++s) superslab(s, std::integral_constant<int, 1>{});
    superslab(ns - 2, std::integral_constant<int, 2>{});
    superslab(ns - 1, std::integral_constant<int, 3>{});
  };
  bool ran_x = false;
  if constexpr (kExt) {
    if (ext) {
      kloop_x();
      ran_x = true;
    }
  }
  if (!ran_x) {
    if (mfma_on) kloop(std::true_type{});
    else kloop(std::false_type{});
  }

  // K pieces of a tail tile meet through the workspace: each writes its
  // sums, then bumps the tile's arrival counter; the last to arrive adds the
  // pieces up and finishes the tile. Nobody waits on anybody. The sums move
  // with device-coherent (sc1) stores and loads, so no L2 write-back or
  // invalidation is needed; the counter is an agent-scope atomic issued after
  // this workgroup's stores have completed. Two pieces: the last adds the
  // other's sums to its own (two addends commute, so the result does not
  // depend on which came last); more: the last re-reads all of them and adds
  // them in piece order, so the result is the same whichever came last.
  constexpr int kSC1 = 16;  // cache-policy operand: sc1
  // register order: per lane 32 float4, one wave instruction = 1 KB contiguous
  auto part_off = [&](int i, int j, int v4) __attribute__((always_inline)) {
    return (uint32_t)((((wave * 32 + (i * kMT + j) * 4 + v4) * 64) + lane) * 16);
  };
  if (kSplit != 1 && pieces > 1) {
    if (!late) lds_barrier();  // both groups in step from here on
    const __amdgpu_buffer_rsrc_t prs =
        make_rsrc(a.part + (int64_t)slot * pieces * (256 * 256), (uint32_t)pieces * (256 * 256 * 4));
    const uint32_t mine = (uint32_t)piece * (256 * 256 * 4);
#pragma unroll
    for (int i = 0; i < kMW; ++i)
#pragma unroll
      for (int j = 0; j < kMT; ++j)
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
          const u32x4_t x = {__float_as_uint(acc[i][j][4 * v4]), __float_as_uint(acc[i][j][4 * v4 + 1]),
                             __float_as_uint(acc[i][j][4 * v4 + 2]), __float_as_uint(acc[i][j][4 * v4 + 3])};
          __builtin_amdgcn_raw_buffer_store_b128(x, prs, (int)(mine + part_off(i, j, v4)), 0, kSC1);
        }
    wait_vmcnt<0>();  // this wave's sums have reached the coherence point
    __syncthreads();
    int* const arrived = reinterpret_cast<int*>(smem);  // the rings are no longer read
    if (tid == 0)
      arrived[0] = __hip_atomic_fetch_add(a.tile_cnt + slot, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const int order = arrived[0];
    __syncthreads();  // read by every wave before the epilogue reuses the LDS
    if (order != pieces - 1) return;  // another piece finishes the tile
    // the sums are added row block by row block in the epilogue (merge_block)
  }
  // row block j of the tile: adds the other pieces' sums (see above), one
  // 32-row block at a time, 4 float4 loads per piece and two pieces in flight
  // (32 registers next to the 128 accumulators and the residual values)
  auto merge_block = [&](int j) __attribute__((always_inline)) {
    if (kSplit == 1 || pieces <= 1) return;
    const __amdgpu_buffer_rsrc_t prs =
        make_rsrc(a.part + (int64_t)slot * pieces * (256 * 256), (uint32_t)pieces * (256 * 256 * 4));
    auto load4 = [&](u32x4_t (&y)[4], int p, int i) __attribute__((always_inline)) {
      const uint32_t base = (uint32_t)p * (256 * 256 * 4);
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4)
        y[v4] = __builtin_bit_cast(
            u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(prs, (int)(base + part_off(i, j, v4)), 0, kSC1));
    };
    auto add4 = [&](const u32x4_t (&y)[4], int i, bool first) __attribute__((always_inline)) {
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        const f32x4_t v = {__uint_as_float(y[v4].x), __uint_as_float(y[v4].y), __uint_as_float(y[v4].z),
                           __uint_as_float(y[v4].w)};
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[i][j][4 * v4 + e] = first ? v[e] : acc[i][j][4 * v4 + e] + v[e];
      }
    };
    // two pieces: the other piece's sums, two 32-row feature blocks per
    // batch; more: acc = p_0 + p_1 + ... + p_{S-1}, one feature block per
    // batch and two pieces' loads in flight. Both use 32 registers.
    const bool two = kSplit == 2;
#pragma unroll
    for (int i = 0; i < kMW; i += 2) {
      u32x4_t y[2][4];
      if (two) {
        load4(y[0], piece ^ 1, i);
        load4(y[1], piece ^ 1, i + 1);
        add4(y[0], i, false);
        add4(y[1], i + 1, false);
      } else {
#pragma unroll
        for (int h = 0; h < 2; ++h)
          for (int p = 0; p < pieces; p += 2) {
            load4(y[0], p, i + h);
            if (p + 1 < pieces) load4(y[1], p + 1, i + h);
            add4(y[0], i + h, p == 0);
            if (p + 1 < pieces) add4(y[1], i + h, false);
          }
      }
      // the sums are materialized here: otherwise the compiler sinks the
      // adds to the epilogue's stores and keeps every loaded value live
      // (spilling) until then
      asm volatile("" : "+v"(acc[i][j]), "+v"(acc[i + 1][j])::"memory");
    }
  };

  if constexpr (kMode == 0) {
    // SwiGLU tile staged in LDS (the rings are no longer read: group B's last
    // fragment reads ended before the barrier group A last passed), then
    // written out in whole cache lines. Layout: [256 token rows][128
    // features] bf16, 16-byte chunk c of row r at chunk c ^ (r & 15).
    // Group A stages while group B runs its last compute phase; one barrier
    // later group B stages; after the next barrier every wave writes out.
    char* const ost = smem;
    auto stage = [&]() __attribute__((always_inline)) {
#pragma unroll
      for (int j = 0; j < kMT; ++j) {
        const int r = wt * 64 + 32 * j + lrow;
#pragma unroll
        for (int p = 0; p < kMW / 2; ++p)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const f32x16_t& ag = acc[2 * p][j];
            const f32x16_t& au = acc[2 * p + 1][j];
            u32x2_t v;
            v.x = pack_bf16(silu_f32(ag[4 * g + 0]) * au[4 * g + 0], silu_f32(ag[4 * g + 1]) * au[4 * g + 1]);
            v.y = pack_bf16(silu_f32(ag[4 * g + 2]) * au[4 * g + 2], silu_f32(ag[4 * g + 3]) * au[4 * g + 3]);
            const int c = 4 * (2 * ww + p) + g;  // 16-byte chunk of features 8c .. 8c + 7
            *reinterpret_cast<u32x2_t*>(ost + r * 256 + ((c ^ (r & 15)) << 4) + 8 * lhalf) = v;
          }
      }
    };
    // absorbed rows: each up wave (odd wt) leaves its block in LDS past the
    // staged tile, lane-major, for the gate wave of the same features
    float* const xst = reinterpret_cast<float*>(smem + 65536) + (2 * ww + (wt >> 1)) * 1024;
    auto stage_x = [&]() __attribute__((always_inline)) {
      if constexpr (kExt) {
        if (ext && (wt & 1)) {
#pragma unroll
          for (int e = 0; e < 16; ++e) xst[e * 64 + lane] = accx[e];
        }
      }
    };
    if (kSplit != 1 && pieces > 1) {
      // last piece of a split tile: every wave is in step and past the rings
      merge_block(0);
      merge_block(1);
      stage();
      lds_barrier();
    } else if (!late) {
      stage();
      stage_x();
      lds_barrier();
      lds_barrier();
    } else {
      stage();
      stage_x();
      lds_barrier();
    }
    // write-out: wave w stores rows 32w .. 32w + 31, 4 rows (16 lanes x 16
    // bytes each) per instruction
    const int cc = lane & 15;
    const bool fok = f0 + 8 * cc < n_feat;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int r = 32 * wave + 4 * q + (lane >> 4);
      const int jr = row_lo + r;
      const u32x4_t v = *reinterpret_cast<const u32x4_t*>(ost + r * 256 + ((cc ^ (r & 15)) << 4));
      if (jr < row_hi && fok)
        *reinterpret_cast<u32x4_t*>(a.out + (int64_t)map_row(jr, a.omap1, a.omap2) * a.out_ld +
                                    (int64_t)(f0 + 8 * cc) * 2) = v;
    }
    if constexpr (kExt) {
      // absorbed rows: the gate waves (even wt) apply SwiGLU with the up
      // values of their partner and store rows row_lo + 256 + (lane & 31)
      const int jr = row_lo + kTR + lrow;
      if (ext && !(wt & 1) && jr < row_hi) {
        const int fb = f0 + 32 * (2 * ww + (wt >> 1)) + 4 * lhalf;
        char* const orow = a.out + (int64_t)map_row(jr, a.omap1, a.omap2) * a.out_ld;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          if (fb + 8 * g >= n_feat) continue;
          float v[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) v[k] = silu_f32(accx[4 * g + k]) * xst[(4 * g + k) * 64 + lane];
          u32x2_t o;
          o.x = pack_bf16(v[0], v[1]);
          o.y = pack_bf16(v[2], v[3]);
          *reinterpret_cast<u32x2_t*>(orow + (int64_t)(fb + 8 * g) * 2) = o;
        }
      }
    }
    if (a.sal_part) {
      // ---- FFN-pruning signal (Eq. 8): per segment of the tile (a run of
      //      rows of one sequence) and feature, the sum of |z| over its rows,
      //      from the staged tile (the values just written, after rounding).
      //      Scratch after the staged tile: row keys [256], segment starts
      //      [kSalSegs + 2], per-wave start counts [4], sums [8][128] ----
      int* const keys = reinterpret_cast<int*>(smem + 65536);
      int* const seg = keys + 256;
      int* const wcnt = seg + kSalSegs + 2;
      static_assert(kMode != 0 || (kWBufs + kTBufs) * kSlab >= 131072, "saliency reads past the staged tile");
      float* const red = reinterpret_cast<float*>(smem + 65536 + 2048);
      const int nvalid = min(256, row_hi - row_lo);
      if constexpr (kSplit == 2) load_sal_key();
      if (tid >= 256) keys[tid - 256] = sal_key;
      lds_barrier();
      bool st = false;
      uint64_t sm = 0;
      if (tid < 256) {
        const int key = keys[tid];
        st = key >= 0 && (tid == 0 || keys[tid - 1] != key);
        sm = __ballot(st);
        if (lane == 0) wcnt[wave] = __popcll(sm);
      }
      lds_barrier();
      if (tid < 256) {
        int k = 0;
        for (int w2 = 0; w2 < wave; ++w2) k += wcnt[w2];
        k += __popcll(sm & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
        if (st && k < kSalSegs) seg[k] = tid;
        if (tid == 0) seg[kSalSegs + 1] = (wcnt[0] + wcnt[1]) + (wcnt[2] + wcnt[3]);
      }
      lds_barrier();
      const int nseg = seg[kSalSegs + 1];
      if (nseg <= kSalSegs) {
        // thread: features 8 cf .. 8 cf + 7 (one 16-byte chunk) of the rows
        // rg, rg + 32, ...; the 32 row classes are added in a fixed order
        // (lanes xor 16 and 32 in the wave, then the 8 waves in turn)
        const int cf = lane & 15;
        const int rg = 4 * wave + (lane >> 4);
        for (int k = 0; k < nseg; ++k) {
          const int r0 = seg[k], r1 = k + 1 < nseg ? seg[k + 1] : nvalid;
          float sum[8] = {};
          // rows rs, rs + 32, ... below r1 (rs: the first row >= r0 of this
          // class); all share the swizzle rs & 15, so they lie 8 KB apart
          const int rs = r0 + ((rg - r0) & 31);
          const int nr = rs < r1 ? (r1 - rs + 31) >> 5 : 0;
          // All eight reads are issued, then the ones past r1 are masked:
          // they stay inside the LDS block (rows < 255 + 32 + 7 * 32 of 256
          // bytes = 128 KB), and reading them costs less than waiting for
          // each read in turn.
          const char* const src = ost + rs * 256 + ((cf ^ (rs & 15)) << 4);
          u32x4_t v[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) v[i] = *reinterpret_cast<const u32x4_t*>(src + i * 8192);
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const uint32_t keep = i < nr ? 0xffffffffu : 0u;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const uint32_t w = v[i][e] & keep;
              sum[2 * e] += fabsf(__uint_as_float(w << 16));
              sum[2 * e + 1] += fabsf(__uint_as_float(w & 0xffff0000u));
            }
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            sum[e] += __shfl_xor(sum[e], 16);
            sum[e] += __shfl_xor(sum[e], 32);
          }
          float* const rk = red + (k & 1) * 1024;  // two buffers: one barrier per segment
          if (lane < 16) {
#pragma unroll
            for (int e = 0; e < 8; ++e) rk[wave * 128 + 8 * cf + e] = sum[e];
          }
          lds_barrier();
          if (tid < 128 && f0 + tid < n_feat) {
            float t = 0.0f;
#pragma unroll
            for (int w2 = 0; w2 < 8; ++w2) t += rk[w2 * 128 + tid];
            a.sal_part[((int64_t)tt * kSalSegs + k) * n_feat + f0 + tid] = t;
          }
        }
      }
      if (ft == 0 && tid <= kSalSegs) {
        int32_t* meta = a.sal_meta + (int64_t)tt * (kSalSegs + 1);
        if (tid == 0) meta[0] = nseg;
        else if (tid - 1 < nseg) meta[tid] = keys[seg[tid - 1]];
      }
    }
  } else {
    __builtin_amdgcn_sched_barrier(0);  // keep the residual loads out of the split-K merge above
    char* orow[kMT];
    const char* rrow[kMT];
#pragma unroll
    for (int j = 0; j < kMT; ++j) {
      const int jr = row_lo + wt * 64 + 32 * j + lrow;
      const int oi = jr < row_hi ? map_row(jr, a.omap1, a.omap2) : 0;
      orow[j] = jr < row_hi ? a.out + (int64_t)oi * a.out_ld : nullptr;
      rrow[j] = (jr < row_hi && a.res) ? a.res + (int64_t)oi * a.res_ld : nullptr;
    }
    // The residual rows are usually the output rows themselves (in-place
    // scatter), so the compiler keeps every residual load behind the stores
    // before it: all of a row block's residual values are loaded before its
    // first store (each lane reads and writes only its own elements).
#pragma unroll
    for (int j = 0; j < kMT; ++j) {
      if (!orow[j]) continue;
      // residual loads first: their latency overlaps the merge's
      u32x2_t rv[kMW][4];
      if (rrow[j]) {
#pragma unroll
        for (int i = 0; i < kMW; ++i) {
          const int fb0_ = f0 + ww * 128 + 32 * i + 4 * lhalf;
#pragma unroll
          for (int g = 0; g < 4; ++g)
            rv[i][g] = fb0_ < n_feat ? *reinterpret_cast<const u32x2_t*>(rrow[j] + (int64_t)(fb0_ + 8 * g) * 2)
                                     : u32x2_t{0u, 0u};
        }
      }
      merge_block(j);
      double gdot = 0.0, gin = 0.0, gout = 0.0;  // layer-gap sums over this lane's features
#pragma unroll
      for (int i = 0; i < kMW; ++i) {
        const int fb0_ = f0 + ww * 128 + 32 * i + 4 * lhalf;
        if (fb0_ >= n_feat) continue;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float v0 = acc[i][j][4 * g + 0], v1 = acc[i][j][4 * g + 1];
          float v2 = acc[i][j][4 * g + 2], v3 = acc[i][j][4 * g + 3];
          float r[4] = {0.0f, 0.0f, 0.0f, 0.0f};
          if (rrow[j]) {
            r[0] = bf16_to_f32(rv[i][g].x & 0xffffu);
            r[1] = bf16_to_f32(rv[i][g].x >> 16);
            r[2] = bf16_to_f32(rv[i][g].y & 0xffffu);
            r[3] = bf16_to_f32(rv[i][g].y >> 16);
            v0 += r[0]; v1 += r[1]; v2 += r[2]; v3 += r[3];
          }
          u32x2_t pk;
          pk.x = pack_bf16(v0, v1);
          pk.y = pack_bf16(v2, v3);
          *reinterpret_cast<u32x2_t*>(orow[j] + (int64_t)(fb0_ + 8 * g) * 2) = pk;
          if (a.gap_part) {
            // the values as stored, after the one rounding
            const float y[4] = {bf16_to_f32(pk.x & 0xffffu), bf16_to_f32(pk.x >> 16), bf16_to_f32(pk.y & 0xffffu),
                                bf16_to_f32(pk.y >> 16)};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              gdot = fma((double)r[e], (double)y[e], gdot);
              gin = fma((double)r[e], (double)r[e], gin);
              gout = fma((double)y[e], (double)y[e], gout);
            }
          }
        }
      }
      if (a.gap_part) {
        // lanes l and l ^ 32 hold the same token's other features
        gdot += __shfl_xor(gdot, 32);
        gin += __shfl_xor(gin, 32);
        gout += __shfl_xor(gout, 32);
        // a wave whose features all lie past the last one has no slot
        if (lhalf == 0 && f0 + ww * 128 < n_feat) {
          const int jr = row_lo + wt * 64 + 32 * j + lrow;
          const int prow = a.omap1 ? a.omap1[jr] : jr;
          double* gp = a.gap_part + ((int64_t)prow * a.gap_np + (f0 + ww * 128) / 128) * 4;
          gp[0] = gdot;
          gp[1] = gin;
          gp[2] = gout;
        }
      }
    }
  }
  // group A's extra barrier at the end matches group B's at the start (the
  // gate/up path above already ends in step)
  if (kMode == 1 && (kSplit == 1 || pieces == 1) && !late) lds_barrier();
}

__global__ __launch_bounds__(256) void zero_i32_kernel(int32_t* __restrict__ p, int n) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0;
}

// Split plan of a ping-pong launch: whole tiles in full rounds per XCD, the
// partial last round as K pieces when the workspace holds their partial sums
// (see GemmSplit).
// Gate/up without the pruning sums absorbs a short last token tile
// (gateup_token_tiles) when its plan runs whole tiles only.
template <int kMode>
GemmSplit pp2_plan(const FfnGemmArgs& a, int* n_tt, int* n_ft) {
  constexpr int kFTile = (kMode == 0) ? 128 : 256;
  *n_ft = (a.n_feat + kFTile - 1) / kFTile;
  auto plan = [&](int ntt) {
    const int64_t items = (int64_t)ntt * *n_ft;
    if (a.part && a.tile_cnt) return gemm_split(items, a.k_bytes / 128);
    GemmSplit sp;
    sp.per_x = (int)((items + kXcds - 1) / kXcds);
    sp.whole_x = sp.per_x;
    sp.tail_x = 0;
    sp.pieces = 1;
    sp.absorb = 0;
    return sp;
  };
  if (kMode == 0 && !a.sal_part) {
    const int ntt = gateup_token_tiles(a.cap, true) + (a.n_sets - 1);
    GemmSplit sp = plan(ntt);
    if (sp.pieces == 1) {
      sp.absorb = 1;
      *n_tt = ntt;
      return sp;
    }
  }
  *n_tt = (a.cap + 255) / 256 + (a.n_sets - 1);
  return plan(*n_tt);
}

template <int kMode, int kGroup, bool kPrio, int kWBufs = 2, bool kSpreadW = true, bool kSpreadT = true,
          bool kPrune = false>
hipError_t launch_pp2(const FfnGemmArgs& a, const GemmSplit& sp, int n_tt, int n_ft, hipStream_t stream,
                      bool counters_clear) {
  if (n_tt <= 0 || n_ft <= 0) return hipSuccess;
  if (sp.pieces > 1 && !counters_clear) {
    // arrival counters start at zero: cleared by the preceding kernel, else
    // by a fill kernel (no memset nodes in a captured stream)
    hipLaunchKernelGGL(zero_i32_kernel, dim3(1), dim3(256), 0, stream, a.tile_cnt, kXcds * sp.tail_x);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int grid = kXcds * (sp.whole_x + sp.tail_x * sp.pieces);
  if (sp.pieces == 1)
    hipLaunchKernelGGL((ffn_gemm_pp2_kernel<kMode, kGroup, kPrio, 1, kWBufs, kSpreadW, kSpreadT, kPrune>), dim3(grid),
                       dim3(512), 0, stream, a, n_tt, n_ft, sp);
  else if (sp.pieces == 2)
    hipLaunchKernelGGL((ffn_gemm_pp2_kernel<kMode, kGroup, kPrio, 2, kWBufs, kSpreadW, kSpreadT, kPrune>), dim3(grid),
                       dim3(512), 0, stream, a, n_tt, n_ft, sp);
  else
    hipLaunchKernelGGL((ffn_gemm_pp2_kernel<kMode, kGroup, kPrio, 0, kWBufs, kSpreadW, kSpreadT, kPrune>), dim3(grid),
                       dim3(512), 0, stream, a, n_tt, n_ft, sp);
  return hipGetLastError();
}

// The large-tile kernels address every operand with 32-bit buffer offsets and
// need at least a few K slabs; callers fall back to ffn_gemm_kernel otherwise.
inline bool big_ok(const FfnGemmArgs& a) {
  const int64_t lim = (int64_t)1 << 31;
  return a.k_bytes >= 2 * kKB && (int64_t)a.tok_rows * a.tok_ld < lim &&
         (int64_t)a.n_feat * a.w_ld < lim;
}
inline bool pp2_ok(const FfnGemmArgs& a) { return big_ok(a) && a.k_bytes % 128 == 0 && a.k_bytes >= 3 * 128; }

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
//   gate/up: the full-line ping-pong kernel (128 output features x 256 tokens,
//            groups of 8 feature tiles); fallback 8-wave 256 x 256 register-staged;
//   down:    the full-line ping-pong kernel (256 x 256, groups of 8 feature
//            tiles) when its plan splits the last round or the tiles number
//            >= 200, else 256 x 128 (4 x 2 waves) for d < 3072 and 128 x 128
//            (2 x 2 waves) for the 7B width, token-tile-major order (every
//            weight tile of a token tile stays in one XCD's L2).
// Both ping-pong launches split the tiles of their last, partial round over K
// (GemmSplit) when the workspace holds the partial sums: 3108 gate/up tiles at
// the 7B width are 12 full rounds plus 36 tiles, 294 down tiles one round plus
// 38, the 108 down tiles of the understanding workload less than one round.
// fp32 data (tiny workloads) uses 128 x 128 tiles, or smaller ones when those
// would leave most of the chip idle (fp32 MFMAs run at 1/16 of the bf16 rate,
// so a handful of large tiles would each take tens of microseconds).
inline int64_t grid_tiles(const FfnGemmArgs& a, int feat_tile, int tok_tile) {
  return (int64_t)((a.cap + tok_tile - 1) / tok_tile + a.n_sets - 1) * ((a.n_feat + feat_tile - 1) / feat_tile);
}

hipError_t launch_ffn_gateup(const FfnGemmArgs& a, bool bf16, hipStream_t stream, bool counters_clear) {
  if (bf16) {
    if (pp2_ok(a)) {
      int n_tt, n_ft;
      const GemmSplit sp = pp2_plan<0>(a, &n_tt, &n_ft);
      return launch_pp2<0, 8, true>(a, sp, n_tt, n_ft, stream, counters_clear);
    }
    return launch_cfg<true, 0, 256, 256, 4, 2, 1, 1, 4>(a, stream);
  }
  if (grid_tiles(a, 64, 128) < 128) return launch_cfg<false, 0, 64, 64, 1, 2, 2>(a, stream);
  return launch_cfg<false, 0, 128, 128, 2, 2, 2>(a, stream);
}

// the down GEMM runs on the ping-pong kernel when it splits or has >= 200 tiles
inline bool down_on_pp2(const FfnGemmArgs& a, const GemmSplit& sp, int n_tt, int n_ft) {
  return pp2_ok(a) && (sp.pieces > 1 || (int64_t)n_tt * n_ft >= 200);
}

int ffn_split_counters(const FfnGemmArgs& a, int mode, bool bf16) {
  if (!bf16 || !pp2_ok(a) || !a.part || !a.tile_cnt) return 0;
  int n_tt, n_ft;
  const GemmSplit sp = mode == 0 ? pp2_plan<0>(a, &n_tt, &n_ft) : pp2_plan<1>(a, &n_tt, &n_ft);
  if (mode == 1 && !down_on_pp2(a, sp, n_tt, n_ft)) return 0;
  return sp.pieces > 1 ? kXcds * sp.tail_x : 0;
}

bool ffn_pruned_ok(const FfnGemmArgs& g, const FfnGemmArgs& dn) { return pp2_ok(g) && pp2_ok(dn); }

hipError_t launch_ffn_down_pruned(const FfnGemmArgs& a, hipStream_t stream, bool counters_clear) {
  int n_tt, n_ft;
  const GemmSplit sp = pp2_plan<1>(a, &n_tt, &n_ft);
  return launch_pp2<1, 8, true, 2, true, true, true>(a, sp, n_tt, n_ft, stream, counters_clear);
}

int ffn_down_gap_slots(const FfnGemmArgs& a, bool bf16) {
  int fpw;  // output features per wave of the kernel launch_ffn_down picks
  if (bf16) {
    int n_tt, n_ft;
    const GemmSplit sp = pp2_plan<1>(a, &n_tt, &n_ft);
    if (down_on_pp2(a, sp, n_tt, n_ft)) fpw = 128;
    else fpw = 64;  // 256 x 128 tiles on 4 x 2 waves, 128 x 128 on 2 x 2
  } else {
    fpw = grid_tiles(a, 128, 128) < 128 ? 32 : 64;
  }
  return (a.n_feat + fpw - 1) / fpw;
}

hipError_t launch_ffn_down(const FfnGemmArgs& a, bool bf16, hipStream_t stream, bool counters_clear) {
  if (bf16) {
    int n_tt, n_ft;
    const GemmSplit sp = pp2_plan<1>(a, &n_tt, &n_ft);
    if (down_on_pp2(a, sp, n_tt, n_ft)) return launch_pp2<1, 8, true>(a, sp, n_tt, n_ft, stream, counters_clear);
    if (a.n_feat < 3072) return launch_cfg<true, 1, 256, 128, 4, 2, 2, 1, 64>(a, stream);
    return launch_cfg<true, 1, 128, 128, 2, 2, 2, 1, 64>(a, stream);
  }
  if (grid_tiles(a, 128, 128) < 128) return launch_cfg<false, 1, 32, 32, 1, 1, 2>(a, stream);
  return launch_cfg<false, 1, 128, 128, 2, 2, 2>(a, stream);
}

}  // namespace ce
