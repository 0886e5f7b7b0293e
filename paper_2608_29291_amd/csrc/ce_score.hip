// Core + expansion routing logits (paper section 3.2, Eq. 4) and sigmoid
// scores (section 3.4, Eq. 6).
//
//   understanding token:  l = c(h)            c(h) = w2c . SiLU(W1c h + b1c) + b2c
//   generation token:     l = c(h) + e_m(h)   e_m(h) = w2e[m] . SiLU(W1e[m] h + b1e[m]) + b2e[m]
//   m = min(floor(n_seg * t_b), n_seg - 1), t_b the timestep of the token's sequence.
//
// One launch. A workgroup scores a tile of up to 32 consecutive tokens of one
// sequence (tiles never straddle sequences, so the segment m is uniform). The
// first layer is an MFMA GEMM of the W1 rows (A operand, blocks of 32 ranks:
// all core blocks, then the active expansion's blocks when the tile holds a
// generation token) against the 32 token rows (B operand). Wave w owns the
// rank blocks w, w + 4, ...; its epilogue applies b1, SiLU and the w2 dot in
// fp32 over its blocks, the four waves' partial sums meet in LDS in a fixed
// order, and the tile's logits and scores are written directly. Always-kept
// tokens get +inf / 1 and their hidden rows are never read.
//
// K is streamed in 128-byte slabs (64 bf16 or 32 fp32 values per row) by
// buffer loads with the LDS bit: one wave instruction fetches 8 rows x 128
// bytes, whole cache lines, into LDS. A slab holds the 32 token rows and the
// tile's weight rows; the ring holds as many slabs as fit in 160 KB (at most
// 8). Chunk c of row r is stored at chunk c ^ ((r >> 1) & 7): each group of 16
// consecutive rows read by a 16-byte fragment load (16 lanes per LDS clock)
// then covers all 64 banks, so the reads are free of bank conflicts.
#include <type_traits>

#include "ce_device.hpp"
#include "ce_launch.hpp"
#include "ce_host.hpp"
#include "ce_router.h"

namespace ce {

namespace {

constexpr int kSlabRow = 128;    // bytes of K per staged row
constexpr int kMaxBlocks = 16;   // (r_core + r_exp) / 32 <= 512 / 32

// s_waitcnt with a run-time vmcnt (0..63): the immediate is chosen by a switch.
template <int N>
__device__ __forceinline__ void wait_vm_upto(int n) {
  if constexpr (N < 63) {
    if (n > N) {
      wait_vm_upto<N + 1>(n);
      return;
    }
  }
  wait_vmcnt<N>();
}
__device__ __forceinline__ void wait_vm(int n) {
  n = n < 0 ? 0 : (n > 63 ? 63 : n);
  // split first so the chain of compares stays short
  if (n < 16) wait_vm_upto<0>(n);
  else if (n < 32) wait_vm_upto<16>(n);
  else if (n < 48) wait_vm_upto<32>(n);
  else wait_vm_upto<48>(n);
}


// Exclusive prefix sum over the 256 threads of a workgroup (4 waves), plus
// the total; scr: 4 ints of LDS. Every thread must call it.
__device__ __forceinline__ int block_excl_scan(int v, int* scr, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) scr[wave] = x;
  __syncthreads();
  int before = 0;
  for (int w = 0; w < wave; ++w) before += scr[w];
  total = (scr[0] + scr[1]) + (scr[2] + scr[3]);
  __syncthreads();  // scr is free again
  return before + x - v;
}

// Sequence b and token range [lo, hi) of token tile `tile`: the tiles of a
// sequence are ceil(len / kTile) consecutive ones, sequences in order. The
// walk takes 256 sequences at a time: one tile count per thread, a block scan,
// and a chunk whose total lies below `tile` is skipped whole (the next
// chunk's offsets are loaded before the scan, so their latency overlaps it).
// Offsets are clamped into [0, T] and an end below its start counts as an
// empty sequence. Every thread must call it; sh: 260 ints of LDS.
template <int kTile>
__device__ __forceinline__ void find_tile(const ScoreArgs& a, int tile, int* sh, int& b, int& lo, int& hi) {
  const int tid = threadIdx.x;
  auto clampT = [&](int o) { return o < 0 ? 0 : (o > a.T ? a.T : o); };
  if (a.tile_start) {
    // the first tiles of the sequences in the workspace (non-decreasing):
    // sequence b is the last with tile_start[b] <= tile, found in two steps
    // over 256 entries each (a count of the entries at or below `tile`)
    const int* ts = a.tile_start;
    const int C = (a.B + 256) / 256;  // entries 0 .. B in 256 runs of C
    const int i0 = tid * C;
    const int c1 = __syncthreads_count(i0 <= a.B && ts[min(i0, a.B)] <= tile);
    const int r0 = (c1 - 1) * C;  // the answer lies in [r0, r0 + C)
    const int j = r0 + tid;
    const int c2 = __syncthreads_count(tid < C && j <= a.B && ts[min(j, a.B)] <= tile);
    const int s = r0 + c2 - 1;
    if (c1 == 0 || s >= a.B) {
      b = -1;
      lo = hi = 0;
      return;
    }
    b = s;
    const int s0 = clampT(a.seq_offsets[s]);
    int s1 = clampT(a.seq_offsets[s + 1]);
    s1 = s1 < s0 ? s0 : s1;
    lo = s0 + (tile - ts[s]) * kTile;
    hi = min(lo + kTile, s1);
    return;
  }
  int base = 0;  // tiles before the current chunk of sequences
  int l0 = 0, l1 = 0;
  if (tid < a.B) {
    l0 = clampT(a.seq_offsets[tid]);
    l1 = clampT(a.seq_offsets[tid + 1]);
  }
  for (int s0 = 0; s0 < a.B; s0 += 256) {
    const int cnt = min(256, a.B - s0);
    const int c0 = l0, c1 = l1 < l0 ? l0 : l1;
    // the next chunk's offsets
    if (s0 + 256 + tid < a.B) {
      l0 = clampT(a.seq_offsets[s0 + 256 + tid]);
      l1 = clampT(a.seq_offsets[s0 + 256 + tid + 1]);
    }
    const int nt = tid < cnt ? (c1 - c0 + kTile - 1) / kTile : 0;
    int total;
    const int ex = block_excl_scan(nt, sh + 256, total);
    if (tile < base + total) {
      if (tid < cnt && tile >= base + ex && tile < base + ex + nt) {
        const int t0 = c0 + (tile - base - ex) * kTile;
        sh[0] = s0 + tid;
        sh[1] = t0;
        sh[2] = min(t0 + kTile, c1);
      }
      __syncthreads();
      b = sh[0];
      lo = sh[1];
      hi = sh[2];
      __syncthreads();  // sh is free again
      return;
    }
    base += total;
  }
  b = -1;
  lo = hi = 0;
}

// The rank-tiled scorer's live work items. A token tile (kTile tokens of one
// sequence, sequences tiled in order) holds n_ct core items if any of its
// tokens is scored (not always-kept) and n_rt - n_ct expansion items if any
// scored token is a generation token; the other items have nothing to do.
// Live items are numbered tile by tile, core before expansion; the grid slot
// `slot` takes live item w = (slot % 8) * ceil(n_live / 8) + slot / 8, so each
// XCD (workgroup L runs on XCD L % 8) gets a contiguous range. Returns w and
// the item (sequence b, tokens [lo, hi), rank tile q), or b = -1.
// Every thread walks the same tiles: sequences 256 at a time (tile counts and
// their prefix sums in LDS), their tiles 256 at a time (thread per tile: its
// sequence by binary search, its flags by 16-byte loads all issued at once),
// live counts by a prefix sum. When the tiles fit one such round (the usual
// case) the item is found from the registers of that round; otherwise a
// second walk finds it. scr: LDS of at least 3 * 257 + 8 ints.
template <int kTile>
__device__ void live_item(const ScoreArgs& a, int slot, int* scr, int& w, int& b, int& lo, int& hi, int& q) {
  const int tid = threadIdx.x;
  int* const t0s = scr;          // [257] first tile of each sequence of the chunk (chunk-relative)
  int* const los = scr + 257;    // [257] clamped start of each sequence
  int* const his = scr + 514;    // [257] clamped end
  int* const res = scr + 771;    // [4] the wanted item
  int* const sc4 = scr + 775;    // [4] scan scratch
  const __amdgpu_buffer_rsrc_t frs = make_rsrc(a.flags, (uint32_t)a.T);
  const int n_exp = a.n_rt - a.n_ct;
  constexpr int kChunks = kTile / 16 + 1;  // 16-byte flag chunks a tile can touch
  int live = 0, lex = 0, tlo = 0, thi = 0, jg = 0, rounds = 0;
  // one round of a walk: tiles tb .. tb + 255 of sequence chunk s0
  auto tile_round = [&](int s0, int cnt, int ctiles, int tb) __attribute__((always_inline)) {
    const int t = tb + tid;
    live = 0;
    tlo = thi = 0;
    jg = 0;
    if (t < ctiles) {
      // sequence of tile t: the last j with t0s[j] <= t
      int l = 0, h = cnt;  // answer in [l, h)
      while (h - l > 1) {
        const int mid = (l + h) >> 1;
        if (t0s[mid] <= t) l = mid;
        else h = mid;
      }
      jg = s0 + l;
      tlo = los[l] + (t - t0s[l]) * kTile;
      thi = min(tlo + kTile, his[l]);
    }
    const int c0 = tlo & ~15;
    u32x4_t v[kChunks];
#pragma unroll
    for (int i = 0; i < kChunks; ++i) v[i] = bload16(frs, (uint32_t)(c0 + 16 * i), 0);  // past T: zeros
    // KEEP is bit 1, GEN bit 0 of each flag byte
    uint32_t scored = 0, gscored = 0;
#pragma unroll
    for (int i = 0; i < kChunks; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        uint32_t valid = 0;
#pragma unroll
        for (int y = 0; y < 4; ++y) {
          const int idx = c0 + 16 * i + 4 * e + y;
          valid |= (idx >= tlo && idx < thi) ? (0xffu << (8 * y)) : 0u;
        }
        const uint32_t nk = ~v[i][e] & valid;  // bit 1 of a byte: not always-kept
        scored |= nk & 0x02020202u;
        gscored |= v[i][e] & (nk >> 1) & 0x01010101u;
      }
    live = scored ? a.n_ct + (gscored ? n_exp : 0) : 0;
  };
  // want < 0: count only; else also record live item `want`
  auto walk = [&](int want) __attribute__((always_inline)) {
    int total = 0;
    rounds = 0;
    for (int s0 = 0; s0 < a.B; s0 += 256) {
      const int cnt = min(256, a.B - s0);
      int nt = 0;
      if (tid < cnt) {
        int l0 = a.seq_offsets[s0 + tid], l1 = a.seq_offsets[s0 + tid + 1];
        l0 = l0 < 0 ? 0 : (l0 > a.T ? a.T : l0);
        l1 = l1 < l0 ? l0 : (l1 > a.T ? a.T : l1);
        los[tid] = l0;
        his[tid] = l1;
        nt = (l1 - l0 + kTile - 1) / kTile;
      }
      int ctiles;
      const int ex = block_excl_scan(nt, sc4, ctiles);
      if (tid < cnt) t0s[tid] = ex;
      if (tid == 0) t0s[cnt] = ctiles;
      __syncthreads();
      for (int tb = 0; tb < ctiles; tb += 256) {
        tile_round(s0, cnt, ctiles, tb);
        int ltotal;
        lex = total + block_excl_scan(live, sc4, ltotal);
        if (want >= 0 && live > 0 && want >= lex && want < lex + live) {
          res[0] = jg;
          res[1] = tlo;
          res[2] = thi;
          res[3] = want - lex;  // core items first, then the expansion items
        }
        total += ltotal;
        ++rounds;
      }
      __syncthreads();  // the chunk's arrays are refilled by the next chunk
    }
    return total;
  };
  if (tid == 0) res[0] = -1;
  const int n_live = walk(-1);
  const int per = (n_live + 7) / 8;
  w = (slot & 7) * per + (slot >> 3);
  if ((slot >> 3) >= per || w >= n_live) {  // the grid is sized for every item: the rest exit
    b = -1;
    return;
  }
  if (rounds == 1) {
    // the registers of the only round still describe every tile
    if (live > 0 && w >= lex && w < lex + live) {
      res[0] = jg;
      res[1] = tlo;
      res[2] = thi;
      res[3] = w - lex;
    }
  } else {
    walk(w);
  }
  __syncthreads();
  b = res[0];
  lo = res[1];
  hi = res[2];
  q = res[3];
  __syncthreads();
}

template <bool kBF16, int kTM>
__global__ __launch_bounds__(256) void score_kernel(ScoreArgs a) {
  static_assert(kTM == 32 || kTM == 128, "token tiles of 32 or 128");
  constexpr int MB = kTM / 32;  // token blocks of the tile
  // ring bytes: the rest of the 160 KB holds the small arrays (more of them
  // for 128-token tiles)
  constexpr int kLds = kTM == 32 ? 152 * 1024 : 144 * 1024;
  __shared__ __attribute__((aligned(1024))) char smem[kLds];
  __shared__ __attribute__((aligned(8))) int sh[260];  // also the summary's int64 scratch
  __shared__ float red[4][2][kTM];
  __shared__ uint8_t keep_s[kTM];
  __shared__ float ep[4][kMaxBlocks / 4][64];  // per wave and block: b1 (32 ranks), w2 (32 ranks)

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  int tile = blockIdx.x;
  if (a.info) {
    // the first B workgroups write the per-sequence summaries the TopK step
    // reads (they run on CUs the scoring tiles leave free)
    if (tile < a.B) {
      seq_summary(a.seq_offsets, a.flags, a.B, a.T, tile, a.info, reinterpret_cast<int64_t*>(sh));
      return;
    }
    tile -= a.B;
  }
  int b, lo, hi;
  find_tile<kTM>(a, tile, sh, b, lo, hi);
  // the same for every lane (read from LDS after a barrier): keep them scalar
  b = __builtin_amdgcn_readfirstlane(b);
  lo = __builtin_amdgcn_readfirstlane(lo);
  hi = __builtin_amdgcn_readfirstlane(hi);
  if (b < 0) return;  // past the last tile
  const int n = hi - lo;

  // ---- token kinds ----
  bool kp = true, gen = false;
  if (tid < n) {
    const uint8_t f = a.flags[lo + tid];
    kp = (f & CE_TOK_KEEP) != 0;
    gen = ((f & CE_TOK_GEN) != 0) && !kp;
  }
  if (tid < kTM) keep_s[tid] = kp ? 1 : 0;
  const int any_scored = __syncthreads_or(!kp);
  const bool any_gen = __syncthreads_or(gen) && a.r_exp > 0;
  if (!any_scored) {
    if (tid < n) {
      a.logits[lo + tid] = __builtin_inff();
      if (a.probs) a.probs[lo + tid] = 1.0f;
    }
    return;
  }
  int m = 0;
  if (any_gen) {
    // exact product in double: floor(n_seg * t) never rounds across a bin edge
    const double mf = floor((double)a.n_seg * (double)a.t[b]);
    m = (mf >= 0.0) ? (int)fmin(mf, (double)(a.n_seg - 1)) : 0;  // NaN -> 0
    m = __builtin_amdgcn_readfirstlane(m);  // uniform (one t per sequence): keep it scalar
  }
  const int nbc = a.r_core / 32;
  const int nb = nbc + (any_gen ? a.r_exp / 32 : 0);  // weight blocks of this tile (<= 16)
  const int stage = (kTM + 32 * nb) * kSlabRow;
  // two slabs in flight: deeper rings measured slower (the extra LDS DMA in
  // flight only adds queueing); a stage is at most (32 + 512) x 128 B = 68 KB
  // for 32-token tiles and (128 + 384) x 128 B = 64 KB for 128-token tiles
  // (the launcher takes those only for r_core + r_exp <= 384)
  int nstage = kLds / stage;
  nstage = nstage > 3 ? 3 : nstage;
  const int per_slab = MB + nb;      // DMA instructions per wave per slab

  // ---- DMA plan: instruction i of a slab covers stage rows 8i .. 8i + 7 and
  //      belongs to wave i % 4: wave w fetches token rows 8w .. 8w + 7 and rows
  //      8w .. 8w + 7 of every weight block ----
  const int r8 = lane >> 3;
  const int pch = lane & 7;
  const int trow = 8 * wave + r8;  // this lane's row inside a 32-row block
  const uint32_t chunk_off = (uint32_t)((pch ^ ((trow >> 1) & 7)) << 4);
  // rows that are never scored read past the resource end: zeros, no traffic
  uint32_t t_voff[MB];
#pragma unroll
  for (int j = 0; j < MB; ++j) {
    const int r = 32 * j + trow;
    t_voff[j] = (r < n && !keep_s[r]) ? (uint32_t)(r * a.h_ld) + chunk_off : 0x7ffffff0u;
  }
  const uint32_t w_voff = (uint32_t)(trow * a.h_ld) + chunk_off;
  const __amdgpu_buffer_rsrc_t trs = make_rsrc(a.hidden + (int64_t)lo * a.h_ld, (uint32_t)(n * a.h_ld));
  const __amdgpu_buffer_rsrc_t crs = make_rsrc(a.w1c, (uint32_t)(a.r_core * a.h_ld));
  const __amdgpu_buffer_rsrc_t ers =
      make_rsrc(any_gen ? a.w1e + (int64_t)m * a.r_exp * a.h_ld : a.w1c,
                (uint32_t)((any_gen ? a.r_exp : a.r_core) * a.h_ld));
  // The ring base passes through an empty asm: the compiler then cannot tie the
  // DMA writes to the fragment reads and leaves their ordering to the explicit
  // vmcnt waits and barriers of the loop, instead of draining every load in
  // flight before each slab's first LDS read (which would serialize the ring).
  typedef __attribute__((address_space(3))) char lds_char;
  lds_char* ring = (lds_char*)smem;
  asm volatile("" : "+s"(ring));
  // Each tile walks K starting from its own slab, so the workgroups running
  // at the same time fetch different weight lines instead of all hitting the
  // same L2 lines. The start follows the tile's index, not the workgroup's,
  // so the sum order is fixed per tile whether or not the launch has the
  // summary workgroups in front.
  const int nk_all = a.k_bytes / kSlabRow;
  const int rot = (int)((unsigned)tile % (unsigned)nk_all);
  auto dma = [&](int kb, int buf) __attribute__((always_inline)) {
    lds_char* st = ring + buf * stage;
    int ks = kb + rot;
    ks = ks >= nk_all ? ks - nk_all : ks;
    const int soff = ks * kSlabRow;
#pragma unroll
    for (int j = 0; j < MB; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(trs, st + (32 * j + 8 * wave) * kSlabRow, 16, (int)t_voff[j], soff, 0,
                                               0);
    // one loop per weight matrix: each instruction's resource is fixed
    for (int blk = 0; blk < nbc; ++blk)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(crs, st + (kTM + 32 * blk + 8 * wave) * kSlabRow, 16,
                                               (int)w_voff, soff + (int)(32 * blk * a.h_ld), 0, 0);
    for (int blk = nbc; blk < nb; ++blk)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ers, st + (kTM + 32 * blk + 8 * wave) * kSlabRow, 16,
                                               (int)w_voff, soff + (int)(32 * (blk - nbc) * a.h_ld), 0, 0);
  };

  // ---- main loop: wave w accumulates its blocks w, w + 4, w + 8, w + 12;
  //      the block count is a compile-time constant of each variant, so a
  //      slab's fragments are all read before its MFMAs are issued ----
  const int lrow = lane & 31;
  const int lhalf = lane >> 5;
  const uint32_t rkey = (uint32_t)((lrow >> 1) & 7);
  const int nk = a.k_bytes / kSlabRow;
  const int nbw = (nb - wave + 3) / 4;  // blocks of this wave (0..4)
  // the epilogue's b1 / w2 values (lane l < 32: b1 of rank l of the block,
  // l >= 32: w2 of rank l - 32), loaded now and parked in LDS after the loop
  float epv[kMaxBlocks / 4];
#pragma unroll
  for (int i = 0; i < kMaxBlocks / 4; ++i) {
    epv[i] = 0.0f;
    const int blk = wave + 4 * i;
    if (blk < nb) {
      const bool core = blk < nbc;
      const int r = (core ? 32 * blk : 32 * (blk - nbc)) + lrow;
      const float* b1 = core ? a.b1c : (a.b1e ? a.b1e + m * a.r_exp : nullptr);
      const float* w2 = core ? a.w2c : a.w2e + m * a.r_exp;
      epv[i] = lhalf ? w2[r] : (b1 ? b1[r] : 0.0f);
    }
  }
  const int pre = min(nk, nstage - 1);
  for (int s = 0; s < pre; ++s) dma(s, s);
  float pc[MB], pe[MB];
#pragma unroll
  for (int j = 0; j < MB; ++j) pc[j] = pe[j] = 0.0f;
  auto run = [&](auto nbw_c) __attribute__((always_inline)) {
    constexpr int NBW = decltype(nbw_c)::value;
    // a 32-token tile keeps two accumulators per block (even and odd K steps),
    // halving the chain of dependent MFMAs; they are added before the epilogue
    constexpr int NACC = MB == 1 ? 2 : 1;
    f32x16_t acc[NBW > 0 ? NBW : 1][MB][NACC];
#pragma unroll
    for (int i = 0; i < NBW; ++i)
#pragma unroll
      for (int j = 0; j < MB; ++j)
#pragma unroll
        for (int e = 0; e < NACC; ++e) acc[i][j][e] = f32x16_t{};
    int buf = 0;
    for (int kb = 0; kb < nk; ++kb) {
      // slab kb must have landed; the later slabs already issued may stay in flight
      const int ahead = min(nk - 1 - kb, nstage - 2);
      wait_vm(ahead * per_slab);
      lds_barrier();
      if constexpr (NBW > 0) {
        const char* st = smem + buf * stage;
        u32x4_t fb[4][MB], fa[4][NBW];
#pragma unroll
        for (int step = 0; step < 4; ++step) {
          const uint32_t off = (((uint32_t)(2 * step + lhalf)) ^ rkey) << 4;
#pragma unroll
          for (int j = 0; j < MB; ++j)
            fb[step][j] = *reinterpret_cast<const u32x4_t*>(st + (32 * j + lrow) * kSlabRow + off);
#pragma unroll
          for (int i = 0; i < NBW; ++i)
            fa[step][i] = *reinterpret_cast<const u32x4_t*>(
                st + (kTM + 32 * (wave + 4 * i) + lrow) * kSlabRow + off);
        }
#pragma unroll
        for (int step = 0; step < 4; ++step)
#pragma unroll
          for (int i = 0; i < NBW; ++i)
#pragma unroll
            for (int j = 0; j < MB; ++j) mfma_step<kBF16>(acc[i][j][NACC == 2 ? (step & 1) : 0], fa[step][i], fb[step][j]);
      }
      // every wave is past slab kb - 1 (the barrier above): its buffer receives
      // slab kb + nstage - 1. Issued after this slab's fragment reads, so no
      // LDS read follows a DMA without a barrier in between.
      if (kb + nstage - 1 < nk) {
        int nbuf = buf + nstage - 1;
        nbuf = nbuf >= nstage ? nbuf - nstage : nbuf;
        dma(kb + nstage - 1, nbuf);
      }
      buf = buf + 1 == nstage ? 0 : buf + 1;
    }
    // ---- epilogue: b1, SiLU, w2 over this wave's blocks; core and expansion kept apart ----
#pragma unroll
    for (int i = 0; i < NBW; ++i) ep[wave][i][lane] = epv[i];
#pragma unroll
    for (int i = 0; i < NBW; ++i) {
      const int blk = wave + 4 * i;
      const bool hb = (blk >= nbc ? a.b1e : a.b1c) != nullptr;
#pragma unroll
      for (int j = 0; j < MB; ++j) {
        float p = 0.0f;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = 8 * (v >> 2) + 4 * lhalf + (v & 3);  // rank inside the block
          float z = acc[i][j][0][v];
          if constexpr (NACC == 2) z += acc[i][j][1][v];
          if (hb) z += ep[wave][i][r];
          p += ep[wave][i][32 + r] * silu_f32(z);
        }
        if (blk < nbc) pc[j] += p;
        else pe[j] += p;
      }
    }
  };
  switch (nbw) {
    case 0: run(std::integral_constant<int, 0>{}); break;
    case 1: run(std::integral_constant<int, 1>{}); break;
    case 2: run(std::integral_constant<int, 2>{}); break;
    case 3: run(std::integral_constant<int, 3>{}); break;
    default:
      // 128-token tiles are launched for at most 12 rank blocks (3 per wave)
      if constexpr (kTM == 32) run(std::integral_constant<int, 4>{});
      break;
  }
#pragma unroll
  for (int j = 0; j < MB; ++j) {
    pc[j] += __shfl_xor(pc[j], 32);
    pe[j] += __shfl_xor(pe[j], 32);
    if (lhalf == 0) {
      red[wave][0][32 * j + lrow] = pc[j];
      red[wave][1][32 * j + lrow] = pe[j];
    }
  }
  __syncthreads();
  if (tid < n) {
    const int i = lo + tid;
    const uint8_t f = a.flags[i];
    float l;
    if (f & CE_TOK_KEEP) {
      l = __builtin_inff();
    } else {
      l = ((red[0][0][tid] + red[1][0][tid]) + (red[2][0][tid] + red[3][0][tid])) + a.b2c;
      if ((f & CE_TOK_GEN) && a.r_exp > 0) {
        float e = (red[0][1][tid] + red[1][1][tid]) + (red[2][1][tid] + red[3][1][tid]);
        if (a.b2e) e += a.b2e[m];
        l += e;
      }
    }
    a.logits[i] = l;
    if (a.probs) a.probs[i] = (f & CE_TOK_KEEP) ? 1.0f : 1.0f / (1.0f + expf(-l));
  }
}

// ---- rank-tiled scorer (bf16) ----
//
// The single-launch kernel above streams every rank of W1 for each 32-token
// tile, so at the 7B width (384 ranks x 7 KB) a workgroup moves 2.8 MB from
// L2 for 32 tokens, and L2-to-CU bytes per workgroup set the time. Here a
// workgroup owns a tile of TM tokens of one sequence x TN ranks (core or the
// active expansion, never both) and writes, per token, the partial logit
// sum over its ranks of w2 . SiLU(W1 h + b1); the TopK step adds the tiles'
// partials in a fixed order. Per workgroup TM token rows and TN rank rows
// stream through LDS by the same whole-line DMA as above; the four waves form
// a 2 x 2 grid over the rank and token halves of the tile. Tiles without a
// scored token, and expansion tiles without a generation token, exit at once
// (their partials are never read). The token rows come from HBM on first
// touch and the rank rows mostly from L2, so each operand has a ring of its
// own: tokens run kTokRing - 1 slabs ahead, ranks kRankRing - 1.
constexpr int kTokRing = 6;
constexpr int kRankRing = 3;

template <int TM, int TN>
__global__ __launch_bounds__(256) void score_tile_kernel(ScoreArgs a) {
  constexpr int MBW = TM / 64;  // token blocks per wave
  constexpr int NBW = TN / 64;  // rank blocks per wave
  constexpr int kTokB = TM * kSlabRow;   // one token slab
  constexpr int kRankB = TN * kSlabRow;  // one rank slab
  constexpr int IT = TM / 32;            // token DMA instructions per wave per slab (8 rows each)
  constexpr int IR = TN / 32;            // rank DMA instructions per wave per slab
  constexpr bool kTwoAcc = MBW * NBW == 1;  // a lone block keeps two accumulators (even / odd K steps)
  constexpr int NACC = kTwoAcc ? 2 : 1;
  __shared__ __attribute__((aligned(1024))) char smem[kTokRing * kTokB + kRankRing * kRankB];
  __shared__ __attribute__((aligned(8))) int sh[260];
  __shared__ float red[2][TM];
  __shared__ float ep[4][NBW][64];
  __shared__ uint8_t keep_s[TM];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave & 1;   // rank half of the tile
  const int wk = wave >> 1;  // token half of the tile

  int item = blockIdx.x;
  if (a.info) {
    if (item < a.B) {
      seq_summary(a.seq_offsets, a.flags, a.B, a.T, item, a.info, reinterpret_cast<int64_t*>(sh));
      return;
    }
    item -= a.B;
  }
  // Only live items get a workgroup (expansion items of tiles without a
  // generation token, and tiles of always-kept tokens only, have nothing to
  // do), so the grid's first round of 256 is not spent on them while live
  // items wait for a second. XCD-aware order: live items are numbered tile by
  // tile and each XCD (workgroup L runs on XCD L % 8) takes a contiguous
  // range, so the rank tiles of a token tile run next to each other on one
  // XCD and its token rows are read from HBM once and from that XCD's L2
  // after. The ring's LDS is the scratch of the walk.
  int* const scr = reinterpret_cast<int*>(smem);
  int w, b, lo, hi, q;
  live_item<TM>(a, item, scr, w, b, lo, hi, q);
  if (b < 0) return;  // the whole workgroup: b is the same in every thread
  b = __builtin_amdgcn_readfirstlane(b);
  lo = __builtin_amdgcn_readfirstlane(lo);
  hi = __builtin_amdgcn_readfirstlane(hi);
  q = __builtin_amdgcn_readfirstlane(q);
  if (b < 0) return;
  const int n = hi - lo;

  bool kp = true, gen = false;
  if (tid < n) {
    const uint8_t f = a.flags[lo + tid];
    kp = (f & CE_TOK_KEEP) != 0;
    gen = ((f & CE_TOK_GEN) != 0) && !kp;
  }
  if (tid < TM) keep_s[tid] = kp ? 1 : 0;
  const int any_scored = __syncthreads_or(!kp);
  const bool any_gen = __syncthreads_or(gen) && a.r_exp > 0;
  const bool exp_tile = q >= a.n_ct;
  if (!any_scored || (exp_tile && !any_gen)) return;
  int m = 0;
  if (exp_tile) {
    const double mf = floor((double)a.n_seg * (double)a.t[b]);
    m = (mf >= 0.0) ? (int)fmin(mf, (double)(a.n_seg - 1)) : 0;  // NaN -> 0
    m = __builtin_amdgcn_readfirstlane(m);
  }
  const int rank0 = (exp_tile ? q - a.n_ct : q) * TN;  // first rank of the tile
  const int nranks = exp_tile ? a.r_exp : a.r_core;
  const int tranks = min(TN, nranks - rank0);        // ranks of this tile (> 0)
  const char* w1 = exp_tile ? a.w1e + ((int64_t)m * a.r_exp + rank0) * a.h_ld : a.w1c + (int64_t)rank0 * a.h_ld;
  const float* b1 = exp_tile ? (a.b1e ? a.b1e + m * a.r_exp : nullptr) : a.b1c;
  const float* w2 = exp_tile ? a.w2e + m * a.r_exp : a.w2c;

  const int lrow = lane & 31;
  const int lhalf = lane >> 5;
  // epilogue values of this wave's rank blocks (lane l < 32: b1 of rank l of
  // the block, l >= 32: w2), zero for ranks past the tile's end
  float epv[NBW];
#pragma unroll
  for (int i = 0; i < NBW; ++i) {
    const int r = rank0 + 32 * (wr * NBW + i) + lrow;
    epv[i] = 0.0f;
    if (r - rank0 < tranks) epv[i] = lhalf ? w2[r] : (b1 ? b1[r] : 0.0f);
  }

  // ---- DMA plan: instruction i of a wave covers rows 32i + 8w .. +7 of a
  //      token slab (i < IT) or of a rank slab ----
  const __amdgpu_buffer_rsrc_t trs = make_rsrc(a.hidden + (int64_t)lo * a.h_ld, (uint32_t)(n * a.h_ld));
  const __amdgpu_buffer_rsrc_t wrs = make_rsrc(w1, (uint32_t)(tranks * a.h_ld));
  uint32_t tvo[IT], rvo[IR];
#pragma unroll
  for (int i = 0; i < IT; ++i) {
    const int r = 32 * i + 8 * wave + (lane >> 3);
    const uint32_t c = (uint32_t)(((lane & 7) ^ ((r >> 1) & 7)) << 4);
    // rows past the tile and always-kept rows read past the resource: zeros, no traffic
    tvo[i] = (r < n && !keep_s[r]) ? (uint32_t)(r * a.h_ld) + c : 0x7ffffff0u;
  }
#pragma unroll
  for (int i = 0; i < IR; ++i) {
    const int r = 32 * i + 8 * wave + (lane >> 3);
    const uint32_t c = (uint32_t)(((lane & 7) ^ ((r >> 1) & 7)) << 4);
    rvo[i] = (uint32_t)(r * a.h_ld) + c;  // ranks past the tile: past the resource
  }
  typedef __attribute__((address_space(3))) char lds_char;
  lds_char* ring = (lds_char*)smem;
  asm volatile("" : "+s"(ring));
  const int nk = a.k_bytes / kSlabRow;
  // each work item walks K from its own slab, so the workgroups running at
  // the same time read different lines instead of the same slab column of
  // every row (the sum order is fixed per item, with or without the summary
  // workgroups in front of the launch)
  const int rot = (int)((unsigned)w % (unsigned)nk);
  auto slab_off = [&](int k) __attribute__((always_inline)) {
    int ks = k + rot;
    ks = ks >= nk ? ks - nk : ks;
    return k < nk ? ks * kSlabRow : 0x40000000;  // past the last slab: past the resources, zeros
  };
  auto dma_t = [&](int k, int st) __attribute__((always_inline)) {
    const int so = slab_off(k);
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      lds_char* dst = ring + st * kTokB + (32 * i + 8 * wave) * kSlabRow;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(trs, dst, 16, (int)tvo[i], so, 0, 0);
    }
  };
  auto dma_r = [&](int k, int st) __attribute__((always_inline)) {
    const int so = slab_off(k);
#pragma unroll
    for (int i = 0; i < IR; ++i) {
      lds_char* dst = ring + kTokRing * kTokB + st * kRankB + (32 * i + 8 * wave) * kSlabRow;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wrs, dst, 16, (int)rvo[i], so, 0, 0);
    }
  };

  f32x16_t acc[NBW][MBW][NACC];
#pragma unroll
  for (int i = 0; i < NBW; ++i)
#pragma unroll
    for (int j = 0; j < MBW; ++j)
#pragma unroll
      for (int e = 0; e < NACC; ++e) acc[i][j][e] = f32x16_t{};

  // Issue order: iteration k issues rank slab k + kRankRing - 1, then token
  // slab k + kTokRing - 1; the prologue runs the same pattern for
  // k = -(kTokRing - 1) .. -1 (negative slabs skipped). Operations complete
  // in order, and rank slab k is issued after token slab k (kTokRing >
  // kRankRing), so "slab k has landed" is "rank slab k has landed": at most
  // the token part of its own iteration and (kRankRing - 2) whole iterations
  // are in flight. Token rows, which come from HBM, thus have kTokRing - 1
  // iterations to land and rank rows, mostly L2 hits, kRankRing - 1 (issuing
  // the tokens first would make each rank slab wait for the token slab issued
  // just before it, leaving the tokens only kRankRing - 1 iterations).
  static_assert(kTokRing > kRankRing, "token slabs run further ahead");
  for (int k = -(kTokRing - 1); k < 0; ++k) {
    if (k + kRankRing - 1 >= 0) dma_r(k + kRankRing - 1, k + kRankRing - 1);
    dma_t(k + kTokRing - 1, k + kTokRing - 1);
  }
  const uint32_t rkey = (uint32_t)((lrow >> 1) & 7);
  int tst = 0, rst = 0;  // ring stages of slab k
  for (int k = 0; k < nk; ++k) {
    wait_vmcnt<IT + (kRankRing - 2) * (IT + IR)>();
    lds_barrier();
    __builtin_amdgcn_sched_barrier(0);
    const char* sa = smem + kTokRing * kTokB + rst * kRankB;
    const char* sb = smem + tst * kTokB;
    u32x4_t fa[4][NBW], fb[4][MBW];
#pragma unroll
    for (int step = 0; step < 4; ++step) {
      const uint32_t off = (((uint32_t)(2 * step + lhalf)) ^ rkey) << 4;
#pragma unroll
      for (int i = 0; i < NBW; ++i)
        fa[step][i] = *reinterpret_cast<const u32x4_t*>(sa + (32 * (wr * NBW + i) + lrow) * kSlabRow + off);
#pragma unroll
      for (int j = 0; j < MBW; ++j)
        fb[step][j] = *reinterpret_cast<const u32x4_t*>(sb + (32 * (wk * MBW + j) + lrow) * kSlabRow + off);
    }
    // every wave is past slab k - 1 (the barrier above): its stages receive
    // rank slab k + kRankRing - 1 and token slab k + kTokRing - 1, in that
    // order. The wave issues in order, and a DMA instruction waits while the
    // memory pipe's queue is full: issued all at once they held back the
    // MFMAs behind them (each slab cost its DMA issue plus its MFMAs), so
    // they go out one at a time between the MFMAs.
    const int rso = slab_off(k + kRankRing - 1), tso = slab_off(k + kTokRing - 1);
    const int rnext = rst == 0 ? kRankRing - 1 : rst - 1, tnext = tst == 0 ? kTokRing - 1 : tst - 1;
    __builtin_amdgcn_sched_barrier(0);
    constexpr int kM = 4 * NBW * MBW;  // MFMAs of the slab
#pragma unroll
    for (int mi = 0; mi < kM; ++mi) {
      const int step = mi / (NBW * MBW), i = (mi / MBW) % NBW, j = mi % MBW;
      mfma_step<true>(acc[i][j][kTwoAcc ? (step & 1) : 0], fa[step][i], fb[step][j]);
      // DMA instructions (IR + IT) * mi / kM .. (IR + IT) * (mi + 1) / kM: rank first
#pragma unroll
      for (int x = (IR + IT) * mi / kM; x < (IR + IT) * (mi + 1) / kM; ++x) {
        if (x < IR) {
          lds_char* dst = ring + kTokRing * kTokB + rnext * kRankB + (32 * x + 8 * wave) * kSlabRow;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(wrs, dst, 16, (int)rvo[x], rso, 0, 0);
        } else {
          lds_char* dst = ring + tnext * kTokB + (32 * (x - IR) + 8 * wave) * kSlabRow;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(trs, dst, 16, (int)tvo[x - IR], tso, 0, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    tst = tst + 1 == kTokRing ? 0 : tst + 1;
    rst = rst + 1 == kRankRing ? 0 : rst + 1;
  }
  wait_vmcnt<0>();  // the slabs issued past the end (zeros) land before the workgroup ends

  // ---- epilogue: b1, SiLU, w2 over this wave's ranks; the two rank halves
  //      meet in LDS in a fixed order ----
#pragma unroll
  for (int i = 0; i < NBW; ++i) ep[wave][i][lane] = epv[i];
#pragma unroll
  for (int j = 0; j < MBW; ++j) {
    float p = 0.0f;
#pragma unroll
    for (int i = 0; i < NBW; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = 8 * (v >> 2) + 4 * lhalf + (v & 3);  // rank inside the block
        float z = acc[i][j][0][v];
        if constexpr (kTwoAcc) z += acc[i][j][NACC - 1][v];
        p += ep[wave][i][32 + r] * silu_f32(z + ep[wave][i][r]);
      }
    p += __shfl_xor(p, 32);
    if (lhalf == 0) red[wr][32 * (wk * MBW + j) + lrow] = p;
  }
  __syncthreads();
  if (tid < n) a.part[(int64_t)q * a.T + lo + tid] = red[0][tid] + red[1][tid];
}

}  // namespace

// First token tile of each sequence into out[0 .. B] (out[B] = all tiles),
// in one workgroup: thread t takes a run of ceil(B / 1024) sequences, the runs
// are scanned in order. Offsets are clamped as find_tile clamps them.
__global__ __launch_bounds__(1024) void tile_start_kernel(const int32_t* __restrict__ offs, int B, int T,
                                                         int tile, int32_t* __restrict__ out) {
  __shared__ int wsum[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  auto clampT = [&](int o) { return o < 0 ? 0 : (o > T ? T : o); };
  auto tiles_of = [&](int s) {
    const int s0 = clampT(offs[s]);
    int s1 = clampT(offs[s + 1]);
    s1 = s1 < s0 ? s0 : s1;
    return (s1 - s0 + tile - 1) / tile;
  };
  const int per = (B + 1023) / 1024;
  const int r0 = min(tid * per, B), r1 = min(r0 + per, B);
  int loc = 0;
  for (int s = r0; s < r1; ++s) loc += tiles_of(s);
  int incl = loc;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  int before = 0, total = 0;
  for (int w = 0; w < 16; ++w) {
    before += w < wave ? wsum[w] : 0;
    total += wsum[w];
  }
  int run = before + incl - loc;
  for (int s = r0; s < r1; ++s) {
    out[s] = run;
    run += tiles_of(s);
  }
  if (tid == 0) out[B] = total;
}

// Batches above this many sequences look their tiles up in tile_start.
constexpr int kTileScanMinB = 1024;

hipError_t launch_score(const ScoreArgs& a0, bool bf16, hipStream_t stream) {
  if (a0.T == 0 && !a0.info) return hipSuccess;
  ScoreArgs a = a0;
  const int tm = score_token_tile(a.B, a.T, a.k_bytes / (bf16 ? 2 : 4), a.r_core, a.r_exp, bf16 ? 2 : 4);
  if (a.tile_start && a.B > kTileScanMinB) {
    hipLaunchKernelGGL(tile_start_kernel, dim3(1), dim3(1024), 0, stream, a.seq_offsets, a.B, a.T, tm,
                       a.tile_start);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  } else {
    a.tile_start = nullptr;
  }
  const int tiles = (a.T + tm - 1) / tm + a.B + (a.info ? a.B : 0);  // >= the tile count (+ summaries)
  if (bf16 && tm == 128)
    hipLaunchKernelGGL((score_kernel<true, 128>), dim3(tiles), dim3(256), 0, stream, a);
  else if (bf16)
    hipLaunchKernelGGL((score_kernel<true, 32>), dim3(tiles), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((score_kernel<false, 32>), dim3(tiles), dim3(256), 0, stream, a);
  return hipGetLastError();
}

// Logits (Eq. 4) and scores (Eq. 6) from the rank-tiled scorer's partial
// sums, added in the order the TopK step of the fused block adds them (core
// tiles, b2_core, then for generation tokens the expansion tiles plus
// b2_exp[m]), so both paths give the same logits bit for bit. Workgroup
// (x, b): the tokens of sequence b, strided over gridDim.x workgroups.
__global__ __launch_bounds__(256) void score_assemble_kernel(ScoreArgs a) {
  const int b = blockIdx.y;
  int lo = a.seq_offsets[b], hi = a.seq_offsets[b + 1];
  lo = lo < 0 ? 0 : (lo > a.T ? a.T : lo);
  hi = hi < lo ? lo : (hi > a.T ? a.T : hi);
  float b2e_m = 0.0f;
  if (a.r_exp > 0 && a.b2e) {
    const double mf = floor((double)a.n_seg * (double)a.t[b]);
    const int m = (mf >= 0.0) ? (int)fmin(mf, (double)(a.n_seg - 1)) : 0;  // NaN -> 0
    b2e_m = a.b2e[m];
  }
  const bool has_exp = a.r_exp > 0 && a.n_rt > a.n_ct;
  for (int i = lo + blockIdx.x * 256 + (int)threadIdx.x; i < hi; i += gridDim.x * 256) {
    const uint8_t f = a.flags[i];
    float l;
    if (f & CE_TOK_KEEP) {
      l = __builtin_inff();
    } else {
      const float* pp = a.part + i;
      l = pp[0];
      for (int q = 1; q < a.n_ct; ++q) l += pp[(int64_t)q * a.T];
      l += a.b2c;
      if ((f & CE_TOK_GEN) && has_exp) {
        float e = pp[(int64_t)a.n_ct * a.T];
        for (int q = a.n_ct + 1; q < a.n_rt; ++q) e += pp[(int64_t)q * a.T];
        l += e + b2e_m;
      }
    }
    a.logits[i] = l;
    if (a.probs) a.probs[i] = (f & CE_TOK_KEEP) ? 1.0f : 1.0f / (1.0f + expf(-l));
  }
}

hipError_t launch_score_assemble(const ScoreArgs& a, hipStream_t stream) {
  if (!a.part || a.n_rt <= 0 || a.B <= 0) return hipErrorInvalidValue;
  // about one workgroup per 256 tokens of an average sequence, at most 64
  int gx = (int)(((int64_t)a.T + (int64_t)a.B * 256 - 1) / ((int64_t)a.B * 256));
  gx = gx < 1 ? 1 : (gx > 64 ? 64 : gx);
  hipLaunchKernelGGL(score_assemble_kernel, dim3(gx, a.B), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_score_tiles(const ScoreArgs& a, int tm, int tn, hipStream_t stream) {
  if (!a.part || a.n_rt <= 0) return hipErrorInvalidValue;
  const int items = (a.T / tm + a.B) * a.n_rt;
  const int grid = (a.info ? a.B : 0) + (items + 7) / 8 * 8;
  if (tm == 64 && tn == 64) hipLaunchKernelGGL((score_tile_kernel<64, 64>), dim3(grid), dim3(256), 0, stream, a);
  else if (tm == 128 && tn == 64) hipLaunchKernelGGL((score_tile_kernel<128, 64>), dim3(grid), dim3(256), 0, stream, a);
  else if (tm == 64 && tn == 128) hipLaunchKernelGGL((score_tile_kernel<64, 128>), dim3(grid), dim3(256), 0, stream, a);
  else if (tm == 128 && tn == 128) hipLaunchKernelGGL((score_tile_kernel<128, 128>), dim3(grid), dim3(256), 0, stream, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace ce
