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
#include "ce_router.h"

namespace ce {

namespace {

constexpr int kTok = 32;         // tokens per tile
constexpr int kSlabRow = 128;    // bytes of K per staged row
constexpr int kLds = 152 * 1024;  // ring bytes (the rest of the 160 KB holds the small arrays)
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

// Locate tile `tile` among the per-sequence tilings: sequence b, tokens [lo, hi).
// The offsets are read into LDS 256 sequences at a time (one load per thread),
// then every thread walks them: one memory latency plus a few LDS reads per
// sequence.
__device__ void find_tile(const ScoreArgs& a, int tile, int* sh, int& b, int& lo, int& hi) {
  const int tid = threadIdx.x;
  int base = 0;  // tiles before the current chunk of sequences
  b = -1;
  lo = hi = 0;
  for (int s0 = 0; s0 < a.B; s0 += 256) {
    const int cnt = min(256, a.B - s0);
    if (tid <= cnt) {
      int o = a.seq_offsets[s0 + tid];
      sh[tid] = o < 0 ? 0 : (o > a.T ? a.T : o);
    }
    __syncthreads();
    int prev = sh[0];
    for (int j = 0; j < cnt; ++j) {
      int se = sh[j + 1];
      se = se < prev ? prev : se;
      const int nt = (se - prev + kTok - 1) / kTok;
      if (b < 0 && tile < base + nt) {
        b = s0 + j;
        lo = prev + (tile - base) * kTok;
        hi = min(lo + kTok, se);
      }
      base += nt;
      prev = se;
    }
    __syncthreads();  // sh is refilled by the next chunk
    if (b >= 0) return;
  }
}

template <bool kBF16>
__global__ __launch_bounds__(256) void score_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[kLds];
  __shared__ __attribute__((aligned(8))) int sh[260];  // also the summary's int64 scratch
  __shared__ float red[4][2][kTok];
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
  find_tile(a, tile, sh, b, lo, hi);
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
  const int stage = (kTok + 32 * nb) * kSlabRow;
  // two slabs in flight: deeper rings measured slower (the extra LDS DMA in
  // flight only adds queueing)
  int nstage = kLds / stage;         // >= 2: a stage is at most (32 + 512) x 128 B = 68 KB
  nstage = nstage > 3 ? 3 : nstage;
  const int per_slab = 1 + nb;       // DMA instructions per wave per slab

  // ---- DMA plan: instruction i of a slab covers stage rows 8i .. 8i + 7 and
  //      belongs to wave i % 4: wave w fetches token rows 8w .. 8w + 7 and rows
  //      8w .. 8w + 7 of every weight block ----
  const int r8 = lane >> 3;
  const int pch = lane & 7;
  const int trow = 8 * wave + r8;  // this lane's row inside a 32-row block
  const bool tlive = trow < n && !(a.flags[lo + (trow < n ? trow : 0)] & CE_TOK_KEEP);
  const uint32_t chunk_off = (uint32_t)((pch ^ ((trow >> 1) & 7)) << 4);
  // rows that are never scored read past the resource end: zeros, no traffic
  const uint32_t t_voff = tlive ? (uint32_t)(trow * a.h_ld) + chunk_off : 0x7ffffff0u;
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
  // same L2 lines (the sum order is fixed per tile).
  const int nk_all = a.k_bytes / kSlabRow;
  const int rot = (int)(blockIdx.x % (unsigned)nk_all);
  auto dma = [&](int kb, int buf) __attribute__((always_inline)) {
    lds_char* st = ring + buf * stage;
    int ks = kb + rot;
    ks = ks >= nk_all ? ks - nk_all : ks;
    const int soff = ks * kSlabRow;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(trs, st + 8 * wave * kSlabRow, 16, (int)t_voff, soff, 0, 0);
    // one loop per weight matrix: each instruction's resource is fixed
    for (int blk = 0; blk < nbc; ++blk)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(crs, st + (kTok + 32 * blk + 8 * wave) * kSlabRow, 16,
                                               (int)w_voff, soff + (int)(32 * blk * a.h_ld), 0, 0);
    for (int blk = nbc; blk < nb; ++blk)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ers, st + (kTok + 32 * blk + 8 * wave) * kSlabRow, 16,
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
  float pc = 0.0f, pe = 0.0f;
  auto run = [&](auto nbw_c) __attribute__((always_inline)) {
    constexpr int NBW = decltype(nbw_c)::value;
    // two accumulators per block (even and odd K steps) halve the chain of
    // dependent MFMAs; they are added before the epilogue
    f32x16_t acc[NBW > 0 ? NBW : 1][2];
#pragma unroll
    for (int i = 0; i < NBW; ++i) acc[i][0] = acc[i][1] = f32x16_t{};
    int buf = 0;
    for (int kb = 0; kb < nk; ++kb) {
      // slab kb must have landed; the later slabs already issued may stay in flight
      const int ahead = min(nk - 1 - kb, nstage - 2);
      wait_vm(ahead * per_slab);
      lds_barrier();
      if constexpr (NBW > 0) {
        const char* st = smem + buf * stage;
        u32x4_t fb[4], fa[4][NBW];
#pragma unroll
        for (int step = 0; step < 4; ++step) {
          const uint32_t off = (((uint32_t)(2 * step + lhalf)) ^ rkey) << 4;
          fb[step] = *reinterpret_cast<const u32x4_t*>(st + lrow * kSlabRow + off);
#pragma unroll
          for (int i = 0; i < NBW; ++i)
            fa[step][i] = *reinterpret_cast<const u32x4_t*>(
                st + (kTok + 32 * (wave + 4 * i) + lrow) * kSlabRow + off);
        }
#pragma unroll
        for (int step = 0; step < 4; ++step)
#pragma unroll
          for (int i = 0; i < NBW; ++i) mfma_step<kBF16>(acc[i][step & 1], fa[step][i], fb[step]);
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
      float p = 0.0f;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = 8 * (v >> 2) + 4 * lhalf + (v & 3);  // rank inside the block
        float z = acc[i][0][v] + acc[i][1][v];
        if (hb) z += ep[wave][i][r];
        p += ep[wave][i][32 + r] * silu_f32(z);
      }
      if (blk < nbc) pc += p;
      else pe += p;
    }
  };
  switch (nbw) {
    case 0: run(std::integral_constant<int, 0>{}); break;
    case 1: run(std::integral_constant<int, 1>{}); break;
    case 2: run(std::integral_constant<int, 2>{}); break;
    case 3: run(std::integral_constant<int, 3>{}); break;
    default: run(std::integral_constant<int, 4>{}); break;
  }
  pc += __shfl_xor(pc, 32);
  pe += __shfl_xor(pe, 32);
  if (lhalf == 0) {
    red[wave][0][lrow] = pc;
    red[wave][1][lrow] = pe;
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

}  // namespace

hipError_t launch_score(const ScoreArgs& a, bool bf16, hipStream_t stream) {
  if (a.T == 0 && !a.info) return hipSuccess;
  const int tiles = (a.T + kTok - 1) / kTok + a.B + (a.info ? a.B : 0);  // >= the tile count (+ summaries)
  if (bf16)
    hipLaunchKernelGGL(score_kernel<true>, dim3(tiles), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(score_kernel<false>, dim3(tiles), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ce
