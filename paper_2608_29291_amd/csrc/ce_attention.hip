// Attention over the packed retained tokens of a routed layer (paper section
// 3.4, task-adaptive token compaction: the retained tokens are packed into a
// shorter sequence for the layer's attention and FFN; for understanding the
// packed keys / values of the routed layers are the compressed key-value cache
// that decoding reuses).
//
//   O_b[:, h] = softmax(scale * Q_b[:, h] K_b[:, kv(h)]^T + M) V_b[:, kv(h)]
//
// per sequence b (packed rows q_offsets[b] .. q_offsets[b+1] of Q / O and
// kv_offsets[b] .. of K / V), query head h, key/value head kv(h) = h / (H / H_kv).
// M is 0, or with causal masking -inf for keys after the query, end-aligned:
// query i of n_q sits at key position n_kv - n_q + i. A query that sees no key
// outputs zeros.
//
// Kernel (bf16 in and out, fp32 accumulation, head_dim 128): a workgroup of 4
// waves takes 128 queries of one (sequence, head), 32 per wave, and streams the
// keys in tiles of 64:
//   * S^T = K Q^T on MFMA 32x32x16 (keys are the A operand, queries the B
//     operand, held in registers for the whole loop), so each lane owns one
//     query: its 32 scores of the tile sit in the lane and its partner lane
//     l ^ 32, and the online softmax (running max m, running sum l, rescale
//     of the output by 2^(m_old - m_new)) needs one cross-lane exchange;
//   * P (bf16, the lane's probabilities in MFMA operand order) times V^T:
//     O^T = V^T P^T with the key index of the product permuted to match the
//     layout of the score accumulators;
//   * K tiles reach LDS by whole-line DMA (a key row of 128 bf16 is 256 bytes:
//     chunk c of row r stored at c ^ (r & 15), so 16 consecutive rows read by
//     one 16-byte fragment load cover all 64 banks); V tiles are loaded to
//     registers and written transposed, [dim][key], 8-byte units u of row d at
//     u ^ ((d >> 1) & 15) (16 consecutive rows of one parity get distinct
//     units); blocks of 32 rows sit 32 x 128 + 8 bytes apart, an offset the
//     compiler cannot fold into one paired read (pairing rows of two blocks
//     would put two reads on one bank); each write instruction covers rows of
//     both parities;
//   * each stage issues the score MFMAs of key tile t + 1 before the softmax
//     of tile t (they are independent, so the matrix pipe can run while the
//     VALU computes exponentials), then P V of tile t; K and V are
//     double-buffered, one barrier per tile. With causal masking the tiles
//     after the block's last query are skipped, and only tiles that reach past
//     a wave's first visible limit are masked element by element;
//   * the scale is folded into the exponent, p = 2^(s c - m c) with c = scale
//     log2 e > 0 and m a running maximum of the raw scores that moves (and
//     rescales the output and the sum) only when some lane's tile maximum
//     exceeds it by more than 8 / c, so p < 2^8 and most tiles skip the
//     rescale.
#include <type_traits>

#include "ce_device.hpp"
#include "ce_launch.hpp"

namespace ce {

namespace {

constexpr int kDh = 128;       // head dimension
constexpr int kQT = 128;       // queries per workgroup
constexpr int kKT = 64;        // keys per tile
constexpr int kKRow = kDh * 2; // bytes per key row
constexpr int kKBytes = kKT * kKRow;       // 16 KB
constexpr int kVRow = kKT * 2;             // bytes per row of V^T (64 keys)
constexpr int kVBlk = 32 * kVRow + 8;      // 32 rows of V^T, padded
constexpr int kVBytes = 4 * kVBlk;         // 16 KB + 32
constexpr float kLazy = 8.0f;              // headroom of the running maximum (exponent of 2)

struct AttnArgs {
  const char* q;
  const char* k;
  const char* v;
  char* o;
  const int32_t* qo;
  const int32_t* ko;
  int B, H, Hkv, q_cap, kv_cap, causal;
  float scale_log2;  // scale * log2(e)
};

__device__ __forceinline__ int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }

// Exclusive prefix sum over the 256 threads of the workgroup, plus the total
// (scr: 4 ints of LDS). Every thread must call it.
__device__ __forceinline__ int excl_scan256(int v, int* scr, int& total) {
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
  __syncthreads();
  return before + x - v;
}

__device__ __forceinline__ uint32_t vkey_of(int d) { return (uint32_t)((d >> 1) & 15); }
__device__ __forceinline__ uint32_t vt_off(int d, uint32_t unit) {  // byte offset of V^T row d, unit
  return (uint32_t)((d >> 5) * kVBlk + (d & 31) * kVRow) + ((unit ^ vkey_of(d)) << 3);
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void attention_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[2 * kKBytes + 2 * kVBytes];
  char* const kbuf = smem;
  char* const vbuf = smem + 2 * kKBytes;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.y;
  const int kvh = h / (a.H / a.Hkv);

  // ---- which sequence and query tile: the per-sequence tile counts; for
  //      more than 32 sequences 256 at a time (one per thread, a block scan;
  //      a chunk below this workgroup's tile is skipped whole, and the next
  //      chunk's offsets are loaded before the scan). The LDS is free until
  //      the first K tile. ----
  const int t = blockIdx.x;
  int b = -1, q0 = 0, nq = 0, qbase = 0;
  if (a.B <= 32) {
    // a few sequences: every thread walks them (no barrier)
    int tt = t;
    for (int s = 0; s < a.B; ++s) {
      const int lo = clampi(a.qo[s], 0, a.q_cap), hi = clampi(a.qo[s + 1], lo, a.q_cap);
      const int tiles = (hi - lo + kQT - 1) / kQT;
      if (tt < tiles) {
        b = s;
        q0 = (tiles - 1 - tt) * kQT;  // last tiles first: under a causal mask they see the most keys
        nq = hi - lo;
        qbase = lo;
        break;
      }
      tt -= tiles;
    }
  } else {
    int* const wsh = reinterpret_cast<int*>(smem);
    int lo = 0, hi = 0;
    if (tid < a.B) {
      lo = clampi(a.qo[tid], 0, a.q_cap);
      hi = clampi(a.qo[tid + 1], lo, a.q_cap);
    }
    int base = 0;  // tiles of the chunks before
    for (int s0 = 0; s0 < a.B; s0 += 256) {
      const int cnt = min(256, a.B - s0);
      const int clo = lo, chi = hi;
      if (s0 + 256 + tid < a.B) {
        lo = clampi(a.qo[s0 + 256 + tid], 0, a.q_cap);
        hi = clampi(a.qo[s0 + 256 + tid + 1], lo, a.q_cap);
      }
      const int nt = tid < cnt ? (chi - clo + kQT - 1) / kQT : 0;
      int total;
      const int ex = excl_scan256(nt, wsh, total);
      if (t < base + total) {
        if (tid < cnt && t >= base + ex && t < base + ex + nt) {
          wsh[4] = s0 + tid;
          wsh[5] = (nt - 1 - (t - base - ex)) * kQT;  // last tiles first: under a causal mask they see the most keys
          wsh[6] = chi - clo;
          wsh[7] = clo;
        }
        __syncthreads();
        b = wsh[4];
        q0 = wsh[5];
        nq = wsh[6];
        qbase = wsh[7];
        __syncthreads();  // the LDS goes to the K / V tiles
        break;
      }
      base += total;
    }
  }
  if (b < 0) return;
  b = __builtin_amdgcn_readfirstlane(b);
  const int klo = clampi(a.ko[b], 0, a.kv_cap), khi = clampi(a.ko[b + 1], klo, a.kv_cap);
  const int nk = khi - klo;
  const int off = nk - nq;  // end alignment of the causal mask

  // tiles of keys this query block can see
  int ntiles = (nk + kKT - 1) / kKT;
  if (a.causal) {
    const int jmax = min(nq - 1, q0 + kQT - 1) + off;  // last key the block's last query sees
    ntiles = jmax < 0 ? 0 : min(ntiles, jmax / kKT + 1);
  }

  // ---- queries of this lane: row q0 + 32 wave + (lane % 32), K-chunks of (lane / 32) ----
  const int lrow = lane & 31;
  const int lhalf = lane >> 5;
  const int qi = q0 + 32 * wave + lrow;  // query index inside the sequence
  const int qr = min(qi, nq - 1);
  u32x4_t qf[8];
  {
    const char* qp = a.q + ((int64_t)(qbase + qr) * a.H + h) * kKRow + lhalf * 16;
#pragma unroll
    for (int s = 0; s < 8; ++s) qf[s] = *reinterpret_cast<const u32x4_t*>(qp + s * 32);
  }

  auto opaque = [](uint32_t x) __attribute__((always_inline)) {
    asm volatile("" : "+v"(x));
    return x;
  };
  const int64_t kv_row = (int64_t)a.Hkv * kKRow;  // bytes between consecutive keys
  const int64_t tile_bytes = kKT * kv_row;

  // ---- K tile DMA: wave w fetches key rows 16 w .. +15, four rows of 256 B
  //      per instruction; full tiles add the tile offset as a scalar ----
  const __amdgpu_buffer_rsrc_t krs = make_rsrc(a.k, (uint32_t)((int64_t)a.kv_cap * kv_row));
  const int kr_sub = lane >> 4;   // row within the instruction
  const int kpc = lane & 15;      // physical chunk this lane fills
  uint32_t kvo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 16 * wave + 4 * i + kr_sub;
    kvo[i] = (uint32_t)((int64_t)klo * kv_row + (int64_t)kvh * kKRow + (int64_t)r * kv_row + ((kpc ^ (r & 15)) << 4));
  }
  // Keys of a ragged last tile past the sequence's end are fetched as they
  // are (the next sequence's rows, or zeros past the buffer): every score of
  // a key at or past n_kv is replaced by -inf before the softmax reads it.
  auto dma_k = [&](int tile, int buf) __attribute__((always_inline)) {
    char* region = kbuf + buf * kKBytes + 16 * wave * kKRow;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(krs, (__attribute__((address_space(3))) void*)(region + 4 * i * kKRow),
                                               16, (int)kvo[i], (int)(tile * tile_bytes), 0, 0);
  };
  // ---- V tile: thread (kg = tid % 16, dg = tid / 16) loads keys 4 kg .. +3 of
  //      dims 8 dg .. +7 and writes them transposed (one byte permute per
  //      output dword) ----
  const int vkg = tid & 15;
  const int vdg = tid >> 4;
  // keys of a ragged last tile past the sequence's end read its last key
  // instead (finite values: their probabilities are 0, and 0 * NaN is not)
  const char* vsrc = a.v + (int64_t)klo * kv_row + (int64_t)kvh * kKRow + vdg * 16;
  u32x4_t vreg[4];
  auto load_v = [&](int tile) __attribute__((always_inline)) {
    const int k0 = tile * kKT + 4 * vkg;
    const int kmax = nk - 1;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      vreg[i] = *reinterpret_cast<const u32x4_t*>(vsrc + (int64_t)min(k0 + i, kmax) * kv_row);
  };
  // odd dim groups take the dims of each pair in the other order, so one
  // instruction writes rows of both parities
  uint32_t vst[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int d = 8 * vdg + (e ^ (vdg & 1));
    vst[e] = vt_off(d, (uint32_t)vkg);
  }
  const uint32_t sel_even = (vdg & 1) ? 0x07060302u : 0x05040100u;  // low or high halves
  const uint32_t sel_odd = (vdg & 1) ? 0x05040100u : 0x07060302u;
  auto store_v = [&](auto buf_c) __attribute__((always_inline)) {
    constexpr int kBuf = decltype(buf_c)::value;
    char* vb = vbuf + kBuf * kVBytes;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t sel = (e & 1) ? sel_odd : sel_even;
      const u32x2_t w = {__builtin_amdgcn_perm(vreg[1][e >> 1], vreg[0][e >> 1], sel),
                         __builtin_amdgcn_perm(vreg[3][e >> 1], vreg[2][e >> 1], sel)};
      *reinterpret_cast<u32x2_t*>(vb + vst[e]) = w;
    }
  };

  // ---- per-lane LDS fragment offsets, fixed over the loop ----
  uint32_t koff[8];  // K: row lrow, chunk (2 s + lhalf), swizzled
#pragma unroll
  for (int s2 = 0; s2 < 8; ++s2)
    koff[s2] = opaque((uint32_t)(lrow * kKRow + ((((uint32_t)(2 * s2 + lhalf)) ^ (uint32_t)(lrow & 15)) << 4)));
  uint32_t voff8[8];  // V^T: row lrow, logical unit lhalf + 2 i (block db adds db * kVBlk)
#pragma unroll
  for (int i = 0; i < 8; ++i) voff8[i] = opaque(vt_off(lrow, (uint32_t)(lhalf + 2 * i)));

  f32x16_t oacc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) oacc[i] = f32x16_t{};
  float m_run = -__builtin_inff(), l_run = 0.0f;
  const int vis = a.causal ? min(nk, qi + off + 1) : nk;              // keys [0, vis) are visible
  const int vis0 = a.causal ? min(nk, q0 + 32 * wave + off + 1) : nk;  // the wave's smallest

  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  // scores of one key tile: S^T = K Q^T, two blocks of 32 keys, two chains
  auto scores = [&](int kbuf_i, f32x16_t (&sc)[2]) __attribute__((always_inline)) {
    const char* kb = kbuf + kbuf_i * kKBytes;
    sc[0] = f32x16_t{};
    sc[1] = f32x16_t{};
#pragma unroll
    for (int s2 = 0; s2 < 8; ++s2)
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2) {
        const u32x4_t kf = *reinterpret_cast<const u32x4_t*>(kb + koff[s2] + 32 * kb2 * kKRow);
        mfma_step<true>(sc[kb2], kf, qf[s2]);
      }
  };
  // hide the keys of tile `tile` this lane may not see (ragged end, causal cut)
  auto mask = [&](int tile, f32x16_t (&sc)[2]) __attribute__((always_inline)) {
    const int kbase = tile * kKT;
    if (kbase + kKT > vis0) {
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int j = kbase + 32 * kb2 + 8 * (v >> 2) + 4 * lhalf + (v & 3);
          if (j >= vis) sc[kb2][v] = -__builtin_inff();
        }
    }
  };
  // one pipeline stage: scores of tile + 1 (into sn) under the softmax of
  // tile (from sc), then P V of tile
  auto body = [&](auto cur_c, int tile, f32x16_t (&sc)[2], f32x16_t (&sn)[2]) __attribute__((always_inline)) {
    constexpr int kCur = decltype(cur_c)::value;
    const bool more = tile + 1 < ntiles;
    if (tile + 2 < ntiles) dma_k(tile + 2, kCur);  // K of tile was read one stage ago
    if (more) load_v(tile + 1);
    // ---- scores of tile + 1 ----
    if (more) scores(kCur ^ 1, sn);
    // ---- online softmax of tile (lane = query) ----
    float mt = -__builtin_inff();
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sc[kb2][v]);
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    // The running maximum moves (and the output is rescaled) only when some
    // lane's tile maximum exceeds it by more than kLazy in the exponent, so
    // probabilities stay below 2^kLazy; the sum l uses the same maximum, so
    // the quotient O / l does not depend on it.
    if (__builtin_amdgcn_ballot_w64((mt - m_run) * a.scale_log2 > kLazy)) {
      const float m_new = fmaxf(m_run, mt);
      const float alpha =
          m_new == -__builtin_inff() ? 1.0f : __builtin_amdgcn_exp2f((m_run - m_new) * a.scale_log2);
#pragma unroll
      for (int i = 0; i < 4; ++i) oacc[i] *= alpha;
      l_run *= alpha;
      m_run = m_new;
    }
    const float mc = m_run == -__builtin_inff() ? 0.0f : m_run * a.scale_log2;
    float rs = 0.0f;
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sc[kb2][v], a.scale_log2, -mc));
        sc[kb2][v] = p;
        rs += p;
      }
    rs += __shfl_xor(rs, 32);
    u32x4_t pf[4];
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        pf[st][i] = pack_bf16(sc[st >> 1][8 * (st & 1) + 2 * i], sc[st >> 1][8 * (st & 1) + 2 * i + 1]);
    l_run += rs;
    // ---- O^T += V^T P^T over 4 steps of 16 keys ----
    const char* vb = vbuf + kCur * kVBytes;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const int kb2 = st >> 1, h2 = st & 1;
      const int i0 = (8 * kb2 + 4 * h2) >> 1;  // logical units (8 kb2 + 4 h2 + lhalf) and +2
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const u32x2_t lo = *reinterpret_cast<const u32x2_t*>(vb + db * kVBlk + voff8[i0]);
        const u32x2_t hi = *reinterpret_cast<const u32x2_t*>(vb + db * kVBlk + voff8[i0 + 1]);
        const u32x4_t vf = {lo.x, lo.y, hi.x, hi.y};
        mfma_step<true>(oacc[db], vf, pf[st]);
      }
    }
    if (more) {
      mask(tile + 1, sn);
      store_v(std::integral_constant<int, kCur ^ 1>{});
    }
    wait_vmcnt<0>();
    __syncthreads();
  };

  f32x16_t sa[2], sb[2];
  if (ntiles > 0) {
    dma_k(0, 0);
    if (ntiles > 1) dma_k(1, 1);
    load_v(0);
    store_v(B0{});
    wait_vmcnt<0>();
    __syncthreads();
    scores(0, sa);
    mask(0, sa);
    lds_barrier();  // every wave has read K of tile 0 before the first stage refills it
  }
  int tile = 0;
  for (; tile + 1 < ntiles; tile += 2) {
    body(B0{}, tile, sa, sb);
    body(B1{}, tile + 1, sb, sa);
  }
  if (tile < ntiles) body(B0{}, tile, sa, sb);

  // ---- epilogue: O = O^T / l, rows of real queries only ----
  if (qi >= nq) return;
  const float inv = l_run > 0.0f ? 1.0f / l_run : 0.0f;
  char* op = a.o + ((int64_t)(qbase + qi) * a.H + h) * kKRow;
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int d0 = 32 * db + 8 * g + 4 * lhalf;
      store4<true>(op + d0 * 2, oacc[db][4 * g] * inv, oacc[db][4 * g + 1] * inv, oacc[db][4 * g + 2] * inv,
                   oacc[db][4 * g + 3] * inv);
    }
}

}  // namespace

hipError_t launch_attention(const char* q, const char* k, const char* v, char* o, const int32_t* q_offsets,
                            const int32_t* kv_offsets, int B, int H, int Hkv, int q_cap, int kv_cap, bool causal,
                            float scale, hipStream_t stream) {
  if (q_cap <= 0) return hipSuccess;
  const int tiles = (q_cap + kQT - 1) / kQT + B;  // each sequence adds at most one partial tile
  AttnArgs args{q, k, v, o, q_offsets, kv_offsets, B, H, Hkv, q_cap, kv_cap, causal ? 1 : 0,
                scale * 1.4426950408889634f};
  hipLaunchKernelGGL(attention_kernel, dim3(tiles, H), dim3(256), 0, stream, args);
  return hipGetLastError();
}

}  // namespace ce
