// Per-sequence TopK over the routing logits (paper section 3.4, Eq. 6) and the
// packed index maps that drive compaction.
//
// Selection is exact and deterministic: each float32 logit becomes an
// order-preserving uint32 key (-0 == +0, NaN lowest); a radix select finds the
// key theta of the k-th retained routable token; then one sweep in token order
// retains every always-kept token, every key > theta and the first
// (k - #{key > theta}) tokens with key == theta (lower index wins). The same
// sweep assigns packed positions with wavefront ballot / popcount prefix sums,
// so kept_idx comes out ascending within each sequence.
//
// One 1024-thread workgroup per sequence. Sequences of up to 16384 tokens keep
// their keys in LDS: the loads of eight 1024-token chunks (four when the
// scorer left partial sums over more than four tiles) are in flight together,
// one wave sums the packed offset meanwhile, three radix passes of 12, 10 and
// 10 bits take two barriers each, and the sweep ranks all chunks with one
// scan. Longer sequences re-read logits and flags from global memory on each
// of four 8-bit passes.
#include "ce_device.hpp"
#include "ce_launch.hpp"

namespace ce {

namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kMaxChunks = 16;  // keys held in LDS: up to 16 x 1024 tokens

__global__ __launch_bounds__(256) void seq_info_kernel(const int32_t* __restrict__ offs,
                                                       const uint8_t* __restrict__ flags, int B,
                                                       int T, int32_t* __restrict__ info) {
  __shared__ int64_t scratch[4];
  seq_summary(offs, flags, B, T, blockIdx.x, info, scratch);
}

constexpr uint32_t kKeptKey = 0xffffffffu;  // LDS path: an always-kept token's key (logit keys stop at +inf's)
constexpr int kBins0 = 4096;  // LDS path, pass 0: key bits 31..20
constexpr int kBins1 = 1024;  // LDS path, passes 1 and 2: bits 19..10, then 9..0

struct SelShared {
  uint32_t keys[kMaxChunks * kSelThreads];
  uint32_t hist[256];         // global-memory path
  alignas(16) uint32_t hA[kBins0];  // LDS path: passes 0 and 2
  alignas(16) uint32_t hB[kBins1];  // LDS path: pass 1
  uint32_t slot_cnt[kMaxChunks * kSelWaves];  // LDS path sweep: per (chunk, wave) counts
  int32_t wsum_s[kSelWaves];
  int32_t wsum_e[kSelWaves];
  int64_t scratch[kSelWaves];
  int64_t off_b;
  uint32_t sel_digit;
  int32_t sel_above;
};

// Retained rows of sequence s: its always-kept tokens plus ceil(keep * routable).
__device__ __forceinline__ int64_t seq_kept(const SelectArgs& a, int len, int w) {
  const int nk = w & 0x7fffffff;
  return nk + num_keep_dev(a.keep, len - nk);
}

// Packed offset of sequence b (sum of K_b' over b' < b) by one wave, given
// the sizes of sequence `lane` (loaded early by the caller, zero past b).
__device__ __forceinline__ int64_t seq_offset_wave(const SelectArgs& a, int b, int lane, int len0, int w0) {
  if (a.offs_ready) return (int64_t)a.kept_offsets[b];  // from the sequence-offset scan
  int64_t part = lane < b ? seq_kept(a, len0, w0) : 0;
  for (int s = lane + 64; s < b; s += 64) part += seq_kept(a, a.info[3 * s + 1], a.info[3 * s + 2]);
  for (int off = 32; off > 0; off >>= 1) part += __shfl_xor(part, off);
  return part;
}

// Batch status by one wave: bit 0 = offsets out of order or not covering
// [0, T), bit 1 = more retained rows than the capacity. len0 / w0: the sizes
// of sequence `lane` (loaded early by the caller when lane < B).
__device__ __forceinline__ void batch_status_wave(const SelectArgs& a, int lane, int len0, int w0) {
  int64_t tot = 0;
  int bad = 0;
  for (int s = lane; s < a.B; s += 64) {
    const int l2 = s == lane ? len0 : a.info[3 * s + 1];
    const int w = s == lane ? w0 : a.info[3 * s + 2];
    bad |= (w < 0) ? 1 : 0;
    tot += seq_kept(a, l2, w);
  }
  for (int off = 32; off > 0; off >>= 1) tot += __shfl_xor(tot, off);
  const bool any_bad = __ballot(bad != 0) != 0ull;
  if (lane == 0) {
    uint32_t st = 0;
    if (any_bad) st |= 1u;
    if (tot > a.cap) st |= 2u;
    *a.status = st;
  }
}

// Wave 0: the digit of the krem-th largest key in histogram h (lane l owns
// digits 4l .. 4l+3) and the number of keys with a larger digit.
__device__ __forceinline__ void find_digit(const uint32_t* h, int krem, int lane, SelShared& sh) {
  const uint32_t h0 = h[4 * lane + 0], h1 = h[4 * lane + 1];
  const uint32_t h2 = h[4 * lane + 2], h3 = h[4 * lane + 3];
  const int s = (int)(h0 + h1 + h2 + h3);
  int incl = s;  // inclusive suffix sum over lanes >= lane
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_down(incl, o);
    if (lane + o < 64) incl += y;
  }
  int cum = incl - s;  // keys with a larger digit (higher lanes)
  const uint32_t hh[4] = {h0, h1, h2, h3};
#pragma unroll
  for (int dd = 3; dd >= 0; --dd) {
    const int hv = (int)hh[dd];
    if (cum < krem && cum + hv >= krem) {
      sh.sel_digit = (uint32_t)(4 * lane + dd);
      sh.sel_above = cum;
    }
    cum += hv;
  }
}

// Inclusive prefix sum over the 64 lanes of a wave (lane i: lanes 0..i), with
// DPP row shifts inside each row of 16 lanes, then the row-15 and row-31
// broadcasts.
__device__ __forceinline__ int wave_prefix_incl(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);  // row_bcast:15 into rows 1, 3
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);  // row_bcast:31 into rows 2, 3
  return v;
}

// Wave 0: the bin of the krem-th largest key in histogram h of 64 * kPer
// bins, and the number of keys in higher bins. Lane l first sums bins
// [kPer * l, kPer * (l + 1)); the range that holds the krem-th key is then
// searched one bin per lane. Needs 1 <= krem <= the histogram's total.
template <int kPer>
__device__ __forceinline__ void find_bin(const uint32_t* h, int krem, int lane, SelShared& sh) {
  constexpr int kQ = kPer / 4;  // 16-byte reads per lane
  static_assert(kQ == 4 || kQ % 16 == 0, "bin range of 16 or a multiple of 64");
  // each lane starts its reads at a different 16-byte column, so that a
  // wave's reads spread over all banks
  const int rot = kQ >= 16 ? lane : lane / (16 / kQ);
  const uint4* h4 = reinterpret_cast<const uint4*>(h + kPer * lane);
  uint32_t s = 0;
#pragma unroll
  for (int j = 0; j < kQ; ++j) {
    const uint4 v = h4[(j + rot) & (kQ - 1)];
    s += (v.x + v.y) + (v.z + v.w);
  }
  const int pre = wave_prefix_incl((int)s);
  const int above = __builtin_amdgcn_readlane(pre, 63) - pre;  // keys in higher lanes' ranges
  const uint64_t hit = __ballot(above < krem && above + (int)s >= krem);
  const int L = hit ? __builtin_ctzll(hit) : 0;
  const int above_l = __builtin_amdgcn_readlane(above, L);
  const int v = lane < kPer ? (int)h[kPer * L + lane] : 0;
  const int pre2 = wave_prefix_incl(v);
  const int above2 = above_l + (__builtin_amdgcn_readlane(pre2, 63) - pre2);
  const uint64_t hit2 = __ballot(lane < kPer && above2 < krem && above2 + v >= krem);
  const int j = hit2 ? __builtin_ctzll(hit2) : 0;
  if (lane == j) {
    sh.sel_digit = (uint32_t)(kPer * L + j);
    sh.sel_above = above2;
  }
}

// Keys of the 1024-token chunks [c0, c0 + kC) from the rank-tiled scorer's
// partial sums (n_tiles <= kQ tiles): the loads of every tile for the kC
// chunks are in flight together, then each logit is summed in a fixed order:
// core tiles, b2c, then (generation tokens) the expansion tiles and b2e[m].
template <int kC, int kQ>
__device__ __forceinline__ void assemble_keys(const SelectArgs& a, SelShared& sh, int c0, int lo, int len,
                                              int n_tiles, bool has_exp, float b2e_m) {
  const int tid = threadIdx.x;
  const int64_t T = a.T;
  const float* pp = a.part + lo;
  int ic[kC];
  uint32_t fc[kC];
  float pc[kQ][kC];
#pragma unroll
  for (int j = 0; j < kC; ++j) {
    ic[j] = min((c0 + j) * kSelThreads + tid, len - 1);
    fc[j] = a.flags[lo + ic[j]];
  }
#pragma unroll
  for (int q = 0; q < kQ; ++q)
    if (q < n_tiles) {
#pragma unroll
      for (int j = 0; j < kC; ++j) pc[q][j] = pp[q * T + ic[j]];
    }
#pragma unroll
  for (int j = 0; j < kC; ++j) {
    float l = pc[0][j];
#pragma unroll
    for (int q = 1; q < kQ; ++q)
      if (q < a.n_ct) l += pc[q][j];
    l += a.b2c;
    if (has_exp) {
      float e = 0.0f;
#pragma unroll
      for (int q = 1; q < kQ; ++q) {
        if (q == a.n_ct) e = pc[q][j];
        else if (q > a.n_ct && q < a.n_rt) e += pc[q][j];
      }
      if (fc[j] & 1u) l += e + b2e_m;
    }
    const int i = (c0 + j) * kSelThreads + tid;
    const bool kp = (fc[j] & 2u) != 0;
    if (i < len) {
      sh.keys[i] = kp ? kKeptKey : logit_key(l);
      a.logits_w[lo + i] = kp ? __builtin_inff() : l;
    }
  }
}

// Sequences of at most kMaxChunks * kSelThreads tokens: keys in LDS, an
// always-kept token's key above every logit's (kKeptKey), so one histogram
// counts both and krem starts at k + (always-kept count). Three passes on key
// bits 31..20 (sign, exponent, three mantissa bits: routing logits spread
// over many of these bins, where an 8-bit top digit puts most keys in one or
// two bins and the LDS atomics serialize), 19..10 and 9..0. The loops stay
// loops, each handling four tokens per thread at a time: each workgroup runs
// this code once on a cold instruction cache.
__device__ __forceinline__ void select_body_lds(const SelectArgs& a, SelShared& sh, int b, int lo, int len,
                                                int nkeep) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int nc = (len + kSelThreads - 1) / kSelThreads;  // chunks of 1024 tokens (wave-uniform)

  // wave 15 sums the packed offset of this sequence and wave 14 (sequence 0)
  // the batch status; the sizes of sequence `lane` are loaded now, so that
  // their latency overlaps the key loads below
  const bool off_wave = wave == kSelWaves - 1, st_wave = wave == kSelWaves - 2 && b == 0 && !a.offs_ready;
  int len0 = 0, w0 = 0;
  if ((off_wave && lane < b && !a.offs_ready) || (st_wave && lane < a.B)) {
    len0 = a.info[3 * lane + 1];
    w0 = a.info[3 * lane + 2];
  }

  // ---- keys: token c * 1024 + tid of chunk c; eight chunks per round with
  //      their loads in flight together (clamped into the sequence) ----
  if (!a.part) {
#pragma unroll 1
    for (int c0 = 0; c0 < nc; c0 += 8) {
      uint32_t f8[8];
      float l8[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int i = min((c0 + j) * kSelThreads + tid, len - 1);
        f8[j] = a.flags[lo + i];
        l8[j] = a.logits[lo + i];
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int i = (c0 + j) * kSelThreads + tid;
        if (i < len) sh.keys[i] = (f8[j] & 2u) ? kKeptKey : logit_key(l8[j]);
      }
    }
  } else {
    // logits from the rank-tiled scorer's partial sums: eight chunks per
    // round with up to four tiles, else four
    float b2e_m = 0.0f;
    if (a.r_exp > 0 && a.b2e) {
      const double mf = floor((double)a.n_seg * (double)a.t[b]);
      const int m = (mf >= 0.0) ? (int)fmin(mf, (double)(a.n_seg - 1)) : 0;  // NaN -> 0
      b2e_m = a.b2e[m];
    }
    const bool has_exp = a.r_exp > 0 && a.n_rt > a.n_ct;
    const int n_tiles = has_exp ? a.n_rt : a.n_ct;
    if (n_tiles <= 4) {
#pragma unroll 1
      for (int c0 = 0; c0 < nc; c0 += 8) assemble_keys<8, 4>(a, sh, c0, lo, len, n_tiles, has_exp, b2e_m);
    } else {
#pragma unroll 1
      for (int c0 = 0; c0 < nc; c0 += 4)
        assemble_keys<4, kScoreMaxTiles>(a, sh, c0, lo, len, n_tiles, has_exp, b2e_m);
    }
  }

  if (off_wave) {
    const int64_t off = seq_offset_wave(a, b, lane, len0, w0);
    if (lane == 0) sh.off_b = off;
  } else if (st_wave) {
    batch_status_wave(a, lane, len0, w0);
  }
  // pass 0 counts into hA, pass 1 into hB, pass 2 into hA's first kBins1
  // bins (cleared by wave 1 while wave 0 scans hB)
#pragma unroll
  for (int j = 0; j < kBins0 / kSelThreads; ++j) sh.hA[j * kSelThreads + tid] = 0u;
  sh.hB[tid] = 0u;
  __syncthreads();

  const int n_r = len - nkeep;
  const int k = num_keep_dev(a.keep, n_r);
  // mode: 0 = none of the routable tokens, 1 = all of them, 2 = threshold
  const int mode = (k <= 0) ? 0 : (k >= n_r ? 1 : 2);

  // Adds the keys of the sequence whose bits above `shift_m` equal `match` to
  // h[(key >> shift) & mask], four tokens per thread at a time.
  auto count_pass = [&](uint32_t* h, int shift_m, uint32_t match, int shift, uint32_t mask) {
#pragma unroll 1
    for (int c0 = 0; c0 < nc; c0 += 4) {
      uint32_t k4[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) k4[j] = sh.keys[min((c0 + j) * kSelThreads + tid, len - 1)];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool in = (c0 + j) * kSelThreads + tid < len;
        const bool sel = shift_m >= 32 || (k4[j] >> shift_m) == match;
        if (in && sel) atomicAdd(&h[(k4[j] >> shift) & mask], 1u);
      }
    }
  };

  uint32_t theta = 0;
  int krem = k + nkeep;  // the always-kept keys are the nkeep largest
  if (mode == 2) {
    count_pass(sh.hA, 32, 0u, 20, kBins0 - 1);
    lds_barrier();
    if (wave == 0) find_bin<kBins0 / 64>(sh.hA, krem, lane, sh);
    lds_barrier();
    uint32_t prefix = sh.sel_digit << 20;
    krem -= sh.sel_above;
    count_pass(sh.hB, 20, prefix >> 20, 10, kBins1 - 1);
    lds_barrier();
    if (wave == 0) {
      find_bin<kBins1 / 64>(sh.hB, krem, lane, sh);
    } else if (wave == 1) {
      uint4* z = reinterpret_cast<uint4*>(sh.hA) + lane * (kBins1 / 256);
#pragma unroll
      for (int j = 0; j < kBins1 / 256; ++j) z[j] = make_uint4(0u, 0u, 0u, 0u);
    }
    lds_barrier();
    prefix |= sh.sel_digit << 10;
    krem -= sh.sel_above;
    count_pass(sh.hA, 10, prefix >> 10, 0, kBins1 - 1);
    lds_barrier();
    if (wave == 0) find_bin<kBins1 / 64>(sh.hA, krem, lane, sh);
    lds_barrier();
    theta = prefix | sh.sel_digit;
    krem -= sh.sel_above;
  }
  // krem = number of theta-equal routable tokens to retain (lowest indices
  // first); theta < kKeptKey, so the always-kept tokens count as strong

  // ---- sweep: strong (always kept) and tie tokens counted per (chunk, wave)
  //      in token order, one scan over those counts, then packed positions ----
  auto classify = [&](uint32_t key, bool in, bool& st, bool& eq) {
    st = in && (mode == 1 || (mode == 0 ? key == kKeptKey : key > theta));
    eq = in && mode == 2 && key == theta;
  };
#pragma unroll 1
  for (int c0 = 0; c0 < nc; c0 += 4) {
    uint32_t k4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) k4[j] = sh.keys[min((c0 + j) * kSelThreads + tid, len - 1)];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      bool st, eq;
      classify(k4[j], (c0 + j) * kSelThreads + tid < len, st, eq);
      const uint64_t bs = __ballot(st), be = __ballot(eq);
      // strong count in the low 16 bits, ties in the high 16 (each at most 16384)
      if (lane == 0 && c0 + j < nc)
        sh.slot_cnt[(c0 + j) * kSelWaves + wave] = (uint32_t)__popcll(bs) | ((uint32_t)__popcll(be) << 16);
    }
  }
  __syncthreads();
  if (wave == 0) {
    // exclusive prefix over the (chunk, wave) entries in token order; lane l
    // owns entries 4l .. 4l+3
    const int n_ent = nc * kSelWaves;
    uint32_t v4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) v4[j] = (4 * lane + j < n_ent) ? sh.slot_cnt[4 * lane + j] : 0u;
    const uint32_t tot = v4[0] + v4[1] + v4[2] + v4[3];
    // both 16-bit halves stay below 2^15, so the packed sums fit an int
    uint32_t run = (uint32_t)wave_prefix_incl((int)tot) - tot;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (4 * lane + j < n_ent) sh.slot_cnt[4 * lane + j] = run;
      run += v4[j];
    }
  }
  __syncthreads();
  const int64_t off_b = sh.off_b;
#pragma unroll 1
  for (int c0 = 0; c0 < nc; c0 += 4) {
    uint32_t k4[4], pre4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      k4[j] = sh.keys[min((c0 + j) * kSelThreads + tid, len - 1)];
      pre4[j] = sh.slot_cnt[min(c0 + j, nc - 1) * kSelWaves + wave];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = (c0 + j) * kSelThreads + tid;
      bool st, eq;
      classify(k4[j], i < len, st, eq);
      const uint64_t bs = __ballot(st), be = __ballot(eq);
      const int s_before = (int)(pre4[j] & 0xffffu) + __popcll(bs & lt_mask);
      const int e_before = (int)(pre4[j] >> 16) + __popcll(be & lt_mask);
      const bool kept = st || (eq && e_before < krem);
      const int64_t pos = off_b + s_before + (e_before < krem ? e_before : krem);
      if (i < len) {
        if (kept && pos >= 0 && pos < a.cap) a.kept_idx[pos] = lo + i;
        if (a.token_pos) a.token_pos[lo + i] = kept ? (int32_t)(pos < 0x7fffffff ? pos : 0x7fffffff) : -1;
      }
    }
  }
  if (tid == 0) {
    const int64_t k_b = nkeep + k;
    a.kept_offsets[b] = (int32_t)(off_b < 0x7fffffff ? off_b : 0x7fffffff);
    if (b == a.B - 1) {
      const int64_t tot = off_b + k_b;
      a.kept_offsets[a.B] = (int32_t)(tot < 0x7fffffff ? tot : 0x7fffffff);
    }
  }
}

// Sequences longer than the LDS key buffer holds: keys and KEEP bits are
// re-read from global memory on every pass.
__device__ __forceinline__ void select_body_global(const SelectArgs& a, SelShared& sh, int lo, int len, int nkeep,
                                   int64_t off_b) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));

  // ---- logits from the rank-tiled scorer's partial sums (fixed order) ----
  if (a.part) {
    float b2e_m = 0.0f;
    if (a.r_exp > 0 && a.b2e) {
      const double mf = floor((double)a.n_seg * (double)a.t[blockIdx.x]);
      const int m = (mf >= 0.0) ? (int)fmin(mf, (double)(a.n_seg - 1)) : 0;  // NaN -> 0
      b2e_m = a.b2e[m];
    }
    for (int i = tid; i < len; i += kSelThreads) {
      const uint8_t f = a.flags[lo + i];
      float l;
      if (f & 2) {
        l = __builtin_inff();
      } else {
        const float* pp = a.part + lo + i;
        l = pp[0];
        for (int qq = 1; qq < a.n_ct; ++qq) l += pp[(int64_t)qq * a.T];
        l += a.b2c;
        if ((f & 1) && a.r_exp > 0 && a.n_rt > a.n_ct) {
          float e = pp[(int64_t)a.n_ct * a.T];
          for (int qq = a.n_ct + 1; qq < a.n_rt; ++qq) e += pp[(int64_t)qq * a.T];
          l += e + b2e_m;
        }
      }
      a.logits_w[lo + i] = l;
    }
    __threadfence_block();
    __syncthreads();
  }
  const float* logits = a.part ? a.logits_w : a.logits;
  auto key_of = [&](int i) -> uint32_t { return logit_key(logits[lo + i]); };
  auto keep_of = [&](int i) -> bool { return (a.flags[lo + i] & 2) != 0; };

  const int n_r = len - nkeep;
  const int k = num_keep_dev(a.keep, n_r);
  // mode: 0 = none of the routable tokens, 1 = all of them, 2 = threshold
  const int mode = (k <= 0) ? 0 : (k >= n_r ? 1 : 2);

  uint32_t theta = 0;
  int krem = k;
  if (mode == 2) {
    uint32_t prefix = 0, pmask = 0;
    for (int shift = 24; shift >= 0; shift -= 8) {
      if (tid < 256) sh.hist[tid] = 0;
      __syncthreads();
      for (int i = tid; i < len; i += kSelThreads) {
        if (keep_of(i)) continue;
        const uint32_t key = key_of(i);
        if ((key & pmask) == prefix) atomicAdd(&sh.hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (wave == 0) find_digit(sh.hist, krem, lane, sh);
      __syncthreads();
      prefix |= sh.sel_digit << shift;
      pmask |= 255u << shift;
      krem -= sh.sel_above;
      __syncthreads();
    }
    theta = prefix;
  }
  // krem = number of theta-equal routable tokens to retain (lowest indices first)

  // ---- sweep: retain + packed positions ----
  int64_t kept_base = 0;
  int eq_base = 0;
  for (int base = 0; base < len; base += kSelThreads) {
    const int i = base + tid;
    const bool valid = i < len;
    bool strong = false, eq = false;
    if (valid) {
      const bool kp = keep_of(i);
      if (kp) {
        strong = true;
      } else if (mode == 1) {
        strong = true;
      } else if (mode == 2) {
        const uint32_t key = key_of(i);
        strong = key > theta;
        eq = key == theta;
      }
    }
    const uint64_t bs = __ballot(strong);
    const uint64_t be = __ballot(eq);
    const int ps = __popcll(bs & lt_mask);
    const int pe = __popcll(be & lt_mask);
    if (lane == 0) {
      sh.wsum_s[wave] = __popcll(bs);
      sh.wsum_e[wave] = __popcll(be);
    }
    __syncthreads();
    int ws_s = 0, ws_e = 0, tot_s = 0, tot_e = 0;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
      const int vs = sh.wsum_s[w], ve = sh.wsum_e[w];
      if (w < wave) {
        ws_s += vs;
        ws_e += ve;
      }
      tot_s += vs;
      tot_e += ve;
    }
    const int rem = krem - eq_base > 0 ? krem - eq_base : 0;  // ties still to take
    const int eq_before = ws_e + pe;                           // ties before i in this chunk
    const bool kept = strong || (eq && eq_before < rem);
    const int ties_kept_before = eq_before < rem ? eq_before : rem;
    const int64_t pos = off_b + kept_base + ws_s + ps + ties_kept_before;
    if (valid) {
      if (kept && pos < a.cap) a.kept_idx[pos] = lo + i;
      if (a.token_pos) a.token_pos[lo + i] = kept ? (int32_t)(pos < 0x7fffffff ? pos : 0x7fffffff) : -1;
    }
    kept_base += tot_s + (tot_e < rem ? tot_e : rem);
    eq_base += tot_e;
    __syncthreads();
  }
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectArgs a) {
  __shared__ SelShared sh;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  // the following gate/up launch's arrival counters start at zero
  if (a.clear_cnt && b == 0)
    for (int i = tid; i < a.clear_n; i += kSelThreads) a.clear_cnt[i] = 0;
  const int lo = a.info[3 * b + 0];
  const int len = a.info[3 * b + 1];
  const int nkeep = a.info[3 * b + 2] & 0x7fffffff;
  if (len <= kMaxChunks * kSelThreads) {
    select_body_lds(a, sh, b, lo, len, nkeep);
    return;
  }

  // ---- long sequence: packed offset of this sequence first ----
  int64_t off_b;
  if (a.offs_ready) {
    off_b = (int64_t)a.kept_offsets[b];
  } else {
    int64_t part = 0;
    for (int s = tid; s < b; s += kSelThreads) part += seq_kept(a, a.info[3 * s + 1], a.info[3 * s + 2]);
    off_b = block_sum_i64(part, sh.scratch);
  }
  const int64_t k_b = nkeep + num_keep_dev(a.keep, len - nkeep);
  if (tid == 0) {
    a.kept_offsets[b] = (int32_t)(off_b < 0x7fffffff ? off_b : 0x7fffffff);
    if (b == a.B - 1) {
      const int64_t tot = off_b + k_b;
      a.kept_offsets[a.B] = (int32_t)(tot < 0x7fffffff ? tot : 0x7fffffff);
    }
  }
  if (b == 0 && (tid >> 6) == 0 && !a.offs_ready) {
    const int l0 = (tid < a.B) ? a.info[3 * tid + 1] : 0, w0 = (tid < a.B) ? a.info[3 * tid + 2] : 0;
    batch_status_wave(a, tid & 63, l0, w0);
  }
  select_body_global(a, sh, lo, len, nkeep, off_b);
}

// Packed offset of every sequence for large batches, in one workgroup:
// kept_offsets[b] = sum of the retained rows of sequences 0 .. b - 1 (the
// value the select kernel writes there too), kept_offsets[B] = the total, and
// the batch status word. Without it each select workgroup sums its earlier
// sequences itself, which costs O(B) per workgroup. Thread t takes a run of
// ceil(B / 1024) consecutive sequences; the runs are scanned in order.
__global__ __launch_bounds__(1024) void seq_offsets_kernel(SelectArgs a) {
  __shared__ int64_t wsum[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int per = (a.B + 1023) / 1024;
  const int s0 = min(tid * per, a.B), s1 = min(s0 + per, a.B);
  int64_t loc = 0;
  int bad = 0;
  for (int s = s0; s < s1; ++s) {
    const int w = a.info[3 * s + 2];
    bad |= w < 0 ? 1 : 0;
    loc += seq_kept(a, a.info[3 * s + 1], w);
  }
  int64_t incl = loc;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) wsum[wave] = incl;
  const int any_bad = __syncthreads_or(bad);
  int64_t before = 0, total = 0;
  for (int w = 0; w < 16; ++w) {
    before += w < wave ? wsum[w] : 0;
    total += wsum[w];
  }
  int64_t run = before + incl - loc;
  for (int s = s0; s < s1; ++s) {
    a.kept_offsets[s] = (int32_t)(run < 0x7fffffff ? run : 0x7fffffff);
    run += seq_kept(a, a.info[3 * s + 1], a.info[3 * s + 2]);
  }
  if (tid == 0) {
    a.kept_offsets[a.B] = (int32_t)(total < 0x7fffffff ? total : 0x7fffffff);
    uint32_t st = 0;
    if (any_bad) st |= 1u;
    if (total > a.cap) st |= 2u;
    *a.status = st;
  }
}

// Stable partition of packed rows by FFN set: grp_rows lists set-0 rows first
// (in packed order), then set-1 rows; n0 = number of set-0 rows.
__global__ __launch_bounds__(1024) void group_kernel(const int32_t* __restrict__ kept_idx,
                                                     const int32_t* __restrict__ kept_offsets,
                                                     int B, int cap, int T,
                                                     const uint8_t* __restrict__ flags,
                                                     int32_t* __restrict__ grp_rows,
                                                     int32_t* __restrict__ n0_out) {
  __shared__ int64_t scratch[16];
  __shared__ int32_t w0s[16], w1s[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int kt = kept_offsets[B];
  kt = kt < 0 ? 0 : (kt > cap ? cap : kt);
  auto is_set1 = [&](int j) -> bool {
    const int tok = kept_idx[j];
    return tok >= 0 && tok < T && (flags[tok] & 1);
  };
  int64_t c0 = 0;
  for (int j = tid; j < kt; j += 1024) c0 += is_set1(j) ? 0 : 1;
  const int n0 = (int)block_sum_i64(c0, scratch);
  int base0 = 0, base1 = 0;
  for (int base = 0; base < kt; base += 1024) {
    const int j = base + tid;
    const bool valid = j < kt;
    const bool s1 = valid && is_set1(j);
    const bool s0 = valid && !s1;
    const uint64_t b0 = __ballot(s0), b1 = __ballot(s1);
    if (lane == 0) {
      w0s[wave] = __popcll(b0);
      w1s[wave] = __popcll(b1);
    }
    __syncthreads();
    int p0 = 0, p1 = 0, t0 = 0, t1 = 0;
    for (int w = 0; w < 16; ++w) {
      if (w < wave) {
        p0 += w0s[w];
        p1 += w1s[w];
      }
      t0 += w0s[w];
      t1 += w1s[w];
    }
    if (s0) grp_rows[base0 + p0 + __popcll(b0 & lt_mask)] = j;
    if (s1) grp_rows[n0 + base1 + p1 + __popcll(b1 & lt_mask)] = j;
    base0 += t0;
    base1 += t1;
    __syncthreads();
  }
  if (tid == 0) *n0_out = n0;
}

// compact[j] = hidden[kept_idx[j]]: one wave per row, 16-byte chunks.
__global__ __launch_bounds__(256) void gather_kernel(const char* __restrict__ hidden,
                                                     int64_t row_bytes,
                                                     const int32_t* __restrict__ kept_idx,
                                                     const int32_t* __restrict__ kept_offsets,
                                                     int B, int cap, char* __restrict__ compact) {
  int kt = kept_offsets[B];
  kt = kt < 0 ? 0 : (kt > cap ? cap : kt);
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= kt) return;
  const char* src = hidden + (int64_t)kept_idx[j] * row_bytes;
  char* dst = compact + (int64_t)j * row_bytes;
  for (int64_t o = (threadIdx.x & 63) * 16; o < row_bytes; o += 64 * 16)
    *reinterpret_cast<u32x4_t*>(dst + o) = *reinterpret_cast<const u32x4_t*>(src + o);
}

}  // namespace

hipError_t launch_seq_info(const int32_t* seq_offsets, const uint8_t* flags, int B, int T,
                           int32_t* info, hipStream_t stream) {
  hipLaunchKernelGGL(seq_info_kernel, dim3(B), dim3(256), 0, stream, seq_offsets, flags, B, T, info);
  return hipGetLastError();
}

// Batches above this many sequences get the sequence-offset scan first.
constexpr int kSeqScanMinB = 1024;

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  SelectArgs s = a;
  s.offs_ready = 0;
  if (a.B > kSeqScanMinB) {
    hipLaunchKernelGGL(seq_offsets_kernel, dim3(1), dim3(1024), 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    s.offs_ready = 1;
  }
  hipLaunchKernelGGL(select_kernel, dim3(s.B), dim3(kSelThreads), 0, stream, s);
  return hipGetLastError();
}

hipError_t launch_group(const int32_t* kept_idx, const int32_t* kept_offsets, int B, int cap,
                        int T, const uint8_t* flags, int32_t* grp_rows, int32_t* n0,
                        hipStream_t stream) {
  hipLaunchKernelGGL(group_kernel, dim3(1), dim3(1024), 0, stream, kept_idx, kept_offsets, B, cap,
                     T, flags, grp_rows, n0);
  return hipGetLastError();
}

hipError_t launch_gather(const char* hidden, int64_t row_bytes, const int32_t* kept_idx,
                         const int32_t* kept_offsets, int B, int cap, char* compact,
                         hipStream_t stream) {
  if (cap <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_kernel, dim3((cap + 3) / 4), dim3(256), 0, stream, hidden, row_bytes,
                     kept_idx, kept_offsets, B, cap, compact);
  return hipGetLastError();
}

}  // namespace ce
