// Per-sequence TopK over the routing logits (paper section 3.4, Eq. 6) and the
// packed index maps that drive compaction.
//
// Selection is exact and deterministic: each float32 logit becomes an
// order-preserving uint32 key (-0 == +0, NaN lowest); a 4-pass 8-bit radix
// select finds the key theta of the k-th retained routable token; then one
// sweep in token order retains every always-kept token, every key > theta and
// the first (k - #{key > theta}) tokens with key == theta (lower index wins).
// The same sweep assigns packed positions with wavefront ballot / popcount
// prefix sums, so kept_idx comes out ascending within each sequence.
//
// One 1024-thread workgroup per sequence; sequences of up to 16384 tokens keep
// their keys and KEEP bits in LDS, longer ones re-read logits and flags from
// global memory on every pass.
#include "ce_device.hpp"
#include "ce_launch.hpp"

namespace ce {

namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kLdsKeys = 16384;

__global__ __launch_bounds__(256) void seq_info_kernel(const int32_t* __restrict__ offs,
                                                       const uint8_t* __restrict__ flags, int B,
                                                       int T, int32_t* __restrict__ info) {
  __shared__ int64_t scratch[4];
  seq_summary(offs, flags, B, T, blockIdx.x, info, scratch);
}

struct SelShared {
  uint32_t keys[kLdsKeys];
  uint64_t keepmask[kLdsKeys / 64];
  uint32_t hist[256];
  int32_t wsum_s[kSelWaves];
  int32_t wsum_e[kSelWaves];
  int64_t scratch[kSelWaves];
  uint32_t sel_digit;
  int32_t sel_above;
};

template <bool kLds>
__device__ void select_body(const SelectArgs& a, SelShared& sh, int lo, int len, int nkeep,
                            int64_t off_b) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));

  // ---- logits from the rank-tiled scorer's partial sums (fixed order) ----
  float b2e_m = 0.0f;
  if (a.part && a.r_exp > 0 && a.b2e) {
    const double mf = floor((double)a.n_seg * (double)a.t[blockIdx.x]);
    const int m = (mf >= 0.0) ? (int)fmin(mf, (double)(a.n_seg - 1)) : 0;  // NaN -> 0
    b2e_m = a.b2e[m];
  }
  auto assemble = [&](int i) -> float {
    const uint8_t f = a.flags[lo + i];
    if (f & 2) return __builtin_inff();
    const float* pp = a.part + lo + i;
    float l = pp[0];
    for (int qq = 1; qq < a.n_ct; ++qq) l += pp[(int64_t)qq * a.T];
    l += a.b2c;
    if ((f & 1) && a.r_exp > 0) {
      float e = pp[(int64_t)a.n_ct * a.T];
      for (int qq = a.n_ct + 1; qq < a.n_rt; ++qq) e += pp[(int64_t)qq * a.T];
      l += e + b2e_m;
    }
    return l;
  };
  if (!kLds && a.part) {
    for (int i = tid; i < len; i += kSelThreads) a.logits_w[lo + i] = assemble(i);
    __threadfence_block();
    __syncthreads();
  }

  // ---- keys ----
  if constexpr (kLds) {
    for (int base = 0; base < len; base += kSelThreads) {
      const int i = base + tid;
      bool kp = false;
      if (i < len) {
        kp = (a.flags[lo + i] & 2) != 0;
        float l;
        if (a.part) {
          l = assemble(i);
          a.logits_w[lo + i] = l;
        } else {
          l = a.logits[lo + i];
        }
        sh.keys[i] = logit_key(l);
      }
      const uint64_t bal = __ballot(kp);
      if (lane == 0 && base + wave * 64 < len) sh.keepmask[(base >> 6) + wave] = bal;
    }
    __syncthreads();
  }
  auto key_of = [&](int i) -> uint32_t {
    if constexpr (kLds) return sh.keys[i];
    else return logit_key(a.logits[lo + i]);
  };
  auto keep_of = [&](int i) -> bool {
    if constexpr (kLds) return (sh.keepmask[i >> 6] >> (i & 63)) & 1ull;
    else return (a.flags[lo + i] & 2) != 0;
  };

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
      if (wave == 0) {
        // lane l owns digits 4l .. 4l+3; find the digit holding the krem-th largest
        const uint32_t h0 = sh.hist[4 * lane + 0], h1 = sh.hist[4 * lane + 1];
        const uint32_t h2 = sh.hist[4 * lane + 2], h3 = sh.hist[4 * lane + 3];
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
          const int h = (int)hh[dd];
          if (cum < krem && cum + h >= krem) {
            sh.sel_digit = (uint32_t)(4 * lane + dd);
            sh.sel_above = cum;
          }
          cum += h;
        }
      }
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

  // ---- packed offset of this sequence: sum of K_b' over b' < b ----
  int64_t part = 0;
  for (int s = tid; s < b; s += kSelThreads) {
    const int len = a.info[3 * s + 1];
    const int nk = a.info[3 * s + 2] & 0x7fffffff;
    part += nk + num_keep_dev(a.keep, len - nk);
  }
  const int64_t off_b = block_sum_i64(part, sh.scratch);

  const int lo = a.info[3 * b + 0];
  const int len = a.info[3 * b + 1];
  const int nkeep = a.info[3 * b + 2] & 0x7fffffff;
  const int64_t k_b = nkeep + num_keep_dev(a.keep, len - nkeep);
  if (tid == 0) {
    a.kept_offsets[b] = (int32_t)(off_b < 0x7fffffff ? off_b : 0x7fffffff);
    if (b == a.B - 1) {
      const int64_t tot = off_b + k_b;
      a.kept_offsets[a.B] = (int32_t)(tot < 0x7fffffff ? tot : 0x7fffffff);
    }
  }
  if (b == 0) {
    // status: one writer, no atomics; covers every sequence
    int64_t tot = 0;
    int bad = 0;
    for (int s = tid; s < a.B; s += kSelThreads) {
      const int l2 = a.info[3 * s + 1];
      const int w = a.info[3 * s + 2];
      const int nk = w & 0x7fffffff;
      bad |= (w < 0) ? 1 : 0;
      tot += nk + num_keep_dev(a.keep, l2 - nk);
    }
    const int any_bad = __syncthreads_or(bad);
    tot = block_sum_i64(tot, sh.scratch);
    if (tid == 0) {
      uint32_t st = 0;
      if (any_bad) st |= 1u;
      if (tot > a.cap) st |= 2u;
      *a.status = st;
    }
  }

  if (len <= kLdsKeys) select_body<true>(a, sh, lo, len, nkeep, off_b);
  else select_body<false>(a, sh, lo, len, nkeep, off_b);
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

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(select_kernel, dim3(a.B), dim3(kSelThreads), 0, stream, a);
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
