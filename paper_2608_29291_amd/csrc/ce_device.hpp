// Device helpers shared by the CE-Router kernels (gfx950 / CDNA4 only).
//
// Tiles are staged through LDS in 16-byte chunks: one tile row holds
// KB = 128 bytes of the contraction dimension (64 bf16 or 32 fp32 values) as
// 8 chunks, stored at an XOR-swizzled chunk slot (lds_chunk_off) so that the
// 16-byte MFMA fragment reads of consecutive rows hit distinct LDS banks.
//
// MFMA operand convention used everywhere: the "A" operand (output rows) is a
// weight matrix row block (features / scorer ranks), the "B" operand (output
// columns) is a block of 32 token rows. Both are K-contiguous in memory. For a
// 32-byte step of K, lane l supplies chunk (2*s + l/32) of row (l % 32) for both
// operands, so A and B always agree on which K values meet. The 32x32 output
// block then holds, in lane l and accumulator v:
//   column (token)  = l % 32
//   row (feature)   = 8*(v/4) + 4*(l/32) + (v%4)
// i.e. 4 consecutive features per (lane, v/4): outputs are stored as 8-byte
// (bf16) or 16-byte (fp32) vectors.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ce {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kKB = 128;     // bytes of K per staged tile row
constexpr int kChunks = 8;   // 16-byte chunks per staged tile row

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two float32 -> packed bf16 (low = a), round to nearest even, one
// v_cvt_pk_bf16_f32; NaN stays NaN.
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// float32 -> bf16 bits (low 16 bits of the result).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) { return pack_bf16(f, 0.0f) & 0xffffu; }

// SiLU(x) = x * sigmoid(x) with the hardware exp2 and reciprocal (about one
// ulp each): x * rcp(1 + 2^(-x log2 e)).
__device__ __forceinline__ float silu_f32(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * x));
}

// LDS byte offset of chunk c of tile row r (XOR swizzle over 8 chunks).
// The XOR key (r ^ r>>3) & 7 differs for any 8 consecutive rows and also for
// the 8 even (or 8 odd) rows of any 16 consecutive rows, so a 16-byte
// fragment read of 8 or of 16 consecutive rows touches distinct banks whether
// the LDS serves 128 or 256 bytes per clock.
__device__ __forceinline__ int lds_chunk_off(int r, int c) {
  return (r * kChunks + (c ^ ((r ^ (r >> 3)) & 7))) * 16;
}

// One 32-byte K step on a 32x32 block. `a` and `b` are this lane's 16-byte
// chunks of the A (weights) and B (tokens) operands.
template <bool kBF16>
__device__ __forceinline__ void mfma_step(f32x16_t& acc, const u32x4_t& a, const u32x4_t& b) {
  if constexpr (kBF16) {
    bf16x8_t av = __builtin_bit_cast(bf16x8_t, a);
    bf16x8_t bv = __builtin_bit_cast(bf16x8_t, b);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc, 0, 0, 0);
  } else {
    // fp32: each 16-byte chunk holds 4 K values; 4 MFMAs of K = 2 (one value
    // per lane half) cover the 8 values of the step.
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
  }
}

__device__ __forceinline__ u32x4_t lds_read16(const char* lds, int off) {
  return *reinterpret_cast<const u32x4_t*>(lds + off);
}

__device__ __forceinline__ void lds_write16(char* lds, int off, const u32x4_t& v) {
  *reinterpret_cast<u32x4_t*>(lds + off) = v;
}

__device__ __forceinline__ u32x4_t gload16(const char* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
}

__device__ __forceinline__ u32x4_t gload16_cached(const char* p) {
  return *reinterpret_cast<const u32x4_t*>(p);
}

// Workgroup barrier for LDS-only hand-offs: waits for this wave's own LDS
// operations, then s_barrier, with a compiler memory clobber so no memory
// access moves across it. Unlike __syncthreads() it carries no memory fence,
// so loads still in flight to LDS (buffer loads with the LDS bit) are not
// drained here; their consumers wait for them explicitly with vmcnt.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until at most N vector memory operations of this wave are in flight
// (vmcnt only; the export and LDS/scalar counters are left alone).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // vmcnt lives in bits [3:0] and [15:14]; expcnt = 7 and lgkmcnt = 15 mean "no wait"
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Raw buffer resource over [base, base + bytes): 16-byte loads through it take
// a per-lane 32-bit offset plus a wave-uniform offset, and return zeros past
// `bytes` (the hardware range check).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ u32x4_t bload16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0));
}

// Store 4 consecutive output values (fp32 accumulators) as dtype.
template <bool kBF16>
__device__ __forceinline__ void store4(char* p, float a, float b, float c, float d) {
  if constexpr (kBF16) {
    u32x2_t v;
    v.x = pack_bf16(a, b);
    v.y = pack_bf16(c, d);
    *reinterpret_cast<u32x2_t*>(p) = v;
  } else {
    f32x4_t v = {a, b, c, d};
    *reinterpret_cast<f32x4_t*>(p) = v;
  }
}

// Load 4 consecutive values of dtype as fp32.
template <bool kBF16>
__device__ __forceinline__ f32x4_t load4(const char* p) {
  f32x4_t r;
  if constexpr (kBF16) {
    u32x2_t v = *reinterpret_cast<const u32x2_t*>(p);
    r.x = bf16_to_f32(v.x & 0xffffu);
    r.y = bf16_to_f32(v.x >> 16);
    r.z = bf16_to_f32(v.y & 0xffffu);
    r.w = bf16_to_f32(v.y >> 16);
  } else {
    r = *reinterpret_cast<const f32x4_t*>(p);
  }
  return r;
}

// Order-preserving uint32 key of a float32 logit: larger logit -> larger key;
// -0 and +0 share a key; every NaN maps to 0, below -inf (0x007fffff).
__device__ __forceinline__ uint32_t logit_key(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// k = ceil(keep * n), exact, on the float32 bit pattern of keep (keep in [0, 1]).
__device__ __forceinline__ int32_t num_keep_dev(float keep, int32_t n) {
  if (n <= 0) return 0;
  uint32_t u = __float_as_uint(keep);
  if (u == 0u || u == 0x80000000u) return 0;
  int e = (int)((u >> 23) & 0xffu);
  uint64_t m = u & 0x7fffffu;
  int ex;
  if (e == 0) {
    ex = -149;
  } else {
    m |= 0x800000u;
    ex = e - 150;
  }
  uint64_t p = m * (uint64_t)(uint32_t)n;
  if (ex >= 0) return (int32_t)(p << ex);
  int s = -ex;
  if (s >= 63) return p ? 1 : 0;
  uint64_t k = (p + ((1ull << s) - 1ull)) >> s;
  return (int32_t)k;
}

// Sum of one int64 per thread over the workgroup (wave reduction, then LDS
// across waves; scratch holds one value per wave).
__device__ __forceinline__ int64_t block_sum_i64(int64_t v, int64_t* scratch) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) scratch[wave] = v;
  __syncthreads();
  int64_t s = 0;
  const int nw = blockDim.x >> 6;
  for (int w = 0; w < nw; ++w) s += scratch[w];
  return s;
}

// Per-sequence summary of sequence b, computed by one workgroup:
// info[3b] = lo (clamped), info[3b+1] = len (clamped), info[3b+2] = number of
// always-kept tokens | bad << 31 (offsets out of order or not covering [0, T)).
__device__ __forceinline__ void seq_summary(const int32_t* __restrict__ offs, const uint8_t* __restrict__ flags,
                                            int B, int T, int b, int32_t* __restrict__ info, int64_t* scratch) {
  const int o0 = offs[b], o1 = offs[b + 1];
  const bool bad = o0 < 0 || o1 < o0 || o1 > T || (b == 0 && o0 != 0) || (b == B - 1 && o1 != T);
  const int lo = o0 < 0 ? 0 : (o0 > T ? T : o0);
  const int hi = o1 < lo ? lo : (o1 > T ? T : o1);
  // KEEP bits of [lo, hi): the 16-byte-aligned middle in 16-byte loads (one
  // or two per thread for sequences of a few thousand tokens), the ends bytewise
  int m0 = lo + (int)((16u - (uint32_t)(((uintptr_t)flags + (uintptr_t)lo) & 15u)) & 15u);
  m0 = m0 > hi ? hi : m0;
  const int m1 = m0 + ((hi - m0) & ~15);
  int c = 0;
  for (int i = lo + (int)threadIdx.x; i < m0; i += blockDim.x) c += (flags[i] >> 1) & 1;
  for (int i = m1 + (int)threadIdx.x; i < hi; i += blockDim.x) c += (flags[i] >> 1) & 1;
  const uint4* fw = reinterpret_cast<const uint4*>(flags + m0);
  for (int i = threadIdx.x; i < (m1 - m0) >> 4; i += blockDim.x) {
    const uint4 v = fw[i];
    c += __popc(v.x & 0x02020202u) + __popc(v.y & 0x02020202u) + __popc(v.z & 0x02020202u) +
         __popc(v.w & 0x02020202u);
  }
  const int64_t n_keep = block_sum_i64(c, scratch);
  if (threadIdx.x == 0) {
    info[3 * b + 0] = lo;
    info[3 * b + 1] = hi - lo;
    info[3 * b + 2] = (int32_t)n_keep | (bad ? (int32_t)0x80000000 : 0);
  }
}

}  // namespace ce
