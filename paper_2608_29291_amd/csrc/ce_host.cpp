// Host-only part of the C ABI (validation, workspace layout, keep-count rule,
// status strings). Pure C++: no HIP headers.
#include "ce_host.hpp"

#include <math.h>
#include <string.h>

namespace ce {

static size_t align_up(size_t x) { return (x + kWsAlign - 1) / kWsAlign * kWsAlign; }

int elem_size(int dtype) {
  if (dtype == CE_BF16) return 2;
  if (dtype == CE_F32) return 4;
  return 0;
}

int down_split_tiles(int cap, int d, int d_ff, int n_sets, int elem) {
  if (elem != 2 || cap <= 0 || d <= 0 || d_ff <= 0 || n_sets < 1) return 0;
  const int64_t k_bytes = (int64_t)d_ff * 2;
  const int64_t lim = (int64_t)1 << 31;
  // the ping-pong kernel's limits: whole 128-byte K superslabs, at least 3 of
  // them per K half, 32-bit buffer offsets
  if (k_bytes % 128 != 0 || k_bytes < 6 * 128) return 0;
  if ((int64_t)cap * k_bytes >= lim || (int64_t)d * k_bytes >= lim) return 0;
  const int64_t tiles = (int64_t)((cap + 255) / 256 + n_sets - 1) * ((d + 255) / 256);
  if (tiles > kSplitMaxTiles) return 0;
  // Launch cost in units of the K-loop time of one 128-byte superslab (one
  // workgroup per CU, rounds of 256), from measured per-workgroup timelines:
  // a whole tile adds its prologue and residual epilogue (~5.6 superslabs), a
  // half adds the partial sums written and read back besides (~14.1).
  const int64_t ns = k_bytes / 128;
  auto rounds = [](int64_t n) { return (n + 255) / 256; };
  const double whole = (double)rounds(tiles) * ((double)ns + 5.6);
  const double halves = (double)rounds(2 * tiles) * ((double)ns / 2.0 + 14.1);
  return halves < whole ? (int)tiles : 0;
}

int score_token_tile(int B, int T, int d, int r_core, int r_exp, int elem) {
  const int r = r_core + (r_exp > 0 ? r_exp : 0);
  if (elem != 2 || B < 1 || T < 1 || d < 1 || r > 384) return 32;
  auto rounds = [](int64_t items) { return (items + 255) / 256; };
  const int64_t c32 = rounds(((int64_t)T + 31) / 32) * (32 + r);
  const int64_t c128 = rounds(((int64_t)T + 127) / 128) * (128 + r);
  return c128 < c32 ? 128 : 32;
}

int score_tiling(int B, int T, int d, int r_core, int r_exp, int elem, int* tm, int* tn, int* n_ct, int* n_rt) {
  if (elem != 2 || B < 1 || T < 1 || d < 1 || r_core < 32) return 0;
  auto rounds = [](int64_t items) { return (items + 255) / 256; };
  // The host sees neither the always-kept nor the generation tokens, so both
  // costs count every token as scored, once with the expansion ranks active
  // (generation batches) and once without (understanding batches, where the
  // expansion tiles exit at once); the rank tiles must win both ways.
  auto single = [&](int re) {
    // the single-launch kernel: tiles of t1 tokens x every active rank; with
    // only two slabs in its LDS ring (stages over 48 KB: 128 tokens + more
    // than 256 ranks) a slab lands while the previous one is multiplied,
    // measured about 1.5x slower per byte than the deeper rings
    const int t1 = score_token_tile(B, T, d, r_core, r_exp, elem);
    const int r = r_core + re;
    int64_t c = rounds(((int64_t)T + t1 - 1) / t1) * (t1 + r);
    if ((t1 + r) * 128 > 48 * 1024) c = c * 3 / 2;
    return c;
  };
  auto tiled = [&](int m, int rt, int re) {
    const int ct = (r_core + rt - 1) / rt;
    const int et = re > 0 ? (re + rt - 1) / rt : 0;
    return rounds(((int64_t)T + m - 1) / m * (ct + et)) * (m + rt);
  };
  int64_t best = -1;
  for (int m = 64; m <= 128; m += 64)
    for (int rt = 64; rt <= 128; rt += 64) {
      const int ct = (r_core + rt - 1) / rt;
      const int et = r_exp > 0 ? (r_exp + rt - 1) / rt : 0;
      if (ct + et > kScoreMaxTiles) continue;
      const int64_t cost = tiled(m, rt, r_exp);
      if (best < 0 || cost < best) {
        best = cost;
        *tm = m;
        *tn = rt;
        *n_ct = ct;
        *n_rt = ct + et;
      }
    }
  if (best < 0) return 0;
  return best < single(r_exp) && tiled(*tm, *tn, 0) < single(0);
}

WsLayout ws_layout(int which, int B, int T, int cap, int d, int d_ff, int elem) {
  WsLayout L;
  memset(&L, 0, sizeof(L));
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + (bytes ? bytes : 1));
    return at;
  };
  const size_t sB = (size_t)(B < 0 ? 0 : B);
  const size_t sT = (size_t)(T < 0 ? 0 : T);
  const size_t sC = (size_t)(cap < 0 ? 0 : cap);
  const size_t sF = (size_t)(d_ff < 0 ? 0 : d_ff);
  L.status = take(16);
  if (which == CE_WS_TOPK || which == CE_WS_BLOCK) L.seq_info = take(3 * sB * 4);
  if (which == CE_WS_BLOCK) {
    L.kept_off = take((sB + 1) * 4);
    L.kept_idx = take(sC * 4);
    L.token_pos = take(sT * 4);
    L.logits = take(sT * 4);
    L.score_part = take((size_t)kScoreMaxTiles * sT * 4);
  }
  if (which == CE_WS_FFN || which == CE_WS_BLOCK) {
    L.grp_rows = take(sC * 4);
    L.grp_n0 = take(4);
    L.act = take(sC * sF * (size_t)elem);
    int tiles = 0;
    for (int n_sets = 1; n_sets <= 2; ++n_sets) {
      const int t = down_split_tiles(cap, d, d_ff, n_sets, elem);
      tiles = t > tiles ? t : tiles;
    }
    if (tiles > 0) {
      L.down_part = take((size_t)tiles * 2 * 256 * 256 * 4);
      L.down_cnt = take((size_t)tiles * 4);
    }
    L.sal_part = take(((size_t)kSalSplits * sB * sF + sB * ((sF + 255) / 256) * 2) * 4);
  }
  L.total = off;
  return L;
}

int32_t num_keep_host(float keep, int32_t n) {
  if (n < 0) return -1;
  if (!(keep >= 0.0f && keep <= 1.0f)) return -1;  // also rejects NaN
  if (n == 0 || keep == 0.0f) return 0;
  uint32_t u;
  memcpy(&u, &keep, 4);
  const int e = (int)((u >> 23) & 0xffu);
  uint64_t m = u & 0x7fffffu;
  int ex;
  if (e == 0) {
    ex = -149;
  } else {
    m |= 0x800000u;
    ex = e - 150;
  }
  // keep = m * 2^ex exactly; k = ceil(m * n / 2^-ex) in 64-bit integers
  const uint64_t p = m * (uint64_t)(uint32_t)n;  // < 2^55
  if (ex >= 0) return (int32_t)(p << ex);
  const int s = -ex;
  if (s >= 63) return p ? 1 : 0;
  return (int32_t)((p + ((1ull << s) - 1ull)) >> s);
}

int check_batch(const ce_batch* b, bool need_t) {
  if (!b) return CE_ERR_INVALID_ARG;
  if (b->B < 1 || b->T < 0 || b->kept_capacity < 0) return CE_ERR_INVALID_ARG;
  if (!b->seq_offsets) return CE_ERR_INVALID_ARG;
  if (b->T > 0 && !b->flags) return CE_ERR_INVALID_ARG;
  if (need_t && !b->t) return CE_ERR_INVALID_ARG;
  if (!(b->keep >= 0.0f && b->keep <= 1.0f)) return CE_ERR_INVALID_ARG;
  return CE_OK;
}

int check_dtype_d(int dtype, int32_t d) {
  if (dtype != CE_F32 && dtype != CE_BF16) return CE_ERR_UNSUPPORTED;
  if (d <= 0 || (d % 64) != 0) return CE_ERR_UNSUPPORTED;
  return CE_OK;
}

int check_scorer(const ce_scorer_w* w) {
  if (!w) return CE_ERR_INVALID_ARG;
  int st = check_dtype_d(w->dtype, w->d);
  if (st != CE_OK) return st;
  if (w->r_core < 32 || (w->r_core % 32) != 0) return CE_ERR_UNSUPPORTED;
  if (w->r_exp < 0 || (w->r_exp % 32) != 0) return CE_ERR_UNSUPPORTED;
  if (w->r_core + w->r_exp > kMaxRanks) return CE_ERR_UNSUPPORTED;
  if (w->n_seg < 1 || w->n_seg > kMaxSeg) return CE_ERR_UNSUPPORTED;
  if (!w->w1_core || !w->w2_core) return CE_ERR_INVALID_ARG;
  if (w->r_exp > 0 && (!w->w1_exp || !w->w2_exp)) return CE_ERR_INVALID_ARG;
  if (!isfinite(w->b2_core)) return CE_ERR_INVALID_ARG;
  return CE_OK;
}

int check_ffn(const ce_ffn_w* w) {
  if (!w) return CE_ERR_INVALID_ARG;
  int st = check_dtype_d(w->dtype, w->d);
  if (st != CE_OK) return st;
  if (w->d_ff <= 0 || (w->d_ff % 64) != 0) return CE_ERR_UNSUPPORTED;
  if (w->n_sets != 1 && w->n_sets != 2) return CE_ERR_UNSUPPORTED;
  for (int s = 0; s < w->n_sets; ++s)
    if (!w->w_gate[s] || !w->w_up[s] || !w->w_down[s]) return CE_ERR_INVALID_ARG;
  return CE_OK;
}

int check_ws(const void* ws, size_t ws_bytes, size_t need) {
  if (!ws || ws_bytes < need) return CE_ERR_WORKSPACE;
  if (((uintptr_t)ws % kWsAlign) != 0) return CE_ERR_WORKSPACE;
  return CE_OK;
}

}  // namespace ce

extern "C" {

const char* ce_status_string(int status) {
  switch (status) {
    case CE_OK: return "CE_OK";
    case CE_ERR_INVALID_ARG: return "CE_ERR_INVALID_ARG: null pointer, bad size or value out of range";
    case CE_ERR_UNSUPPORTED: return "CE_ERR_UNSUPPORTED: shape or dtype outside the supported limits";
    case CE_ERR_WORKSPACE: return "CE_ERR_WORKSPACE: workspace missing, misaligned or too small";
    case CE_ERR_HIP: return "CE_ERR_HIP: a HIP runtime call failed";
    default: return "unknown ce_router status";
  }
}

const char* ce_version(void) { return "ce_router 0.1.0 gfx950"; }

int32_t ce_num_keep(float keep, int32_t n_routable) { return ce::num_keep_host(keep, n_routable); }

int64_t ce_kept_count_host(int32_t B, int32_t T, const int32_t* offs, const uint8_t* flags,
                           float keep) {
  if (B < 1 || T < 0 || !offs || (T > 0 && !flags)) return -1;
  if (!(keep >= 0.0f && keep <= 1.0f)) return -1;
  if (offs[0] != 0 || offs[B] != T) return -1;
  int64_t total = 0;
  for (int b = 0; b < B; ++b) {
    const int lo = offs[b], hi = offs[b + 1];
    if (hi < lo || lo < 0 || hi > T) return -1;
    int a = 0;
    for (int i = lo; i < hi; ++i) a += (flags[i] & CE_TOK_KEEP) ? 1 : 0;
    total += a + ce::num_keep_host(keep, hi - lo - a);
  }
  return total;
}

size_t ce_workspace_size(int which, const ce_batch* batch, int32_t d, int32_t d_ff, int dtype) {
  if (!batch || (which != CE_WS_TOPK && which != CE_WS_FFN && which != CE_WS_BLOCK)) return 0;
  const int elem = ce::elem_size(dtype);
  if (!elem) return 0;
  return ce::ws_layout(which, batch->B, batch->T, batch->kept_capacity, d, d_ff, elem).total;
}

}  // extern "C"
