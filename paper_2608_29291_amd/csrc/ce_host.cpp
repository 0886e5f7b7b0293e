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

GemmSplit gemm_split(int64_t items, int ns) {
  GemmSplit sp;
  sp.per_x = (int)((items + kXcdCount - 1) / kXcdCount);
  sp.whole_x = sp.per_x;
  sp.tail_x = 0;
  sp.pieces = 1;
  sp.absorb = 0;
  if (items <= 0 || ns < 6) return sp;
  const int full = sp.per_x / kCusPerXcd * kCusPerXcd;
  const int tail = sp.per_x - full;
  // after more than two full rounds the workgroups' finishing times spread
  // out enough that the dispatcher fills the last round's gaps by itself
  // (measured: splitting the 7B-width gate/up tail, 12 rounds + 5 tiles per
  // XCD, gained nothing)
  if (tail == 0 || full > 2 * kCusPerXcd) return sp;
  const double whole = (double)ns + 3.5;
  double best = whole;
  int best_s = 1;
  for (int s = 2; s * tail <= kCusPerXcd && s * 3 <= ns; ++s) {
    const double cost = (double)ns / s + 2.0 + 2.5 * (s == 2 ? 1 : s);
    if (cost < best) {
      best = cost;
      best_s = s;
    }
  }
  if (best_s == 1) return sp;
  sp.whole_x = full;
  sp.tail_x = tail;
  sp.pieces = best_s;
  return sp;
}

void gemm_items(int mode, int cap, int d, int d_ff, int n_sets, int elem, int64_t* items, int* ns) {
  *items = 0;
  *ns = 0;
  if (elem != 2 || cap <= 0 || d <= 0 || d_ff <= 0 || n_sets < 1) return;
  const int64_t k_bytes = (int64_t)(mode == 0 ? d : d_ff) * 2;
  const int n_feat = mode == 0 ? d_ff : d;
  const int64_t lim = (int64_t)1 << 31;
  if (k_bytes % 128 != 0 || k_bytes < 3 * 128) return;
  // rows of the token operand: the hidden states (T rows, gate/up on the
  // block path) or the packed rows; cap bounds the packed ones, and the
  // launcher checks the actual operand before it relies on this
  if ((int64_t)cap * k_bytes >= lim || (int64_t)n_feat * k_bytes >= lim) return;
  const int ftile = mode == 0 ? 128 : 256;
  *items = (int64_t)((cap + 255) / 256 + n_sets - 1) * ((n_feat + ftile - 1) / ftile);
  *ns = (int)(k_bytes / 128);
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
  const bool block = which == CE_WS_BLOCK || which == CE_WS_BLOCK_GAP;
  L.status = take(16);
  if (which == CE_WS_TOPK || block) L.seq_info = take(3 * sB * 4);
  if (which == CE_WS_SCORE) L.score_part = take((size_t)kScoreMaxTiles * sT * 4);
  if (which == CE_WS_SCORE || block) L.tile_start = take((sB + 1) * 4);
  if (block) {
    L.kept_off = take((sB + 1) * 4);
    L.kept_idx = take(sC * 4);
    L.token_pos = take(sT * 4);
    L.logits = take(sT * 4);
    L.score_part = take((size_t)kScoreMaxTiles * sT * 4);
  }
  const bool pruned = which == CE_WS_FFN_PRUNED;
  if (which == CE_WS_FFN || block || pruned) {
    L.grp_rows = take(sC * 4);
    L.grp_n0 = take(4);
    L.act = take(sC * sF * (size_t)elem);
    // partial-sum tiles of the split tails of both GEMMs (they run one after
    // the other, so they share the region), for either number of weight sets
    int slots = 0;
    for (int n_sets = 1; n_sets <= 2; ++n_sets)
      for (int mode = 0; mode <= 1; ++mode) {
        int64_t items;
        int ns;
        gemm_items(mode, cap, d, d_ff, n_sets, elem, &items, &ns);
        const GemmSplit sp = gemm_split(items, ns);
        const int n = kXcdCount * sp.tail_x * sp.pieces;
        slots = n > slots ? n : slots;
      }
    if (slots > 0) {
      L.gemm_part = take((size_t)slots * 256 * 256 * 4);
      L.gu_cnt = take((size_t)kSplitMaxSlots * 4);
      L.dn_cnt = take((size_t)kSplitMaxSlots * 4);
    }
    L.sal_part = take(((size_t)kSalSplits * sB * sF + sB * ((sF + 255) / 256) * 2) * 4);
  }
  if (pruned) {
    const size_t tiles = (sC + 255) / 256 + 1;  // token tiles of either number of weight sets
    L.row_seq = take(sC * 4);
    L.sal_seg = take(tiles * kSalSegs * sF * 4);
    L.sal_meta = take(tiles * (kSalSegs + 1) * 4);
    L.row_flag = take(sC);
    L.seq_cnt = take(sB * 4);
  }
  if (which == CE_WS_BLOCK_GAP) {
    // one slot per wave of the down GEMM and row; waves cover >= 32 features
    const size_t sD = (size_t)(d < 0 ? 0 : d);
    L.gap_part = take(sC * ((sD + 31) / 32) * 4 * sizeof(double));
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
  if (b->B > kMaxBatch) return CE_ERR_UNSUPPORTED;  // sequence index in a grid's y dimension
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
  if (!batch || which < CE_WS_TOPK || which > CE_WS_SCORE) return 0;
  const int elem = ce::elem_size(dtype);
  if (!elem) return 0;
  return ce::ws_layout(which, batch->B, batch->T, batch->kept_capacity, d, d_ff, elem).total;
}

}  // extern "C"
