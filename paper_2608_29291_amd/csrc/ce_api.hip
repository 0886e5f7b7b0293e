// C-ABI entry points of the CE-Router routed-block library (declared in
// include/ce_router.h). Each entry point validates on the host, carves the
// caller's workspace, then enqueues its kernels on the caller's stream.
#include <hip/hip_runtime.h>

#include "ce_host.hpp"
#include <math.h>

#include "ce_launch.hpp"

using namespace ce;

namespace {

inline int hip_status(hipError_t e) { return e == hipSuccess ? CE_OK : CE_ERR_HIP; }

#define CE_TRY(expr)                          \
  do {                                        \
    const hipError_t _e = (expr);             \
    if (_e != hipSuccess) return CE_ERR_HIP;  \
  } while (0)

#define CE_CHECK(expr)               \
  do {                               \
    const int _s = (expr);           \
    if (_s != CE_OK) return _s;      \
  } while (0)

template <typename T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

ScoreArgs make_score_args(const ce_batch* b, const void* hidden, const ce_scorer_w* w, float* logits,
                          float* probs) {
  const int elem = elem_size(w->dtype);
  ScoreArgs a{};
  a.hidden = static_cast<const char*>(hidden);
  a.h_ld = (int64_t)w->d * elem;
  a.k_bytes = w->d * elem;
  a.B = b->B;
  a.T = b->T;
  a.seq_offsets = b->seq_offsets;
  a.flags = b->flags;
  a.t = b->t;
  a.w1c = static_cast<const char*>(w->w1_core);
  a.b1c = w->b1_core;
  a.w2c = w->w2_core;
  a.b2c = w->b2_core;
  a.w1e = static_cast<const char*>(w->w1_exp);
  a.b1e = w->b1_exp;
  a.w2e = w->w2_exp;
  a.b2e = w->b2_exp;
  a.r_core = w->r_core;
  a.r_exp = w->r_exp;
  a.n_seg = w->n_seg;
  a.logits = logits;
  a.probs = probs;
  a.info = nullptr;
  return a;
}

// gate/up: tokens (row map2[map1[j]] of `tok`) -> act[omap1[j]] (or act[j])
FfnGemmArgs gateup_args(const ce_ffn_w* w, const ce_batch* b, const char* tok, const int32_t* map1,
                        const int32_t* map2, char* act, const int32_t* omap1, const int32_t* kt,
                        const int32_t* n0) {
  const int elem = elem_size(w->dtype);
  FfnGemmArgs a = {};
  for (int s = 0; s < 2; ++s) {
    const int ss = s < w->n_sets ? s : 0;
    a.w0[s] = static_cast<const char*>(w->w_gate[ss]);
    a.w1[s] = static_cast<const char*>(w->w_up[ss]);
  }
  a.w_ld = (int64_t)w->d * elem;
  a.n_feat = w->d_ff;
  a.k_bytes = w->d * elem;
  a.tok = tok;
  a.tok_ld = (int64_t)w->d * elem;
  a.tok_rows = map2 ? b->T : b->kept_capacity;  // hidden rows, or packed rows
  a.map1 = map1;
  a.map2 = map2;
  a.out = act;
  a.out_ld = (int64_t)w->d_ff * elem;
  a.omap1 = omap1;
  a.omap2 = nullptr;
  a.kt_ptr = kt;
  a.cap = b->kept_capacity;
  a.n0_ptr = n0;
  a.n_sets = w->n_sets;
  return a;
}

// down: act[map1[j]] (or act[j]) -> out[omap2[omap1[j]]] (+ res at the same row)
FfnGemmArgs down_args(const ce_ffn_w* w, const ce_batch* b, const char* act, const int32_t* map1,
                      char* out, const int32_t* omap1, const int32_t* omap2, const char* res,
                      const int32_t* kt, const int32_t* n0) {
  const int elem = elem_size(w->dtype);
  FfnGemmArgs a = {};
  for (int s = 0; s < 2; ++s) {
    const int ss = s < w->n_sets ? s : 0;
    a.w0[s] = static_cast<const char*>(w->w_down[ss]);
    a.w1[s] = nullptr;
  }
  a.w_ld = (int64_t)w->d_ff * elem;
  a.n_feat = w->d;
  a.k_bytes = w->d_ff * elem;
  a.tok = act;
  a.tok_ld = (int64_t)w->d_ff * elem;
  a.tok_rows = b->kept_capacity;
  a.map1 = map1;
  a.map2 = nullptr;
  a.out = out;
  a.out_ld = (int64_t)w->d * elem;
  a.omap1 = omap1;
  a.omap2 = omap2;
  a.res = res;
  a.res_ld = (int64_t)w->d * elem;
  a.kt_ptr = kt;
  a.cap = b->kept_capacity;
  a.n0_ptr = n0;
  a.n_sets = w->n_sets;
  return a;
}

// Partial sums and arrival counters of a GEMM launch's split tail tiles
// (present when the layout reserved them); mode 0 = gate/up, 1 = down.
void set_split(FfnGemmArgs& a, void* ws, const WsLayout& L, int mode) {
  a.part = L.gemm_part ? at<float>(ws, L.gemm_part) : nullptr;
  const size_t cnt = mode == 0 ? L.gu_cnt : L.dn_cnt;
  a.tile_cnt = (L.gemm_part && cnt) ? at<int32_t>(ws, cnt) : nullptr;
}

// Shared argument checks of the staged FFN calls; on success fills the
// MoT grouping (launching the group kernel when there are two weight sets).
int ffn_prologue(const ce_batch* batch, const void* in, const int32_t* kept_idx,
                 const int32_t* kept_offsets, const ce_ffn_w* w, const void* out, void* ws,
                 size_t ws_bytes, hipStream_t s, int32_t** grp, int32_t** n0) {
  CE_CHECK(check_batch(batch, false));
  CE_CHECK(check_ffn(w));
  if (!kept_offsets) return CE_ERR_INVALID_ARG;
  if (batch->kept_capacity > 0 && (!in || !kept_idx || !out)) return CE_ERR_INVALID_ARG;
  const WsLayout L = ws_layout(CE_WS_FFN, batch->B, batch->T, batch->kept_capacity, w->d, w->d_ff,
                               elem_size(w->dtype));
  CE_CHECK(check_ws(ws, ws_bytes, L.total));
  *grp = nullptr;
  *n0 = nullptr;
  if (batch->kept_capacity == 0) return CE_OK;
  if (w->n_sets == 2) {
    *grp = at<int32_t>(ws, L.grp_rows);
    *n0 = at<int32_t>(ws, L.grp_n0);
    CE_TRY(launch_group(kept_idx, kept_offsets, batch->B, batch->kept_capacity, batch->T,
                        batch->flags, *grp, *n0, s));
  }
  return CE_OK;
}

// Arguments of ce_topk_compact / ce_topk_compact_noalloc shared by both (the
// workspace and the scratch are checked by the callers).
int topk_args_ok(const ce_batch* batch, const float* logits, const void* hidden, int dtype, int32_t d,
                 const int32_t* kept_idx, const int32_t* kept_offsets, const void* compact) {
  CE_CHECK(check_batch(batch, false));
  if (!kept_offsets) return CE_ERR_INVALID_ARG;
  if (batch->T > 0 && !logits) return CE_ERR_INVALID_ARG;
  if (batch->kept_capacity > 0 && !kept_idx) return CE_ERR_INVALID_ARG;
  if (compact) {
    CE_CHECK(check_dtype_d(dtype, d));
    if (batch->T > 0 && !hidden) return CE_ERR_INVALID_ARG;
  }
  return CE_OK;
}

// The TopK launches: per-sequence summaries into `info` [3 B], selection and
// index maps (status word into `status`), optional gather.
int topk_launch(const ce_batch* batch, const float* logits, const void* hidden, int dtype, int32_t d,
                int32_t* kept_idx, int32_t* kept_offsets, int32_t* token_pos, void* compact, int32_t* info,
                uint32_t* status, hipStream_t s) {
  CE_TRY(launch_seq_info(batch->seq_offsets, batch->flags, batch->B, batch->T, info, s));
  SelectArgs sa{};
  sa.logits = logits;
  sa.flags = batch->flags;
  sa.info = info;
  sa.B = batch->B;
  sa.keep = batch->keep;
  sa.cap = batch->kept_capacity;
  sa.kept_idx = kept_idx;
  sa.kept_offsets = kept_offsets;
  sa.token_pos = token_pos;
  sa.status = status;
  CE_TRY(launch_select(sa, s));
  if (compact)
    CE_TRY(launch_gather(static_cast<const char*>(hidden), (int64_t)d * elem_size(dtype), kept_idx, kept_offsets,
                         batch->B, batch->kept_capacity, static_cast<char*>(compact), s));
  return CE_OK;
}

// Outputs of the layer-skipping gap computed with the routed block.
struct GapOut {
  float delta;
  float* cos;
  float* rho_all;
  float* rho_ret;
  float* gap;
  uint8_t* skip;
};

// The routed block; with `go` also the layer-skipping gap from the down
// GEMM's per-row sums (the caller's workspace has the CE_WS_BLOCK_GAP layout).
int routed_block_impl(const ce_batch* batch, const void* hidden_in, void* hidden_out, const ce_scorer_w* scorer,
                      const ce_ffn_w* ffn, float* logits_out, int32_t* kept_idx_out, int32_t* kept_offsets_out,
                      const GapOut* go, void* ws, size_t ws_bytes, void* stream) {
  CE_CHECK(check_batch(batch, scorer != nullptr && scorer->r_exp > 0));
  CE_CHECK(check_scorer(scorer));
  CE_CHECK(check_ffn(ffn));
  if (scorer->d != ffn->d || scorer->dtype != ffn->dtype) return CE_ERR_INVALID_ARG;
  if (batch->T > 0 && (!hidden_in || !hidden_out)) return CE_ERR_INVALID_ARG;
  const int elem = elem_size(ffn->dtype);
  const WsLayout L = ws_layout(go ? CE_WS_BLOCK_GAP : CE_WS_BLOCK, batch->B, batch->T, batch->kept_capacity, ffn->d,
                               ffn->d_ff, elem);
  CE_CHECK(check_ws(ws, ws_bytes, L.total));
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool bf16 = ffn->dtype == CE_BF16;
  float* logits = logits_out ? logits_out : at<float>(ws, L.logits);
  int32_t* kept_idx = kept_idx_out ? kept_idx_out : at<int32_t>(ws, L.kept_idx);
  int32_t* kept_off = kept_offsets_out ? kept_offsets_out : at<int32_t>(ws, L.kept_off);
  int32_t* token_pos = at<int32_t>(ws, L.token_pos);
  int32_t* info = at<int32_t>(ws, L.seq_info);

  // 1. routing logits (Eq. 4); the same launch writes the per-sequence
  //    summaries. bf16: rank-tiled partial logits when that moves fewer
  //    bytes per workgroup; the TopK step adds them up.
  ScoreArgs sa = make_score_args(batch, hidden_in, scorer, logits, nullptr);
  sa.info = info;
  sa.tile_start = at<int32_t>(ws, L.tile_start);
  int tm = 0, tn = 0;
  const bool tiled = bf16 && score_tiling(batch->B, batch->T, scorer->d, scorer->r_core, scorer->r_exp, elem,
                                          &tm, &tn, &sa.n_ct, &sa.n_rt);
  if (tiled) {
    sa.part = at<float>(ws, L.score_part);
    CE_TRY(launch_score_tiles(sa, tm, tn, s));
  } else {
    CE_TRY(launch_score(sa, bf16, s));
  }
  // FFN launch arguments (host-known; the row counts stay on the device)
  const int32_t* kt = kept_off + batch->B;
  int32_t* grp = ffn->n_sets == 2 ? at<int32_t>(ws, L.grp_rows) : nullptr;
  int32_t* n0 = ffn->n_sets == 2 ? at<int32_t>(ws, L.grp_n0) : nullptr;
  char* act = at<char>(ws, L.act);
  FfnGemmArgs dn = down_args(ffn, batch, act, nullptr, static_cast<char*>(hidden_out), grp,
                             kept_idx, static_cast<const char*>(hidden_in), kt, n0);
  set_split(dn, ws, L, 1);
  double* gap_part = go ? at<double>(ws, L.gap_part) : nullptr;
  if (go) {
    dn.gap_part = gap_part;
    dn.gap_np = ffn_down_gap_slots(dn, bf16);
  }
  FfnGemmArgs g = gateup_args(ffn, batch, static_cast<const char*>(hidden_in), grp, kept_idx, act,
                              nullptr, kt, n0);
  set_split(g, ws, L, 0);
  g.clear_n = ffn_split_counters(dn, 1, bf16);
  g.clear_cnt = g.clear_n > 0 ? dn.tile_cnt : nullptr;
  const int gu_counters = ffn_split_counters(g, 0, bf16);

  // 2-3. per-sequence TopK + packed index maps (Eq. 6); the select launch
  //      also clears the gate/up launch's arrival counters
  SelectArgs sel{};
  sel.logits = logits;
  if (tiled) {
    sel.part = sa.part;
    sel.logits_w = logits;
    sel.n_ct = sa.n_ct;
    sel.n_rt = sa.n_rt;
    sel.T = batch->T;
    sel.r_exp = scorer->r_exp;
    sel.n_seg = scorer->n_seg;
    sel.b2c = scorer->b2_core;
    sel.b2e = scorer->b2_exp;
    sel.t = batch->t;
  }
  sel.flags = batch->flags;
  sel.info = info;
  sel.B = batch->B;
  sel.keep = batch->keep;
  sel.cap = batch->kept_capacity;
  sel.kept_idx = kept_idx;
  sel.kept_offsets = kept_off;
  sel.token_pos = token_pos;
  sel.status = at<uint32_t>(ws, L.status);
  sel.clear_cnt = gu_counters > 0 ? g.tile_cnt : nullptr;
  sel.clear_n = gu_counters;
  CE_TRY(launch_select(sel, s));
  // bypass path for a separate output buffer: dropped rows copied unchanged
  if (hidden_in != hidden_out)
    CE_TRY(launch_copy_rows(static_cast<const char*>(hidden_in), static_cast<char*>(hidden_out),
                            (int64_t)ffn->d * elem, batch->T, token_pos, s));
  // layer gap (Eq. 7) from the down GEMM's per-row sums, after the block
  auto finish_gap = [&]() -> int {
    if (!go) return CE_OK;
    CE_TRY(launch_gap_from_parts(gap_part, dn.gap_np, batch->kept_capacity, batch->seq_offsets, batch->B,
                                 batch->T, token_pos, go->delta, go->cos, go->rho_all, go->rho_ret, go->gap,
                                 go->skip, s));
    return CE_OK;
  };
  if (batch->kept_capacity == 0) return finish_gap();
  // 4. SwiGLU FFN on the retained rows, gathered straight from hidden_in
  if (ffn->n_sets == 2)
    CE_TRY(launch_group(kept_idx, kept_off, batch->B, batch->kept_capacity, batch->T, batch->flags,
                        grp, n0, s));
  CE_TRY(launch_ffn_gateup(g, bf16, s, gu_counters > 0));
  // 5. down projection + residual, scattered straight into the token rows
  CE_TRY(launch_ffn_down(dn, bf16, s, g.clear_cnt != nullptr));
  return finish_gap();
}

}  // namespace

extern "C" {

int ce_workspace_status(const void* ws, uint32_t* status_out, void* stream) {
  if (!ws || !status_out) return CE_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  CE_TRY(hipMemcpyAsync(status_out, ws, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
  CE_TRY(hipStreamSynchronize(s));
  return CE_OK;
}

int ce_score(const ce_batch* batch, const void* hidden, const ce_scorer_w* w, float* logits,
             float* probs, void* stream) {
  CE_CHECK(check_batch(batch, w != nullptr && w->r_exp > 0));
  CE_CHECK(check_scorer(w));
  if (batch->T > 0 && (!hidden || !logits)) return CE_ERR_INVALID_ARG;
  if (batch->T == 0) return CE_OK;
  const ScoreArgs a = make_score_args(batch, hidden, w, logits, probs);
  return hip_status(launch_score(a, w->dtype == CE_BF16, static_cast<hipStream_t>(stream)));
}

int ce_score_ws(const ce_batch* batch, const void* hidden, const ce_scorer_w* w, float* logits, float* probs,
                void* ws, size_t ws_bytes, void* stream) {
  CE_CHECK(check_batch(batch, w != nullptr && w->r_exp > 0));
  CE_CHECK(check_scorer(w));
  if (batch->T > 0 && (!hidden || !logits)) return CE_ERR_INVALID_ARG;
  const int elem = elem_size(w->dtype);
  const WsLayout L = ws_layout(CE_WS_SCORE, batch->B, batch->T, batch->kept_capacity, w->d, 0, elem);
  CE_CHECK(check_ws(ws, ws_bytes, L.total));
  if (batch->T == 0) return CE_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  ScoreArgs a = make_score_args(batch, hidden, w, logits, probs);
  a.tile_start = at<int32_t>(ws, L.tile_start);
  const bool bf16 = w->dtype == CE_BF16;
  int tm = 0, tn = 0;
  if (!(bf16 && score_tiling(batch->B, batch->T, w->d, w->r_core, w->r_exp, elem, &tm, &tn, &a.n_ct, &a.n_rt)))
    return hip_status(launch_score(a, bf16, s));
  a.part = at<float>(ws, L.score_part);
  CE_TRY(launch_score_tiles(a, tm, tn, s));
  CE_TRY(launch_score_assemble(a, s));
  return CE_OK;
}

int ce_topk_compact(const ce_batch* batch, const float* logits, const void* hidden, int dtype,
                    int32_t d, int32_t* kept_idx, int32_t* kept_offsets, int32_t* token_pos,
                    void* compact, void* ws, size_t ws_bytes, void* stream) {
  CE_CHECK(topk_args_ok(batch, logits, hidden, dtype, d, kept_idx, kept_offsets, compact));
  const int elem = compact ? elem_size(dtype) : 4;
  const WsLayout L = ws_layout(CE_WS_TOPK, batch->B, batch->T, batch->kept_capacity, 0, 0, elem);
  CE_CHECK(check_ws(ws, ws_bytes, L.total));
  return topk_launch(batch, logits, hidden, dtype, d, kept_idx, kept_offsets, token_pos, compact,
                     at<int32_t>(ws, L.seq_info), at<uint32_t>(ws, L.status), static_cast<hipStream_t>(stream));
}

int ce_ffn_gateup(const ce_batch* batch, const void* compact, const int32_t* kept_idx,
                  const int32_t* kept_offsets, const ce_ffn_w* w, void* act, void* ws,
                  size_t ws_bytes, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t *grp, *n0;
  CE_CHECK(ffn_prologue(batch, compact, kept_idx, kept_offsets, w, act, ws, ws_bytes, s, &grp, &n0));
  if (batch->kept_capacity == 0) return CE_OK;
  const WsLayout L = ws_layout(CE_WS_FFN, batch->B, batch->T, batch->kept_capacity, w->d, w->d_ff,
                               elem_size(w->dtype));
  FfnGemmArgs g = gateup_args(w, batch, static_cast<const char*>(compact), grp, nullptr,
                              static_cast<char*>(act), grp, kept_offsets + batch->B, n0);
  set_split(g, ws, L, 0);
  CE_TRY(launch_ffn_gateup(g, w->dtype == CE_BF16, s));
  return CE_OK;
}

int ce_ffn_down(const ce_batch* batch, const void* act, const int32_t* kept_idx,
                const int32_t* kept_offsets, const ce_ffn_w* w, void* ffn_out, void* ws,
                size_t ws_bytes, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t *grp, *n0;
  CE_CHECK(ffn_prologue(batch, act, kept_idx, kept_offsets, w, ffn_out, ws, ws_bytes, s, &grp, &n0));
  if (batch->kept_capacity == 0) return CE_OK;
  const WsLayout L = ws_layout(CE_WS_FFN, batch->B, batch->T, batch->kept_capacity, w->d, w->d_ff,
                               elem_size(w->dtype));
  FfnGemmArgs dn = down_args(w, batch, static_cast<const char*>(act), grp,
                             static_cast<char*>(ffn_out), grp, nullptr, nullptr,
                             kept_offsets + batch->B, n0);
  set_split(dn, ws, L, 1);
  CE_TRY(launch_ffn_down(dn, w->dtype == CE_BF16, s));
  return CE_OK;
}

int ce_routed_ffn(const ce_batch* batch, const void* compact, const int32_t* kept_idx,
                  const int32_t* kept_offsets, const ce_ffn_w* w, void* ffn_out, void* ws,
                  size_t ws_bytes, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t *grp, *n0;
  CE_CHECK(ffn_prologue(batch, compact, kept_idx, kept_offsets, w, ffn_out, ws, ws_bytes, s, &grp,
                        &n0));
  if (batch->kept_capacity == 0) return CE_OK;
  const WsLayout L = ws_layout(CE_WS_FFN, batch->B, batch->T, batch->kept_capacity, w->d, w->d_ff,
                               elem_size(w->dtype));
  const bool bf16 = w->dtype == CE_BF16;
  const int32_t* kt = kept_offsets + batch->B;
  // activations stay in grouped GEMM order inside the workspace
  char* act = at<char>(ws, L.act);
  FfnGemmArgs dn = down_args(w, batch, act, nullptr, static_cast<char*>(ffn_out), grp, nullptr,
                             nullptr, kt, n0);
  set_split(dn, ws, L, 1);
  FfnGemmArgs g = gateup_args(w, batch, static_cast<const char*>(compact), grp, nullptr, act,
                              nullptr, kt, n0);
  set_split(g, ws, L, 0);
  g.clear_n = ffn_split_counters(dn, 1, bf16);
  g.clear_cnt = g.clear_n > 0 ? dn.tile_cnt : nullptr;
  CE_TRY(launch_ffn_gateup(g, bf16, s));
  CE_TRY(launch_ffn_down(dn, bf16, s, g.clear_cnt != nullptr));
  return CE_OK;
}

int ce_routed_ffn_pruned(const ce_batch* batch, const void* compact, const int32_t* kept_idx,
                         const int32_t* kept_offsets, const ce_ffn_w* w, const float* norms, int32_t n_keep,
                         float delta, void* ffn_out, float* saliency, float* leakage, uint8_t* use_pruned,
                         void* ws, size_t ws_bytes, void* stream) {
  CE_CHECK(check_batch(batch, false));
  CE_CHECK(check_ffn(w));
  if (!kept_offsets || !norms || !saliency || !leakage || !use_pruned) return CE_ERR_INVALID_ARG;
  if (batch->kept_capacity > 0 && (!compact || !kept_idx || !ffn_out)) return CE_ERR_INVALID_ARG;
  if (!isfinite(delta)) return CE_ERR_INVALID_ARG;
  if (w->dtype != CE_BF16) return CE_ERR_UNSUPPORTED;
  if (n_keep < 0 || n_keep > w->d_ff || (n_keep % 64) != 0) return CE_ERR_UNSUPPORTED;
  const WsLayout L = ws_layout(CE_WS_FFN_PRUNED, batch->B, batch->T, batch->kept_capacity, w->d, w->d_ff, 2);
  CE_CHECK(check_ws(ws, ws_bytes, L.total));
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int32_t* kt = kept_offsets + batch->B;
  int32_t* grp = w->n_sets == 2 ? at<int32_t>(ws, L.grp_rows) : nullptr;
  int32_t* n0 = w->n_sets == 2 ? at<int32_t>(ws, L.grp_n0) : nullptr;
  char* act = at<char>(ws, L.act);
  int32_t* row_seq = at<int32_t>(ws, L.row_seq);
  FfnGemmArgs g = gateup_args(w, batch, static_cast<const char*>(compact), grp, nullptr, act, nullptr, kt, n0);
  set_split(g, ws, L, 0);
  g.row_seq = row_seq;
  g.sal_part = at<float>(ws, L.sal_seg);
  g.sal_meta = at<int32_t>(ws, L.sal_meta);
  FfnGemmArgs dn = down_args(w, batch, act, nullptr, static_cast<char*>(ffn_out), grp, nullptr, nullptr, kt, n0);
  set_split(dn, ws, L, 1);
  uint8_t* row_flag = at<uint8_t>(ws, L.row_flag);
  dn.row_flag = row_flag;
  dn.ns_keep = n_keep * 2 / 128;
  if (batch->kept_capacity > 0 && !ffn_pruned_ok(g, dn)) return CE_ERR_UNSUPPORTED;
  float* chunk_tot = at<float>(ws, L.sal_part) + (size_t)kSalSplits * batch->B * w->d_ff;
  int32_t* seq_cnt = at<int32_t>(ws, L.seq_cnt);
  CE_TRY(launch_row_seq(kept_offsets, batch->B, batch->kept_capacity, row_seq, seq_cnt, s));
  if (batch->kept_capacity == 0) {
    // no rows: zero saliency, leakage 0 (the pruned FFN runs, on nothing)
    return hip_status(launch_saliency_segments(g, kept_offsets, norms, batch->B, n_keep, delta, chunk_tot,
                                               saliency, leakage, use_pruned, row_flag, seq_cnt, s));
  }
  if (w->n_sets == 2)
    CE_TRY(launch_group(kept_idx, kept_offsets, batch->B, batch->kept_capacity, batch->T, batch->flags, grp, n0,
                        s));
  g.clear_n = ffn_split_counters(dn, 1, true);
  g.clear_cnt = g.clear_n > 0 ? dn.tile_cnt : nullptr;
  // 1. gate/up + SwiGLU, with the per-segment |z| sums
  CE_TRY(launch_ffn_gateup(g, true, s));
  // 2. saliency (Eq. 8), leakage (Eq. 9) and the pruned/full choice per sequence
  CE_TRY(launch_saliency_segments(g, kept_offsets, norms, batch->B, n_keep, delta, chunk_tot, saliency, leakage,
                                  use_pruned, row_flag, seq_cnt, s));
  // 3. down, skipping the channels of P on the rows that run pruned
  CE_TRY(launch_ffn_down_pruned(dn, s, g.clear_cnt != nullptr));
  return CE_OK;
}

int ce_scatter_residual(const ce_batch* batch, const void* ffn_out, const int32_t* kept_idx,
                        const int32_t* kept_offsets, int dtype, int32_t d, const void* hidden_in,
                        void* hidden_out, void* stream) {
  CE_CHECK(check_batch(batch, false));
  CE_CHECK(check_dtype_d(dtype, d));
  if (!kept_offsets) return CE_ERR_INVALID_ARG;
  if (batch->T > 0 && (!hidden_in || !hidden_out)) return CE_ERR_INVALID_ARG;
  if (batch->kept_capacity > 0 && (!ffn_out || !kept_idx)) return CE_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int elem = elem_size(dtype);
  if (hidden_in != hidden_out)
    CE_TRY(launch_copy_rows(static_cast<const char*>(hidden_in), static_cast<char*>(hidden_out),
                            (int64_t)d * elem, batch->T, nullptr, s));
  CE_TRY(launch_scatter(static_cast<const char*>(ffn_out), kept_idx, kept_offsets, batch->B,
                        batch->kept_capacity, batch->T, d, dtype == CE_BF16,
                        static_cast<const char*>(hidden_in), static_cast<char*>(hidden_out), s));
  return CE_OK;
}

int ce_routed_block(const ce_batch* batch, const void* hidden_in, void* hidden_out,
                    const ce_scorer_w* scorer, const ce_ffn_w* ffn, float* logits_out,
                    int32_t* kept_idx_out, int32_t* kept_offsets_out, void* ws, size_t ws_bytes,
                    void* stream) {
  return routed_block_impl(batch, hidden_in, hidden_out, scorer, ffn, logits_out, kept_idx_out, kept_offsets_out,
                           nullptr, ws, ws_bytes, stream);
}

int ce_routed_block_gap(const ce_batch* batch, const void* hidden_in, void* hidden_out,
                        const ce_scorer_w* scorer, const ce_ffn_w* ffn, float* logits_out,
                        int32_t* kept_idx_out, int32_t* kept_offsets_out, float delta, float* cos,
                        float* rho_all, float* rho_ret, float* gap, uint8_t* skip, void* ws,
                        size_t ws_bytes, void* stream) {
  if (!rho_all || !rho_ret || !gap) return CE_ERR_INVALID_ARG;
  if (!isfinite(delta)) return CE_ERR_INVALID_ARG;
  if (batch && batch->T > 0 && !cos) return CE_ERR_INVALID_ARG;
  const GapOut go{delta, cos, rho_all, rho_ret, gap, skip};
  return routed_block_impl(batch, hidden_in, hidden_out, scorer, ffn, logits_out, kept_idx_out, kept_offsets_out,
                           &go, ws, ws_bytes, stream);
}

int ce_score_tiling(const ce_batch* batch, const ce_scorer_w* scorer, int32_t* tile_out) {
  if (!batch || batch->B < 1 || batch->T < 0) return CE_ERR_INVALID_ARG;
  CE_CHECK(check_scorer(scorer));
  int tm = 0, tn = 0, n_ct = 0, n_rt = 0;
  const int elem = elem_size(scorer->dtype);
  const int tiled = score_tiling(batch->B, batch->T, scorer->d, scorer->r_core, scorer->r_exp, elem, &tm, &tn,
                                 &n_ct, &n_rt);
  if (tile_out) {
    tile_out[0] = tiled ? tm : score_token_tile(batch->B, batch->T, scorer->d, scorer->r_core, scorer->r_exp, elem);
    tile_out[1] = tiled ? tn : 0;
  }
  return tiled;
}

int ce_drop_stability(const ce_batch* batch, const int32_t* token_pos_t,
                      const int32_t* token_pos_ref, float* jaccard, float* j_rand, float* rda,
                      void* stream) {
  CE_CHECK(check_batch(batch, false));
  if (!jaccard) return CE_ERR_INVALID_ARG;
  if (batch->T > 0 && (!token_pos_t || !token_pos_ref)) return CE_ERR_INVALID_ARG;
  return hip_status(launch_stability(batch->seq_offsets, batch->flags, batch->B, batch->T, token_pos_t,
                                     token_pos_ref, jaccard, j_rand, rda,
                                     static_cast<hipStream_t>(stream)));
}

int ce_ffn_down_colnorms(const ce_ffn_w* w, float* norms, void* stream) {
  CE_CHECK(check_ffn(w));
  if (!norms) return CE_ERR_INVALID_ARG;
  return hip_status(launch_colnorms(static_cast<const char*>(w->w_down[0]),
                                    static_cast<const char*>(w->n_sets == 2 ? w->w_down[1] : w->w_down[0]),
                                    w->n_sets, w->d, w->d_ff, w->dtype == CE_BF16, norms,
                                    static_cast<hipStream_t>(stream)));
}

int ce_ffn_saliency(const ce_batch* batch, const void* act, const int32_t* kept_idx,
                    const int32_t* kept_offsets, const ce_ffn_w* w, const float* norms,
                    const uint8_t* prune_mask, float delta, float* saliency, float* leakage,
                    uint8_t* use_pruned, void* ws, size_t ws_bytes, void* stream) {
  CE_CHECK(check_batch(batch, false));
  CE_CHECK(check_ffn(w));
  if (!kept_offsets || !norms || !prune_mask || !saliency || !leakage) return CE_ERR_INVALID_ARG;
  if (!isfinite(delta)) return CE_ERR_INVALID_ARG;
  if (batch->kept_capacity > 0 && (!act || !kept_idx)) return CE_ERR_INVALID_ARG;
  const WsLayout L = ws_layout(CE_WS_FFN, batch->B, batch->T, batch->kept_capacity, w->d, w->d_ff,
                               elem_size(w->dtype));
  CE_CHECK(check_ws(ws, ws_bytes, L.total));
  return hip_status(launch_saliency(static_cast<const char*>(act), kept_idx, kept_offsets, batch->flags,
                                    norms, batch->B, batch->T, batch->kept_capacity, w->d_ff, w->n_sets,
                                    w->dtype == CE_BF16, prune_mask, delta, at<float>(ws, L.sal_part),
                                    saliency, leakage, use_pruned, static_cast<hipStream_t>(stream)));
}

int ce_ffn_mask_channels(const ce_batch* batch, void* act, const int32_t* kept_offsets, int dtype,
                         int32_t d_ff, const uint8_t* prune_mask, const uint8_t* use_pruned,
                         void* stream) {
  CE_CHECK(check_batch(batch, false));
  if (dtype != CE_F32 && dtype != CE_BF16) return CE_ERR_UNSUPPORTED;
  if (d_ff <= 0 || (d_ff % 64) != 0) return CE_ERR_UNSUPPORTED;
  if (!kept_offsets || !prune_mask || !use_pruned) return CE_ERR_INVALID_ARG;
  if (batch->kept_capacity > 0 && !act) return CE_ERR_INVALID_ARG;
  return hip_status(launch_mask_channels(static_cast<char*>(act), kept_offsets, batch->B,
                                         batch->kept_capacity, d_ff, dtype == CE_BF16, prune_mask, use_pruned,
                                         static_cast<hipStream_t>(stream)));
}

int ce_layer_gap(const ce_batch* batch, const void* x_in, const void* x_out, int dtype, int32_t d,
                 const int32_t* token_pos, float delta, float* cos, float* rho_all, float* rho_ret,
                 float* gap, uint8_t* skip, void* stream) {
  CE_CHECK(check_batch(batch, false));
  CE_CHECK(check_dtype_d(dtype, d));
  if (!rho_all || !rho_ret || !gap) return CE_ERR_INVALID_ARG;
  if (!isfinite(delta)) return CE_ERR_INVALID_ARG;
  if (batch->T > 0 && (!x_in || !x_out || !token_pos || !cos)) return CE_ERR_INVALID_ARG;
  return hip_status(launch_layer_gap(static_cast<const char*>(x_in), static_cast<const char*>(x_out),
                                     batch->seq_offsets, batch->B, batch->T, d, dtype == CE_BF16, token_pos,
                                     delta, cos, rho_all, rho_ret, gap, skip, static_cast<hipStream_t>(stream)));
}

int ce_routed_attention(const ce_attn* at, const void* q, const void* k, const void* v, void* o, void* stream) {
  if (!at) return CE_ERR_INVALID_ARG;
  if (at->B < 1 || at->n_heads < 1 || at->n_kv_heads < 1 || at->q_capacity < 0 || at->kv_capacity < 0)
    return CE_ERR_INVALID_ARG;
  if (at->n_heads % at->n_kv_heads != 0) return CE_ERR_INVALID_ARG;
  if (at->causal != 0 && at->causal != 1) return CE_ERR_INVALID_ARG;
  if (!isfinite(at->scale) || !(at->scale > 0.0f)) return CE_ERR_INVALID_ARG;
  if (!at->q_offsets || !at->kv_offsets) return CE_ERR_INVALID_ARG;
  if (at->dtype != CE_BF16 || at->head_dim != 128) return CE_ERR_UNSUPPORTED;
  const int64_t lim = (int64_t)1 << 31;
  if ((int64_t)at->q_capacity * at->n_heads * 256 >= lim || (int64_t)at->kv_capacity * at->n_kv_heads * 256 >= lim)
    return CE_ERR_UNSUPPORTED;
  if (at->q_capacity > 0 && (!q || !o)) return CE_ERR_INVALID_ARG;
  if (at->q_capacity > 0 && at->kv_capacity > 0 && (!k || !v)) return CE_ERR_INVALID_ARG;
  return hip_status(launch_attention(static_cast<const char*>(q), static_cast<const char*>(k),
                                     static_cast<const char*>(v), static_cast<char*>(o), at->q_offsets,
                                     at->kv_offsets, at->B, at->n_heads, at->n_kv_heads, at->q_capacity,
                                     at->kv_capacity, at->causal != 0, at->scale, static_cast<hipStream_t>(stream)));
}

}  // extern "C"

// ---------------------------------------------------------------------------
// TopK and packing without a workspace, for callers that cannot allocate
// (code under HIP graph capture, serving loops that forbid hipMalloc). The
// summaries and the status word live in a fixed array in device memory instead
// of the caller's workspace; every call on a GPU shares that GPU's copy, so
// calls that overlap on one GPU race.
// ---------------------------------------------------------------------------
#include <atomic>
#include <mutex>

namespace {

// Layout of `scratch`: the status word (padded to 256 bytes), then the
// per-sequence summaries, 3 int32 per sequence, for at most CE_NOALLOC_MAX_B
// sequences: 786,688 bytes per GPU, held until the process ends.
constexpr size_t kScratchStatusBytes = 256;
constexpr size_t kScratchBytes = kScratchStatusBytes + (size_t)3 * CE_NOALLOC_MAX_B * sizeof(int32_t);
static __device__ __align__(256) char scratch[kScratchBytes];

// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is looked up once per device (with that device current) and
// only that address is passed to kernels.
constexpr int kMaxDevices = 64;
std::atomic<char*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

int scratch_of_current_device(char** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return CE_ERR_HIP;
  char* p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
      void* addr = nullptr;
      if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || !addr) return CE_ERR_HIP;
      p = static_cast<char*>(addr);
      g_scratch[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return CE_OK;
}

}  // namespace

extern "C" int ce_topk_compact_noalloc(const ce_batch* batch, const float* logits, const void* hidden,
                                       int dtype, int32_t d, int32_t* kept_idx, int32_t* kept_offsets,
                                       int32_t* token_pos, void* compact, uint32_t* status, void* stream) {
  CE_CHECK(topk_args_ok(batch, logits, hidden, dtype, d, kept_idx, kept_offsets, compact));
  if (batch->B > CE_NOALLOC_MAX_B) return CE_ERR_UNSUPPORTED;
  char* sc = nullptr;
  CE_CHECK(scratch_of_current_device(&sc));
  // the summaries are written in full by the first launch and the status
  // word by the second, so nothing left by an earlier call is read
  uint32_t* st = status ? status : reinterpret_cast<uint32_t*>(sc);
  return topk_launch(batch, logits, hidden, dtype, d, kept_idx, kept_offsets, token_pos, compact,
                     reinterpret_cast<int32_t*>(sc + kScratchStatusBytes), st, static_cast<hipStream_t>(stream));
}
