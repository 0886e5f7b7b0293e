// Internal launcher interface between the C-ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ce_host.hpp"

namespace ce {

// One "weights x tokens" FFN GEMM (see ce_ffn.hip).
struct FfnGemmArgs {
  // weights: rows = output features, K-contiguous; per set.
  //   gate/up mode: w0 = W_gate, w1 = W_up; down mode: w0 = W_down.
  const char* w0[2];
  const char* w1[2];
  int64_t w_ld;     // bytes per weight row
  int n_feat;       // output features (d_ff or d)
  int k_bytes;      // bytes of the contraction per row (multiple of 128)
  // tokens: GEMM row j reads row map2[map1[j]] of `tok`
  const char* tok;
  int64_t tok_ld;
  int64_t tok_rows;  // rows of `tok` (bounds the 32-bit offsets of the large-tile kernel)
  const int32_t* map1;
  const int32_t* map2;
  // output: row omap2[omap1[j]] of `out` (each level skipped when NULL)
  char* out;
  int64_t out_ld;
  const int32_t* omap1;
  const int32_t* omap2;
  const char* res;  // down only: residual rows (same row map as out), or NULL
  int64_t res_ld;
  // sizes on the device
  const int32_t* kt_ptr;  // number of packed rows (clamped to cap)
  int cap;
  const int32_t* n0_ptr;  // rows in the first weight set (MoT), or NULL
  int n_sets;
  // tail tiles split over K (see GemmSplit): fp32 partial sums [slots x 256 x
  // 256] and this launch's arrival counters, zero on entry (both NULL: no split)
  float* part;
  int32_t* tile_cnt;
  // the following GEMM launch's arrival counters, cleared by the first
  // workgroup (NULL: none), so that launch needs no fill kernel
  int32_t* clear_cnt;
  int clear_n;
  // down only: per-row partial sums of the layer-skipping gap (NULL: none).
  // For packed row p the epilogue of each wave writes, at slot q = (first
  // feature of the wave) / (features per wave), the fp64 sums over its
  // features of in*out, in*in and out*out (in = residual, out = the stored
  // output): gap_part[(p * gap_np + q) * 4 + {0, 1, 2}]
  double* gap_part;
  int gap_np;
  // FFN pruning (ce_routed_ffn_pruned). row_seq[p]: sequence of packed row p.
  // gate/up: per token tile tt, the epilogue sums |z| over each run of rows of
  // one sequence (a segment, at most kSalSegs per tile) into
  // sal_part[(tt * kSalSegs + k) * d_ff + c]; sal_meta[tt * (kSalSegs + 1)] =
  // the tile's segment count (more than kSalSegs: no partials), then each
  // segment's sequence (NULL: none).
  // down: packed rows p with row_flag[p] != 0 (their sequence runs pruned)
  // read zeros from K superslab ns_keep on (the channels of P, the tail); a
  // whole tile whose rows all run pruned stops its K loop there (NULL: no
  // pruning).
  const int32_t* row_seq;
  float* sal_part;
  int32_t* sal_meta;
  const uint8_t* row_flag;
  int ns_keep;
};

// counters_clear: this launch's arrival counters (tile_cnt) were already
// cleared on this stream (by the previous kernel through clear_cnt); else a
// fill kernel clears them first when the launch splits.
hipError_t launch_ffn_gateup(const FfnGemmArgs& a, bool bf16, hipStream_t stream, bool counters_clear = false);
hipError_t launch_ffn_down(const FfnGemmArgs& a, bool bf16, hipStream_t stream, bool counters_clear = false);
// Number of arrival counters a GEMM launch with these arguments uses (0: no
// split); mode 0 = gate/up, 1 = down.
int ffn_split_counters(const FfnGemmArgs& a, int mode, bool bf16);
// Down GEMM of the pruned FFN: always the ping-pong kernel (the pruning
// logic lives there); the caller checks ffn_pruned_ok first.
hipError_t launch_ffn_down_pruned(const FfnGemmArgs& a, hipStream_t stream, bool counters_clear);
bool ffn_pruned_ok(const FfnGemmArgs& gateup, const FfnGemmArgs& down);

// Pruned FFN: row_seq[p] = b for the packed rows p of each sequence b.
// Also zeroes seq_cnt [B] (the saliency kernel's arrival counters).
hipError_t launch_row_seq(const int32_t* kept_offsets, int B, int cap, int32_t* row_seq, int32_t* seq_cnt,
                          hipStream_t stream);
// Saliency (Eq. 8) of each sequence from the gate/up epilogue's segment sums
// (falling back to act for tiles with more than kSalSegs segments) and the
// leakage (Eq. 9) of the tail channels [n_keep, d_ff); use_pruned = leakage <= delta,
// also written to row_flag for every packed row of the sequence. One launch:
// the last workgroup of each sequence (seq_cnt, zeroed by launch_row_seq)
// forms its leakage.
hipError_t launch_saliency_segments(const FfnGemmArgs& gateup, const int32_t* kept_offsets, const float* norms,
                                    int B, int n_keep, float delta, float* chunk_tot, float* saliency, float* lambda,
                                    uint8_t* use_pruned, uint8_t* row_flag, int32_t* seq_cnt, hipStream_t stream);

// Gap partial-sum slots per row (gap_np) of the down kernel that
// launch_ffn_down picks for these arguments: ceil(d / features per wave).
int ffn_down_gap_slots(const FfnGemmArgs& a, bool bf16);

struct ScoreArgs {
  const char* hidden;
  int64_t h_ld;        // bytes per hidden row
  int k_bytes;         // d * elem
  int B, T;
  const int32_t* seq_offsets;
  const uint8_t* flags;
  const float* t;
  const char* w1c;     // [r_core x d]
  const float* b1c;
  const float* w2c;
  float b2c;
  const char* w1e;     // [n_seg x r_exp x d]
  const float* b1e;
  const float* w2e;
  const float* b2e;
  int r_core, r_exp, n_seg;
  float* logits;
  float* probs;
  int32_t* info;  // if set, B extra workgroups also write the per-sequence summary (seq_info layout)
  // rank-tiled scorer only: per-token partial logits [n_rt x T], rank tiles
  // 0 .. n_ct - 1 over the core ranks, the rest over the expansion ranks
  float* part;
  int n_ct, n_rt;
  // single-launch scorer: room for the first token tile of each sequence
  // [B + 1] (or NULL); above 1024 sequences launch_score fills it first and
  // each workgroup looks its tile up there instead of walking the sequences
  int32_t* tile_start;
};
hipError_t launch_score(const ScoreArgs& a, bool bf16, hipStream_t stream);
// Rank-tiled scorer (bf16): tiles of tm tokens x tn ranks (tm, tn in {64, 128})
// write per-token partial logits to a.part; the TopK step adds them up.
hipError_t launch_score_tiles(const ScoreArgs& a, int tm, int tn, hipStream_t stream);
// Logits (and probs) from a.part in the TopK step's order (the staged
// rank-tiled path).
hipError_t launch_score_assemble(const ScoreArgs& a, hipStream_t stream);

// Per-sequence summary written by the count kernel: {lo, len, keep_count | bad<<31}.
hipError_t launch_seq_info(const int32_t* seq_offsets, const uint8_t* flags, int B, int T,
                           int32_t* info, hipStream_t stream);

struct SelectArgs {
  const float* logits;
  // When part is set, the logits are first assembled from the rank-tiled
  // scorer's partial sums [n_rt x T] (fixed order: core tiles, b2c, then for
  // generation tokens the expansion tiles and b2e[m]) and written to logits_w.
  const float* part;
  float* logits_w;
  int n_ct, n_rt, T, r_exp, n_seg;
  float b2c;
  const float* b2e;
  const float* t;
  const uint8_t* flags;
  const int32_t* info;
  int B;
  float keep;
  int cap;
  int32_t* kept_idx;
  int32_t* kept_offsets;
  int32_t* token_pos;  // or NULL
  uint32_t* status;
  // counters of the following gate/up launch, cleared by workgroup 0 (or NULL)
  int32_t* clear_cnt;
  int clear_n;
  // set by launch_select: kept_offsets[b] and the status word were already
  // written by the sequence-offset scan (large batches)
  int offs_ready;
};
hipError_t launch_select(const SelectArgs& a, hipStream_t stream);

// MoT: stable partition of the packed rows by FFN set (GEN bit).
// Entries of kept_idx outside [0, T) count as weight set 0.
hipError_t launch_group(const int32_t* kept_idx, const int32_t* kept_offsets, int B, int cap,
                        int T, const uint8_t* flags, int32_t* grp_rows, int32_t* n0,
                        hipStream_t stream);

// compact[j] = hidden[kept_idx[j]] for j < Kt
hipError_t launch_gather(const char* hidden, int64_t row_bytes, const int32_t* kept_idx,
                         const int32_t* kept_offsets, int B, int cap, char* compact,
                         hipStream_t stream);

// out[kept_idx[j]] = in[kept_idx[j]] + ffn[j] for j < Kt (entries outside [0, T) skipped)
hipError_t launch_scatter(const char* ffn_out, const int32_t* kept_idx, const int32_t* kept_offsets,
                          int B, int cap, int T, int d, bool bf16, const char* h_in, char* h_out,
                          hipStream_t stream);

// out[i] = in[i] for every row (token_pos == NULL) or for rows with token_pos[i] < 0
hipError_t launch_copy_rows(const char* h_in, char* h_out, int64_t row_bytes, int T,
                            const int32_t* token_pos, hipStream_t stream);

// Drop-set Jaccard / random baseline / RDA per sequence (see ce_stability.hip).
hipError_t launch_stability(const int32_t* seq_offsets, const uint8_t* flags, int B, int T,
                            const int32_t* tp_t, const int32_t* tp_ref, float* jaccard, float* j_rand,
                            float* rda, hipStream_t stream);

// FFN-pruning signal: down-projection column norms, per-sequence saliency +
// leakage, channel masking (see ce_ucs_ffn.hip).
hipError_t launch_colnorms(const char* w0, const char* w1, int n_sets, int d, int d_ff, bool bf16,
                           float* norms, hipStream_t stream);
hipError_t launch_saliency(const char* act, const int32_t* kept_idx, const int32_t* kept_offsets,
                           const uint8_t* flags, const float* norms, int B, int T, int cap, int d_ff,
                           int n_sets, bool bf16, const uint8_t* mask, float delta, float* part,
                           float* saliency, float* lambda, uint8_t* use_pruned, hipStream_t stream);
hipError_t launch_mask_channels(char* act, const int32_t* kept_offsets, int B, int cap, int d_ff, bool bf16,
                                const uint8_t* mask, const uint8_t* use_pruned, hipStream_t stream);

// Layer gap of a routed block from the down GEMM's per-row partial sums:
// cos = 1 for dropped tokens (they bypass the layer), else from the slots of
// the token's packed row; then the per-sequence means, gap and skip.
// Packed rows at or past cap (an overflowing batch) get cos = NaN.
hipError_t launch_gap_from_parts(const double* gap_part, int gap_np, int cap, const int32_t* seq_offsets, int B,
                                 int T, const int32_t* token_pos, float delta, float* cos_tok, float* rho_all,
                                 float* rho_ret, float* gap, uint8_t* skip, hipStream_t stream);

hipError_t launch_layer_gap(const char* x_in, const char* x_out, const int32_t* seq_offsets, int B, int T, int d,
                            bool bf16, const int32_t* token_pos, float delta, float* cos_tok, float* rho_all,
                            float* rho_ret, float* gap, uint8_t* skip, hipStream_t stream);

hipError_t launch_attention(const char* q, const char* k, const char* v, char* o, const int32_t* q_offsets,
                            const int32_t* kv_offsets, int B, int H, int Hkv, int q_cap, int kv_cap, bool causal,
                            float scale, hipStream_t stream);

}  // namespace ce
