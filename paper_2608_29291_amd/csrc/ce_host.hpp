// Host-only logic of the C ABI: argument validation, workspace layout and the
// exact keep-count rule. No HIP calls here, so this part also builds and runs
// on a machine without a GPU.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "ce_router.h"

namespace ce {

constexpr size_t kWsAlign = 256;
constexpr int kMaxRanks = 512;
constexpr int kMaxSeg = 16;

// Byte offsets of each workspace region (0 = region absent for that kind).
struct WsLayout {
  size_t status;     // uint32 status word (+ padding)
  size_t seq_info;   // int32 [3 * B]
  size_t kept_off;   // int32 [B + 1]  (block path, when the caller passes none)
  size_t kept_idx;   // int32 [cap]    (block path)
  size_t token_pos;  // int32 [T]      (block path)
  size_t logits;     // float [T]      (block path)
  size_t score_part; // float [kScoreMaxTiles x T] rank-tiled scorer partial logits (block path)
  size_t grp_rows;   // int32 [cap]    (MoT grouping)
  size_t grp_n0;     // int32          (MoT group size)
  size_t act;        // dtype [cap * d_ff] SwiGLU activations
  size_t down_part;  // float [2 x tiles x 256 x 256] split-K partial sums of the down GEMM
  size_t down_cnt;   // int32 [tiles] arrival counters of the split-K down GEMM
  size_t sal_part;   // float [kSalSplits x B x d_ff] FFN-saliency partial sums, then
                     // float [B x ceil(d_ff / 256) x 2] per-chunk totals
  size_t total;
};

WsLayout ws_layout(int which, int B, int T, int cap, int d, int d_ff, int elem);

// The down GEMM (d outputs, contraction d_ff) runs as two K halves when its
// 256 x 256 tiles fill the chip's rounds of 256 workgroups so unevenly that
// twice the workgroups, each with half of K plus the partial-sum exchange,
// finish sooner (a cost model); returns that tile count, or 0 when the down
// GEMM is not split. Shared by the launcher and the workspace layout so both
// agree. At most kSplitMaxTiles tiles (512 MB of partial sums).
constexpr int kSplitMaxTiles = 1024;
// The FFN-saliency reduction splits each sequence's rows over at most this
// many workgroups (partial sums in the workspace, summed in a fixed order).
constexpr int kSalSplits = 16;
int down_split_tiles(int cap, int d, int d_ff, int n_sets, int elem);

// Token tile of the single-launch scorer: 32, or (bf16, r_core + r_exp <=
// 384) 128 when that takes fewer rounds of 256 workgroups x rows of K each
// workgroup streams (tile tokens + every rank; the expansion ranks counted
// whenever r_exp > 0). 128-token tiles move the W1 rows once per 128 tokens
// instead of once per 32.
int score_token_tile(int B, int T, int d, int r_core, int r_exp, int elem);

// The fused block's rank-tiled scorer (bf16): tiles of tm tokens x tn ranks,
// tm, tn in {64, 128}, with n_ct core and n_rt - n_ct expansion rank tiles,
// writing partial logits that the TopK step assembles. Chosen (returns 1)
// when it takes fewer rounds of 256 workgroups x rows of K per workgroup than
// the single-launch scorer with score_token_tile's tile (weighted 1.5x when
// only two of its slabs fit in LDS), counting every token as scored, both
// with the expansion ranks active and without them.
constexpr int kScoreMaxTiles = 10;  // ceil(r_core / 64) + ceil(r_exp / 64) with r_core + r_exp <= 512
int score_tiling(int B, int T, int d, int r_core, int r_exp, int elem, int* tm, int* tn, int* n_ct, int* n_rt);

int elem_size(int dtype);  // 2 for bf16, 4 for f32, 0 if unknown

int32_t num_keep_host(float keep, int32_t n);

// Validation: each returns CE_OK or a negative status.
int check_batch(const ce_batch* b, bool need_t);
int check_dtype_d(int dtype, int32_t d);
int check_scorer(const ce_scorer_w* w);
int check_ffn(const ce_ffn_w* w);
int check_ws(const void* ws, size_t ws_bytes, size_t need);

}  // namespace ce
