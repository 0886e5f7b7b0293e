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
  size_t tile_start; // int32 [B + 1] first token tile of each sequence (single-launch scorer, B > 1024)
  size_t kept_off;   // int32 [B + 1]  (block path, when the caller passes none)
  size_t kept_idx;   // int32 [cap]    (block path)
  size_t token_pos;  // int32 [T]      (block path)
  size_t logits;     // float [T]      (block path)
  size_t score_part; // float [kScoreMaxTiles x T] rank-tiled scorer partial logits (block path)
  size_t grp_rows;   // int32 [cap]    (MoT grouping)
  size_t grp_n0;     // int32          (MoT group size)
  size_t act;        // dtype [cap * d_ff] SwiGLU activations
  size_t gemm_part;  // float [slots x 256 x 256] K-piece partial sums of the FFN GEMMs' tail tiles
  size_t gu_cnt;     // int32 [kSplitMaxSlots] arrival counters of the gate/up tail tiles
  size_t dn_cnt;     // int32 [kSplitMaxSlots] arrival counters of the down tail tiles
  size_t gap_part;   // double [cap x ceil(d / 32) x 4] layer-gap partial sums (CE_WS_BLOCK_GAP)
  size_t row_seq;    // int32 [cap] sequence of each packed row (CE_WS_FFN_PRUNED)
  size_t sal_seg;    // float [tiles x kSalSegs x d_ff] per-segment |z| sums (CE_WS_FFN_PRUNED)
  size_t sal_meta;   // int32 [tiles x (kSalSegs + 1)] segment counts and sequences (CE_WS_FFN_PRUNED)
  size_t row_flag;   // uint8 [cap] 1 where the packed row's sequence runs pruned (CE_WS_FFN_PRUNED)
  size_t seq_cnt;    // int32 [B] arrival counters of the saliency kernel (CE_WS_FFN_PRUNED)
  size_t sal_part;   // float [kSalSplits x B x d_ff] FFN-saliency partial sums, then
                     // float [B x ceil(d_ff / 256) x 2] per-chunk totals
  size_t total;
};

WsLayout ws_layout(int which, int B, int T, int cap, int d, int d_ff, int elem);

// Work split of one 256 x 256-tile FFN GEMM launch (the ping-pong kernel) over
// the chip's 8 XCDs of 32 CUs, one workgroup per CU at a time. Work item w
// (a tile) runs on XCD w / per_x. On each XCD the first whole_x items run as
// whole tiles, in full rounds of 32; the remaining tail_x items (the last,
// partial round) run as `pieces` workgroups each, over equal ranges of the
// K superslabs, whose fp32 partial sums meet through the workspace: the last
// piece to arrive adds them up in piece order and runs the epilogue.
// pieces == 1: no split (whole_x = per_x, tail_x = 0).
constexpr int kXcdCount = 8;
constexpr int kCusPerXcd = 32;
constexpr int kSplitMaxSlots = kXcdCount * kCusPerXcd;  // partial-sum tiles: 256 x 256 KB = 64 MB
struct GemmSplit {
  int per_x;    // items per XCD (the last XCD may have fewer)
  int whole_x;  // whole items per XCD
  int tail_x;   // split items per XCD
  int pieces;   // workgroups per split item
  int absorb;   // gate/up, whole tiles only: a last token tile of at most 32
                // rows joins the tile before it (see gateup_token_tiles)
};
// Chosen by a cost model in units of one superslab's K-loop time: a whole
// tile costs ns + 3.5 (prologue, epilogue); a piece ns / S + 2 (its partial
// sums written) + the last arriver's reads (2.5 per partial tile read: one for
// S = 2, whose two addends commute; all S otherwise, summed in piece order).
// Splits only when that beats running the tail as whole tiles, after at most
// two full rounds; S * tail_x <= 32 and at least 3 superslabs per piece.
GemmSplit gemm_split(int64_t items, int ns);
// Item and superslab counts of the gate/up (mode 0: 128 output features per
// tile) and down (mode 1: 256) launches over kept_capacity rows, or 0 items
// when the ping-pong kernel does not apply (fp32, K not in whole 128-byte
// superslabs, fewer than 3 of them, or 32-bit offsets overflowing).
void gemm_items(int mode, int cap, int d, int d_ff, int n_sets, int elem, int64_t* items, int* ns);

// Sequences per batch: some grids put the sequence index in their y dimension.
constexpr int kMaxBatch = 65535;
// The FFN-saliency reduction splits each sequence's rows over at most this
// many workgroups (partial sums in the workspace, summed in a fixed order).
constexpr int kSalSplits = 16;
// The pruned FFN's gate/up epilogue keeps |z| sums for at most this many
// segments (runs of rows of one sequence) per 256-row token tile.
constexpr int kSalSegs = 8;

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
