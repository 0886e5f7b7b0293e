/*
 * ce_router.h -- C ABI of the CE-Router routed-block library for MI355X (gfx950).
 *
 * One routed layer of a unified multimodal backbone, as defined in the paper
 * "Accelerating Unified Multimodal Models with Core-Expansion Routing and
 * Unified Computation Scheduling":
 *
 *   1. score     core + expansion routing logits per token       (section 3.2, Eq. 4)
 *   2. topk      per-sequence TopK of the logits -> retained set  (section 3.4, Eq. 6)
 *   3. compact   retained tokens packed into a shorter sequence   (section 3.4, after Eq. 6)
 *   4. ffn       SwiGLU FFN on the packed rows only              (section 3.4, after Eq. 6:
 *                the retained tokens form a shorter sequence for the layer's
 *                attention and FFN)
 *   5. scatter   residual merge; dropped tokens take the bypass   (section 3.4, after Eq. 6)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every pointer argument documented as "device" is GPU memory on the current
 *   HIP device, owned by the caller, contiguous, 16-byte aligned. "host"
 *   pointers are ordinary CPU memory, read before the call returns.
 * - The library allocates no memory and keeps no pointer after a call
 *   returns. All work is enqueued on `stream` (a hipStream_t; NULL = the
 *   default stream); calls return without waiting for it. There are no
 *   device-to-host copies and no synchronisation on the hot path.
 * - Arguments are validated on the host before anything is launched: a
 *   validation error (CE_ERR_INVALID_ARG, CE_ERR_UNSUPPORTED,
 *   CE_ERR_WORKSPACE) means nothing was enqueued. CE_ERR_HIP reports a failed
 *   launch; entry points with several launches may already have enqueued the
 *   earlier ones, so after CE_ERR_HIP the outputs and workspace are undefined.
 * - Values known only on the device (how many tokens each sequence keeps,
 *   the packed row count Kt, MoT group sizes) never leave the device. Grids
 *   are sized from host-known upper bounds (kept_capacity); surplus tiles
 *   exit early. If the device finds inconsistent data (bad seq_offsets,
 *   Kt > kept_capacity) it never reads or writes out of bounds; it records
 *   the problem in the workspace status word (ce_workspace_status).
 * - Element types: hidden states and the scorer/FFN weight matrices share
 *   one dtype (CE_F32 or CE_BF16); biases, second-layer scorer vectors,
 *   timesteps and logits are float32; indices are int32.
 * - Shape limits: d % 64 == 0, d_ff % 64 == 0, scorer ranks % 32 == 0 and
 *   r_core + r_exp <= 512, 1 <= n_seg <= 16, 1 <= B <= 65535 (more
 *   sequences: CE_ERR_UNSUPPORTED), 0 <= T < 2^31.
 * - Matrices are row-major in the nn.Linear layout [out_features x in_features].
 * - Functions are stateless; concurrent calls on different streams are safe
 *   as long as they use different workspaces and outputs.
 */
#ifndef CE_ROUTER_H
#define CE_ROUTER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
enum {
    CE_OK = 0,
    CE_ERR_INVALID_ARG = -1, /* null pointer, bad size, value out of range     */
    CE_ERR_UNSUPPORTED = -2, /* shape/dtype outside the supported limits      */
    CE_ERR_WORKSPACE = -3,   /* workspace pointer null or smaller than needed */
    CE_ERR_HIP = -4          /* a HIP runtime call failed (launch, query)     */
};

/* ---- element types ----------------------------------------------------- */
enum { CE_F32 = 0, CE_BF16 = 1 };

/* ---- per-token flags (uint8) ------------------------------------------- */
enum {
    CE_TOK_GEN = 1,  /* generation token: scored by core + expansion e_{m(t)}  */
                     /* (Eq. 4); in a two-set MoT FFN it uses weight set 1.   */
                     /* Clear: understanding token, core only, weight set 0.  */
    CE_TOK_KEEP = 2  /* always retained (text / structure token); not scored, */
                     /* not counted in K; its logit is reported as +inf.       */
};

/* ---- device status word bits (ce_workspace_status) ---------------------- */
enum {
    CE_DEV_BAD_OFFSETS = 1,  /* seq_offsets not non-decreasing within [0, T]   */
    CE_DEV_OVERFLOW = 2      /* total retained rows Kt exceeded kept_capacity  */
};

/* ---- workspace kinds ---------------------------------------------------- */
enum { CE_WS_TOPK = 0, CE_WS_FFN = 1, CE_WS_BLOCK = 2, CE_WS_BLOCK_GAP = 3, CE_WS_FFN_PRUNED = 4, CE_WS_SCORE = 5 };

/*
 * A ragged batch of B sequences packed back to back: sequence b owns tokens
 * [seq_offsets[b], seq_offsets[b+1]).
 *   seq_offsets   device int32 [B+1], seq_offsets[0] = 0, non-decreasing, last = T
 *   flags         device uint8 [T], CE_TOK_* bits; other bits ignored
 *   t             device float32 [B], denoising timestep of sequence b in [0, 1]
 *                 (read only for sequences holding generation tokens; values
 *                 outside [0, 1] are clamped to the first / last segment)
 *   keep          keep ratio r in [0, 1]: sequence b retains its KEEP tokens
 *                 plus k_b = ceil(keep * n_b) of its n_b routable tokens
 *                 (ce_num_keep), exactly, on the float32 value of keep
 *   kept_capacity host upper bound on Kt = sum_b (A_b + k_b) (A_b = KEEP count);
 *                 sizes kept_idx / compact / FFN buffers; T always suffices
 */
typedef struct ce_batch {
    int32_t B;
    int32_t T;
    const int32_t* seq_offsets;
    const uint8_t* flags;
    const float* t;
    float keep;
    int32_t kept_capacity;
} ce_batch;

/*
 * Router of one layer (section 3.2): one core scorer shared by both tasks and
 * every generation segment, plus n_seg generation expansion scorers, each a
 * token-wise two-layer MLP with a scalar output:
 *     s(h) = w2 . SiLU(W1 h + b1) + b2
 * Understanding tokens: l = c(h). Generation tokens: l = c(h) + e_{m(t)}(h),
 * with m(t) = min(floor(n_seg * t), n_seg - 1) (equal-width segments of t).
 *   w1_core  device dtype   [r_core x d]
 *   b1_core  device float32 [r_core] or NULL (zero)
 *   w2_core  device float32 [r_core]
 *   b2_core  host scalar
 *   w1_exp   device dtype   [n_seg x r_exp x d]   (may be NULL if r_exp == 0)
 *   b1_exp   device float32 [n_seg x r_exp] or NULL
 *   w2_exp   device float32 [n_seg x r_exp]
 *   b2_exp   device float32 [n_seg] or NULL
 */
typedef struct ce_scorer_w {
    int32_t d, r_core, r_exp, n_seg;
    int32_t dtype;
    const void* w1_core;
    const float* b1_core;
    const float* w2_core;
    float b2_core;
    const void* w1_exp;
    const float* b1_exp;
    const float* w2_exp;
    const float* b2_exp;
} ce_scorer_w;

/*
 * SwiGLU FFN weight sets: y = W_down (SiLU(W_gate x) * (W_up x)).
 * n_sets = 1, or 2 for a mixture-of-transformers block where each retained
 * token uses set (flags & CE_TOK_GEN).
 *   w_gate[s], w_up[s]  device dtype [d_ff x d]
 *   w_down[s]           device dtype [d x d_ff]
 */
typedef struct ce_ffn_w {
    int32_t d, d_ff, n_sets;
    int32_t dtype;
    const void* w_gate[2];
    const void* w_up[2];
    const void* w_down[2];
} ce_ffn_w;

/* Human-readable name of a status code (static string). */
const char* ce_status_string(int status);

/* Library version string, e.g. "ce_router 0.1.0 gfx950". */
const char* ce_version(void);

/*
 * k = ceil(keep * n) evaluated exactly on the float32 value of keep (section
 * 3.4 / appendix A.2 define r = K / N; the rounding is this library's
 * reading). Returns -1 if keep is outside [0, 1] or NaN, or n < 0.
 */
int32_t ce_num_keep(float keep, int32_t n_routable);

/*
 * Host helper: exact Kt = sum_b (A_b + ce_num_keep(keep, n_b - A_b)) from
 * host copies of seq_offsets [B+1] and flags [T]. Returns -1 on bad input.
 */
int64_t ce_kept_count_host(int32_t B, int32_t T, const int32_t* seq_offsets_host,
                           const uint8_t* flags_host, float keep);

/*
 * Workspace bytes needed by an entry point (which = CE_WS_*), for this batch
 * (B, T, kept_capacity), hidden size d, FFN width d_ff and dtype. The
 * workspace is caller-owned device memory, 256-byte aligned; its contents on
 * entry do not matter.
 */
size_t ce_workspace_size(int which, const ce_batch* batch, int32_t d, int32_t d_ff, int dtype);

/*
 * Read the device status word (CE_DEV_* bits) written into a workspace by
 * the last ce_topk_compact / ce_routed_block call that used it. Synchronises
 * `stream`. Debug / test helper, not for the hot path.
 */
int ce_workspace_status(const void* ws, uint32_t* status_out, void* stream);

/*
 * Step 1 -- routing logits (section 3.2, Eq. 4) and scores (Eq. 6).
 *   hidden  device dtype [T x d]
 *   logits  device float32 [T] out: Eq. 4 logit; +inf for KEEP tokens
 *   probs   device float32 [T] out or NULL: sigmoid(logit) (Eq. 6); 1 for KEEP
 * Deterministic: every logit is summed in a fixed order.
 * Errors: CE_ERR_INVALID_ARG for null pointers / sizes, CE_ERR_UNSUPPORTED
 * for shapes outside the limits, CE_ERR_HIP on a failed launch.
 */
int ce_score(const ce_batch* batch, const void* hidden, const ce_scorer_w* w,
             float* logits, float* probs, void* stream);

/*
 * Step 1 with a workspace (section 3.2, Eq. 4 and Eq. 6): the scorer
 * ce_routed_block uses. Where ce_score_tiling returns 1 (large bf16 batches
 * with many ranks) the rank-tiled kernel writes per-token partial sums into
 * the workspace and a second launch adds them in the fused block's TopK
 * order, so the logits equal that block's bit for bit; otherwise this is
 * ce_score. Arguments as ce_score;
 *   ws  device workspace of ce_workspace_size(CE_WS_SCORE, ...) bytes
 *       (d = the scorer's hidden size; d_ff is not read)
 * Errors as ce_score; CE_ERR_WORKSPACE for a missing or short workspace.
 */
int ce_score_ws(const ce_batch* batch, const void* hidden, const ce_scorer_w* w,
                float* logits, float* probs, void* ws, size_t ws_bytes, void* stream);

/*
 * Steps 2-3 -- per-sequence TopK and packing (section 3.4, Eq. 6).
 * Among the routable (non-KEEP) tokens of each sequence, the k_b tokens
 * first in the order (larger logit first; equal logits -> lower token index;
 * -0 == +0; NaN below -inf) are retained, together with every KEEP token.
 *   logits       device float32 [T] (values of KEEP tokens are ignored)
 *   hidden       device dtype [T x d], read only if compact != NULL
 *   kept_idx     device int32 [kept_capacity] out: retained token indices,
 *                ascending within each sequence, sequences in order
 *   kept_offsets device int32 [B+1] out: sequence b's retained tokens are
 *                kept_idx[kept_offsets[b] .. kept_offsets[b+1])
 *   token_pos    device int32 [T] out or NULL: position of each token in
 *                kept_idx, -1 for dropped tokens
 *   compact      device dtype [kept_capacity x d] out or NULL: row j = hidden[kept_idx[j]]
 *   ws           device workspace of ce_workspace_size(CE_WS_TOPK, ...) bytes
 */
int ce_topk_compact(const ce_batch* batch, const float* logits, const void* hidden,
                    int dtype, int32_t d, int32_t* kept_idx, int32_t* kept_offsets,
                    int32_t* token_pos, void* compact, void* ws, size_t ws_bytes,
                    void* stream);

/*
 * ce_topk_compact without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, serving loops or harnesses that forbid
 * hipMalloc). Same arguments and results as ce_topk_compact, except:
 *   - no ws / ws_bytes: the per-sequence summaries live in a fixed array of
 *     786,688 bytes in device memory that the library holds on each GPU it
 *     runs on until the process ends (looked up on the first call on a
 *     device); calls that overlap on one GPU share it and race;
 *   - status  device uint32 [1] out, or NULL: the status word (CE_DEV_* bits)
 *             that ce_topk_compact writes into its workspace;
 *   - at most CE_NOALLOC_MAX_B sequences: larger batches return
 *     CE_ERR_UNSUPPORTED before anything is enqueued.
 * Allocates nothing: no hipMalloc, no hipFree, no allocating library call.
 */
enum { CE_NOALLOC_MAX_B = 65536 };
int ce_topk_compact_noalloc(const ce_batch* batch, const float* logits, const void* hidden,
                            int dtype, int32_t d, int32_t* kept_idx, int32_t* kept_offsets,
                            int32_t* token_pos, void* compact, uint32_t* status, void* stream);

/*
 * Step 4 -- SwiGLU FFN on the packed rows (section 3.4, after Eq. 6: the
 * retained tokens are packed into a shorter sequence and only that sequence
 * runs through the layer's FFN; in a mixture-of-transformers backbone, section
 * 4.1, each retained token uses the FFN weight set of its task).
 *   compact      device dtype [kept_capacity x d]: packed rows (row j is token kept_idx[j])
 *   kept_idx     device int32 [kept_capacity] (needed for the MoT set choice)
 *   kept_offsets device int32 [B+1]: Kt = kept_offsets[B] rows are processed
 *   ffn_out      device dtype [kept_capacity x d] out: FFN(row j), no residual
 *   ws           device workspace of ce_workspace_size(CE_WS_FFN, ...) bytes
 *                (holds the [kept_capacity x d_ff] SwiGLU activations)
 */
int ce_routed_ffn(const ce_batch* batch, const void* compact, const int32_t* kept_idx,
                  const int32_t* kept_offsets, const ce_ffn_w* w, void* ffn_out,
                  void* ws, size_t ws_bytes, void* stream);

/*
 * Step 4 in two launches (same result as ce_routed_ffn; section 3.4, FFN over
 * the packed retained rows):
 *   ce_ffn_gateup  act[j] = SiLU(W_gate x_j) * (W_up x_j), x_j = compact[j]; act is the
 *                  intermediate activation z of the FFN (section 3.4, Eq. 8 scores FFN
 *                  channels from it). act: device dtype [kept_capacity x d_ff], packed order.
 *   ce_ffn_down    ffn_out[j] = W_down act[j]; ffn_out: device dtype [kept_capacity x d].
 * Arguments otherwise as ce_routed_ffn; ws: ce_workspace_size(CE_WS_FFN, ...) bytes
 * (the act region of the workspace is not used by these two calls).
 */
int ce_ffn_gateup(const ce_batch* batch, const void* compact, const int32_t* kept_idx,
                  const int32_t* kept_offsets, const ce_ffn_w* w, void* act, void* ws,
                  size_t ws_bytes, void* stream);
int ce_ffn_down(const ce_batch* batch, const void* act, const int32_t* kept_idx,
                const int32_t* kept_offsets, const ce_ffn_w* w, void* ffn_out, void* ws,
                size_t ws_bytes, void* stream);

/*
 * Step 5 -- residual merge (section 3.4: dropped tokens take the bypass path):
 *   hidden_out[kept_idx[j]] = hidden_in[kept_idx[j]] + ffn_out[j]   (fp32 add, one rounding)
 *   hidden_out[i] = hidden_in[i] for dropped i
 * hidden_in == hidden_out is allowed (in place: dropped rows are not touched);
 * out of place, every dropped row is copied (extra traffic).
 */
int ce_scatter_residual(const ce_batch* batch, const void* ffn_out, const int32_t* kept_idx,
                        const int32_t* kept_offsets, int dtype, int32_t d,
                        const void* hidden_in, void* hidden_out, void* stream);

/*
 * Steps 1-5 fused (section 3.2 Eq. 4, section 3.4 Eq. 6 and the packing /
 * bypass rule after it): score -> TopK -> SwiGLU FFN over the retained rows
 * (gathered directly from hidden_in) -> residual scatter into hidden_out;
 * dropped tokens take the bypass path (their rows are never written in place,
 * copied unchanged out of place).
 *   hidden_in / hidden_out  device dtype [T x d] (may alias: in place)
 *   logits_out       device float32 [T] or NULL
 *   kept_idx_out     device int32 [kept_capacity] or NULL
 *   kept_offsets_out device int32 [B+1] or NULL
 *   ws               device workspace of ce_workspace_size(CE_WS_BLOCK, ...) bytes
 * Scorer and FFN must agree on d and dtype.
 */
int ce_routed_block(const ce_batch* batch, const void* hidden_in, void* hidden_out,
                    const ce_scorer_w* scorer, const ce_ffn_w* ffn, float* logits_out,
                    int32_t* kept_idx_out, int32_t* kept_offsets_out, void* ws,
                    size_t ws_bytes, void* stream);

/*
 * ce_routed_block plus the layer-skipping redundancy gap of the block
 * (section 3.4, UCS operator (1), Eq. 7), with x_in = hidden_in and x_out =
 * hidden_out as ce_layer_gap defines it, without reading either [T x d]
 * matrix again: the down GEMM's epilogue, which holds each retained row's
 * residual and output, adds up the fp64 sums of in*out, in*in and out*out per
 * row, and a dropped token, which bypasses the block unchanged, has cos = 1.
 * Same arguments and results as ce_routed_block (the outputs are bit for bit
 * those of ce_routed_block), plus
 *   delta     skip threshold delta_LS (the paper's is 0.0040), finite
 *   cos       device float32 [T] out: per-token cosine (NaN past an overflowing
 *             capacity, see CE_DEV_OVERFLOW)
 *   rho_all, rho_ret, gap  device float32 [B] out; skip device uint8 [B] out or NULL
 *   ws        device workspace of ce_workspace_size(CE_WS_BLOCK_GAP, ...) bytes
 * The sums add the per-row partials in a fixed order (deterministic); they
 * differ from ce_layer_gap's only in the order of the fp64 additions.
 */
int ce_routed_block_gap(const ce_batch* batch, const void* hidden_in, void* hidden_out,
                        const ce_scorer_w* scorer, const ce_ffn_w* ffn, float* logits_out,
                        int32_t* kept_idx_out, int32_t* kept_offsets_out, float delta, float* cos,
                        float* rho_all, float* rho_ret, float* gap, uint8_t* skip, void* ws,
                        size_t ws_bytes, void* stream);

/*
 * Host query: how the routing logits (section 3.2, Eq. 4) are computed for
 * this batch. ce_score runs the single-launch scorer: tiles of 32 or 128
 * tokens of one sequence, each streaming every active rank of W1 (128 for
 * bf16 batches large enough that 32-token tiles would need several rounds of
 * workgroups). For large bf16 batches with many ranks, ce_routed_block
 * instead scores tiles of tm tokens x tn ranks (tm, tn in {64, 128}; a tile
 * covers core or expansion ranks, never both), each writing per-token
 * partial sums of w2 . SiLU(W1 h + b1) over its ranks into the workspace,
 * and the TopK step assembles the logits from them in a fixed order (core
 * tiles, b2_core, then for generation tokens the expansion tiles and
 * b2_exp[m]). The choice depends only on B, T, d, r_core, r_exp and dtype.
 *   tile_out  host int32 [2] or NULL: {tm, tn} of the block's rank tiles, or
 *             {token tile, 0} for the single-launch scorer
 * Returns 1 (rank-tiled block), 0 (single-launch scorer) or a negative
 * status for an invalid batch or scorer description (device pointers are not
 * read).
 */
int ce_score_tiling(const ce_batch* batch, const ce_scorer_w* scorer, int32_t* tile_out);

/*
 * Drop-set stability between two timesteps (section 3.4, UCS operators (3)
 * diffusion-head cache reuse and (4) denoising-step early exit; Eq. 10-11).
 * For each sequence b the drop set D of a timestep is its routable tokens
 * (CE_TOK_KEEP clear) whose packed position is negative (dropped):
 *   jaccard[b] = |D_t n D_ref| / |D_t u D_ref|            (1 when both are empty)
 *   j_rand[b]  = expected Jaccard of two independent, uniformly random subsets
 *                of the sequence's routable tokens with the same two sizes
 *                (hypergeometric overlap, evaluated in fp64)
 *   rda[b]     = (jaccard - j_rand) / (1 - j_rand)       (1 when j_rand = 1)
 * The early-exit signal is the pair (t, t - 1); cache reuse compares with the
 * timestep of the last refresh. Thresholds and the decisions they drive stay
 * with the caller.
 *   token_pos_t, token_pos_ref  device int32 [T]: ce_topk_compact's token_pos
 *                               at the two timesteps (same batch layout)
 *   jaccard                     device float32 [B] out
 *   j_rand, rda                 device float32 [B] out, or NULL
 * Deterministic. Errors: CE_ERR_INVALID_ARG for null pointers / sizes,
 * CE_ERR_HIP on a failed launch.
 */
int ce_drop_stability(const ce_batch* batch, const int32_t* token_pos_t,
                      const int32_t* token_pos_ref, float* jaccard, float* j_rand, float* rda,
                      void* stream);

/*
 * FFN pruning on the retained rows (section 3.4, UCS operator (2); Eq. 8-9).
 * The pruned FFN is the FFN without the channels of a static mask P; it runs
 * for a sequence when the saliency leakage of P on that sequence's retained
 * tokens is at most delta (the paper's delta_FFN is 0.150).
 *
 * ce_ffn_down_colnorms: norms[s * d_ff + c] = ||W_down[s][:, c]||_2 in fp32 for
 *   each weight set s of w (W_down is [d x d_ff]); computed once per layer.
 *   norms  device float32 [n_sets x d_ff] out
 *
 * ce_ffn_saliency: for each sequence b, over its packed rows j (kept_offsets),
 *   saliency[b * d_ff + c] = mean_j |act[j][c]| * norms[set(j) * d_ff + c]   (Eq. 8)
 *   leakage[b] = sum_{c: prune_mask[c]} saliency[b][c] / sum_c saliency[b][c]  (Eq. 9)
 *   use_pruned[b] = leakage[b] <= delta
 *   act         device dtype [kept_capacity x d_ff]: SwiGLU activations in packed
 *               row order (the output of ce_ffn_gateup)
 *   kept_idx    device int32 [kept_capacity] (the MoT set of row j is the GEN
 *               bit of token kept_idx[j] when w->n_sets == 2)
 *   prune_mask  device uint8 [d_ff], nonzero = channel in P
 *   saliency    device float32 [B x d_ff] out; leakage device float32 [B] out
 *   use_pruned  device uint8 [B] out, or NULL
 *   ws          the FFN workspace (ce_workspace_size(CE_WS_FFN, ...)); holds the
 *               per-row-split partial sums (each sequence's rows are split over
 *               up to 16 workgroups), summed in a fixed order
 *   A sequence with no retained rows (or zero total saliency) has leakage 0.
 *
 * ce_ffn_mask_channels: act[j][c] = 0 for every c in P on the rows j of the
 *   sequences with use_pruned[b] != 0, in place; ce_ffn_down on the result is
 *   the pruned FFN for those sequences and the full FFN for the others.
 *
 * All three are deterministic (fixed summation order). Errors:
 * CE_ERR_INVALID_ARG for null pointers / sizes / a non-finite delta,
 * CE_ERR_UNSUPPORTED for dtypes or widths outside the limits, CE_ERR_WORKSPACE
 * (ce_ffn_saliency), CE_ERR_HIP.
 */
int ce_ffn_down_colnorms(const ce_ffn_w* w, float* norms, void* stream);
int ce_ffn_saliency(const ce_batch* batch, const void* act, const int32_t* kept_idx,
                    const int32_t* kept_offsets, const ce_ffn_w* w, const float* norms,
                    const uint8_t* prune_mask, float delta, float* saliency, float* leakage,
                    uint8_t* use_pruned, void* ws, size_t ws_bytes, void* stream);
int ce_ffn_mask_channels(const ce_batch* batch, void* act, const int32_t* kept_offsets, int dtype,
                         int32_t d_ff, const uint8_t* prune_mask, const uint8_t* use_pruned,
                         void* stream);

/*
 * The FFN on the packed rows with the pruning decision taken on the fly and
 * the pruned FFN doing less work (section 3.4, UCS operator (2); Eq. 8-9).
 * P is the tail of the channels, [n_keep, d_ff): a layer whose static mask is
 * another set permutes its FFN channels once (W_gate / W_up rows and W_down
 * columns together, which leaves the FFN unchanged) so that P comes last.
 *   1. gate/up + SwiGLU as ce_ffn_gateup; its epilogue also adds up |z| per
 *      channel over each run of rows of one sequence (no second pass over the
 *      [Kt x d_ff] activations);
 *   2. saliency[b][c] = mean_j |z[j][c]| * norms[set(j)][c] over the packed rows of
 *      sequence b (Eq. 8), leakage[b] = sum_{c >= n_keep} saliency[b][c] /
 *      sum_c saliency[b][c] (Eq. 9; 0 when the sum is 0), use_pruned[b] =
 *      leakage[b] <= delta;
 *   3. down: rows of sequences with use_pruned skip the channels of P (they
 *      read zeros there, and a 256-row tile whose rows all run pruned stops
 *      its K loop at n_keep), so ffn_out is the pruned FFN for those sequences
 *      and the full FFN for the others, as ce_ffn_mask_channels + ce_ffn_down.
 * Arguments as ce_routed_ffn, plus
 *   norms       device float32 [n_sets x d_ff]: ce_ffn_down_colnorms of w
 *   n_keep      channels kept by the pruned FFN: 0 <= n_keep <= d_ff, n_keep % 64 == 0
 *   delta       leakage threshold (the paper's delta_FFN is 0.150), finite
 *   saliency    device float32 [B x d_ff] out; leakage device float32 [B] out
 *   use_pruned  device uint8 [B] out (read back by step 3)
 *   ws          device workspace of ce_workspace_size(CE_WS_FFN_PRUNED, ...) bytes
 * bf16 only, with d and d_ff such that both GEMMs run on the ping-pong kernel
 * (K at least 3 x 64 elements); else CE_ERR_UNSUPPORTED. Deterministic.
 */
int ce_routed_ffn_pruned(const ce_batch* batch, const void* compact, const int32_t* kept_idx,
                         const int32_t* kept_offsets, const ce_ffn_w* w, const float* norms,
                         int32_t n_keep, float delta, void* ffn_out, float* saliency, float* leakage,
                         uint8_t* use_pruned, void* ws, size_t ws_bytes, void* stream);

/*
 * Layer-skipping redundancy gap (section 3.4, UCS operator (1); Eq. 7). For a
 * candidate layer with input x_in and output x_out (the same batch layout),
 * per token i and sequence b:
 *   cos[i]     = <x_in[i], x_out[i]> / (||x_in[i]|| ||x_out[i]||)
 *                (1 when both rows are zero, 0 when exactly one is)
 *   rho_all[b] = mean cos over the sequence's tokens          (1 for an empty sequence)
 *   rho_ret[b] = mean cos over its retained tokens, token_pos >= 0
 *                (rho_all[b] when none is retained)
 *   gap[b]     = rho_all[b] - rho_ret[b]                       (Eq. 7)
 *   skip[b]    = gap[b] <= delta (the paper's delta_LS is 0.0040)
 *   x_in, x_out  device dtype [T x d] row-major (CE_BF16 or CE_F32; d % 64 == 0)
 *   token_pos    device int32 [T]: ce_topk_compact's token_pos for this layer
 *   cos          device float32 [T] out (also the per-token stage's result)
 *   rho_all, rho_ret, gap  device float32 [B] out; skip device uint8 [B] out, or NULL
 * Sums run in fp64 in a fixed order (deterministic). Errors: CE_ERR_INVALID_ARG
 * for null pointers / sizes / a non-finite delta, CE_ERR_UNSUPPORTED for the
 * dtype or d, CE_ERR_HIP.
 */
int ce_layer_gap(const ce_batch* batch, const void* x_in, const void* x_out, int dtype, int32_t d,
                 const int32_t* token_pos, float delta, float* cos, float* rho_all, float* rho_ret,
                 float* gap, uint8_t* skip, void* stream);

/*
 * Attention over the packed retained tokens of a routed layer (section 3.4,
 * task-adaptive token compaction: retained tokens are packed into a shorter
 * sequence for the layer's attention and FFN; for understanding, the packed
 * keys / values are the compressed key-value cache that decoding reuses).
 * For each sequence b and query head h, with kv(h) = h / (n_heads / n_kv_heads):
 *   O_b[:, h] = softmax(scale * Q_b[:, h] K_b[:, kv(h)]^T + M) V_b[:, kv(h)]
 * M = 0, or with causal != 0, -inf for key j > i + (n_kv - n_q) (end-aligned:
 * prefill has n_q = n_kv, a decode step n_q = 1 over the whole cache). A query
 * that sees no key outputs zeros. Sequences never attend to each other.
 */
typedef struct ce_attn {
  int32_t B;                  /* sequences, >= 1 */
  int32_t n_heads;            /* query heads H */
  int32_t n_kv_heads;         /* key/value heads; divides H */
  int32_t head_dim;           /* 128 */
  const int32_t* q_offsets;   /* device int32 [B+1]: packed query rows of each sequence */
  const int32_t* kv_offsets;  /* device int32 [B+1]: packed key/value rows of each sequence */
  int32_t q_capacity;         /* rows of q and o (grid bound; offsets are clamped to it) */
  int32_t kv_capacity;        /* rows of k and v */
  int32_t causal;             /* 0 or 1 */
  float scale;                /* softmax scale > 0, e.g. 1 / sqrt(head_dim) */
  int32_t dtype;              /* CE_BF16 */
} ce_attn;

/*
 *   q, o   device bf16 [q_capacity x n_heads x head_dim], row-major (o written
 *          for the rows of real queries only)
 *   k, v   device bf16 [kv_capacity x n_kv_heads x head_dim], row-major
 * fp32 accumulation; the probabilities are rounded to bf16 for the product
 * with V. Deterministic. Errors: CE_ERR_INVALID_ARG for null pointers, sizes,
 * a scale that is not a positive finite number or causal outside {0, 1}; CE_ERR_UNSUPPORTED for another
 * dtype or head_dim, or buffers of 2 GiB or more; CE_ERR_HIP.
 */
int ce_routed_attention(const ce_attn* attn, const void* q, const void* k, const void* v, void* o,
                        void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CE_ROUTER_H */
