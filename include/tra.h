/*
 * tra.h -- C ABI of the Token Radius Attention (TRA) hot path on MI355X (gfx950).
 *
 * The path (Sec. 3 of the paper) runs in four steps, one entry point each:
 *
 *   tra_entropy           per-query attention entropy H_i (Sec. 2.2, Eq. 2),
 *                         accumulated inside an online-softmax pass (App. C.2,
 *                         Alg. 2), optionally fused with the dense output O.
 *   tra_budget_radius     entropy -> budget K_hat = ceil(tau * exp(H))
 *                         (Sec. 3.1, Eq. 8; or the entropy-identified
 *                         lognormal mapping of App. A.2) -> smallest
 *                         boundary-aware squared radius reaching it
 *                         (Sec. 3.2, Eqs. 13-14).
 *   tra_build_block_mask  per-token radii -> Boolean query-block x key-block
 *                         mask by the token vote of Alg. 1 (App. C.1), plus
 *                         per-row lists of retained key blocks.
 *   tra_sparse_attention  block-sparse attention over the retained blocks
 *                         (Sec. 3.2, Eq. 16, executed at block granularity).
 *   tra_token_attention   the same over the retained blocks with the token
 *                         mask of Eq. 15 applied inside them (Eq. 16 exactly).
 *   tra_dense_attention   dense attention (Sec. 2.1, Eq. 1), the baseline.
 *
 * Tensors and layout
 * ------------------
 * All tensor arguments are DEVICE pointers to contiguous row-major buffers on
 * the device that was current when the plan was created.  Q, K, V and O are
 * [batch][heads][S][head_dim].  The first N = F*H*W tokens are the video
 * tokens in RASTER order of the F x H x W latent grid, token
 * i = (f*H + x)*W + y (Sec. 2.1); the last text_tokens tokens (S = N +
 * text_tokens) are the text tokens of joint text-video attention (Sec. 3.2),
 * in the caller's order.  Element type is bf16 (TRA_BF16) or fp32 (TRA_FP32) as
 * set in the config; pointers must be 16-byte aligned.  Per-token arrays
 * (entropy, budget, radius_sq, lse) are [batch][heads][S] in the same order.
 *
 * The library applies the tile-major token order of Sec. 3.3 internally: each
 * frame is cut into tile_h x tile_w tiles (edge tiles clipped), tokens are
 * listed frame by frame, tile by tile, row-major inside a tile; text tokens
 * follow the video tokens unchanged.  With the packed block layout (default)
 * block u is positions [u*block, min((u+1)*block, S)) of that order and
 * NB = ceil(S / block) (App. C).  With tile-aligned padded blocks
 * (TRA_BLOCKS_TILES) every video block is one whole tile of one frame, padded
 * when the frame edge clips the tile (see tra_block_layout).  A block holding
 * any text token is a text block.  Block-level arrays use row index
 * r = (b*heads + h)*NB + u:
 *   mask [batch][heads][NB][NB] uint8 (1 = retained),
 *   cnt  [batch][heads][NB]     int32 (retained key blocks of row r),
 *   cols [batch][heads][NB][NB] int32 (retained key-block ids, ascending in
 *                               the first cnt entries, -1 after them),
 *   order[batch*heads*NB]       int32 (a permutation of all rows r, heaviest
 *                               first by cnt, ties by ascending r).
 *
 * Calls, ownership, errors
 * ------------------------
 * Every compute call is asynchronous on `stream` (a hipStream_t passed as
 * void*, NULL = the null stream), checks its arguments before launching, and
 * returns a status.  The caller owns every buffer -- tensors and workspaces
 * -- and keeps it alive until the stream has drained.  The plan owns only its
 * device tables (permutation, thresholds, block boxes, key-block distance
 * words and, for the 2-D distance, the per-key vectors of the token-level key
 * test, and the count lookup table of App. C.1: C(n) for every candidate
 * radius at every position of one octant of the grid, ceil(F/2) ceil(H/2)
 * ceil(W/2) (n_cap + 1) ints -- 331 MB at 21 x 45 x 80 -- or, where that
 * would exceed 1 GiB, C(n_cap) per position); no call writes them, so a plan
 * is immutable after creation and may be shared by calls on any number of
 * streams at once.
 *
 * Calls that need scratch device memory take it from the caller as
 * (workspace, workspace_bytes): a device buffer, 256-byte aligned, of at least
 * tra_workspace_size(plan, call) bytes.  Its contents need no initialisation
 * and are undefined after the call.  Calls whose use of one workspace overlaps
 * in time (different streams) race; give each stream its own.  What a bf16
 * plan's workspace holds:
 *   attention calls (tra_entropy, tra_sparse_attention, tra_token_attention,
 *     tra_dense_attention): K and V rewritten in tile-major order (V
 *     transposed in 64-key tiles), 2 x batch x heads x NB x 128 x head_dim x 2
 *     bytes, rewritten by every call, plus 512 bytes of row-queue counters
 *     that the call resets and draws its query-block rows from;
 *   tra_sparse_attention, in addition: the work-unit tables and the split
 *     rows' partial results, (head_dim + 3) x 512 bytes for each of up to
 *     32 G + 1 pieces (G the workgroups the GPU holds at once; 1.65 GB at
 *     head_dim 128 on MI355X, less where the plan has fewer blocks);
 *   tra_build_block_mask with a non-NULL order: the counting-sort histograms
 *     of the row order, 4 x ((NB + 1) x ceil(batch x heads x NB / 256) + 1)
 *     bytes (the only workspace of fp32 plans; with a NULL order the mask call
 *     needs none and the workspace may be NULL).
 * No C++ exception crosses this ABI.  On failure, tra_last_error() returns a
 * message for the calling thread.
 */
#ifndef TRA_H
#define TRA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Squared radius of the full-support candidate radius of Sec. 3.2 (keeps
 * every key of every frame). */
#define TRA_RADIUS_FULL 2147483647

typedef enum {
  TRA_OK = 0,
  TRA_ERR_INVALID_ARG = 1, /* null pointer, bad shape or misaligned buffer   */
  TRA_ERR_UNSUPPORTED = 2, /* head_dim / block / dtype / device not handled   */
  TRA_ERR_DEVICE = 3,      /* a HIP runtime call or kernel launch failed      */
  TRA_ERR_ALLOC = 4        /* plan table allocation failed                    */
} tra_status;

typedef enum { TRA_BF16 = 0, TRA_FP32 = 1 } tra_dtype;

/* Block retention rule.  VOTE is Alg. 1: with c_j the number of valid queries
 * of the query block whose radius covers key j, C = {j : c_j > 0} and
 * C_hi = {j : 3 c_j > n_u} (n_u = valid queries of the block, b/3 for a full
 * block), keep iff |C| > 0 and 10 |C_hi| > 6 |C|.  UNION keeps iff |C| > 0.
 * Under both rules the diagonal block (u, u) is always kept. */
typedef enum { TRA_MASK_VOTE = 0, TRA_MASK_UNION = 1 } tra_mask_rule;

/* Entropy-to-budget mapping.  UNIFORM is the paper's K_hat = ceil(tau e^H)
 * (Sec. 3.1, Eq. 8).  LOGNORMAL is the entropy-identified lognormal mapping of
 * App. A.2: with S keys per attention row, sigma = sqrt(2 (log S - H)) and
 * K_hat = ceil(S * Phibar(sigma - Phi^{-1}(tau))), Phibar = 1 - Phi the
 * standard normal tail; at H = log S both give ceil(tau S). */
typedef enum { TRA_BUDGET_UNIFORM = 0, TRA_BUDGET_LOGNORMAL = 1 } tra_budget_map;

/* Distance of the radius test.  D2 is Eq. 15: the 2-D spatial distance against
 * sqrt(n) phi(delta).  D1 is the sequence-distance ablation (App. C.1,
 * Eq. area-matched-1d): |i - j| between raster indices against the area-matched
 * 1-D radius (pi/2) n phi(delta), n the squared 2-D radius. */
typedef enum { TRA_DIST_2D = 0, TRA_DIST_1D = 1 } tra_distance;

/* Block layout of the block mask and of the block-sparse and token-level
 * calls (the blocks their mask, cnt, cols and order refer to).
 * PACKED: block u is positions [u b, (u+1) b) of the tile-major order, so a
 *   block may hold parts of two tiles, or of two frames; NB = ceil(S / b).
 * TILES: tile-aligned padded blocks.  Every video block is exactly one
 *   tile_h x tile_w tile of one frame (tile_h * tile_w must equal b): frames
 *   in order, tiles in tile-row-major order, tokens row-major inside the tile.
 *   A tile clipped by the frame edge fills the first positions of its block;
 *   the rest are padding, neither queries nor keys.  Text tokens follow in
 *   blocks of b, the last one padded.  NB = F ceil(H / tile_h) ceil(W /
 *   tile_w) + ceil(T / b).  A block then has the smallest spatial footprint b
 *   tokens can have, so fewer of its keys lie outside a query's radius: App. D
 *   names that in-block work as the block-granular method's main limitation.
 * tra_entropy and tra_dense_attention are defined over tokens and give the
 * same results under both layouts. */
typedef enum { TRA_BLOCKS_PACKED = 0, TRA_BLOCKS_TILES = 1 } tra_block_layout;

typedef struct tra_config {
  int32_t batch;     /* >= 1                                                  */
  int32_t heads;     /* >= 1                                                  */
  int32_t frames;    /* F >= 1 (at most 64)                                   */
  int32_t height;    /* H >= 1 (latent rows, at most 1023)                    */
  int32_t width;     /* W >= 1 (latent columns, at most 1023)                 */
  int32_t head_dim;  /* d: 64 or 128                                          */
  int32_t block;     /* b: 64 or 128 (bf16 needs 128)                         */
  int32_t tile_h;    /* tile rows >= 1 (typ. 8)                               */
  int32_t tile_w;    /* tile columns >= 1 (typ. 8 for b=64, 16 for b=128)     */
  int32_t dtype;     /* tra_dtype                                             */
  int32_t rule;      /* tra_mask_rule                                         */
  int32_t budget_map;   /* tra_budget_map                                     */
  int32_t distance;     /* tra_distance                                       */
  int32_t text_tokens;  /* T >= 0 text tokens after the video tokens          */
  int32_t block_layout; /* tra_block_layout                                   */
  double tau;        /* target attention mass, 0 < tau < 1 (paper: 0.9)      */
  double gamma;      /* temporal decay rate of phi(delta) = exp(-gamma delta),
                        gamma >= 0 (Eq. 10; 0.6 Wan, 0.95 HunyuanVideo)       */
} tra_config;

typedef struct tra_plan_s* tra_plan;

/* The calls that take a workspace, for tra_workspace_size. */
typedef enum {
  TRA_CALL_ENTROPY = 0,    /* tra_entropy (entropy only or fused with o)      */
  TRA_CALL_BLOCK_MASK = 1, /* tra_build_block_mask with a non-NULL order      */
  TRA_CALL_SPARSE = 2,     /* tra_sparse_attention                            */
  TRA_CALL_TOKEN = 3,      /* tra_token_attention                             */
  TRA_CALL_DENSE = 4       /* tra_dense_attention                             */
} tra_call;

/* Validates cfg, builds the shape tables on the host in fp64/integer
 * arithmetic (tile-major permutation, squared-radius thresholds
 * thr[n][delta] = floor(n * exp(-2 gamma delta)) for n in [0, n_cap],
 * n_cap = (H-1)^2 + (W-1)^2, for TRA_DIST_1D also the 1-D thresholds
 * thr1[n][delta] = floor((pi/2) n * exp(-gamma delta)), per-block bounding
 * boxes) and copies them to the current device.  *out receives the plan, or
 * NULL on failure. */
tra_status tra_plan_create(const tra_config* cfg, tra_plan* out);

/* Frees the plan's device tables.  NULL is accepted. */
tra_status tra_plan_destroy(tra_plan plan);

/* n_tokens = S = F*H*W + text_tokens (the token count of every per-token
 * tensor), NB of the plan's block layout, n_cap as above.  Any output may be
 * NULL. */
tra_status tra_plan_dims(tra_plan plan, int32_t* n_tokens, int32_t* n_blocks,
                         int32_t* n_cap);

/* Host-only (no device needed): the plan's tables for cfg, for inspection.
 * perm[P]: token index (raster for video, N + t for text token t) of the
 *          token at position p of the block layout's order, -1 at a padding
 *          position; P = S for the packed layout, NB * block for tiles.
 * thr[(n_cap+1) * F]: thr[n*F + delta] (2-D, squared).
 * thr1[(n_cap+1) * F]: thr1[n*F + delta] = floor((pi/2) n exp(-gamma delta)).
 * blocks[NB * 10]: per block {f_min, f_max, x_min, x_max, y_min, y_max,
 *                 n_video, r_min, r_max, n_text} over its video tokens (r the
 *                 raster index) and the count of its text tokens; a block's
 *                 tokens fill its first n_video + n_text positions.
 * Any array pointer may be NULL; *n_cap_out (may be NULL) gets n_cap. */
tra_status tra_plan_host_tables(const tra_config* cfg, int32_t* perm, int32_t* thr,
                                int32_t* thr1, int32_t* blocks, int32_t* n_cap_out);

/* *bytes = the workspace size (bytes) that `call` (a tra_call) needs on this
 * plan; 0 means the call takes none (its workspace may be NULL).  The size
 * depends on the plan only, not on the call's data. */
tra_status tra_workspace_size(tra_plan plan, int32_t call, size_t* bytes);

/* Kernel timing, for benchmarks (not for calls captured into a graph).
 * tra_kernel_timing(call, n): the calling thread's next n calls of kind
 * `call` (TRA_CALL_ENTROPY, TRA_CALL_SPARSE, TRA_CALL_TOKEN or TRA_CALL_DENSE)
 * record a HIP event pair on their stream around their attention kernel
 * alone -- not around the layout pre-pass, nor the work-unit and merge kernels
 * of a block-sparse call.  The n event pairs are created here, on the current
 * device (calls of plans on another device are not timed), and replace the
 * thread's earlier ones; n = 0 releases them.  1 <= n <= 4096.
 * tra_kernel_times(ms, n, got): waits for the recorded calls and writes up to
 * n kernel times (milliseconds, call order) to ms; *got receives how many
 * calls were recorded. */
tra_status tra_kernel_timing(int32_t call, int32_t n);
tra_status tra_kernel_times(float* ms, int32_t n, int32_t* got);

/* Message describing the last failure on the calling thread ("" if none). */
const char* tra_last_error(void);

/* Library version string. */
const char* tra_version(void);

/* Attention entropy H_i = -sum_j p_ij log p_ij in nats over all S keys
 * (Eq. 2; with text tokens the joint attention row), for every token, computed
 * with the online-softmax identity
 * H = log Z - sum_j p_ij s_ij of App. C.2 (Alg. 2).
 * q, k: inputs.  v, o: both NULL (entropy only), or both non-NULL, in which
 * case o also receives dense attention softmax(q k^T / sqrt(d)) v (the fused
 * warm-up step of Alg. 2).  For bf16 plans the fused call runs its own kernel
 * (the key blocks split over two groups of waves and merged), so its o and
 * entropy agree with tra_dense_attention's output and with the entropy-only
 * call up to fp32 rounding, not bit for bit; fp32 plans share one kernel.
 * entropy: fp32 [batch][heads][S] output.  workspace: TRA_CALL_ENTROPY. */
tra_status tra_entropy(tra_plan plan, const void* q, const void* k, const void* v,
                       void* o, float* entropy, void* workspace, size_t workspace_bytes,
                       void* stream);

/* Entropy -> budget -> squared radius, per token (Sec. 3.1-3.2; App. C.1,
 * Eq. implementation-budget-radius: a bisection over the plan's count table).
 * For a video token, K_hat is evaluated in fp64 by the plan's mapping and
 * clamped to [1, S]:
 *   UNIFORM    K_hat = ceil(tau * exp(H));
 *   LOGNORMAL  K_hat = ceil(S * 0.5 erfc((sigma - z) / sqrt 2)),
 *              sigma = sqrt(2 max(0, log S - H)), z = Phi^{-1}(tau)
 *              (z found on the host by bisection on Phi to full fp64 precision).
 * A NaN entropy gives K_hat = S.  radius_sq = the smallest n in [0, n_cap] whose
 * boundary-aware count C(n) = sum_t #{(x', y') : (x-x')^2 + (y-y')^2 <=
 * thr[n][|t - f|]} over the video grid (Eq. 13) reaches K_hat (Eq. 14), else
 * TRA_RADIUS_FULL.  Counts are exact integers.  Text tokens get K_hat = S and
 * TRA_RADIUS_FULL.
 * entropy: fp32 input; budget: int32 output or NULL; radius_sq: int32 output. */
tra_status tra_budget_radius(tra_plan plan, const float* entropy, int32_t* budget,
                             int32_t* radius_sq, void* stream);

/* Alg. 1 block mask from per-token squared radii (raster order).  A video
 * query i covers a video key j iff (x_i-x_j)^2 + (y_i-y_j)^2 <=
 * thr[n_i][|f_i - f_j|] (Eq. 15), or for TRA_DIST_1D iff |i - j| <=
 * thr1[n_i][|f_i - f_j|]; radius values outside [0, n_cap] other than
 * TRA_RADIUS_FULL are clamped (negative -> 0, larger -> FULL).  The rule and
 * distance come from the plan.  Text blocks are retained in every row and a
 * text block's row retains every block (Alg. 1; text keys stay visible). 
 * mask: uint8 output or NULL; cnt, cols: int32 outputs; order: int32 output
 * (the heaviest-first row order, sorted in the workspace) or NULL (not
 * computed).  workspace: TRA_CALL_BLOCK_MASK when order is non-NULL, else
 * unused (may be NULL). */
tra_status tra_build_block_mask(tra_plan plan, const int32_t* radius_sq, uint8_t* mask,
                                int32_t* cnt, int32_t* cols, int32_t* order,
                                void* workspace, size_t workspace_bytes, void* stream);

/* tra_build_block_mask without any allocation, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid it): the same mask, lists and order, bit for bit,
 * but the heaviest-first order sorts in a scratch array that the library
 * holds on each GPU (4 MiB, kept until the process ends) instead of a
 * caller's workspace.  With a non-NULL order it needs (NB + 1) *
 * ceil(batch * heads * NB / 256) <= 2^20 workspace ints and otherwise returns
 * TRA_ERR_UNSUPPORTED before launching anything.  All calls on one GPU share
 * that array: two such calls that overlap in time on that GPU (different
 * streams) race; calls on one stream are ordered and safe.  Nothing here
 * calls hipMalloc or hipFree. */
tra_status tra_build_block_mask_noalloc(tra_plan plan, const int32_t* radius_sq, uint8_t* mask,
                                        int32_t* cnt, int32_t* cols, int32_t* order,
                                        void* stream);

/* Block-sparse attention: a query of block u takes one softmax over every key
 * of the key blocks cols[r][0..cnt[r]) (r its row) and attends to no other key
 * (Eq. 16 at block granularity).  With a non-NULL `order`, only the rows it
 * lists are computed, handed out in that order (entries outside [0, rows) are
 * skipped); with NULL every row is computed.  The schedule never changes a
 * row's result.
 * cnt values are clamped to [0, NB]; column ids outside [0, NB) are skipped.
 * o: output; lse: fp32 natural-log log-sum-exp of the scaled scores over the
 * retained keys, or NULL.  A row with cnt = 0 gets o = 0, lse = -inf.
 * Work is balanced by cutting long lists: with T the total of the (clamped)
 * list lengths of the rows computed and G the number of workgroups the GPU
 * holds at once, a row of more than L = max(48, ceil(T / 16G)) entries
 * is computed as ceil(cnt / L) pieces of consecutive entries whose partial
 * softmax states are merged afterwards, so its result differs from an
 * unsplit computation by rounding only (each piece rounds its probabilities
 * to bf16 relative to its own running maximum); rows of at most 48 entries
 * are never split.  The output is normalised by the sum of the
 * bf16-rounded probabilities that multiply V (lse by the fp32 sum).
 * workspace: TRA_CALL_SPARSE. */
tra_status tra_sparse_attention(tra_plan plan, const void* q, const void* k,
                                const void* v, const int32_t* cnt, const int32_t* cols,
                                const int32_t* order, void* o, float* lse, void* workspace,
                                size_t workspace_bytes, void* stream);

/* Token-level TRA attention inside the retained blocks (Sec. 3.2, Eq. 16 with
 * the -inf bias of the token mask, Eq. 15; App. D names the block-granular
 * execution's redundant in-block work as the method's main limitation).  A
 * video query i of block u takes one softmax over the keys j of the key
 * blocks cols[r][0..cnt[r]) that its radius covers -- the same integer test as
 * tra_build_block_mask: (x_i-x_j)^2 + (y_i-y_j)^2 <= thr[n_i][|f_i-f_j|], or
 * for TRA_DIST_1D |i - j| <= thr1[n_i][|f_i-f_j|] -- plus every text key of
 * those blocks; a text query attends to every key of its retained blocks.
 * With lists from the union rule every covered key lies in a listed block,
 * so this is Eq. 16 over all keys.  radius_sq: int32 [batch][heads][S] input
 * (raster order, as written by tra_budget_radius; values above n_cap mean the
 * full radius, negative ones 0).  q, k, v, cnt, cols, order, o, lse as for
 * tra_sparse_attention; a query's own key is always covered, so a query of a
 * row that lists its own block never has an empty softmax; a query that
 * covers no listed key gets o = 0, lse = -inf.  Whole 128-key tiles that none
 * of a wave's 32 queries covers are skipped.  (bf16, 2-D: the test is
 * evaluated as an exact integer dot product of per-query and per-key vectors on
 * the matrix cores; the decisions are the same.)  bf16 plans need every threshold
 * below 65536 (n_cap <= 65535 for 2-D, floor(pi/2 n_cap) <= 65535 for 1-D)
 * and, with the packed layout, at least one block of video tokens per frame
 * (H*W >= block), else TRA_ERR_UNSUPPORTED.  workspace: TRA_CALL_TOKEN. */
tra_status tra_token_attention(tra_plan plan, const void* q, const void* k, const void* v,
                               const int32_t* radius_sq, const int32_t* cnt,
                               const int32_t* cols, const int32_t* order, void* o,
                               float* lse, void* workspace, size_t workspace_bytes,
                               void* stream);

/* Dense attention o_i = sum_j softmax_j(q_i k_j / sqrt(d)) v_j (Eq. 1), the
 * baseline the sparse call is measured against.  lse as above, or NULL.
 * workspace: TRA_CALL_DENSE. */
tra_status tra_dense_attention(tra_plan plan, const void* q, const void* k,
                               const void* v, void* o, float* lse, void* workspace,
                               size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TRA_H */
