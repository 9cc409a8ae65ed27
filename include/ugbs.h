/*
 * ugbs.h -- uncertainty-gated block-sparse causal prefill attention on
 * AMD Instinct MI355X (gfx950).  Plain C ABI.
 *
 * The method (Appendix A of the paper, steps A.1-A.10): keys are pooled into
 * blocks of 64 tokens; every Q-tile of 64 query rows scores every causally
 * visible block with the maximum over its rows; the sink block 0 and the
 * tile's own block are always kept; a sorted top-2k over the remaining
 * blocks gives both the kept list and the normalised cutoff margin sigma;
 * sigma is averaged over heads, and the tiles whose head mean lies at or
 * below the layer's q-quantile keep 2k blocks while every other tile keeps k
 * (rho = 2, Section 3 step 5); attention then runs only over the kept blocks.
 *
 * Pipeline for one layer, four stream-ordered calls:
 *   ugbs_block_meta   (K)                    -> meta
 *   ugbs_score_select (Q, meta, workspace)   -> idx_sorted, sigma
 *   ugbs_route        (sigma, idx_sorted)    -> kv_idx (may alias idx_sorted)
 *   ugbs_attend       (Q, K, V, kv_idx)      -> O
 * or, with the selection inside the attention kernel (no kv_idx lists):
 *   ugbs_block_meta   (K)                    -> meta
 *   ugbs_score_select (Q, meta, workspace)   -> sigma (idx_sorted NULL)
 *   ugbs_route        (sigma, workspace)     -> trigger flags (kv_idx NULL)
 *   ugbs_attend_select(Q, K, V, workspace)   -> O
 * or with per-row selection into tile bitmaps:
 *   ugbs_select_rows  (Q, meta, trigger)     -> bitmap
 *   ugbs_attend_bitmap(Q, K, V, bitmap)      -> O
 * No call synchronises the device; none allocates device memory.
 *
 * Diagnostics (Appendix D: sigma as a best-arm identification index), off
 * the prefill path, on the score tensor of ugbs_score_select(scores_out):
 *   ugbs_noise_scale  (Q, meta)                 -> rough, tau
 *   ugbs_bai_tiles    (scores, tau, z)          -> per-tile gaps, MC failures
 *   ugbs_bai_heads    (tiles, tau)              -> per-head aggregates
 *
 * Conventions shared by every entry point
 *   - All tensor pointers are device pointers owned by the caller.  The
 *     library never frees, keeps or allocates them.
 *   - Tensors are contiguous, batch-major "BHND": Q and O are
 *     [B, H, N, d], K and V are [B, H_kv, N, d], bf16 (raw 16-bit pattern).
 *     Query head h reads kv head h / (H / H_kv).
 *   - Prefill: the query rows are the key positions 0..N-1 (causal).
 *     N_B = N / 64 key blocks, T = N / 64 Q-tiles (T == N_B).
 *   - `stream` is a hipStream_t (NULL = the default stream).  Every call only
 *     enqueues work and returns; errors from the kernels themselves surface
 *     at the caller's next synchronisation.
 *   - Every argument is validated before anything is enqueued.  On error the
 *     call returns a ugbs_status != UGBS_OK and enqueues nothing.
 *     UGBS_ERR_HIP reports a failed launch (hipGetLastError).
 *   - Inputs must be finite.  Calls on one stream may be issued from any
 *     host thread; the library holds no per-call state.
 *   - The calls enqueue kernels only (no memset, copy, allocation or
 *     synchronisation), so a layer can be captured in a HIP graph and
 *     replayed; make one call of each kind outside the capture first, which
 *     sets the kernels' LDS limits and caches their occupancy.
 */
#ifndef UGBS_H
#define UGBS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__) || defined(__clang__)
#define UGBS_API __attribute__((visibility("default")))
#else
#define UGBS_API
#endif

#define UGBS_ABI_VERSION 10
#define UGBS_BLOCK 64          /* BLOCK_M = BLOCK_N = 64 tokens (Section 3.1, 3.2) */
#define UGBS_MAX_BLOCKS 4096   /* N_B <= 4096, i.e. N <= 262144 */
#define UGBS_MAX_BLOCKS_ROWS 2048 /* ugbs_select_rows, ugbs_bai_tiles, ugbs_bai_heads: N_B <= 2048 */
#define UGBS_MAX_KV_WIDTH 4096 /* kv_width accepted by ugbs_attend; rho * k_budget <= 4096 */
#define UGBS_MAX_RHO 8         /* expansion factor rho in 1..8 */
#define UGBS_ROUTE_SCRATCH_BYTES (1u << 20) /* device scratch of ugbs_route_noalloc, per GPU */

typedef enum {
  UGBS_OK = 0,
  UGBS_ERR_NULL = 1,      /* a required pointer is NULL */
  UGBS_ERR_SHAPE = 2,     /* batch/heads/seq_len/head_dim/block/kv_width invalid */
  UGBS_ERR_BUDGET = 3,    /* k_budget < 3, rho outside [1, 8], or rho k_budget > 4096 */
  UGBS_ERR_Q = 4,         /* q outside [0, 1] or NaN */
  UGBS_ERR_BACKBONE = 5,  /* backbone not one of ugbs_backbone */
  UGBS_ERR_ALIGN = 6,     /* a pointer is not aligned as documented */
  UGBS_ERR_WORKSPACE = 7, /* workspace NULL or smaller than ugbs_workspace_bytes */
  UGBS_ERR_HIP = 8,       /* a HIP launch failed */
  UGBS_ERR_SCALE = 9,     /* softmax_scale negative, NaN or infinite */
  UGBS_ERR_SCRATCH = 10   /* the problem needs more than the static scratch of ugbs_route_noalloc */
} ugbs_status;

/* Block-scoring backbone (Section 3.1).
 * UGBS_KMEAN: mean-pooled keys, Eq. (block-score) / A.1-A.2.
 * UGBS_QUEST: element-wise K-min/K-max bound, Eq. (quest-score). */
typedef enum { UGBS_KMEAN = 0, UGBS_QUEST = 1 } ugbs_backbone;

/* Problem description, following the paper's problem statement:
 * Q, K, V shapes, block size, k_budget, q, the backbone and the expansion
 * factor rho (Section 3 step 5; the paper uses rho = 2).  Every kv_idx row
 * has W = rho * k_budget slots; "2k" below stands for W. */
typedef struct ugbs_problem {
  int32_t batch;        /* B >= 1 */
  int32_t n_heads;      /* H >= 1, a multiple of n_kv_heads */
  int32_t n_kv_heads;   /* H_kv >= 1 */
  int32_t seq_len;      /* N: a positive multiple of 64, N / 64 <= UGBS_MAX_BLOCKS */
  int32_t head_dim;     /* d: 64, 128 or 256 */
  int32_t block;        /* must be 64 */
  int32_t k_budget;     /* k >= 3 with rho k <= UGBS_MAX_KV_WIDTH; counts the forced sink and
                           self blocks; with k >= N_B every tile keeps all visible blocks */
  int32_t backbone;     /* ugbs_backbone */
  double q;             /* trigger fraction, 0 <= q <= 1 */
  float softmax_scale;  /* attention logit scale; 0 means 1/sqrt(head_dim) */
  int32_t rho;          /* expansion factor, 1..UGBS_MAX_RHO; 0 means 2 */
} ugbs_problem;

/* Stage 1 -- block metadata (A.1; Eq. (quest-score) for Quest).
 *   K    : [B, H_kv, N, d] bf16, 16-byte aligned.
 *   meta : UGBS_KMEAN: [B, H_kv, N_B, d] bf16, the mean of the block's 64
 *          keys: the 64 values of a channel are summed in fp64 and the
 *          mean is rounded once to nearest-even bf16.  The fp64 sum is
 *          exact (so the result is the correctly rounded exact mean, for
 *          any order of summation) whenever the nonzero values of the
 *          channel within the block have binary exponents at most 39
 *          apart (8 significant bits each, 64 terms: every partial sum then
 *          fits in 53 bits).  Beyond that range the sum may round in its
 *          last fp64 bit, which changes the bf16 mean only when it lies
 *          within that rounding of a bf16 rounding boundary.
 *          UGBS_QUEST: [B, H_kv, N_B, d, 2] bf16: for every channel the
 *          pair (element-wise minimum, element-wise maximum) over the
 *          block's 64 keys, adjacent (the order in which the scoring
 *          kernel's 2:4-sparse contraction reads them).
 *          16-byte aligned.  A zero is always written as +0. */
UGBS_API int ugbs_block_meta(const ugbs_problem* p, const void* K, void* meta, void* stream);

/* Stages 2+3 -- tile scores, forcing, sorted top-2k and sigma
 * (A.2-A.6; Eqs. (tile-score), (sigma-def)).
 *   For every Q-tile t and query head h, the candidate blocks are the
 *   causally visible, non-forced ones C(t) = {1, ..., t-1}.  Their tile score
 *   is the maximum over the 64 rows of the tile of
 *     K-mean: q_r . kbar_b            Quest: sum_d max(q_rd kmax_bd, q_rd kmin_bd)
 *   (no 1/sqrt(d): a positive scale changes neither the order nor sigma),
 *   accumulated in fp32 from bf16 products.
 *   Q          : [B, H, N, d] bf16, 16-byte aligned.
 *   meta       : output of ugbs_block_meta for the same problem.
 *   scores_in  : NULL, or [B, H, T, N_B] fp32 tile scores that replace the
 *                computed ones (only entries in C(t) are read).
 *   scores_out : NULL, or [B, H, T, N_B] fp32; receives the tile scores,
 *                -inf outside C(t).
 *   idx_sorted : [B, H, T, 2k] int32, or NULL (sigma only).  Row (t, h) is
 *                [0] (t = 0) or [0, t], then C(t) ordered by score
 *                descending, lower block index first on equal scores
 *                (-0 == +0), cut at 2k slots and padded with the sentinel
 *                N_B.
 *   sigma      : [B, H, T] fp32.  With F the forced list and m = k - |F|:
 *                sigma = (c[m-1] - c[m]) / (c[0] - c[m]) over the sorted
 *                candidate scores c (fp32 arithmetic), 0 when the
 *                denominator is 0, and -1 when |C(t)| <= m (a saturated
 *                tile: it keeps every visible block).
 *   workspace  : needed only when scores_in and scores_out are both NULL
 *                (the tile scores then pass through it, and stay there for
 *                ugbs_attend_select): device memory of at least
 *                ugbs_workspace_bytes(p) bytes, 256-byte aligned, owned by
 *                the caller, contents on entry ignored; otherwise may be
 *                NULL.  Two calls that overlap in time must not share a
 *                workspace.
 *   Q and meta are read-only; idx_sorted/sigma/scores_out are fully written. */
UGBS_API int ugbs_score_select(const ugbs_problem* p, const void* Q, const void* meta,
                      const float* scores_in, float* scores_out,
                      int32_t* idx_sorted, float* sigma,
                      void* workspace, size_t workspace_bytes, void* stream);

/* Stage 4 -- head mean, per-layer quantile trigger and padded expansion
 * (A.7-A.9; Eq. (trigger)).
 *   The quantile population P of a sequence is the set of tiles with more
 *   candidates than kept slots (|C(t)| > k - |F(t)|; it depends only on N
 *   and k).  For t in P, sigma_bar[t] = (sum over h = 0..H-1 of sigma[t,h],
 *   fp32, in head order) / H.  With n = |P| and n_trig = ceil(q n) (computed
 *   in double on the host), tau is the n_trig-th smallest sigma_bar over P,
 *   and tile t triggers iff t in P and sigma_bar[t] <= tau (ties at tau all
 *   trigger).  kv_idx = idx_sorted, with slots k..2k-1 of every row of a
 *   tile that does not trigger overwritten by the sentinel N_B.
 *   sigma      : [B, H, T] fp32 from ugbs_score_select.
 *   idx_sorted : [B, H, T, 2k] int32, or NULL together with kv_idx (then
 *                only the statistics and trigger flags are produced).
 *   kv_idx     : [B, H, T, 2k] int32; may equal idx_sorted (in place: only
 *                the sentinel slots are written).
 *   sigma_bar  : NULL or [B, T] fp32 (-1 outside P).
 *   tau        : NULL or [B] fp32 (-1 when no tile triggers).
 *   trigger    : NULL or [B, T] uint8 (0/1).
 *   workspace  : device memory of at least ugbs_workspace_bytes(p) bytes,
 *                256-byte aligned, owned by the caller.  The route's own
 *                sections are overwritten (the trigger flags stay there for
 *                ugbs_attend_select); the packed tile scores that
 *                ugbs_score_select left there are not touched.  Two calls
 *                that overlap in time must not share a workspace. */
UGBS_API int ugbs_route(const ugbs_problem* p, const float* sigma, const int32_t* idx_sorted,
               int32_t* kv_idx, float* sigma_bar, float* tau, uint8_t* trigger,
               void* workspace, size_t workspace_bytes, void* stream);

/* Quest tile scores on the vector ALU (A.2-A.3 with Eq. (quest-score)), the
 * literal per-channel form, kept for comparison with the matrix-core
 * contraction inside ugbs_score_select (UGBS_QUEST only, else
 * UGBS_ERR_BACKBONE).  For channel c the bound term max(q_c kmax_c,
 * q_c kmin_c) is one two-element bf16 dot product (min(q_c, 0),
 * max(q_c, 0)) . (kmin_c, kmax_c), of which one product is zero; the terms
 * of a row are accumulated in fp32 in channel order and the tile score is
 * the maximum over the 64 rows.  Both forms sum exact bf16 products in
 * fp32, so they agree up to the order of the fp32 additions.
 *   Q          : [B, H, N, d] bf16, 16-byte aligned.
 *   meta       : Quest output of ugbs_block_meta for the same problem.
 *   scores_out : [B, H, T, N_B] fp32, 4-byte aligned, fully written: the
 *                tile score of every candidate of C(t) = {1..t-1}, -inf
 *                elsewhere (the layout of ugbs_score_select's scores_out). */
UGBS_API int ugbs_quest_scores_valu(const ugbs_problem* p, const void* Q, const void* meta,
                                    float* scores_out, void* stream);

/* Stage 4 for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation):
 * ugbs_route without a workspace argument.  Same arguments and results as
 * ugbs_route (every output bit-identical); the route's own sections
 * (sigma_bar | tau | trigger, each 256-byte aligned: 4 B T + 4 B + B T bytes
 * rounded up) live in a static device array of UGBS_ROUTE_SCRATCH_BYTES
 * (1 MiB) that the library holds on each GPU it runs on until the process
 * ends; any batch up to 64 at every supported N fits.  A problem whose
 * sections exceed it returns UGBS_ERR_SCRATCH before anything is enqueued.
 * The call allocates nothing (no hipMalloc, no allocating library routine);
 * on its first call on a device it looks up that device's copy of the array
 * (the current device, which `stream` must belong to).
 *   - Every call on a GPU shares that GPU's array, which keeps the last
 *     call's contents; calls that overlap in time on one GPU (other streams,
 *     other host threads) race on it and must be ordered by the caller.
 *   - The array is written in full for the problem's sections before it is
 *     read, so no clearing is needed between calls.
 *   - The trigger flags stay in the library's array, not in a caller
 *     workspace: a following ugbs_attend_select takes them through its
 *     `trigger` argument (pass this call's `trigger` output).
 * With ugbs_score_select given scores_out (no workspace needed), a layer
 * runs without any workspace: block_meta, score_select, route_noalloc,
 * attend. */
UGBS_API int ugbs_route_noalloc(const ugbs_problem* p, const float* sigma, const int32_t* idx_sorted,
                                int32_t* kv_idx, float* sigma_bar, float* tau, uint8_t* trigger,
                                void* stream);

/* Stage 5 -- block-sparse causal attention over kv_idx (A.10; Eq. (Attn)).
 *   For row i of tile t and query head h, the attended keys are
 *   J_i = { j <= i : block(j) is listed in kv_idx[b, h, t, :] } and
 *   O_i = sum_{j in J_i} softmax_j(scale * q_i . k_j) v_j, computed with bf16
 *   products, fp32 accumulation and an fp32 online softmax.  Entries outside
 *   [0, N_B) (the sentinel N_B included) and blocks after t are skipped, and
 *   a block listed twice counts once (the row is a set, as in J_i).  A row
 *   with no attended key gives O = 0.
 *   kv_idx with every block 0..t listed (kv_width = N_B) is dense causal
 *   attention.
 *   Q, K, V : as in the conventions above, 16-byte aligned.
 *   kv_idx  : [B, H, T, kv_width] int32, 4-byte aligned.
 *   kv_width: 1 <= kv_width <= UGBS_MAX_KV_WIDTH (2k for the pipeline).
 *   O       : [B, H, N, d] bf16, 16-byte aligned; fully written. */
UGBS_API int ugbs_attend(const ugbs_problem* p, const void* Q, const void* K, const void* V,
                const int32_t* kv_idx, int32_t kv_width, void* O, void* stream);

/* ---- Diagnostics (Appendix D) ----------------------------------------------
 * With F(t) the forced list, m = k - |F| kept candidates and
 * R' = rho k - |F| candidates after expansion (rho = 2), a tile enters the
 * diagnostics when |C(t)| >= R' + 1 (at least rho k + 1 visible blocks, the
 * paper's diagnostic mask).  For such a tile, with c the candidate scores
 * sorted as in ugbs_score_select (descending, lower block first on ties):
 *   g = c[m-1] - c[m], G = c[m-1] - c[R'], r = c[0] - c[m]   (Eq. (gaps))
 *   sigma = g / r (0 when r == 0), all fp32 subtract / IEEE divide. */
typedef struct ugbs_bai_tile {
  float g, G, r, sigma;
  float delta2;     /* min over j = 0..R'-1, j != m-1, of c[j] - c[j+1]: the
                       smallest secondary spacing, assumption (A1) */
  int32_t fail_k;   /* Monte Carlo samples in which the empirical top-m set
                       misses the true top-m of mu (see ugbs_bai_tiles) */
  int32_t fail_rk;  /* samples in which the empirical top-R' set misses it */
  int32_t valid;    /* 1 if the tile is in the diagnostic mask; otherwise 0,
                       the floats NaN and the counts 0 */
} ugbs_bai_tile;

/* Per (batch, head) aggregates over the n_tiles valid tiles of a sequence
 * (the empirical recipe of Appendix D).  Fields that are undefined for a
 * head (no valid tile; n_q = 0; tau not positive; n_samples = 0) are NaN. */
typedef struct ugbs_bai_head {
  int32_t n_tiles;     /* valid tiles n */
  int32_t n_q;         /* ceil(q n), the router's trigger count */
  int32_t pad[2];
  double r_mean;       /* mean of r (left-to-right fp64 sum in tile order) / n */
  double r_cv;         /* sqrt(mean (r - r_mean)^2) / r_mean: the proxy for beta in (A2) */
  double sigma_q;      /* the n_q-th smallest sigma (lower tile first on ties) */
  double gamma_q;      /* sigma_q * r_mean */
  double band_mass;    /* fraction of tiles with g in [gamma_q (1-beta), gamma_q (1+beta)] */
  double delta2_p05;   /* delta2 at sorted position floor(0.05 (n-1)): the Delta_2 used */
  double delta2_p50;   /* delta2 at sorted position floor(0.5 (n-1)) */
  double pi2;          /* fraction of tiles with delta2 < delta2_p05 (the pi_2 term) */
  double tau;          /* the noise scale used, as given */
  double chi;          /* sum_{j>=1} (j+1) exp(-j^2 Delta_2^2 / (4 tau^2)); +inf when
                          Delta_2 <= 0 or more than 1e6 terms are needed */
  double eps_bar;      /* chi + (1 + chi) exp(-((rho-1) k Delta_2)^2 / (4 tau^2)) */
  double vbar_gamma;   /* Vbar(gamma_q) = Phi(-gamma_q / (sqrt2 tau)) */
  double C_q;          /* min{1, (1+eps_bar)/2, sqrt2 beta gamma_q / tau
                          phi(gamma_q (1-beta) / (sqrt2 tau)) + eps_bar} */
  double bound;        /* min(q, 1-q) C_q + pi2 (the Proposition, with pi_2) */
  double bound_band;   /* band_mass / 2 C_q + pi2 */
  double mc_err_k;     /* sum fail_k / (n n_samples) */
  double mc_err_rk;    /* sum fail_rk / (n n_samples) */
  double mc_regret;    /* R_q: with V = (fail_k - fail_rk) / n_samples per tile,
                          (sum of the n_q largest V - sum of V over the router's
                          n_q tiles) / n */
} ugbs_bai_head;

/* Noise scale tau from row-to-row score differences (Appendix D, empirical
 * recipe step 3): adjacent query rows of a tile see the same block, so the
 * difference of their scores carries two independent noise draws and
 * E[(s[r+1,b] - s[r,b])^2] = 2 tau^2.
 *   rough : [B, H, T] fp64, 8-byte aligned, fully written.  For tile t:
 *           the sum over candidate blocks b in C(t) = {1..t-1} and the 63
 *           adjacent row pairs (r, r+1) of (s[r+1,b] - s[r,b])^2, where s is
 *           the per-row block score of ugbs_score_select (before the max over
 *           rows), fp32 scores and squares, fp64 accumulation; 0 for t < 2.
 *   tau   : [B, H] fp32, fully written: sqrt(sum_t rough / (2 * 63 *
 *           (T-1)(T-2)/2)), NaN when T < 3.
 *   Q, meta as for ugbs_score_select. */
UGBS_API int ugbs_noise_scale(const ugbs_problem* p, const void* Q, const void* meta,
                              double* rough, float* tau, void* stream);

/* Per-tile gaps and Monte Carlo identification failures (N_B <=
 * UGBS_MAX_BLOCKS_ROWS, else UGBS_ERR_SHAPE).
 *   scores    : [B, H, T, N_B] fp32 tile scores in the layout of
 *               ugbs_score_select's scores_out (entries of C(t) are read).
 *   tau       : [B, H] fp32 noise scale; may be NULL when n_samples == 0.
 *   z         : [N_B, n_samples] fp32 standard normals shared by all tiles
 *               and heads, block-major (draw s of block b at z[b * n_samples
 *               + s]); may be NULL when n_samples == 0.
 *   n_samples : 0 <= n_samples <= 1 << 20.
 *   tiles     : [B, H, T] ugbs_bai_tile, 8-byte aligned, fully written.
 * For sample s the perturbed scores are mu_b = fp32(c_b + fp32(tau z[b, s]))
 * over b in C(t) (c_b with -0 read as +0).  fail_k counts the samples where
 * NOT (min of mu over the empirical top-m > max of mu over the other
 * candidates); fail_rk the samples where fewer than m members of the
 * empirical top-R' exceed every other candidate's mu. */
UGBS_API int ugbs_bai_tiles(const ugbs_problem* p, const float* scores, const float* tau,
                            const float* z, int32_t n_samples, ugbs_bai_tile* tiles, void* stream);

/* Per-head aggregates (ugbs_bai_head) from the tiles of ugbs_bai_tiles (N_B <=
 * UGBS_MAX_BLOCKS_ROWS, else UGBS_ERR_SHAPE); q and
 * k_budget come from p.
 *   tiles     : [B, H, T] from ugbs_bai_tiles for the same problem.
 *   tau       : [B, H] fp32, the noise scale for the closed forms.
 *   n_samples : the value passed to ugbs_bai_tiles.
 *   heads     : [B, H] ugbs_bai_head, 8-byte aligned, fully written. */
UGBS_API int ugbs_bai_heads(const ugbs_problem* p, const ugbs_bai_tile* tiles, const float* tau,
                            int32_t n_samples, ugbs_bai_head* heads, void* stream);

/* Stage 5 with the selection inside the attention kernel (the block
 * selection fused into attention that the Limitations of Section 4 list as
 * engineering work left open): the same output as ugbs_attend
 * on the kv_idx of ugbs_route, without materialising kv_idx.  For every
 * unit (b, h, t) the attended blocks are the forced ones, [0] or [0, t],
 * and the R best candidates of C(t) by (score descending, lower block
 * first, -0 == +0), R = (trigger[b, t] ? 2k : k) - |F|, or all of C(t) when
 * it has at most R; the attention is then as in ugbs_attend (the blocks are
 * visited in the same order, so the two entry points agree bit for bit).
 *   scores   : NULL, or [B, H, T, N_B] fp32 tile scores (entries of C(t)
 *              are read).  NULL: the packed scores that ugbs_score_select
 *              (without scores_in / scores_out) left in `workspace`.
 *   trigger  : NULL, or [B, T] uint8 flags (nonzero = expanded).  NULL: the
 *              flags ugbs_route left in `workspace`.
 *   workspace: needed when scores or trigger is NULL: the workspace of the
 *              ugbs_score_select and ugbs_route calls of the same problem,
 *              issued before this one on the stream.
 *   Q, K, V, O as for ugbs_attend. */
UGBS_API int ugbs_attend_select(const ugbs_problem* p, const void* Q, const void* K, const void* V,
                                const float* scores, const uint8_t* trigger,
                                const void* workspace, size_t workspace_bytes, void* O,
                                void* stream);

/* Per-row selection scattered into tile bitmaps (N_B <= UGBS_MAX_BLOCKS_ROWS,
 * else UGBS_ERR_SHAPE; the per-row variant the
 * Limitations of Section 4 name for the per-tile granularity of Section
 * 3.2).  Every query row r of tile t ranks the candidates C(t) = {1..t-1}
 * by its own score (A.2 before the max over rows: K-mean q_r . kbar_b,
 * Quest sum_d max(q_rd kmax_bd, q_rd kmin_bd); bf16 products, fp32 sums)
 * and keeps the forced blocks [0] or [0, t] and its R best candidates by
 * (score descending, lower block first, -0 == +0), R = (trigger[b, t] ?
 * rho k : k) - |F|, all of C(t) when it has at most R.  The tile's set is
 * the union over its 64 rows.
 *   Q, meta    : as for ugbs_score_select; may be NULL with row_scores.
 *   row_scores : NULL, or [B, H, N, N_B] fp32 per-row scores that replace the
 *                computed ones (entries of C(t) for the rows of tile t are read).
 *   trigger    : [B, T] uint8 flags (nonzero = expanded), e.g. ugbs_route's;
 *                all zero for plain per-row top-k.
 *   bitmap     : [B, H, T, ceil(N_B / 32)] uint32, fully written: bit b % 32
 *                of word b / 32 is set when block b is in the tile's set
 *                (blocks after t never are). */
UGBS_API int ugbs_select_rows(const ugbs_problem* p, const void* Q, const void* meta,
                              const float* row_scores, const uint8_t* trigger, uint32_t* bitmap,
                              void* stream);

/* Stage 5 over tile bitmaps: as ugbs_attend with the set of blocks of tile
 * (b, h, t) given by the set bits of bitmap[b, h, t, :] (bits of blocks
 * after t are ignored).
 *   bitmap : [B, H, T, ceil(N_B / 32)] uint32, 4-byte aligned. */
UGBS_API int ugbs_attend_bitmap(const ugbs_problem* p, const void* Q, const void* K, const void* V,
                                const uint32_t* bitmap, void* O, void* stream);

/* Bytes of device workspace ugbs_score_select (without scores_in/scores_out),
 * ugbs_route and ugbs_attend_select need for problem p; one workspace
 * serves the calls of a layer in sequence on a stream (0 if p is invalid).
 * It holds the route's sections (B T fp32 + B fp32 + B T bytes, each
 * 256-byte aligned), then B H (T-1)(T-2)/2 fp32 packed candidate scores. */
UGBS_API size_t ugbs_workspace_bytes(const ugbs_problem* p);

/* Static, human-readable text for a ugbs_status value. */
UGBS_API const char* ugbs_status_string(int status);

/* UGBS_ABI_VERSION of the loaded library. */
UGBS_API int ugbs_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* UGBS_H */
