/*
 * hwsel.h -- C ABI of the batched candidate-scoring library for MI355X (gfx950).
 *
 * The library ranks GEMM kernel configurations without running them, as in
 * "Hardware-Aware Features for CUTLASS Kernel Selection": every
 * (problem p, candidate c) row gets a statically computed feature vector
 * x = phi(p, c, h) for a target hardware description h; a learned scorer
 * f maps rows to scores; the deployed choice per problem is the
 * highest-scoring candidate; the choice is judged by its selection regret.
 *
 * Conventions for every entry point
 *   - Array arguments are DEVICE pointers (memory of the current HIP device)
 *     unless the comment says "host".  The caller owns every buffer; the
 *     library allocates nothing, frees nothing and keeps no device state
 *     (one exception: the scratch array of hwsel_evaluate_noalloc).
 *   - `stream` is a hipStream_t passed as void*; NULL is the null stream.
 *     Calls only enqueue work on it: they return before the work finishes and
 *     never synchronise.
 *   - Arguments are checked on the host before anything is enqueued.  A
 *     rejected call returns a non-zero status, enqueues nothing and records a
 *     message readable with hwsel_last_error() (per thread).  Device-resident
 *     contents (offsets, indices, knob values) cannot be checked without a
 *     synchronisation; each call states what it assumes of them and what the
 *     kernels do when the assumption is broken (they never read or write out
 *     of the stated bounds).
 *   - All entry points are thread-safe.
 */
#ifndef HWSEL_H
#define HWSEL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    HWSEL_OK = 0,
    HWSEL_EINVAL = 1,       /* a null pointer, a size out of range, misalignment */
    HWSEL_EUNSUPPORTED = 2, /* a valid request the library does not implement */
    HWSEL_EHIP = 3          /* the HIP runtime reported an error at launch */
} hwsel_status;

/* Integer codes used in problem and candidate records. */
enum { HWSEL_LAYOUT_TN = 0, HWSEL_LAYOUT_TT = 1, HWSEL_LAYOUT_NN = 2, HWSEL_LAYOUT_NT = 3 };
enum { HWSEL_DTYPE_BF16 = 0, HWSEL_DTYPE_FP16 = 1, HWSEL_DTYPE_FP8 = 2, HWSEL_DTYPE_FP32 = 3 };
enum { HWSEL_KS_WS = 0, HWSEL_KS_PINGPONG = 1, HWSEL_KS_COOPERATIVE = 2 };
enum { HWSEL_ES_NOSMEM = 0, HWSEL_ES_TMA = 1, HWSEL_ES_TMA_COOPERATIVE = 2 };
enum { HWSEL_TS_PERSISTENT = 0, HWSEL_TS_STREAMK = 1 };

/*
 * Hardware descriptor h of the TARGET the ranked kernels would run on
 * (section "Structural Core": SM count, shared-memory and register-file
 * capacity per SM, LLC capacity, HBM bandwidth, peak throughput of the
 * compute engine).  Exact integers in fixed units: bytes, GB/s (= bytes per
 * ns), GFLOP/s (= flop per ns).  peak_gflops is indexed by the input dtype
 * code (bf16, fp16, fp8).  Passed by value.  Every field must be >= 1 except
 * smem_reserved (>= 0); hwsel_features rejects other values.
 */
typedef struct hwsel_hw {
    int64_t n_sm, smem_per_sm, smem_per_block_max, smem_reserved;
    int64_t regs_per_sm, max_regs_per_thread, max_blocks_per_sm, max_threads_per_sm;
    int64_t arch_id, llc_bytes, hbm_bw_gbps;
    int64_t peak_gflops[3];
} hwsel_hw_t;

/*
 * GEMM problem p = (M, N, K, layout) with its input dtype (section "Problem
 * and Candidate Sets").  The layout tag names the storage of A, then of B,
 * as in the printed kernel's TN = A row-major, B column-major: NN and NT
 * have A column-major; TT and NT have B row-major.  16 bytes per record,
 * array-of-structs on the device.
 */
typedef struct hwsel_problem {
    int32_t M, N, K;
    uint8_t layout, dtype, pad[2];
} hwsel_problem_t;

/*
 * Candidate configurations c, one row each, as a struct of DEVICE arrays of
 * length R (section "Configuration Space", Table "Configuration knobs"):
 * tile shape (T_M, T_N, T_K), instruction tile (16*inst_m_div16, inst_n,
 * inst_k), pipeline stages, cluster (C_M, C_N), swizzle, mainloop schedule,
 * epilogue schedule and tile scheduler codes.  The struct itself is read on
 * the host.  Knob values of 0 are read as 1; schedule codes beyond the last
 * one are read as the last one.
 */
typedef struct hwsel_cands {
    const uint16_t *tile_m, *tile_n, *tile_k, *inst_n;
    const uint8_t *stages, *cluster_m, *cluster_n, *swizzle, *inst_m_div16, *inst_k;
    const uint8_t *kernel_sched, *epi_sched, *tile_sched;
} hwsel_cands_t;

/*
 * Features.  X[r][0..n_features) = phi(p(r), c_r, h) for every row r < R,
 * where p(r) is the problem whose segment [seg_offsets[p], seg_offsets[p+1])
 * holds r (section "Feature Map", Table "Feature groups", and the formulas of
 * "Work Decomposition and Wave Quantization", "Memory Behavior", "Resource
 * Pressure and Occupancy", "Pipeline Balance").  n_features is 64, 96 or 128;
 * the 96- and 128-column schemas extend the 64-column one.
 *
 *   problems     [P] records; M, N, K below 1 are read as 1.
 *   seg_offsets  [P+1] int64, non-decreasing, seg_offsets[0] = 0,
 *                seg_offsets[P] = R (assumed; a row outside every segment is
 *                assigned to the nearest one, never read out of bounds).
 *   X            fp32, row-major, leading dimension ld >= n_features,
 *                ld % 4 == 0, 16-byte aligned.
 * Integer-valued columns are exact integers rounded once to fp32; ratio
 * columns are one binary64 division of exact integers rounded to fp32; the
 * log2 columns are binary64 log2 rounded to fp32.
 * Returns HWSEL_EINVAL for null pointers, P < 1, R < 1, a bad ld or alignment
 * or hardware field; HWSEL_EUNSUPPORTED for another n_features.
 */
int hwsel_features(hwsel_hw_t hw, const hwsel_problem_t *problems, int32_t P,
                   const int64_t *seg_offsets, const hwsel_cands_t *cands, int64_t R,
                   int32_t n_features, float *X, int64_t ld, void *stream);

/*
 * Additive tree ensemble f(x) = base_score + sum_t leaf_t(x) (section
 * "Model A (gradient-boosted ranker)").  n_trees perfect binary trees of the
 * same depth, stored breadth-first per tree: internal node i (0-based) has
 * children 2i+1 (left) and 2i+2 (right); a row goes left iff
 * x[node_feature] < node_threshold, or x is NaN and flags bit 0 is set.
 * Device arrays: node_feature uint8 [n_trees][2^depth - 1] (values must be
 * < n_features; larger ones are read as n_features - 1), node_threshold fp32
 * [n_trees][2^depth - 1], leaf_value fp32 [n_trees][2^depth].
 * The struct itself is read on the host.
 */
typedef struct hwsel_forest {
    int32_t n_trees, depth, n_features;
    uint32_t flags;                /* bit 0: NaN goes left */
    float base_score;
    const uint8_t *node_feature;
    const float *node_threshold;
    const float *leaf_value;
} hwsel_forest_t;

/*
 * Packing: a one-time conversion of a forest into the layout the fast scorer
 * reads (per-feature sorted distinct thresholds, u8 threshold ranks, trees
 * grouped into LDS-sized chunks, see the exact-binning identity in
 * forest.hip).  hwsel_forest_pack reads the forest's device arrays, builds
 * the image on the host and writes `bytes` = hwsel_forest_pack_bytes() bytes
 * to `packed` (device, 16-byte aligned).  It synchronises `stream` (a model
 * is packed once, at load time).  Returns HWSEL_EUNSUPPORTED when a feature
 * has more than 255 distinct thresholds, depth > 10 or n_features > 128 (the
 * unpacked path covers those), HWSEL_EINVAL for a node feature >=
 * n_features or a NaN threshold.
 */
int hwsel_forest_pack_bytes(const hwsel_forest_t *f, size_t *bytes);
int hwsel_forest_pack(const hwsel_forest_t *f, void *packed, size_t bytes, void *stream);
/* The same image built from a forest whose arrays (node_feature,
 * node_threshold, leaf_value) are in HOST memory, written to `image` (host
 * memory of hwsel_forest_pack_bytes() bytes); no HIP call is made, so it
 * runs on a machine without a GPU.  Copy the image to device memory (16-byte
 * aligned) to score with it.  Same status codes as hwsel_forest_pack. */
int hwsel_forest_pack_host(const hwsel_forest_t *f, void *image, size_t bytes);

/* Device workspace (bytes) hwsel_forest_score needs for a packed forest and
 * R rows: u8 bins [R][n_features rounded up to 16] and one fp32 partial sum
 * per tree chunk and row. */
int hwsel_forest_workspace_bytes(const hwsel_forest_t *f, int64_t R, size_t *bytes);

/*
 * scores[r] = f(X[r]) for r < R, accumulated in fp32 in a fixed order (the
 * same inputs give bit-identical scores from run to run).
 *   X: fp32 [R][ld], ld >= n_features, as written by hwsel_features.
 *   packed: NULL for the direct tree walk, or the image hwsel_forest_pack
 *     wrote for this very forest (an image of another shape gives NaN
 *     scores; one of the same shape but other values is not detected); then
 *     `workspace` must hold
 *     hwsel_forest_workspace_bytes(f, R) bytes (device, 256-byte aligned).
 * Returns HWSEL_EINVAL for null pointers, R < 1, n_trees < 1, ld <
 * n_features, a short or misaligned workspace; HWSEL_EUNSUPPORTED for depth
 * outside [1, 12] or n_features outside [1, 256] (and for a packed call on a
 * forest hwsel_forest_pack does not accept).
 */
int hwsel_forest_score(const hwsel_forest_t *f, const void *packed, const float *X, int64_t R, int64_t ld,
                       float *scores, void *workspace, size_t workspace_bytes, void *stream);

/*
 * hwsel_forest_score (packed path only) with check outputs of the same
 * traversal kernels: the scores are bit-identical to hwsel_forest_score's.
 *   leaf_hash  uint64 [R] (nullable, 8-byte aligned): each row's leaf-path
 *              fingerprint, the wrapping 64-bit sum over trees t of
 *              mix(t * 2^32 + leaf_t), with leaf_t the index in [0, 2^depth)
 *              of the leaf the row reaches in tree t and mix the 64-bit
 *              finaliser of SplitMix64 (Steele, Lea, Flood, OOPSLA 2014).
 *              One changed leaf always changes it; tree order does not.
 *   leaf_idx   uint16 [leaf_rows][n_trees] (nullable): leaf_idx[i][t] =
 *              leaf_t of row leaf_row0 + i, for rows [leaf_row0, leaf_row0 +
 *              leaf_rows) within [0, R).
 * For a packed image whose stored shape (trees, depth, features, chunking)
 * differs from the forest's, every score is NaN and nothing else is written
 * (hwsel_forest_score does the same).
 * Returns the status codes of hwsel_forest_score, and HWSEL_EINVAL for a
 * NULL packed image, a misaligned leaf_hash or a row range outside [0, R).
 */
int hwsel_forest_score_checked(const hwsel_forest_t *f, const void *packed, const float *X, int64_t R, int64_t ld,
                               float *scores, void *workspace, size_t workspace_bytes, uint64_t *leaf_hash,
                               uint16_t *leaf_idx, int64_t leaf_row0, int64_t leaf_rows, void *stream);

/*
 * Leaf index of every tree for selected rows: leaf_idx[i][t] = index in
 * [0, 2^depth) of the leaf that row rows[i] reaches in tree t.  A check
 * hook for the traversal (same decision rule as hwsel_forest_score).
 *   rows: int64 [n_rows] (values must lie in [0, R); others are clamped).
 * Same status codes as hwsel_forest_score.
 */
int hwsel_forest_leaves(const hwsel_forest_t *f, const float *X, int64_t R, int64_t ld,
                        const int64_t *rows, int64_t n_rows, uint16_t *leaf_idx, void *stream);

/*
 * Feed-forward ranker (section "Model B (feed-forward ranker)") with widths
 * 128 -> 512 -> 512 -> 256 -> 1 and GELU hidden activations:
 *   h0 = bf16((clean(x) - mean) * inv_std)   (fp32, two operations; clean maps
 *                                            NaN and +-inf to 0)
 *   h_l = bf16(GELU(W_l h_{l-1} + b_l)), l = 1..3, fp32 accumulation
 *   score = W4 h3 + b4 in fp32.
 * GELU(a) = a Phi(a) (the erf form).  The row-block kernel evaluates it with
 * erff; the matrix-core kernel with a fitted approximation whose absolute
 * error is below 1e-6 for every finite a (exactly max(a, 0) for |a| >= 20).
 * Device arrays: mean, inv_std fp32 [128]; W1 [512][128], W2 [512][512],
 * W3 [256][512], W4 [1][256] as bf16 bit patterns (uint16), row-major
 * [out][in]; b1..b4 fp32.  The struct itself is read on the host.
 */
typedef struct hwsel_mlp {
    int32_t n_in, h1, h2, h3;
    const float *mean, *inv_std;
    const uint16_t *W1, *W2, *W3, *W4;
    const float *b1, *b2, *b3, *b4;
} hwsel_mlp_t;

/*
 * Packing: a one-time rearrangement of W1..W3 into the fragment order of the
 * bf16 matrix-core instructions (asynchronous on `stream`; the weights must
 * not change until it has run).  `packed` is device memory of
 * hwsel_mlp_pack_bytes() bytes, 16-byte aligned.  Returns HWSEL_EINVAL for
 * null pointers or a short buffer, HWSEL_EUNSUPPORTED for other widths.
 */
int hwsel_mlp_pack_bytes(const hwsel_mlp_t *m, size_t *bytes);
int hwsel_mlp_pack(const hwsel_mlp_t *m, void *packed, size_t bytes, void *stream);

/*
 * scores[r] = MLP(X[r][0..128)) for r < R.  X: fp32 [R][ld], ld >= 128,
 * ld % 4 == 0, 16-byte aligned.  packed: NULL for the fp32-FMA row-block
 * kernel, or the image hwsel_mlp_pack wrote for these weights (matrix-core
 * kernel; mean, inv_std and b1..b3 must then be 16-byte aligned and W4
 * 8-byte aligned).  Returns HWSEL_EINVAL for null pointers, R < 1, bad
 * ld/alignment; HWSEL_EUNSUPPORTED for other widths.
 */
int hwsel_mlp_score(const hwsel_mlp_t *m, const void *packed, const float *X, int64_t R, int64_t ld,
                    float *scores, void *stream);

/*
 * Per-problem selection, eq. (selection) generalised to the k best:
 * idx[p][j] = local index (0-based within segment p) of the candidate ranked
 * j-th by score descending, ties broken by the lower index; -0 equals +0;
 * NaN ranks below -inf.  Segments with fewer than k rows are padded with
 * index -1 and value -inf.  vals (nullable) receives the scores.
 *   scores [R] fp32 with R = seg_offsets[P]; idx int32 [P][k]; vals fp32 [P][k].
 *   seg_offsets as for hwsel_features (segments longer than 2^31 - 1 rows are
 *   not supported).
 * Returns HWSEL_EINVAL for null pointers, P < 1, k outside [1, 64].
 */
int hwsel_topk_per_problem(const float *scores, const int64_t *seg_offsets, int32_t P, int32_t k,
                           int32_t *idx, float *vals, void *stream);

/*
 * Selection regret, eq. (regret): within a problem the flop count is fixed,
 * so T(c) / T_best = t_best / t(c) for runtimes t.  For each problem p:
 *   t_best          = min runtime of the segment,
 *   regret_top1[p]  = 1 - t_best / t(idx[p][0])          (binary64, then fp32),
 *   regret_bestk[p] = 1 - t_best / min_j t(idx[p][j])    (nullable),
 *   best_idx[p]     = local index of t_best, lowest on ties (nullable).
 * Equal runtimes (inf included) give exactly 0; NaN runtimes rank above +inf
 * and a pick whose runtime is NaN (a kernel that never finishes, T = 0) gives
 * exactly 1, as in hwsel_evaluate; an empty segment or a -1 pick gives NaN,
 * and an empty segment best_idx -1.
 *   runtimes [R] fp32 (seconds), idx int32 [P][k] as from
 *   hwsel_topk_per_problem (entries outside [-1, segment length) are read as
 *   -1).
 * Returns HWSEL_EINVAL for null pointers, P < 1, k outside [1, 64].
 */
int hwsel_regret(const float *runtimes, const int64_t *seg_offsets, int32_t P, const int32_t *idx,
                 int32_t k, float *regret_top1, float *regret_bestk, int32_t *best_idx,
                 void *stream);

/*
 * Fused selection with a packed forest, the scored path in one call (section
 * "Problem Formulation": features, scorer, per-problem argmax generalised to
 * the k best) without materialising the feature matrix: each row's feature
 * vector phi(p, c, h) (n_features columns) is binned against the forest's
 * thresholds as it is computed, the bins are scored, and the scores go to
 * the per-problem top-k.  idx, vals and scores are bit-identical to
 * hwsel_features -> hwsel_forest_score (with `packed`) ->
 * hwsel_topk_per_problem on the same inputs.
 *   Inputs as for hwsel_features and hwsel_forest_score; f->n_features must
 *   be <= n_features.  idx int32 [P][k], vals fp32 [P][k] (nullable), scores
 *   fp32 [R] (nullable); workspace of hwsel_select_forest_workspace_bytes(f,
 *   R) bytes (device, 256-byte aligned).
 * Returns the status codes of those calls, and HWSEL_EINVAL when
 * f->n_features > n_features.
 */
int hwsel_select_forest_workspace_bytes(const hwsel_forest_t *f, int64_t R, size_t *bytes);
int hwsel_select_forest(hwsel_hw_t hw, const hwsel_problem_t *problems, int32_t P, const int64_t *seg_offsets,
                        const hwsel_cands_t *cands, int64_t R, int32_t n_features, const hwsel_forest_t *f,
                        const void *packed, int32_t k, int32_t *idx, float *vals, float *scores, void *workspace,
                        size_t workspace_bytes, void *stream);

/*
 * Linear ridge scorer (section "Linear Ridge Baseline", eq. ridge-loss):
 *   f(x) = bias + sum over numeric columns j of w[j] * z_j
 *              + sum over categorical columns of w_onehot[slot of its level],
 *   z_j  = (clean(x_j) - mean[j]) * inv_std[j]   (fp32, two operations; clean
 *                                                 maps NaN and +-inf to 0).
 * The categorical columns are the layout and schedule fields, one-hot
 * encoded with frozen level sets: column 64 (layout, levels 0..3, slots
 * 0..3), 73 (mainloop schedule, 0..2, slots 4..6), 74 (epilogue schedule,
 * 0..2, slots 7..9), 75 (tile scheduler, 0..1, slots 10..11); they exist for
 * n_features 96 and 128.  A value that is not one of its column's levels
 * encodes to all zeros (adds nothing).  The terms are accumulated in fp32 in a
 * fixed order.  Device arrays: mean, inv_std, w fp32 [n_features] (w of a
 * categorical column is not read), w_onehot fp32 [HWSEL_ONEHOT_SLOTS].  The
 * struct itself is read on the host.
 */
#define HWSEL_ONEHOT_SLOTS 12
typedef struct hwsel_linear {
    int32_t n_features;            /* 64, 96 or 128 */
    float bias;
    const float *mean, *inv_std, *w, *w_onehot;
} hwsel_linear_t;

/*
 * scores[r] = f(X[r]) for r < R.  X: fp32 [R][ld], ld >= n_features,
 * ld % 4 == 0, 16-byte aligned (as written by hwsel_features).
 * Returns HWSEL_EINVAL for null pointers, R < 1, a bad ld or alignment;
 * HWSEL_EUNSUPPORTED for another n_features.
 */
int hwsel_linear_score(const hwsel_linear_t *lin, const float *X, int64_t R, int64_t ld, float *scores,
                       void *stream);

/*
 * The analytic sampling score of section "Candidate Sampling" as a model-free
 * scorer: scores[r] = n_c / (W S_SM c_M c_N) * S * sqrt(T_M T_N T_K) with n_c
 * clusters, S_SM = max(1, floor(n_sm / (c_M c_N))) cluster slots and
 * W = ceil(n_c / S_SM) cluster waves; the same binary64 sequence, and so the
 * same fp32 value, as feature column 58 of hwsel_features, without writing
 * the feature matrix.  Arguments and status codes as for hwsel_features
 * (scores fp32 [R] replaces X, n_features and ld).
 */
int hwsel_sample_score(hwsel_hw_t hw, const hwsel_problem_t *problems, int32_t P, const int64_t *seg_offsets,
                       const hwsel_cands_t *cands, int64_t R, float *scores, void *stream);

/*
 * Selection metrics over problems (section "Selection Regret (The Target
 * Metric)") and the uniform-random baseline (section "Final Fit and Test
 * Protocol").  With y(p,c) = t_best / t_c (1 when t_c == t_best, 0 for a NaN
 * runtime, read as never finishing, also when every runtime is NaN), for each
 * problem p whose segment is non-empty and whose pick c_hat = idx[p][0] is a
 * valid local index ("counted" problems):
 *   regret[p] = 1 - y(p, c_hat)                       binary64
 *   rank[p]   = 1 + #{c : t_c < t(c_hat)}             minimum-rank ties, NaN
 *                                                      slowest; 0 if not counted
 *   ybar[p]   = mean_c y(p, c)                         binary64, NaN if empty
 * and over counted problems, in problem order, binary64:
 *   out[0] mean regret, out[1] median, out[2] 95th percentile, out[3] max,
 *   out[4] Top1 = share with rank 1, out[5] Top5 = share with rank <= 5,
 *   out[6] Within5% = share with regret <= 0.05, out[7] mean of 1 - ybar
 *   (expected regret of a uniform pick), out[8] number of counted problems.
 * Percentiles interpolate linearly between order statistics at position
 * q (n - 1).  With no counted problem out[0..7] are NaN and out[8] is 0.
 * ybar and out[7] are sums whose order differs from a sequential sum; every
 * other output is exact.
 *   runtimes fp32 [R]; seg_offsets [P+1] as for hwsel_features; idx int32
 *   [P][k] as from hwsel_topk_per_problem; out fp64 [HWSEL_EVAL_FIELDS];
 *   regret, rank, ybar [P] (each nullable); workspace of
 *   hwsel_evaluate_workspace_bytes(P) bytes (device, 256-byte aligned).
 * Returns HWSEL_EINVAL for null pointers, P < 1, k outside [1, 64], a short
 * or misaligned workspace.
 */
#define HWSEL_EVAL_FIELDS 9
int hwsel_evaluate_workspace_bytes(int32_t P, size_t *bytes);
int hwsel_evaluate(const float *runtimes, const int64_t *seg_offsets, int32_t P, const int32_t *idx, int32_t k,
                   double *out, double *regret, int32_t *rank, double *ybar, void *workspace,
                   size_t workspace_bytes, void *stream);

/*
 * hwsel_evaluate for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops and harnesses that forbid hipMalloc): no
 * workspace argument, and no allocation of any kind.  The same kernels
 * compute the same outputs, bit for bit, as hwsel_evaluate; the per-problem
 * intermediates live in a device array of the library's code object
 * (HWSEL_EVAL_NOALLOC_SCRATCH_BYTES = 1,835,008 bytes per device, held until
 * the process ends), whose address is looked up once per device, on the
 * first call made with that device current.  All calls on one device share
 * that array: calls that overlap on one device (streams or threads without
 * an order between them) race and their results are undefined.  Nothing
 * carries over from one call to the next.
 *   Arguments as for hwsel_evaluate; P <= HWSEL_EVAL_NOALLOC_MAX_P.
 * Returns HWSEL_EINVAL as hwsel_evaluate does and for P >
 * HWSEL_EVAL_NOALLOC_MAX_P; HWSEL_EHIP when the array's address cannot be
 * looked up or a launch fails.
 */
#define HWSEL_EVAL_NOALLOC_MAX_P 65536
#define HWSEL_EVAL_NOALLOC_SCRATCH_BYTES 1835008
int hwsel_evaluate_noalloc(const float *runtimes, const int64_t *seg_offsets, int32_t P, const int32_t *idx,
                           int32_t k, double *out, double *regret, int32_t *rank, double *ybar, void *stream);

/*
 * Best static configuration (baseline of section "Final Fit and Test
 * Protocol"): among configuration ids that appear in at least 80% of the P
 * problems (5 * count >= 4 * P), the one with the highest mean y over the
 * problems it appears in (y as for hwsel_evaluate; summed in problem order,
 * binary64); ties go to the lower id.  Within a problem only the first row
 * (lowest local index) of an id counts; ids outside [0, n_configs) are
 * ignored.  Results (device): best[0] = id or -1 if none qualifies, best[1] =
 * its problem count, mean_y[0] = its mean y (NaN if none); its mean regret is
 * 1 - mean_y.
 *   config_id int32 [R]: the identity of each row's configuration (e.g. its
 *   catalogue index); workspace of hwsel_static_config_workspace_bytes(P,
 *   n_configs) bytes (device, 256-byte aligned).
 * Returns HWSEL_EINVAL for null pointers, P < 1, n_configs < 1, a short or
 * misaligned workspace.
 */
int hwsel_static_config_workspace_bytes(int32_t P, int32_t n_configs, size_t *bytes);
int hwsel_static_config(const float *runtimes, const int64_t *seg_offsets, int32_t P, const int32_t *config_id,
                        int32_t n_configs, int32_t *best, double *mean_y, void *workspace, size_t workspace_bytes,
                        void *stream);

/*
 * Configuration catalogue (section "Configuration Space", Table
 * "Configuration knobs"): the HWSEL_CATALOGUE_SIZE = 534,600 points of
 * tile_m {64,128,192,256} x tile_n {16,32,48,64,80,96,128,192,256} x tile_k
 * {32,64,128,256,512} x stages {2..12} x cluster (C_M, C_N) in {1,2,4,8,16}^2
 * with C_M C_N <= 16 (15 pairs, C_M slower) x mainloop {WS, Pingpong,
 * Cooperative} x epilogue {NoSmem, TMA, TMA-Cooperative} x scheduler
 * {Persistent, Stream-K} per layout.  Point i is the mixed-radix number of
 * the value positions, first knob slowest.  Fixed fields: swizzle 1,
 * instruction tile 64 x T_N x (32 bytes / input element size).
 *
 * hwsel_catalogue_mask: mask[p][i] = 1 iff point i is valid for problem p
 * (Table "Static validity constraints": Stream-K needs the cooperative
 * mainloop; cooperative needs T_M % 128 == 0; S (T_M + T_N) T_K b + S_epi +
 * smem_reserved <= smem_per_block_max, with the epilogue storage S_epi of
 * feature column 26; A column-major needs T_K <= 256 C_N; B row-major needs
 * T_K <= 256 C_M; with flags bit 0 also the shape guard T_N <= 2M and
 * T_N <= 2N of section "Validity Constraints"), the same predicates as
 * feature columns 86 and 87.  n_valid[p] = number of valid points.
 *   mask uint8 [P][HWSEL_CATALOGUE_SIZE], 4-byte aligned; n_valid int64 [P].
 * Returns HWSEL_EINVAL for null pointers, P < 1, a misaligned mask or a bad
 * hardware field.
 */
#define HWSEL_CATALOGUE_SIZE 534600
int hwsel_catalogue_mask(hwsel_hw_t hw, const hwsel_problem_t *problems, int32_t P, uint32_t flags, uint8_t *mask,
                         int64_t *n_valid, void *stream);

/*
 * Group-contiguous list of the valid points: seg_offsets[0] = 0,
 * seg_offsets[p+1] = seg_offsets[p] + n_valid[p], and point[seg_offsets[p] +
 * j] = the j-th valid point of problem p in ascending order.  Points whose
 * position is >= capacity are not written (seg_offsets[P] tells the caller
 * the size needed).
 *   mask, n_valid as written by hwsel_catalogue_mask; seg_offsets int64 [P+1];
 *   point int32 [capacity].
 * Returns HWSEL_EINVAL for null pointers, P < 1, capacity < 0, a misaligned
 * mask.
 */
int hwsel_catalogue_compact(const uint8_t *mask, const int64_t *n_valid, int32_t P, int64_t *seg_offsets,
                            int32_t *point, int64_t capacity, void *stream);

/*
 * Candidate rows of catalogue points, ready for hwsel_features: row r of
 * problem p (segment as for hwsel_features) gets the knobs of point
 * point[r], or of point r - seg_offsets[p] when point is NULL (the whole
 * catalogue per problem); inst_k follows the problem's input dtype.  Point
 * values outside [0, HWSEL_CATALOGUE_SIZE) are clamped into it.
 *   out: host struct of DEVICE arrays of length R (the field widths of
 *   hwsel_cands_t).
 * Returns HWSEL_EINVAL for null pointers, P < 1, R < 1.
 */
typedef struct hwsel_cands_out {
    uint16_t *tile_m, *tile_n, *tile_k, *inst_n;
    uint8_t *stages, *cluster_m, *cluster_n, *swizzle, *inst_m_div16, *inst_k;
    uint8_t *kernel_sched, *epi_sched, *tile_sched;
} hwsel_cands_out_t;
int hwsel_catalogue_candidates(const hwsel_problem_t *problems, int32_t P, const int64_t *seg_offsets,
                               const int32_t *point, int64_t R, const hwsel_cands_out_t *out, void *stream);

/* Static text for a status code. */
const char *hwsel_status_string(int status);
/* Detail of the last failed call on this thread ("" if none). */
const char *hwsel_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* HWSEL_H */
