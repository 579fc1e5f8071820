// C-ABI entry points: host-side argument checks, then one launch each.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "internal.hpp"

namespace {

thread_local char g_err[512];

int fail(int status, const char *fn, const char *fmt, ...) __attribute__((format(printf, 3, 4)));

int fail(int status, const char *fn, const char *fmt, ...)
{
    int n = snprintf(g_err, sizeof g_err, "%s: ", fn);
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err + n, sizeof g_err - (size_t)n, fmt, ap);
    va_end(ap);
    return status;
}

int launched(hipError_t e, const char *fn)
{
    if (e != hipSuccess) return fail(HWSEL_EHIP, fn, "launch failed: %s", hipGetErrorString(e));
    g_err[0] = 0;
    return HWSEL_OK;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

extern "C" {

const char *hwsel_status_string(int status)
{
    switch (status) {
    case HWSEL_OK: return "ok";
    case HWSEL_EINVAL: return "invalid argument";
    case HWSEL_EUNSUPPORTED: return "unsupported";
    case HWSEL_EHIP: return "HIP runtime error";
    default: return "unknown status";
    }
}

const char *hwsel_last_error(void) { return g_err; }

static int check_hw(const hwsel_hw_t &hw, const char *fn, hwsel::HwDev *h)
{
    const int64_t positive[] = {hw.n_sm, hw.smem_per_sm, hw.smem_per_block_max, hw.regs_per_sm,
                                hw.max_regs_per_thread, hw.max_blocks_per_sm, hw.max_threads_per_sm,
                                hw.arch_id, hw.llc_bytes, hw.hbm_bw_gbps, hw.peak_gflops[0],
                                hw.peak_gflops[1], hw.peak_gflops[2]};
    for (int64_t v : positive)
        if (v < 1) return fail(HWSEL_EINVAL, fn, "hardware field %lld < 1", (long long)v);
    if (hw.smem_reserved < 0) return fail(HWSEL_EINVAL, fn, "smem_reserved < 0");
    *h = hwsel::HwDev{hw.n_sm, hw.smem_per_sm, hw.smem_per_block_max, hw.smem_reserved, hw.regs_per_sm,
                      hw.max_regs_per_thread, hw.max_blocks_per_sm, hw.max_threads_per_sm, hw.arch_id,
                      hw.llc_bytes, hw.hbm_bw_gbps, {hw.peak_gflops[0], hw.peak_gflops[1], hw.peak_gflops[2]}};
    return HWSEL_OK;
}

// Shared checks of the problem/candidate inputs; fills the kernel views.
static int check_rows(const hwsel_hw_t &hw, const hwsel_problem_t *problems, int32_t P, const int64_t *seg_offsets,
                      const hwsel_cands_t *cands, int64_t R, const char *fn, hwsel::HwDev *h, hwsel::CandsDev *c)
{
    if (!problems || !seg_offsets || !cands) return fail(HWSEL_EINVAL, fn, "null pointer");
    const void *fields[] = {cands->tile_m, cands->tile_n, cands->tile_k, cands->inst_n, cands->stages,
                            cands->cluster_m, cands->cluster_n, cands->swizzle, cands->inst_m_div16,
                            cands->inst_k, cands->kernel_sched, cands->epi_sched, cands->tile_sched};
    for (const void *f : fields)
        if (!f) return fail(HWSEL_EINVAL, fn, "null candidate field");
    if (P < 1 || R < 1) return fail(HWSEL_EINVAL, fn, "P=%d R=%lld must be >= 1", P, (long long)R);
    if (int st = check_hw(hw, fn, h)) return st;
    *c = hwsel::CandsDev{cands->tile_m, cands->tile_n, cands->tile_k, cands->inst_n, cands->stages,
                         cands->cluster_m, cands->cluster_n, cands->swizzle, cands->inst_m_div16,
                         cands->inst_k, cands->kernel_sched, cands->epi_sched, cands->tile_sched};
    return HWSEL_OK;
}

int hwsel_features(hwsel_hw_t hw, const hwsel_problem_t *problems, int32_t P, const int64_t *seg_offsets,
                   const hwsel_cands_t *cands, int64_t R, int32_t n_features, float *X, int64_t ld,
                   void *stream)
{
    static const char *fn = "hwsel_features";
    hwsel::HwDev h;
    hwsel::CandsDev c;
    if (int st = check_rows(hw, problems, P, seg_offsets, cands, R, fn, &h, &c)) return st;
    if (!X) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (n_features != 64 && n_features != 96 && n_features != 128)
        return fail(HWSEL_EUNSUPPORTED, fn, "n_features=%d (supported: 64, 96, 128)", n_features);
    if (ld < n_features || ld % 4 != 0) return fail(HWSEL_EINVAL, fn, "ld=%lld", (long long)ld);
    if (!aligned16(X)) return fail(HWSEL_EINVAL, fn, "X not 16-byte aligned");
    return launched(hwsel::launch_features(h, problems, P, seg_offsets, c, R, n_features, X, ld,
                                           (hipStream_t)stream),
                    fn);
}

int hwsel_sample_score(hwsel_hw_t hw, const hwsel_problem_t *problems, int32_t P, const int64_t *seg_offsets,
                       const hwsel_cands_t *cands, int64_t R, float *scores, void *stream)
{
    static const char *fn = "hwsel_sample_score";
    hwsel::HwDev h;
    hwsel::CandsDev c;
    if (int st = check_rows(hw, problems, P, seg_offsets, cands, R, fn, &h, &c)) return st;
    if (!scores) return fail(HWSEL_EINVAL, fn, "null pointer");
    return launched(hwsel::launch_sample_score(h, problems, P, seg_offsets, c, R, scores, (hipStream_t)stream), fn);
}

int hwsel_linear_score(const hwsel_linear_t *lin, const float *X, int64_t R, int64_t ld, float *scores,
                       void *stream)
{
    static const char *fn = "hwsel_linear_score";
    if (!lin || !X || !scores || !lin->mean || !lin->inv_std || !lin->w || !lin->w_onehot)
        return fail(HWSEL_EINVAL, fn, "null pointer");
    if (lin->n_features != 64 && lin->n_features != 96 && lin->n_features != 128)
        return fail(HWSEL_EUNSUPPORTED, fn, "n_features=%d (supported: 64, 96, 128)", lin->n_features);
    if (R < 1) return fail(HWSEL_EINVAL, fn, "R=%lld", (long long)R);
    if (ld < lin->n_features || ld % 4 != 0) return fail(HWSEL_EINVAL, fn, "ld=%lld", (long long)ld);
    if (!aligned16(X)) return fail(HWSEL_EINVAL, fn, "X not 16-byte aligned");
    return launched(hwsel::launch_linear(*lin, X, R, ld, scores, (hipStream_t)stream), fn);
}

int hwsel_evaluate_workspace_bytes(int32_t P, size_t *bytes)
{
    static const char *fn = "hwsel_evaluate_workspace_bytes";
    if (!bytes) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (P < 1) return fail(HWSEL_EINVAL, fn, "P=%d", P);
    *bytes = hwsel::evaluate_workspace_bytes(P);
    g_err[0] = 0;
    return HWSEL_OK;
}

int hwsel_evaluate(const float *runtimes, const int64_t *seg_offsets, int32_t P, const int32_t *idx, int32_t k,
                   double *out, double *regret, int32_t *rank, double *ybar, void *workspace,
                   size_t workspace_bytes, void *stream)
{
    static const char *fn = "hwsel_evaluate";
    if (!runtimes || !seg_offsets || !idx || !out || !workspace) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (P < 1) return fail(HWSEL_EINVAL, fn, "P=%d", P);
    if (k < 1 || k > 64) return fail(HWSEL_EINVAL, fn, "k=%d (1..64)", k);
    const size_t need = hwsel::evaluate_workspace_bytes(P);
    if (workspace_bytes < need) return fail(HWSEL_EINVAL, fn, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
    if (((uintptr_t)workspace & 255u) != 0) return fail(HWSEL_EINVAL, fn, "workspace not 256-byte aligned");
    return launched(hwsel::launch_evaluate(runtimes, seg_offsets, P, idx, k, out, regret, rank, ybar, workspace,
                                           (hipStream_t)stream),
                    fn);
}

int hwsel_evaluate_noalloc(const float *runtimes, const int64_t *seg_offsets, int32_t P, const int32_t *idx,
                           int32_t k, double *out, double *regret, int32_t *rank, double *ybar, void *stream)
{
    static const char *fn = "hwsel_evaluate_noalloc";
    if (!runtimes || !seg_offsets || !idx || !out) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (P < 1 || P > HWSEL_EVAL_NOALLOC_MAX_P)
        return fail(HWSEL_EINVAL, fn, "P=%d (1..%d)", P, HWSEL_EVAL_NOALLOC_MAX_P);
    if (k < 1 || k > 64) return fail(HWSEL_EINVAL, fn, "k=%d (1..64)", k);
    void *scratch = nullptr;
    size_t scratch_bytes = 0;
    const hipError_t e = hwsel::evaluate_noalloc_scratch(&scratch, &scratch_bytes);
    if (e != hipSuccess) return fail(HWSEL_EHIP, fn, "scratch address: %s", hipGetErrorString(e));
    if (scratch_bytes < hwsel::evaluate_workspace_bytes(P) || scratch_bytes != HWSEL_EVAL_NOALLOC_SCRATCH_BYTES)
        return fail(HWSEL_EHIP, fn, "scratch of %zu bytes", scratch_bytes);
    return launched(hwsel::launch_evaluate(runtimes, seg_offsets, P, idx, k, out, regret, rank, ybar, scratch,
                                           (hipStream_t)stream),
                    fn);
}

int hwsel_static_config_workspace_bytes(int32_t P, int32_t n_configs, size_t *bytes)
{
    static const char *fn = "hwsel_static_config_workspace_bytes";
    if (!bytes) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (P < 1 || n_configs < 1) return fail(HWSEL_EINVAL, fn, "P=%d n_configs=%d", P, n_configs);
    *bytes = hwsel::static_config_workspace_bytes(P, n_configs);
    g_err[0] = 0;
    return HWSEL_OK;
}

int hwsel_static_config(const float *runtimes, const int64_t *seg_offsets, int32_t P, const int32_t *config_id,
                        int32_t n_configs, int32_t *best, double *mean_y, void *workspace, size_t workspace_bytes,
                        void *stream)
{
    static const char *fn = "hwsel_static_config";
    if (!runtimes || !seg_offsets || !config_id || !best || !mean_y || !workspace)
        return fail(HWSEL_EINVAL, fn, "null pointer");
    if (P < 1 || n_configs < 1) return fail(HWSEL_EINVAL, fn, "P=%d n_configs=%d", P, n_configs);
    const size_t need = hwsel::static_config_workspace_bytes(P, n_configs);
    if (workspace_bytes < need) return fail(HWSEL_EINVAL, fn, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
    if (((uintptr_t)workspace & 255u) != 0) return fail(HWSEL_EINVAL, fn, "workspace not 256-byte aligned");
    return launched(hwsel::launch_static_config(runtimes, seg_offsets, P, config_id, n_configs, best, mean_y,
                                                workspace, (hipStream_t)stream),
                    fn);
}

int hwsel_catalogue_mask(hwsel_hw_t hw, const hwsel_problem_t *problems, int32_t P, uint32_t flags, uint8_t *mask,
                         int64_t *n_valid, void *stream)
{
    static const char *fn = "hwsel_catalogue_mask";
    hwsel::HwDev h;
    if (!problems || !mask || !n_valid) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (P < 1) return fail(HWSEL_EINVAL, fn, "P=%d", P);
    if (((uintptr_t)mask & 3u) != 0) return fail(HWSEL_EINVAL, fn, "mask not 4-byte aligned");
    if (int st = check_hw(hw, fn, &h)) return st;
    return launched(hwsel::launch_catalogue_mask(h, problems, P, flags, mask, n_valid, (hipStream_t)stream), fn);
}

int hwsel_catalogue_compact(const uint8_t *mask, const int64_t *n_valid, int32_t P, int64_t *seg_offsets,
                            int32_t *point, int64_t capacity, void *stream)
{
    static const char *fn = "hwsel_catalogue_compact";
    if (!mask || !n_valid || !seg_offsets || (!point && capacity > 0)) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (P < 1 || capacity < 0) return fail(HWSEL_EINVAL, fn, "P=%d capacity=%lld", P, (long long)capacity);
    if (((uintptr_t)mask & 3u) != 0) return fail(HWSEL_EINVAL, fn, "mask not 4-byte aligned");
    return launched(hwsel::launch_catalogue_compact(mask, n_valid, P, seg_offsets, point, capacity,
                                                    (hipStream_t)stream),
                    fn);
}

int hwsel_catalogue_candidates(const hwsel_problem_t *problems, int32_t P, const int64_t *seg_offsets,
                               const int32_t *point, int64_t R, const hwsel_cands_out_t *out, void *stream)
{
    static const char *fn = "hwsel_catalogue_candidates";
    if (!problems || !seg_offsets || !out) return fail(HWSEL_EINVAL, fn, "null pointer");
    const void *fields[] = {out->tile_m, out->tile_n, out->tile_k, out->inst_n, out->stages, out->cluster_m,
                            out->cluster_n, out->swizzle, out->inst_m_div16, out->inst_k, out->kernel_sched,
                            out->epi_sched, out->tile_sched};
    for (const void *f : fields)
        if (!f) return fail(HWSEL_EINVAL, fn, "null candidate field");
    if (P < 1 || R < 1) return fail(HWSEL_EINVAL, fn, "P=%d R=%lld", P, (long long)R);
    return launched(hwsel::launch_catalogue_candidates(problems, P, seg_offsets, point, R, *out,
                                                       (hipStream_t)stream),
                    fn);
}

static int check_forest(const hwsel_forest_t *f, const float *X, int64_t R, int64_t ld, const char *fn)
{
    if (!f || !X || !f->node_feature || !f->node_threshold || !f->leaf_value)
        return fail(HWSEL_EINVAL, fn, "null pointer");
    if (R < 1 || f->n_trees < 1) return fail(HWSEL_EINVAL, fn, "R=%lld n_trees=%d", (long long)R, f->n_trees);
    if (f->depth < 1 || f->depth > 12) return fail(HWSEL_EUNSUPPORTED, fn, "depth=%d (1..12)", f->depth);
    if (f->n_features < 1 || f->n_features > 256)
        return fail(HWSEL_EUNSUPPORTED, fn, "n_features=%d (1..256)", f->n_features);
    if (ld < f->n_features) return fail(HWSEL_EINVAL, fn, "ld=%lld < n_features", (long long)ld);
    return HWSEL_OK;
}

int hwsel_forest_pack_bytes(const hwsel_forest_t *f, size_t *bytes)
{
    static const char *fn = "hwsel_forest_pack_bytes";
    if (!f || !bytes) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (f->n_trees < 1) return fail(HWSEL_EINVAL, fn, "n_trees=%d", f->n_trees);
    if (!hwsel::packable(*f))
        return fail(HWSEL_EUNSUPPORTED, fn, "depth=%d n_features=%d (packed: depth <= 10, n_features <= 128)",
                    f->depth, f->n_features);
    *bytes = hwsel::packed_bytes(*f);
    g_err[0] = 0;
    return HWSEL_OK;
}

int hwsel_forest_pack(const hwsel_forest_t *f, void *packed, size_t bytes, void *stream)
{
    static const char *fn = "hwsel_forest_pack";
    size_t need = 0;
    if (int s = hwsel_forest_pack_bytes(f, &need)) return s;
    if (!packed || !f->node_feature || !f->node_threshold || !f->leaf_value)
        return fail(HWSEL_EINVAL, fn, "null pointer");
    if (f->n_features < 1 || f->depth < 1) return fail(HWSEL_EINVAL, fn, "empty forest shape");
    if (bytes < need) return fail(HWSEL_EINVAL, fn, "bytes=%zu < %zu", bytes, need);
    if (!aligned16(packed)) return fail(HWSEL_EINVAL, fn, "packed not 16-byte aligned");
    switch (hwsel::pack_forest(*f, packed, (hipStream_t)stream)) {
    case hwsel::PackStatus::ok: g_err[0] = 0; return HWSEL_OK;
    case hwsel::PackStatus::bad_feature: return fail(HWSEL_EINVAL, fn, "node feature >= n_features");
    case hwsel::PackStatus::nan_threshold: return fail(HWSEL_EINVAL, fn, "NaN threshold");
    case hwsel::PackStatus::too_many_thresholds:
        return fail(HWSEL_EUNSUPPORTED, fn, "a feature has more than 255 distinct thresholds");
    default: return fail(HWSEL_EHIP, fn, "copy failed: %s", hipGetErrorString(hipGetLastError()));
    }
}

int hwsel_forest_pack_host(const hwsel_forest_t *f, void *image, size_t bytes)
{
    static const char *fn = "hwsel_forest_pack_host";
    size_t need = 0;
    if (int s = hwsel_forest_pack_bytes(f, &need)) return s;
    if (!image || !f->node_feature || !f->node_threshold || !f->leaf_value)
        return fail(HWSEL_EINVAL, fn, "null pointer");
    if (f->n_features < 1 || f->depth < 1) return fail(HWSEL_EINVAL, fn, "empty forest shape");
    if (bytes < need) return fail(HWSEL_EINVAL, fn, "bytes=%zu < %zu", bytes, need);
    switch (hwsel::build_image(*f, f->node_feature, f->node_threshold, f->leaf_value, static_cast<uint8_t *>(image))) {
    case hwsel::PackStatus::ok: g_err[0] = 0; return HWSEL_OK;
    case hwsel::PackStatus::bad_feature: return fail(HWSEL_EINVAL, fn, "node feature >= n_features");
    case hwsel::PackStatus::nan_threshold: return fail(HWSEL_EINVAL, fn, "NaN threshold");
    case hwsel::PackStatus::too_many_thresholds:
        return fail(HWSEL_EUNSUPPORTED, fn, "a feature has more than 255 distinct thresholds");
    default: return fail(HWSEL_EINVAL, fn, "cannot pack");
    }
}

int hwsel_forest_workspace_bytes(const hwsel_forest_t *f, int64_t R, size_t *bytes)
{
    static const char *fn = "hwsel_forest_workspace_bytes";
    size_t dummy = 0;
    if (int s = hwsel_forest_pack_bytes(f, &dummy)) return s;
    if (R < 1) return fail(HWSEL_EINVAL, fn, "R=%lld", (long long)R);
    *bytes = hwsel::packed_workspace_bytes(*f, R);
    return HWSEL_OK;
}

int hwsel_forest_score(const hwsel_forest_t *f, const void *packed, const float *X, int64_t R, int64_t ld,
                       float *scores, void *workspace, size_t workspace_bytes, void *stream)
{
    static const char *fn = "hwsel_forest_score";
    if (int s = check_forest(f, X, R, ld, fn)) return s;
    if (!scores) return fail(HWSEL_EINVAL, fn, "null scores");
    if (!packed) return launched(hwsel::launch_forest_score(*f, X, R, ld, scores, (hipStream_t)stream), fn);
    if (!hwsel::packable(*f)) return fail(HWSEL_EUNSUPPORTED, fn, "forest shape cannot be packed");
    if (!aligned16(packed)) return fail(HWSEL_EINVAL, fn, "packed not 16-byte aligned");
    const size_t need = hwsel::packed_workspace_bytes(*f, R);
    if (!workspace || workspace_bytes < need)
        return fail(HWSEL_EINVAL, fn, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
    if (((uintptr_t)workspace & 255u) != 0) return fail(HWSEL_EINVAL, fn, "workspace not 256-byte aligned");
    return launched(hwsel::launch_forest_packed(*f, packed, X, R, ld, scores, workspace, (hipStream_t)stream), fn);
}

int hwsel_forest_score_checked(const hwsel_forest_t *f, const void *packed, const float *X, int64_t R, int64_t ld,
                               float *scores, void *workspace, size_t workspace_bytes, uint64_t *leaf_hash,
                               uint16_t *leaf_idx, int64_t leaf_row0, int64_t leaf_rows, void *stream)
{
    static const char *fn = "hwsel_forest_score_checked";
    if (int s = check_forest(f, X, R, ld, fn)) return s;
    if (!scores || !packed) return fail(HWSEL_EINVAL, fn, "null scores or packed image");
    if (!hwsel::packable(*f)) return fail(HWSEL_EUNSUPPORTED, fn, "forest shape cannot be packed");
    if (!aligned16(packed)) return fail(HWSEL_EINVAL, fn, "packed not 16-byte aligned");
    const size_t need = hwsel::packed_workspace_bytes(*f, R);
    if (!workspace || workspace_bytes < need)
        return fail(HWSEL_EINVAL, fn, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
    if (((uintptr_t)workspace & 255u) != 0) return fail(HWSEL_EINVAL, fn, "workspace not 256-byte aligned");
    if (((uintptr_t)leaf_hash & 7u) != 0) return fail(HWSEL_EINVAL, fn, "leaf_hash not 8-byte aligned");
    if (leaf_idx && (leaf_row0 < 0 || leaf_rows < 1 || leaf_row0 > R - leaf_rows))
        return fail(HWSEL_EINVAL, fn, "leaf rows [%lld, %lld + %lld) outside [0, %lld)", (long long)leaf_row0,
                    (long long)leaf_row0, (long long)leaf_rows, (long long)R);
    return launched(hwsel::launch_forest_checked(*f, packed, X, R, ld, scores, workspace, leaf_hash, leaf_idx,
                                                 leaf_row0, leaf_rows, (hipStream_t)stream),
                    fn);
}

int hwsel_forest_leaves(const hwsel_forest_t *f, const float *X, int64_t R, int64_t ld, const int64_t *rows,
                        int64_t n_rows, uint16_t *leaf_idx, void *stream)
{
    static const char *fn = "hwsel_forest_leaves";
    if (int s = check_forest(f, X, R, ld, fn)) return s;
    if (!rows || !leaf_idx) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (n_rows < 1) return fail(HWSEL_EINVAL, fn, "n_rows=%lld", (long long)n_rows);
    return launched(hwsel::launch_forest_leaves(*f, X, R, ld, rows, n_rows, leaf_idx, (hipStream_t)stream), fn);
}

int hwsel_select_forest_workspace_bytes(const hwsel_forest_t *f, int64_t R, size_t *bytes)
{
    static const char *fn = "hwsel_select_forest_workspace_bytes";
    size_t dummy = 0;
    if (int s = hwsel_forest_pack_bytes(f, &dummy)) return s;
    if (!bytes) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (R < 1) return fail(HWSEL_EINVAL, fn, "R=%lld", (long long)R);
    *bytes = hwsel::packed_workspace_bytes(*f, R) + ((size_t)R * sizeof(float) + 255) / 256 * 256;
    return HWSEL_OK;
}

int hwsel_select_forest(hwsel_hw_t hw, const hwsel_problem_t *problems, int32_t P, const int64_t *seg_offsets,
                        const hwsel_cands_t *cands, int64_t R, int32_t n_features, const hwsel_forest_t *f,
                        const void *packed, int32_t k, int32_t *idx, float *vals, float *scores, void *workspace,
                        size_t workspace_bytes, void *stream)
{
    static const char *fn = "hwsel_select_forest";
    hwsel::HwDev h;
    hwsel::CandsDev c;
    if (int st = check_rows(hw, problems, P, seg_offsets, cands, R, fn, &h, &c)) return st;
    if (n_features != 64 && n_features != 96 && n_features != 128)
        return fail(HWSEL_EUNSUPPORTED, fn, "n_features=%d (supported: 64, 96, 128)", n_features);
    if (!f || !packed || !idx || !workspace || !f->node_feature || !f->node_threshold || !f->leaf_value)
        return fail(HWSEL_EINVAL, fn, "null pointer");
    if (f->n_trees < 1) return fail(HWSEL_EINVAL, fn, "n_trees=%d", f->n_trees);
    if (!hwsel::packable(*f)) return fail(HWSEL_EUNSUPPORTED, fn, "forest shape cannot be packed");
    if (f->n_features < 1 || f->n_features > n_features)
        return fail(HWSEL_EINVAL, fn, "forest n_features=%d, feature map has %d", f->n_features, n_features);
    if (k < 1 || k > 64) return fail(HWSEL_EINVAL, fn, "k=%d (1..64)", k);
    if (!aligned16(packed)) return fail(HWSEL_EINVAL, fn, "packed not 16-byte aligned");
    const size_t base = hwsel::packed_workspace_bytes(*f, R);
    const size_t need = base + ((size_t)R * sizeof(float) + 255) / 256 * 256;
    if (workspace_bytes < need)
        return fail(HWSEL_EINVAL, fn, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
    if (((uintptr_t)workspace & 255u) != 0) return fail(HWSEL_EINVAL, fn, "workspace not 256-byte aligned");
    hipStream_t s = (hipStream_t)stream;
    float *sc = scores ? scores : reinterpret_cast<float *>(static_cast<uint8_t *>(workspace) + base);
    hipError_t e = hwsel::launch_features_bins(h, problems, P, seg_offsets, c, R, n_features,
                                               packed, hwsel::packed_image_id(*f), f->n_features,
                                               hwsel::packed_nan_bin(*f), static_cast<uint8_t *>(workspace),
                                               hwsel::packed_bin_stride(*f), s);
    if (e == hipSuccess) e = hwsel::launch_forest_from_bins(*f, packed, R, sc, workspace, s);
    if (e == hipSuccess) e = hwsel::launch_topk(sc, seg_offsets, P, k, idx, vals, s);
    return launched(e, fn);
}

static int check_mlp(const hwsel_mlp_t *m, const char *fn)
{
    if (!m || !m->mean || !m->inv_std || !m->W1 || !m->W2 || !m->W3 || !m->W4 || !m->b1 || !m->b2 || !m->b3 ||
        !m->b4)
        return fail(HWSEL_EINVAL, fn, "null pointer");
    if (m->n_in != 128 || m->h1 != 512 || m->h2 != 512 || m->h3 != 256)
        return fail(HWSEL_EUNSUPPORTED, fn, "widths %d-%d-%d-%d (supported: 128-512-512-256)", m->n_in, m->h1,
                    m->h2, m->h3);
    return HWSEL_OK;
}

int hwsel_mlp_pack_bytes(const hwsel_mlp_t *m, size_t *bytes)
{
    static const char *fn = "hwsel_mlp_pack_bytes";
    if (!bytes) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (int s = check_mlp(m, fn)) return s;
    *bytes = hwsel::mlp_packed_bytes();
    g_err[0] = 0;
    return HWSEL_OK;
}

int hwsel_mlp_pack(const hwsel_mlp_t *m, void *packed, size_t bytes, void *stream)
{
    static const char *fn = "hwsel_mlp_pack";
    if (int s = check_mlp(m, fn)) return s;
    if (!packed) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (bytes < hwsel::mlp_packed_bytes()) return fail(HWSEL_EINVAL, fn, "bytes=%zu < %zu", bytes, hwsel::mlp_packed_bytes());
    if (!aligned16(packed)) return fail(HWSEL_EINVAL, fn, "packed not 16-byte aligned");
    return launched(hwsel::launch_mlp_pack(*m, packed, (hipStream_t)stream), fn);
}

int hwsel_mlp_score(const hwsel_mlp_t *m, const void *packed, const float *X, int64_t R, int64_t ld, float *scores,
                    void *stream)
{
    static const char *fn = "hwsel_mlp_score";
    if (int s = check_mlp(m, fn)) return s;
    if (!X || !scores) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (R < 1) return fail(HWSEL_EINVAL, fn, "R=%lld", (long long)R);
    if (ld < 128 || ld % 4 != 0) return fail(HWSEL_EINVAL, fn, "ld=%lld", (long long)ld);
    if (!aligned16(X)) return fail(HWSEL_EINVAL, fn, "X not 16-byte aligned");
    if (!packed) return launched(hwsel::launch_mlp(*m, X, R, ld, scores, (hipStream_t)stream), fn);
    if (!aligned16(packed) || !aligned16(m->mean) || !aligned16(m->inv_std) || !aligned16(m->b1) ||
        !aligned16(m->b2) || !aligned16(m->b3) || ((uintptr_t)m->W4 & 7u) != 0)
        return fail(HWSEL_EINVAL, fn, "misaligned packed weights, statistics or biases");
    return launched(hwsel::launch_mlp_packed(*m, packed, X, R, ld, scores, (hipStream_t)stream), fn);
}

int hwsel_topk_per_problem(const float *scores, const int64_t *seg_offsets, int32_t P, int32_t k, int32_t *idx,
                           float *vals, void *stream)
{
    static const char *fn = "hwsel_topk_per_problem";
    if (!scores || !seg_offsets || !idx) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (P < 1) return fail(HWSEL_EINVAL, fn, "P=%d", P);
    if (k < 1 || k > 64) return fail(HWSEL_EINVAL, fn, "k=%d (1..64)", k);
    return launched(hwsel::launch_topk(scores, seg_offsets, P, k, idx, vals, (hipStream_t)stream), fn);
}

int hwsel_regret(const float *runtimes, const int64_t *seg_offsets, int32_t P, const int32_t *idx, int32_t k,
                 float *regret_top1, float *regret_bestk, int32_t *best_idx, void *stream)
{
    static const char *fn = "hwsel_regret";
    if (!runtimes || !seg_offsets || !idx || !regret_top1) return fail(HWSEL_EINVAL, fn, "null pointer");
    if (P < 1) return fail(HWSEL_EINVAL, fn, "P=%d", P);
    if (k < 1 || k > 64) return fail(HWSEL_EINVAL, fn, "k=%d (1..64)", k);
    return launched(hwsel::launch_regret(runtimes, seg_offsets, P, idx, k, regret_top1, regret_bestk, best_idx,
                                         (hipStream_t)stream),
                    fn);
}

}  // extern "C"
