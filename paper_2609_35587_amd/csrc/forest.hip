// Tree-ensemble scoring: s(x) = base + sum_t leaf_t(x).
//
// Generic traversal: one thread per row walks every tree from the root; node
// records (feature byte, fp32 threshold) and leaves come from global memory
// through the caches, the row's feature values are gathered from X.  The leaf
// sum is accumulated in fp32 in tree order, so results are bit-identical from
// run to run.
#include "internal.hpp"

namespace hwsel {
namespace {

struct ForestDev {
    int32_t n_trees, depth, n_features;
    uint32_t nan_left;
    float base;
    const uint8_t *feat;
    const float *thr;
    const float *leaf;
};

// Leaf reached by row x in tree t (index in [0, 2^depth)).
__device__ __forceinline__ int32_t walk(const ForestDev &f, const float *__restrict__ x, int32_t t)
{
    const int64_t n_int = ((int64_t)1 << f.depth) - 1;
    const uint8_t *__restrict__ feat = f.feat + t * n_int;
    const float *__restrict__ thr = f.thr + t * n_int;
    int64_t node = 0;
    for (int32_t l = 0; l < f.depth; ++l) {
        int32_t j = feat[node];
        j = j < f.n_features ? j : f.n_features - 1;
        const float v = x[j];
        const bool left = (v < thr[node]) || (f.nan_left && __builtin_isnan(v));
        node = 2 * node + (left ? 1 : 2);
    }
    return (int32_t)(node - n_int);
}

__global__ __launch_bounds__(256) void k_forest_score(ForestDev f, const float *__restrict__ X, int64_t R,
                                                       int64_t ld, float *__restrict__ scores)
{
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= R) return;
    const float *x = X + r * ld;
    const int64_t n_leaf = (int64_t)1 << f.depth;
    float acc = f.base;
    for (int32_t t = 0; t < f.n_trees; ++t) acc += f.leaf[t * n_leaf + walk(f, x, t)];
    scores[r] = acc;
}

__global__ __launch_bounds__(256) void k_forest_leaves(ForestDev f, const float *__restrict__ X, int64_t R,
                                                        int64_t ld, const int64_t *__restrict__ rows,
                                                        int64_t n_rows, uint16_t *__restrict__ out)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_rows) return;
    int64_t r = rows[i];
    r = r < 0 ? 0 : (r >= R ? R - 1 : r);
    const float *x = X + r * ld;
    for (int32_t t = 0; t < f.n_trees; ++t) out[i * f.n_trees + t] = (uint16_t)walk(f, x, t);
}

ForestDev to_dev(const hwsel_forest_t &f)
{
    return ForestDev{f.n_trees, f.depth, f.n_features, f.flags & 1u, f.base_score,
                     f.node_feature, f.node_threshold, f.leaf_value};
}

}  // namespace

hipError_t launch_forest_score(const hwsel_forest_t &f, const float *X, int64_t R, int64_t ld,
                               float *scores, hipStream_t s)
{
    const dim3 grid((unsigned)((R + 255) / 256)), block(256);
    hipLaunchKernelGGL(k_forest_score, grid, block, 0, s, to_dev(f), X, R, ld, scores);
    return hipGetLastError();
}

hipError_t launch_forest_leaves(const hwsel_forest_t &f, const float *X, int64_t R, int64_t ld,
                                const int64_t *rows, int64_t n_rows, uint16_t *leaf_idx,
                                hipStream_t s)
{
    const dim3 grid((unsigned)((n_rows + 255) / 256)), block(256);
    hipLaunchKernelGGL(k_forest_leaves, grid, block, 0, s, to_dev(f), X, R, ld, rows, n_rows, leaf_idx);
    return hipGetLastError();
}

}  // namespace hwsel
