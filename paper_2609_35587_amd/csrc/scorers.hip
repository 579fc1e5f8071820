// Linear ridge scorer (section "Linear Ridge Baseline"):
//   f(x) = bias + sum_j w_j (clean(x_j) - mean_j) inv_std_j + one-hot terms.
//
// The pass is a GEMV over X and is bound by reading X from HBM (512 bytes per
// 128-column row, 4 bytes out).  Each 16-byte load of a wave covers two rows,
// each lane taking four consecutive columns, and eight such loads are in
// flight per lane.  A lane's column terms, the one-hot weights included,
// sit in registers for the whole pass; the per-lane partial sums of a row
// are combined by DPP within its 32 lanes in a fixed order, so the result
// does not depend on scheduling.
#include "internal.hpp"

namespace hwsel {
namespace {

constexpr int kLinWaves = 4;
constexpr int kIn = 8;         // row pairs per wave step: eight 16-byte loads in flight per lane

// One column's part of the model: numeric (w, mean, inv_std), categorical
// (oh[l], the weight of level l, 0 past the column's levels) or unused (all 0).
struct ColTerm {
    float mean, inv_std, w;
    float oh[4];
};

__device__ __forceinline__ ColTerm column_term(const hwsel_linear_t &lin, int col)
{
    ColTerm t{0.f, 0.f, 0.f, {0.f, 0.f, 0.f, 0.f}};
    if (col >= lin.n_features) return t;
    if (lin.n_features > 64 && (col == 64 || col == 73 || col == 74 || col == 75)) {
        const int slot0 = col == 64 ? 0 : col == 73 ? 4 : col == 74 ? 7 : 10;
        const int levels = col == 64 ? 4 : col == 75 ? 2 : 3;
        for (int l = 0; l < levels; ++l) t.oh[l] = lin.w_onehot[slot0 + l];
        return t;
    }
    t.mean = lin.mean[col];
    t.inv_std = lin.inv_std[col];
    t.w = lin.w[col];
    return t;
}

// Branch-free, since lanes differ in their columns' kinds: the numeric term
// (weight 0 unless numeric) plus the one-hot term (levels 0 unless
// categorical).  A level is an integral x in [0, levels): x equal to 0, 1, 2
// or 3 (NaN equals none of them); levels past the column's own carry 0.
__device__ __forceinline__ float term(const ColTerm &t, float x)
{
    const float z = ((__builtin_isfinite(x) ? x : 0.0f) - t.mean) * t.inv_std;
    float oh = x == 3.0f ? t.oh[3] : 0.0f;
    oh = x == 2.0f ? t.oh[2] : oh;
    oh = x == 1.0f ? t.oh[1] : oh;
    oh = x == 0.0f ? t.oh[0] : oh;
    return fmaf(t.w, z, oh);
}

__global__ __launch_bounds__(64 * kLinWaves) void k_linear(hwsel_linear_t lin, const float *__restrict__ X, int64_t R,
                                                            int64_t ld, float *__restrict__ scores)
{
    const int lane = threadIdx.x & 63;
    const int c0 = 4 * (lane & 31);
    ColTerm t[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) t[j] = column_term(lin, c0 + j);
    // lanes past the model's columns read column 0 (always present) and
    // contribute 0 through their zero terms
    const int cl = c0 < lin.n_features ? c0 : 0;
    // A wave step reads row pairs (2p, 2p + 1): lanes 0-31 the first row,
    // lanes 32-63 the second.  The pair's base address is wave-uniform; a
    // lane adds its own fixed offset.  When 2p + 1 = R (R odd) the second
    // half rereads row 2p, whose score it does not store.
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t off_pair = (lane >> 5) * ld + cl, off_top = cl;
    const int64_t pairs = (R + 1) / 2;
    const int64_t stride = (int64_t)gridDim.x * kLinWaves;
    for (int64_t pr0 = (int64_t)blockIdx.x * kLinWaves + wave; pr0 < pairs; pr0 += kIn * stride) {
        float4 v[kIn];
#pragma unroll
        for (int i = 0; i < kIn; ++i) {
            const int64_t re = 2 * (pr0 + i * stride);
            const int64_t rr = re < R ? re : R - 1;      // pairs past the end (unused) reread row R - 1
            const float *base = X + rr * ld;
            v[i] = *reinterpret_cast<const float4 *>(base + (rr + 1 < R ? off_pair : off_top));
        }
        __builtin_amdgcn_sched_barrier(0);        // all eight loads issue before any use
        float acc[kIn];
#pragma unroll
        for (int i = 0; i < kIn; ++i)
            acc[i] = ((term(t[0], v[i].x) + term(t[1], v[i].y)) + term(t[2], v[i].z)) + term(t[3], v[i].w);
        group_totals<32, kIn>(acc);          // lane 31 / 63: the sum of its 32-lane row
#pragma unroll
        for (int i = 0; i < kIn; ++i) {
            const int64_t r = 2 * (pr0 + i * stride) + (lane >> 5);
            if ((lane & 31) == 31 && r < R) scores[r] = acc[i] + lin.bias;
        }
    }
}

}  // namespace

hipError_t launch_linear(const hwsel_linear_t &lin, const float *X, int64_t R, int64_t ld, float *scores,
                         hipStream_t s)
{
    int dev = 0, n_cu = 256;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n_cu < 1)
        n_cu = 256;
    const int64_t pairs = (R + 1) / 2;
    int64_t blocks = (pairs + kLinWaves - 1) / kLinWaves;
    const int64_t cap = (int64_t)n_cu * 16;
    if (blocks > cap) blocks = cap;
    hipLaunchKernelGGL(k_linear, dim3((unsigned)blocks), dim3(64 * kLinWaves), 0, s, lin, X, R, ld, scores);
    return hipGetLastError();
}

}  // namespace hwsel
