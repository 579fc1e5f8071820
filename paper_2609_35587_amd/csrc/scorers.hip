// Linear ridge scorer (section "Linear Ridge Baseline"):
//   f(x) = bias + sum_j w_j (clean(x_j) - mean_j) inv_std_j + one-hot terms.
//
// The pass is a GEMV over X and is bound by reading X from HBM (512 bytes per
// 128-column row, 4 bytes out).  Each 16-byte load of a wave covers two rows,
// each lane taking four consecutive columns, and four such loads are in
// flight per lane; the per-lane partial sums of a row are combined by a fixed
// butterfly over its 32 lanes, so the result does not depend on scheduling.
#include "internal.hpp"

namespace hwsel {
namespace {

constexpr int kLinWaves = 4;

struct ColTerm {
    int kind;          // 0: unused column, 1: numeric, 2: categorical
    float mean, inv_std, w;
    int slot0, levels;
};

__device__ __forceinline__ ColTerm column_term(const hwsel_linear_t &lin, int col)
{
    ColTerm t{0, 0.f, 0.f, 0.f, 0, 0};
    if (col >= lin.n_features) return t;
    if (lin.n_features > 64 && (col == 64 || col == 73 || col == 74 || col == 75)) {
        t.kind = 2;
        t.slot0 = col == 64 ? 0 : col == 73 ? 4 : col == 74 ? 7 : 10;
        t.levels = col == 64 ? 4 : col == 75 ? 2 : 3;
        return t;
    }
    t.kind = 1;
    t.mean = lin.mean[col];
    t.inv_std = lin.inv_std[col];
    t.w = lin.w[col];
    return t;
}

__device__ __forceinline__ float term(const ColTerm &t, float x, const float *__restrict__ w_onehot)
{
    if (t.kind == 1) {
        const float z = ((__builtin_isfinite(x) ? x : 0.0f) - t.mean) * t.inv_std;
        return t.w * z;
    }
    if (t.kind == 2 && x >= 0.0f && x < (float)t.levels && x == __builtin_floorf(x))
        return w_onehot[t.slot0 + (int)x];
    return 0.0f;
}

__global__ __launch_bounds__(64 * kLinWaves) void k_linear(hwsel_linear_t lin, const float *__restrict__ X, int64_t R,
                                                            int64_t ld, float *__restrict__ scores)
{
    const int lane = threadIdx.x & 63;
    const int c0 = 4 * (lane & 31);
    ColTerm t[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) t[j] = column_term(lin, c0 + j);
    const bool active = c0 < lin.n_features;
    const int64_t pairs = (R + 1) / 2;
    const int64_t stride = (int64_t)gridDim.x * kLinWaves;
    constexpr int kIn = 4;     // row pairs per wave step: four 16-byte loads in flight per lane
    for (int64_t pr0 = (int64_t)blockIdx.x * kLinWaves + (threadIdx.x >> 6); pr0 < pairs; pr0 += kIn * stride) {
        float4 v[kIn];
#pragma unroll
        for (int i = 0; i < kIn; ++i) {
            const int64_t r = 2 * (pr0 + i * stride) + (lane >> 5);
            v[i] = (r < R && active) ? *reinterpret_cast<const float4 *>(X + r * ld + c0)
                                     : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int i = 0; i < kIn; ++i) {
            const int64_t r = 2 * (pr0 + i * stride) + (lane >> 5);
            float acc = 0.0f;
            if (r < R && active) {
                acc = term(t[0], v[i].x, lin.w_onehot);
                acc += term(t[1], v[i].y, lin.w_onehot);
                acc += term(t[2], v[i].z, lin.w_onehot);
                acc += term(t[3], v[i].w, lin.w_onehot);
            }
#pragma unroll
            for (int o = 16; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 32);
            if ((lane & 31) == 0 && r < R) scores[r] = acc + lin.bias;
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
