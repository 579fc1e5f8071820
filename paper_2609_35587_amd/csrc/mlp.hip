// Feed-forward ranker 128 -> 512 -> 512 -> 256 -> 1 (GELU, bf16 activations,
// fp32 accumulation).
//
// Row-block kernel: a workgroup holds the activations of 16 rows in LDS and
// walks the layers; each thread owns output units and reuses every weight it
// loads across the 16 rows.
#include "internal.hpp"

#include <math.h>

namespace hwsel {
namespace {

constexpr int kRows = 16;
constexpr int kThreads = 256;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round fp32 to the nearest bf16 value (ties to even), kept in an fp32.
__device__ __forceinline__ float round_bf16(float v)
{
    uint32_t u = __float_as_uint(v);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return __uint_as_float((u | 0x00400000u) & 0xffff0000u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return __uint_as_float(u & 0xffff0000u);
}

__device__ __forceinline__ float gelu(float a) { return 0.5f * a * (1.0f + erff(a * 0.70710678118654752f)); }

template <int IN, int OUT>
__device__ __forceinline__ void dense_gelu(const uint16_t *__restrict__ W, const float *__restrict__ b,
                                           const float (*in)[IN], float (*out)[OUT])
{
    for (int u = threadIdx.x; u < OUT; u += kThreads) {
        float acc[kRows];
#pragma unroll
        for (int r = 0; r < kRows; ++r) acc[r] = 0.0f;
        const uint16_t *w = W + (int64_t)u * IN;
        for (int j = 0; j < IN; ++j) {
            const float wj = bf16_to_f32(w[j]);
#pragma unroll
            for (int r = 0; r < kRows; ++r) acc[r] = fmaf(wj, in[r][j], acc[r]);
        }
        const float bu = b[u];
#pragma unroll
        for (int r = 0; r < kRows; ++r) out[r][u] = round_bf16(gelu(acc[r] + bu));
    }
}

__global__ __launch_bounds__(kThreads) void k_mlp_rows(hwsel_mlp_t m, const float *__restrict__ X, int64_t R,
                                                        int64_t ld, float *__restrict__ scores)
{
    __shared__ float h0[kRows][128];
    __shared__ float h1[kRows][512];
    __shared__ float h2[kRows][512];
    float (*h3)[256] = reinterpret_cast<float (*)[256]>(&h1[0][0]);   // h1 is dead by then
    const int64_t row0 = (int64_t)blockIdx.x * kRows;
    for (int e = threadIdx.x; e < kRows * 128; e += kThreads) {
        const int r = e >> 7, j = e & 127;
        float v = 0.0f;
        if (row0 + r < R) v = X[(row0 + r) * ld + j];
        if (!__builtin_isfinite(v)) v = 0.0f;
        const float centred = v - m.mean[j];
        h0[r][j] = round_bf16(centred * m.inv_std[j]);
    }
    __syncthreads();
    dense_gelu<128, 512>(m.W1, m.b1, h0, h1);
    __syncthreads();
    dense_gelu<512, 512>(m.W2, m.b2, h1, h2);
    __syncthreads();
    dense_gelu<512, 256>(m.W3, m.b3, h2, h3);
    __syncthreads();
    // output layer: 16 lanes per row
    const int r = threadIdx.x >> 4, part = threadIdx.x & 15;
    float acc = 0.0f;
    for (int j = part; j < 256; j += 16) acc = fmaf(bf16_to_f32(m.W4[j]), h3[r][j], acc);
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 16);
    if (part == 0 && row0 + r < R) scores[row0 + r] = acc + m.b4[0];
}

}  // namespace

hipError_t launch_mlp(const hwsel_mlp_t &m, const float *X, int64_t R, int64_t ld, float *scores,
                      hipStream_t s)
{
    const dim3 grid((unsigned)((R + kRows - 1) / kRows)), block(kThreads);
    hipLaunchKernelGGL(k_mlp_rows, grid, block, 0, s, m, X, R, ld, scores);
    return hipGetLastError();
}

}  // namespace hwsel
