// Measured ceilings for the benchmark's rooflines (libhwsel_ceilings.so; not
// part of the scoring library).  Each kernel runs one unit's work pattern
// with every operand already where the real kernel finds it at best, so its
// rate bounds what that kernel can reach on this device:
//
//   k_visit_ceiling  the depth-10 tree traversal's walk -- per level a u8 bin
//                    gather and a 4-byte sibling-pair gather from LDS,
//                    compare-and-carry descent (the same SDWA sequence), bin
//                    and pair addressing; then the leaf gather and the
//                    16-lane sums -- over 16 trees x 4 rows per group with 4
//                    groups in flight, as the scoring kernel runs it; no bin
//                    rows are refilled and no partial sums stored.
//   k_mfma_ceiling   back-to-back independent v_mfma_f32_32x32x16_bf16 on
//                    register operands (four accumulators per wave).
//   k_copy_ceiling   a streaming device copy, 16 bytes per lane, four in
//                    flight (HBM read + write rate);
//   k_fill_ceiling   a streaming device fill (HBM write rate; the runtime's
//                    own fill is timed beside it and the faster one kept).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.hpp"

namespace {

constexpr int kWaves = 16;
constexpr int kTC = 16;                 // trees per group of lanes
constexpr int kDepth = 10;
constexpr int kNS = 1 << kDepth;        // heap slots per tree
constexpr int kRowB = 128;              // bytes per sibling-pair row: two copies of 16 trees
constexpr int kNodeB = kNS / 2 * kRowB; // 64 KB of sibling pairs (1-based heap nodes 2..2^D - 1)
constexpr int kLeafB = kNS * kTC * 4;   // 64 KB of leaves
constexpr int kRows = 256;              // bin rows of 128 bytes (32 KB)
constexpr int kILP = 4;

__device__ __forceinline__ int descend(int node, uint32_t code, uint32_t bin)
{
    int out;
    asm("v_sub_co_u32_sdwa %0, vcc, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1 src1_sel:DWORD\n\t"
        "v_addc_co_u32_e32 %0, vcc, %3, %3, vcc"
        : "=&v"(out)
        : "v"(code), "v"(bin), "v"(node)
        : "vcc");
    return out;
}

__device__ __forceinline__ void descend_pair(int &node, uint32_t &code, uint32_t bin, uint32_t pair)
{
    int n_out;
    uint32_t c_out, scratch;
    asm("v_sub_co_u32_sdwa %2, vcc, %3, %4 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1 src1_sel:DWORD\n\t"
        "v_cndmask_b32_sdwa %1, %5, %5, vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:WORD_1\n\t"
        "v_addc_co_u32_e32 %0, vcc, %6, %6, vcc"
        : "=&v"(n_out), "=&v"(c_out), "=&v"(scratch)
        : "v"(code), "v"(bin), "v"(pair), "v"(node)
        : "vcc");
    node = n_out;
    code = c_out;
}

__device__ __forceinline__ void descend_root(int &node, uint32_t &code, uint32_t &pair, uint32_t bin, uint32_t p1,
                                             uint32_t p2, uint32_t p3)
{
    int n_out;
    uint32_t c_out, p_out, scratch;
    asm("v_sub_co_u32_sdwa %3, vcc, %4, %5 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1 src1_sel:DWORD\n\t"
        "v_cndmask_b32_sdwa %1, %6, %6, vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:WORD_1\n\t"
        "v_cndmask_b32_e32 %2, %7, %8, vcc\n\t"
        "v_addc_co_u32_e32 %0, vcc, %9, %9, vcc"
        : "=&v"(n_out), "=&v"(c_out), "=&v"(p_out), "=&v"(scratch)
        : "v"(code), "v"(bin), "v"(p1), "v"(p2), "v"(p3), "v"(node)
        : "vcc");
    node = n_out;
    code = c_out;
    pair = p_out;
}

__device__ __forceinline__ uint32_t mix32(uint32_t h)
{
    h ^= h >> 15;
    h *= 2246822519u;
    h ^= h >> 13;
    h *= 3266489917u;
    return h ^ (h >> 16);
}

// The depth-10 traversal's walk, as the scoring kernel runs it with 16 trees
// per chunk: LDS holds 64 KB of sibling-pair codes (two copies of 16 trees,
// each copy's tree in its own 4-byte column), 64 KB of leaves and 256 bin
// rows; a wave walks 4 rows x 16 trees per group, 4 groups in flight; levels
// 0 and 1 take their pairs from registers, levels 2..8 read them from LDS,
// the last level reads none; then the leaves and the 16-lane sums.  Node
// codes hold a feature below 128 in the low byte and a rank in the high
// byte, so every address stays inside the arrays.
__global__ __launch_bounds__(64 * kWaves, 1) void k_visit_ceiling(int iters, uint32_t seed, float *sink)
{
    __shared__ __attribute__((aligned(16))) uint8_t lds[kNodeB + kLeafB + kRows * 128];
    const float *leaves = reinterpret_cast<const float *>(lds + kNodeB);
    uint8_t *bins = lds + kNodeB + kLeafB;
    for (int i = threadIdx.x; i < kNodeB / 4; i += 64 * kWaves) {
        const uint32_t h = mix32((uint32_t)i ^ seed), g = mix32(h);
        reinterpret_cast<uint32_t *>(lds)[i] = ((h & 127u) | (h & 0xff00u)) | (((g & 127u) | (g & 0xff00u)) << 16);
    }
    for (int i = threadIdx.x; i < kLeafB / 4; i += 64 * kWaves)
        reinterpret_cast<float *>(lds + kNodeB)[i] = (float)(mix32((uint32_t)i + seed) & 1023u) * (1.0f / 1024.0f);
    for (int i = threadIdx.x; i < kRows * 128 / 4; i += 64 * kWaves)
        reinterpret_cast<uint32_t *>(bins)[i] = mix32((uint32_t)i * 7u + seed);
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int t = lane % kTC, s = lane / kTC;
    const uint32_t col = 4u * (uint32_t)((s & 1) * 16 + t);
    const uint8_t *region = bins + wave * 16 * 128;        // 16 rows per wave, as in the scoring kernel
    const uint32_t root = *reinterpret_cast<const uint16_t *>(lds + col + 2);
    const uint32_t p1 = *reinterpret_cast<const uint32_t *>(lds + kRowB + col);
    const uint32_t p2 = *reinterpret_cast<const uint32_t *>(lds + 2 * kRowB + col);
    const uint32_t p3 = *reinterpret_cast<const uint32_t *>(lds + 3 * kRowB + col);
    float total = 0.0f;
    for (int it = 0; it < iters; ++it) {
        int node[kILP];
        uint32_t code[kILP], pair[kILP];
        const uint8_t *rowp[kILP];
#pragma unroll
        for (int a = 0; a < kILP; ++a) {
            rowp[a] = region + (a * 4 + s) * 128;
            node[a] = 1;
            code[a] = root;
        }
#pragma unroll
        for (int l = 0; l < kDepth; ++l) {
            uint32_t bin[kILP];
#pragma unroll
            for (int a = 0; a < kILP; ++a) {
                bin[a] = rowp[a][code[a] & 0xffu];
                if (l >= 2 && l < kDepth - 1)
                    pair[a] = *reinterpret_cast<const uint32_t *>(lds + (uint32_t)node[a] * kRowB + col);
            }
#pragma unroll
            for (int a = 0; a < kILP; ++a) {
                if (l == kDepth - 1) node[a] = descend(node[a], code[a], bin[a]);
                else if (l == 0) descend_root(node[a], code[a], pair[a], bin[a], p1, p2, p3);
                else descend_pair(node[a], code[a], bin[a], pair[a]);
            }
        }
        float v[kILP];
#pragma unroll
        for (int a = 0; a < kILP; ++a) v[a] = leaves[(node[a] - kNS) * kTC + t];
        hwsel::group_totals<kTC, kILP>(v);
#pragma unroll
        for (int a = 0; a < kILP; ++a) total += v[a];
    }
    if (total == -1.0f) sink[0] = total;       // keeps the walks live; sums of non-negative leaves never are
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256) void k_mfma_ceiling(int iters, float *sink)
{
    bf16x8 a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = (__bf16)(0.001f * (float)(threadIdx.x + i));
        b[i] = (__bf16)(0.002f * (float)i);
    }
    f32x16 acc[4] = {};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[q], 0, 0, 0);
    }
    float s = 0.0f;
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < 16; ++i) s += acc[q][i];
    if (s == 1234.5f) sink[0] = s;
}

// Streaming copy and fill: each thread moves 4 x 16 bytes per step, all
// loads of a step issued before its stores (the tail is guarded).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void k_copy_ceiling(const u32x4 *__restrict__ src, u32x4 *__restrict__ dst, int64_t n)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += 4 * stride) {
        u32x4 v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (i + q * stride < n) v[q] = __builtin_nontemporal_load(src + i + q * stride);
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (i + q * stride < n) __builtin_nontemporal_store(v[q], dst + i + q * stride);
    }
}

__global__ __launch_bounds__(256) void k_fill_ceiling(u32x4 *__restrict__ dst, int64_t n)
{
    const u32x4 z = {0u, 0u, 0u, 0u};
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        __builtin_nontemporal_store(z, dst + i);
}

int n_cus()
{
    int dev = 0, n = 256;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) !=
                                                 hipSuccess || n < 1)
        n = 256;
    return n;
}

}  // namespace

extern "C" {

// Node visits one launch makes: (workgroups) x 16 waves x 64 lanes x 4 walks x
// 10 levels per iteration.  sink: 4 bytes of device memory.
int64_t hwsel_ceiling_visits_per_launch(int iters) { return (int64_t)n_cus() * kWaves * 64 * kILP * kDepth * iters; }
int hwsel_ceiling_visits(int iters, float *sink, void *stream)
{
    hipLaunchKernelGGL(k_visit_ceiling, dim3(n_cus()), dim3(64 * kWaves), 0, (hipStream_t)stream, iters, 12345u, sink);
    return hipGetLastError() == hipSuccess ? 0 : 3;
}

// bf16 flops one launch makes: (2 workgroups per CU) x 4 waves x 4 products of
// 32 x 32 x 16 per iteration.
double hwsel_ceiling_mfma_flops_per_launch(int iters) { return 2.0 * n_cus() * 4 * 4 * 32768.0 * iters; }
int hwsel_ceiling_mfma(int iters, float *sink, void *stream)
{
    hipLaunchKernelGGL(k_mfma_ceiling, dim3(2 * n_cus()), dim3(256), 0, (hipStream_t)stream, iters, sink);
    return hipGetLastError() == hipSuccess ? 0 : 3;
}

// Copies n16 16-byte elements (both buffers device memory, 16-byte aligned).
int hwsel_ceiling_copy(const void *src, void *dst, int64_t n16, void *stream)
{
    hipLaunchKernelGGL(k_copy_ceiling, dim3(64 * n_cus()), dim3(256), 0, (hipStream_t)stream,
                       static_cast<const u32x4 *>(src), static_cast<u32x4 *>(dst), n16);
    return hipGetLastError() == hipSuccess ? 0 : 3;
}

// Writes n16 16-byte zeros (device memory, 16-byte aligned): with the
// kernel above (runtime = 0) or with the HIP runtime's own fill (runtime = 1,
// hipMemsetD32Async), whichever the caller times.
int hwsel_ceiling_fill(void *dst, int64_t n16, int runtime, void *stream)
{
    if (runtime)
        return hipMemsetD32Async((hipDeviceptr_t)dst, 0, (size_t)n16 * 4, (hipStream_t)stream) == hipSuccess ? 0 : 3;
    hipLaunchKernelGGL(k_fill_ceiling, dim3(64 * n_cus()), dim3(256), 0, (hipStream_t)stream,
                       static_cast<u32x4 *>(dst), n16);
    return hipGetLastError() == hipSuccess ? 0 : 3;
}

}  // extern "C"
