// Configuration catalogue (section "Configuration Space", Table
// "Configuration knobs") and its static validity mask (section "Validity
// Constraints", Table "Static validity constraints").
//
// A point index decodes to its knobs by mixed radix (first knob slowest), so
// the mask pass never stores the catalogue: each thread decodes one group of
// 18 consecutive points (the three fastest knobs' combinations) once and
// tests the 18; a block's mask bytes leave LDS as whole words.  The
// compaction is one workgroup per problem, an ordered scan over its mask.
#include "internal.hpp"

namespace hwsel {
namespace {

constexpr int64_t kCat = HWSEL_CATALOGUE_SIZE;
__constant__ int16_t kTileM[4] = {64, 128, 192, 256};
__constant__ int16_t kTileN[9] = {16, 32, 48, 64, 80, 96, 128, 192, 256};
__constant__ int16_t kTileK[5] = {32, 64, 128, 256, 512};
// (C_M, C_N) in {1,2,4,8,16}^2 with C_M C_N <= 16, C_M slower
__constant__ uint8_t kClusterM[15] = {1, 1, 1, 1, 1, 2, 2, 2, 2, 4, 4, 4, 8, 8, 16};
__constant__ uint8_t kClusterN[15] = {1, 2, 4, 8, 16, 1, 2, 4, 8, 1, 2, 4, 1, 2, 1};

struct Knobs {
    int32_t tm, tn, tk, st, cm, cn, ks, es, ts;
};

// Point index -> knobs (the index fits in 32 bits, so the divisions by
// constants are 32-bit multiply-shifts).
__device__ __forceinline__ Knobs decode(int64_t index)
{
    uint32_t i = (uint32_t)index;
    Knobs k;
    k.ts = (int32_t)(i % 2u); i /= 2u;
    k.es = (int32_t)(i % 3u); i /= 3u;
    k.ks = (int32_t)(i % 3u); i /= 3u;
    const uint32_t cl = i % 15u; i /= 15u;
    k.st = 2 + (int32_t)(i % 11u); i /= 11u;
    k.tk = kTileK[i % 5u]; i /= 5u;
    k.tn = kTileN[i % 9u]; i /= 9u;
    k.tm = kTileM[i];
    k.cm = kClusterM[cl];
    k.cn = kClusterN[cl];
    return k;
}

__device__ __forceinline__ bool valid(const HwDev &h, const hwsel_problem_t &pb, uint32_t flags, const Knobs &k)
{
    const int64_t M = pb.M > 1 ? pb.M : 1, N = pb.N > 1 ? pb.N : 1;
    const int layout = pb.layout < 3 ? pb.layout : 3;
    const int64_t b = (pb.dtype < 2 ? pb.dtype : 2) == 2 ? 1 : 2;
    const int64_t frag = (int64_t)(k.tm < 64 ? k.tm : 64) * (k.tn < 32 ? k.tn : 32) * 2;
    const int64_t epi = k.es == 0 ? 0 : (k.es == 1 ? 2 * frag : 4 * frag);
    bool ok = k.ts != 1 || k.ks == 2;                                   // Stream-K needs cooperative
    ok &= k.ks != 2 || k.tm % 128 == 0;                                 // cooperative splits T_M in two
    ok &= (int64_t)k.st * (k.tm + k.tn) * k.tk * b + epi + h.smem_rsv <= h.smem_block;
    if (layout == 2 || layout == 3) ok &= k.tk <= 256 * k.cn;           // A column-major
    if (layout == 1 || layout == 3) ok &= k.tk <= 256 * k.cm;           // B row-major
    if (flags & 1u) ok &= k.tn <= 2 * M && k.tn <= 2 * N;
    return ok;
}

__global__ void k_zero_i64(int64_t *__restrict__ a, int32_t n)
{
    const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) a[i] = 0;
}

constexpr int kMaskThreads = 256;
constexpr int64_t kWords = (kCat + 3) / 4;
// The three fastest knobs (tile scheduler, epilogue, kernel schedule) take
// 2 x 3 x 3 = 18 values; the 18 consecutive points of a group share every
// other knob, decoded once.
constexpr int kGroup = 18;
constexpr int64_t kGroups = kCat / kGroup;
static_assert(kCat % kGroup == 0 && kCat % 4 == 0, "catalogue groups");
constexpr int kBlockBytes = kMaskThreads * kGroup;           // points (mask bytes) per block

__global__ __launch_bounds__(kMaskThreads) void k_catalogue_mask(HwDev h, const hwsel_problem_t *__restrict__ probs,
                                                                 int32_t P, uint32_t flags, uint8_t *__restrict__ mask,
                                                                 int64_t *__restrict__ n_valid)
{
    __shared__ uint32_t stage[kBlockBytes / 4];
    __shared__ int32_t wave_cnt[kMaskThreads / 64];
    uint8_t *stage_b = reinterpret_cast<uint8_t *>(stage);
    const int64_t g = (int64_t)blockIdx.x * kMaskThreads + threadIdx.x;   // this thread's group
    const int64_t block_point0 = (int64_t)blockIdx.x * kBlockBytes;
    const int block_bytes = (int)(kCat - block_point0 < kBlockBytes ? kCat - block_point0 : kBlockBytes);
    for (int32_t p = blockIdx.y; p < P; p += gridDim.y) {
        const hwsel_problem_t pb = probs[p];
        float cnt = 0.0f;
        if (g < kGroups) {
            Knobs k = decode(g * kGroup);                // the group's first point: fast knobs 0
#pragma unroll
            for (int j = 0; j < kGroup; ++j) {
                k.ts = j % 2;
                k.es = (j / 2) % 3;
                k.ks = j / 6;
                const bool ok = valid(h, pb, flags, k);
                stage_b[threadIdx.x * kGroup + j] = ok ? 1 : 0;
                cnt += ok ? 1.0f : 0.0f;
            }
        }
        // per-wave totals (exact: at most 64 x 18 in fp32), then one LDS step
        float tot[1] = {cnt};
        group_totals<64, 1>(tot);
        if ((threadIdx.x & 63) == 63) wave_cnt[threadIdx.x >> 6] = (int32_t)tot[0];
        __syncthreads();
        uint32_t *row = reinterpret_cast<uint32_t *>(mask + (int64_t)p * kCat + block_point0);
        for (int e = threadIdx.x; e < block_bytes / 4; e += kMaskThreads) row[e] = stage[e];
        if (threadIdx.x == 0) {
            int32_t t = 0;
#pragma unroll
            for (int i = 0; i < kMaskThreads / 64; ++i) t += wave_cnt[i];
            if (t) atomicAdd(reinterpret_cast<unsigned long long *>(n_valid + p), (unsigned long long)t);
        }
        __syncthreads();                                 // stage and wave_cnt are reused for the next problem
    }
}

// seg[0] = 0, seg[p + 1] = seg[p] + max(n_valid[p], 0): one workgroup, each
// thread summing a contiguous range of problems, the range sums scanned in
// LDS (exact integer sums, so the order is free).
constexpr int kOffsetThreads = 1024;

__global__ __launch_bounds__(kOffsetThreads) void k_catalogue_offsets(const int64_t *__restrict__ n_valid, int32_t P,
                                                                      int64_t *__restrict__ seg)
{
    __shared__ int64_t part[kOffsetThreads];
    const int t = threadIdx.x;
    const int64_t per = ((int64_t)P + kOffsetThreads - 1) / kOffsetThreads;
    const int64_t lo = t * per < P ? t * per : P, hi = lo + per < P ? lo + per : P;
    int64_t s = 0;
    for (int64_t i = lo; i < hi; ++i) s += n_valid[i] > 0 ? n_valid[i] : 0;
    part[t] = s;
    __syncthreads();
    for (int d = 1; d < kOffsetThreads; d <<= 1) {      // inclusive scan of the range sums
        const int64_t v = t >= d ? part[t - d] : 0;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    int64_t acc = t > 0 ? part[t - 1] : 0;
    if (t == 0) seg[0] = 0;
    for (int64_t i = lo; i < hi; ++i) {
        acc += n_valid[i] > 0 ? n_valid[i] : 0;
        seg[i + 1] = acc;
    }
}

constexpr int kCompactThreads = 1024;

// Ordered compaction of one problem's mask (one workgroup per problem).  A
// step covers kBlocks consecutive blocks of 1,024 four-byte words (4 points
// each); thread i takes word i of every block, all loads issued together.
// Within a wave, the valid points of lower lanes are counted from one ballot
// per byte position (mbcnt); across the 16 waves and the blocks, the wave
// totals meet in LDS.  Two barriers per step of 16,384 points.
constexpr int kBlocks = 4;

__global__ __launch_bounds__(kCompactThreads) void k_catalogue_compact(const uint8_t *__restrict__ mask,
                                                                       const int64_t *__restrict__ seg,
                                                                       int32_t *__restrict__ point, int64_t cap)
{
    constexpr int kWavesC = kCompactThreads / 64;
    __shared__ int32_t wave_total[kBlocks][kWavesC];
    const int32_t p = blockIdx.x;
    const int wave = threadIdx.x >> 6;
    const uint32_t *row = reinterpret_cast<const uint32_t *>(mask + (int64_t)p * kCat);
    int64_t out = seg[p];
    for (int64_t w0 = 0; w0 < kWords; w0 += kBlocks * kCompactThreads) {
        uint32_t word[kBlocks];
#pragma unroll
        for (int k = 0; k < kBlocks; ++k) {
            const int64_t w = w0 + k * kCompactThreads + threadIdx.x;
            word[k] = w < kWords ? row[w] : 0u;
        }
        int32_t below[kBlocks];              // valid points of block k in lower lanes of this wave
#pragma unroll
        for (int k = 0; k < kBlocks; ++k) {
            int32_t bl = 0, total = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint64_t b = __ballot((word[k] >> (8 * q)) & 1u);
                bl += (int32_t)__builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0u));
                total += __popcll(b);
            }
            below[k] = bl;
            if ((threadIdx.x & 63) == 0) wave_total[k][wave] = total;
        }
        lds_barrier();
        int64_t base = out;                  // points of the earlier blocks of this step
#pragma unroll
        for (int k = 0; k < kBlocks; ++k) {
            int32_t before = 0, all = 0;
#pragma unroll
            for (int i = 0; i < kWavesC; ++i) {
                const int32_t t = wave_total[k][i];
                before += i < wave ? t : 0;
                all += t;
            }
            int64_t pos = base + before + below[k];
            const int64_t w = w0 + k * kCompactThreads + threadIdx.x;
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if ((word[k] >> (8 * q)) & 1u) {
                    if (pos < cap) point[pos] = (int32_t)(4 * w + q);
                    ++pos;
                }
            base += all;
        }
        out = base;
        lds_barrier();                        // wave_total is rewritten by the next step
    }
}

__global__ void k_catalogue_candidates(const hwsel_problem_t *__restrict__ probs, int32_t P,
                                       const int64_t *__restrict__ seg, const int32_t *__restrict__ point, int64_t R,
                                       hwsel_cands_out_t out)
{
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    // the wave's first row (wave-uniform): one scalar search per wave
    const int64_t r_first = (int64_t)blockIdx.x * blockDim.x + __builtin_amdgcn_readfirstlane(threadIdx.x & ~63u);
    if (r >= R) return;
    const int32_t p = segment_of_row_after(seg, P, r, r_first);
    int64_t i = point ? (int64_t)point[r] : r - seg[p];
    i = i < 0 ? 0 : (i >= kCat ? kCat - 1 : i);
    const Knobs k = decode(i);
    const int dt = probs[p].dtype < 2 ? probs[p].dtype : 2;
    out.tile_m[r] = (uint16_t)k.tm;
    out.tile_n[r] = (uint16_t)k.tn;
    out.tile_k[r] = (uint16_t)k.tk;
    out.inst_n[r] = (uint16_t)k.tn;
    out.stages[r] = (uint8_t)k.st;
    out.cluster_m[r] = (uint8_t)k.cm;
    out.cluster_n[r] = (uint8_t)k.cn;
    out.swizzle[r] = 1;
    out.inst_m_div16[r] = 4;
    out.inst_k[r] = dt == 2 ? 32 : 16;
    out.kernel_sched[r] = (uint8_t)k.ks;
    out.epi_sched[r] = (uint8_t)k.es;
    out.tile_sched[r] = (uint8_t)k.ts;
}

// Four consecutive rows per thread, each field written with one 4-byte
// (8-bit fields) or 8-byte (16-bit fields) store; taken when every field
// array is aligned for that (the rows of a partial last quad are stored one
// by one).
__global__ void k_catalogue_candidates4(const hwsel_problem_t *__restrict__ probs, int32_t P,
                                        const int64_t *__restrict__ seg, const int32_t *__restrict__ point,
                                        int64_t R, hwsel_cands_out_t out)
{
    const int64_t r0 = 4 * ((int64_t)blockIdx.x * blockDim.x + threadIdx.x);
    const int64_t r_first = 4 * ((int64_t)blockIdx.x * blockDim.x + __builtin_amdgcn_readfirstlane(threadIdx.x & ~63u));
    if (r0 >= R) return;
    int32_t p = segment_of_row_after(seg, P, r0, r_first);
    uint32_t tm[4], tn[4], tk[4], st[4], cm[4], cn[4], ik[4], ks[4], es[4], ts[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int64_t r = r0 + j < R ? r0 + j : R - 1;
        while (p + 1 < P && seg[p + 1] <= r) ++p;
        int64_t i = point ? (int64_t)point[r] : r - seg[p];
        i = i < 0 ? 0 : (i >= kCat ? kCat - 1 : i);
        const Knobs k = decode(i);
        const int dt = probs[p].dtype < 2 ? probs[p].dtype : 2;
        tm[j] = (uint32_t)k.tm; tn[j] = (uint32_t)k.tn; tk[j] = (uint32_t)k.tk; st[j] = (uint32_t)k.st;
        cm[j] = (uint32_t)k.cm; cn[j] = (uint32_t)k.cn; ik[j] = dt == 2 ? 32u : 16u;
        ks[j] = (uint32_t)k.ks; es[j] = (uint32_t)k.es; ts[j] = (uint32_t)k.ts;
    }
    if (r0 + 3 < R) {
        auto p16 = [](const uint32_t (&v)[4]) {
            return make_uint2(v[0] | (v[1] << 16), v[2] | (v[3] << 16));
        };
        auto p8 = [](const uint32_t (&v)[4]) { return v[0] | (v[1] << 8) | (v[2] << 16) | (v[3] << 24); };
        *reinterpret_cast<uint2 *>(out.tile_m + r0) = p16(tm);
        *reinterpret_cast<uint2 *>(out.tile_n + r0) = p16(tn);
        *reinterpret_cast<uint2 *>(out.tile_k + r0) = p16(tk);
        *reinterpret_cast<uint2 *>(out.inst_n + r0) = p16(tn);
        *reinterpret_cast<uint32_t *>(out.stages + r0) = p8(st);
        *reinterpret_cast<uint32_t *>(out.cluster_m + r0) = p8(cm);
        *reinterpret_cast<uint32_t *>(out.cluster_n + r0) = p8(cn);
        *reinterpret_cast<uint32_t *>(out.swizzle + r0) = 0x01010101u;
        *reinterpret_cast<uint32_t *>(out.inst_m_div16 + r0) = 0x04040404u;
        *reinterpret_cast<uint32_t *>(out.inst_k + r0) = p8(ik);
        *reinterpret_cast<uint32_t *>(out.kernel_sched + r0) = p8(ks);
        *reinterpret_cast<uint32_t *>(out.epi_sched + r0) = p8(es);
        *reinterpret_cast<uint32_t *>(out.tile_sched + r0) = p8(ts);
    } else {
        for (int j = 0; j < 4 && r0 + j < R; ++j) {
            const int64_t r = r0 + j;
            out.tile_m[r] = (uint16_t)tm[j];
            out.tile_n[r] = (uint16_t)tn[j];
            out.tile_k[r] = (uint16_t)tk[j];
            out.inst_n[r] = (uint16_t)tn[j];
            out.stages[r] = (uint8_t)st[j];
            out.cluster_m[r] = (uint8_t)cm[j];
            out.cluster_n[r] = (uint8_t)cn[j];
            out.swizzle[r] = 1;
            out.inst_m_div16[r] = 4;
            out.inst_k[r] = (uint8_t)ik[j];
            out.kernel_sched[r] = (uint8_t)ks[j];
            out.epi_sched[r] = (uint8_t)es[j];
            out.tile_sched[r] = (uint8_t)ts[j];
        }
    }
}

}  // namespace

hipError_t launch_catalogue_mask(const HwDev &h, const hwsel_problem_t *probs, int32_t P, uint32_t flags,
                                 uint8_t *mask, int64_t *n_valid, hipStream_t s)
{
    hipLaunchKernelGGL(k_zero_i64, dim3((P + 255) / 256), dim3(256), 0, s, n_valid, P);
    const dim3 grid((unsigned)((kGroups + kMaskThreads - 1) / kMaskThreads), (unsigned)(P < 65535 ? P : 65535));
    hipLaunchKernelGGL(k_catalogue_mask, grid, dim3(kMaskThreads), 0, s, h, probs, P, flags, mask, n_valid);
    return hipGetLastError();
}

hipError_t launch_catalogue_compact(const uint8_t *mask, const int64_t *n_valid, int32_t P, int64_t *seg,
                                    int32_t *point, int64_t cap, hipStream_t s)
{
    hipLaunchKernelGGL(k_catalogue_offsets, dim3(1), dim3(kOffsetThreads), 0, s, n_valid, P, seg);
    hipLaunchKernelGGL(k_catalogue_compact, dim3(P), dim3(kCompactThreads), 0, s, mask, seg, point, cap);
    return hipGetLastError();
}

hipError_t launch_catalogue_candidates(const hwsel_problem_t *probs, int32_t P, const int64_t *seg,
                                       const int32_t *point, int64_t R, const hwsel_cands_out_t &out, hipStream_t s)
{
    auto al = [](const void *q, uintptr_t a) { return ((uintptr_t)q & (a - 1)) == 0; };
    const bool packed = al(out.tile_m, 8) && al(out.tile_n, 8) && al(out.tile_k, 8) && al(out.inst_n, 8) &&
                        al(out.stages, 4) && al(out.cluster_m, 4) && al(out.cluster_n, 4) && al(out.swizzle, 4) &&
                        al(out.inst_m_div16, 4) && al(out.inst_k, 4) && al(out.kernel_sched, 4) &&
                        al(out.epi_sched, 4) && al(out.tile_sched, 4);
    if (packed) {
        const int64_t quads = (R + 3) / 4;
        hipLaunchKernelGGL(k_catalogue_candidates4, dim3((unsigned)((quads + 255) / 256)), dim3(256), 0, s, probs, P,
                           seg, point, R, out);
    } else {
        hipLaunchKernelGGL(k_catalogue_candidates, dim3((unsigned)((R + 255) / 256)), dim3(256), 0, s, probs, P,
                           seg, point, R, out);
    }
    return hipGetLastError();
}

}  // namespace hwsel
