// Selection metrics and baselines over problems (section "Selection Regret
// (The Target Metric)"; baselines of section "Final Fit and Test Protocol").
//
// Per-problem passes read each segment once (one workgroup per problem);
// the aggregates are exact order statistics and fixed-order binary64 sums
// over at most a few hundred thousand problems.
#include <limits.h>

#include <mutex>

#include "internal.hpp"

namespace hwsel {
namespace {

constexpr int kEvalThreads = 256;

// Strictly faster runtime; NaN is slower than everything, +inf included.
__device__ __forceinline__ bool faster(float a, float b)
{
    const bool na = a != a, nb = b != b;
    if (na || nb) return !na && nb;
    return a < b;
}

// y = t_best / t: 1 for equal runtimes (inf included), 0 for NaN.
__device__ __forceinline__ double y_of(float t_best, float t)
{
    if (t == t_best) return 1.0;
    if (t != t) return 0.0;
    return (double)t_best / (double)t;
}

// Fastest runtime of rows [base, base + n) for a whole workgroup.
__device__ float block_fastest(const float *__restrict__ rt, int64_t base, int64_t n, float *red)
{
    float best = __builtin_nanf("");
    for (int64_t j = threadIdx.x; j < n; j += blockDim.x) {
        const float t = rt[base + j];
        if (faster(t, best)) best = t;
    }
    red[threadIdx.x] = best;
    __syncthreads();
    for (int s = blockDim.x / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s && faster(red[threadIdx.x + s], red[threadIdx.x])) red[threadIdx.x] = red[threadIdx.x + s];
        __syncthreads();
    }
    const float out = red[0];
    __syncthreads();
    return out;
}

// Fixed-shape tree sums over the workgroup (same order every run).
__device__ double block_sum(double v, double *red)
{
    red[threadIdx.x] = v;
    __syncthreads();
    for (int s = blockDim.x / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
        __syncthreads();
    }
    const double out = red[0];
    __syncthreads();
    return out;
}

__device__ int64_t block_count(int64_t v, int64_t *red)
{
    red[threadIdx.x] = v;
    __syncthreads();
    for (int s = blockDim.x / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
        __syncthreads();
    }
    const int64_t out = red[0];
    __syncthreads();
    return out;
}

__global__ __launch_bounds__(kEvalThreads) void k_eval_groups(const float *__restrict__ rt,
                                                              const int64_t *__restrict__ seg, int32_t P,
                                                              const int32_t *__restrict__ idx, int32_t k,
                                                              double *__restrict__ regret, int32_t *__restrict__ rank,
                                                              double *__restrict__ ybar)
{
    __shared__ double red[kEvalThreads];
    const int32_t p = blockIdx.x;
    if (p >= P) return;                                   // one workgroup per problem
    const int64_t base = seg[p], n = seg[p + 1] - seg[p];
    if (n <= 0) {
        if (threadIdx.x == 0) {
            regret[p] = __builtin_nan("");
            rank[p] = 0;
            ybar[p] = __builtin_nan("");
        }
        return;
    }
    const float t_best = block_fastest(rt, base, n, reinterpret_cast<float *>(red));
    const int32_t sel = idx[(int64_t)p * k];
    const bool counted = sel >= 0 && sel < n;
    const float t_sel = counted ? rt[base + sel] : 0.0f;
    double ys = 0.0;
    int64_t nb = 0;
    for (int64_t j = threadIdx.x; j < n; j += kEvalThreads) {
        const float t = rt[base + j];
        ys += y_of(t_best, t);
        nb += faster(t, t_sel) ? 1 : 0;
    }
    ys = block_sum(ys, red);
    nb = block_count(nb, reinterpret_cast<int64_t *>(red));
    if (threadIdx.x == 0) {
        ybar[p] = ys / (double)n;
        regret[p] = counted ? 1.0 - y_of(t_best, t_sel) : __builtin_nan("");
        rank[p] = counted ? (int32_t)(1 + nb) : 0;
    }
}

// Order statistics of the counted regrets by radix selection: for each
// requested rank, eight passes over the 64-bit keys (an order-preserving map
// of the binary64 values), one byte per pass from the top, each counting the
// candidates that still match the prefix.  Linear in P per pass; the counts
// are integers, so the result is exact and independent of scheduling.
// stats[i] = the value of rank ranks[i] (0-based) among the counted regrets,
// for the ranks of the median and the 95th percentile.
__device__ __forceinline__ uint64_t order_key(double v)
{
    const uint64_t b = __builtin_bit_cast(uint64_t, v);
    return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ __forceinline__ double key_value(uint64_t k)
{
    return __builtin_bit_cast(double, (k >> 63) ? (k & 0x7fffffffffffffffull) : ~k);
}

constexpr int kSelectThreads = 1024;

__global__ __launch_bounds__(kSelectThreads) void k_eval_select(const double *__restrict__ regret,
                                                                const int32_t *__restrict__ rank, int32_t P,
                                                                double *__restrict__ stats)
{
    __shared__ int64_t hist[256];
    __shared__ int64_t cnt_s;
    __shared__ uint64_t prefix_s;
    __shared__ int64_t k_s;
    // number of counted problems
    if (threadIdx.x == 0) cnt_s = 0;
    __syncthreads();
    int64_t local = 0;
    for (int32_t i = threadIdx.x; i < P; i += kSelectThreads) local += rank[i] != 0;
    atomicAdd(reinterpret_cast<unsigned long long *>(&cnt_s), (unsigned long long)local);
    __syncthreads();
    const int64_t n = cnt_s;
    if (n == 0) return;
    // ranks: floor and ceil positions of q (n - 1) for q = 0.5, 0.95
    int64_t want[4];
    {
        const double p50 = 0.5 * (double)(n - 1), p95 = 0.95 * (double)(n - 1);
        const int64_t l50 = (int64_t)__builtin_floor(p50), l95 = (int64_t)__builtin_floor(p95);
        want[0] = l50;
        want[1] = l50 + 1 < n ? l50 + 1 : n - 1;
        want[2] = l95;
        want[3] = l95 + 1 < n ? l95 + 1 : n - 1;
    }
    for (int t = 0; t < 4; ++t) {
        uint64_t prefix = 0, mask = 0;
        int64_t k = want[t];
        for (int shift = 56; shift >= 0; shift -= 8) {
            for (int b = threadIdx.x; b < 256; b += kSelectThreads) hist[b] = 0;
            __syncthreads();
            for (int32_t i = threadIdx.x; i < P; i += kSelectThreads) {
                if (rank[i] == 0) continue;
                const uint64_t key = order_key(regret[i]);
                if ((key & mask) == prefix)
                    atomicAdd(reinterpret_cast<unsigned long long *>(&hist[(key >> shift) & 255u]), 1ull);
            }
            __syncthreads();
            if (threadIdx.x == 0) {
                int64_t acc = 0;
                int d = 0;
                for (; d < 255; ++d) {
                    if (acc + hist[d] > k) break;
                    acc += hist[d];
                }
                k_s = k - acc;
                prefix_s = prefix | ((uint64_t)d << shift);
            }
            __syncthreads();
            prefix = prefix_s;
            k = k_s;
            mask |= 0xffull << shift;
            __syncthreads();
        }
        if (threadIdx.x == 0) stats[t] = key_value(prefix);
    }
}

// value at position q (n - 1) by linear interpolation between its two
// neighbouring order statistics
__device__ double interpolate(double lo_v, double hi_v, int64_t n, double q)
{
    const double pos = q * (double)(n - 1);
    const double lo = __builtin_floor(pos);
    return lo_v + (pos - lo) * (hi_v - lo_v);
}

__global__ void k_eval_aggregate(const double *__restrict__ regret, const int32_t *__restrict__ rank,
                                 const double *__restrict__ ybar, const double *__restrict__ stats, int32_t P,
                                 double *__restrict__ out, double *__restrict__ regret_out,
                                 int32_t *__restrict__ rank_out, double *__restrict__ ybar_out)
{
    if (threadIdx.x == 0) {
        int64_t cnt = 0, top1 = 0, top5 = 0, w5 = 0;
        double sum = 0.0, rsum = 0.0, mx = -__builtin_inf();
        for (int32_t p = 0; p < P; ++p) {
            if (rank[p] == 0) continue;
            const double r = regret[p];
            ++cnt;
            sum += r;
            rsum += 1.0 - ybar[p];
            mx = r > mx ? r : mx;
            top1 += rank[p] == 1;
            top5 += rank[p] <= 5;
            w5 += r <= 0.05;
        }
        if (cnt == 0) {
            for (int i = 0; i < 8; ++i) out[i] = __builtin_nan("");
            out[8] = 0.0;
        } else {
            out[0] = sum / (double)cnt;
            out[1] = interpolate(stats[0], stats[1], cnt, 0.5);
            out[2] = interpolate(stats[2], stats[3], cnt, 0.95);
            out[3] = mx;
            out[4] = (double)top1 / (double)cnt;
            out[5] = (double)top5 / (double)cnt;
            out[6] = (double)w5 / (double)cnt;
            out[7] = rsum / (double)cnt;
            out[8] = (double)cnt;
        }
    }
    for (int32_t p = threadIdx.x; p < P; p += blockDim.x) {
        if (regret_out) regret_out[p] = regret[p];
        if (rank_out) rank_out[p] = rank[p];
        if (ybar_out) ybar_out[p] = ybar[p];
    }
}

// Up to kSmallP problems: one workgroup stages the per-problem values in LDS,
// sorts the counted regrets with a bitonic network held in registers (element
// tid + 1024 m in thread tid; partners less than 64 apart are exchanged
// inside the wave, the others through LDS or within the thread), counts in
// parallel, and wave 0 takes the two sums in problem order; the same outputs
// as k_eval_select + k_eval_aggregate.
constexpr int kSmallP = 4096;
constexpr int kSmallT = 1024, kSmallM = kSmallP / kSmallT;

// Lane l's double as a wave-uniform value.
__device__ __forceinline__ double bcast_lane(double v, int l)
{
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)u, l), hi = __builtin_amdgcn_readlane((uint32_t)(u >> 32), l);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// One compare-exchange of the network as seen from element i, which holds
// `own` and whose partner (index i ^ j) holds `other`: the lower index keeps
// the smaller value when the block of size k runs upwards.
__device__ __forceinline__ double bitonic_keep(double own, double other, int32_t i, int32_t j, int32_t k)
{
    const bool up = (i & k) == 0;
    const bool lower = (i & j) == 0;
    const double a = lower ? own : other, b = lower ? other : own;   // a at the lower index
    const bool swap = (a > b) == up;
    return lower ? (swap ? b : a) : (swap ? a : b);
}

__global__ __launch_bounds__(kSmallT) void k_eval_small(const double *__restrict__ regret,
                                                        const int32_t *__restrict__ rank,
                                                        const double *__restrict__ ybar, int32_t P,
                                                        double *__restrict__ out, double *__restrict__ regret_out,
                                                        int32_t *__restrict__ rank_out, double *__restrict__ ybar_out)
{
    __shared__ double reg_s[kSmallP], yb_s[kSmallP], sorted[kSmallP];
    __shared__ int32_t rank_s[kSmallP];
    __shared__ double wmax[kSmallT / 64];
    __shared__ int64_t wcnt[4][kSmallT / 64];
    const int32_t tid = threadIdx.x;
    int32_t n2 = 2;
    while (n2 < P) n2 <<= 1;
    const int32_t mcount = (n2 + kSmallT - 1) / kSmallT;      // register slots in use (uniform)
    double v[kSmallM];
    int64_t cnt = 0, top1 = 0, top5 = 0, w5 = 0;
    double mx = -__builtin_inf();
#pragma unroll
    for (int m = 0; m < kSmallM; ++m) {
        const int32_t i = tid + kSmallT * m;
        const bool in = i < P;
        const double r = in ? regret[i] : 0.0;
        const int32_t rk = in ? rank[i] : 0;
        reg_s[i] = r;
        yb_s[i] = in ? ybar[i] : 0.0;
        rank_s[i] = rk;
        const bool c = rk != 0;
        v[m] = c ? r : __builtin_inf();                          // uncounted sort last
        cnt += c;
        top1 += c && rk == 1;
        top5 += c && rk <= 5;
        w5 += c && r <= 0.05;
        mx = (c && r > mx) ? r : mx;
    }
    for (int32_t k = 2; k <= n2; k <<= 1)
        for (int32_t j = k >> 1; j > 0; j >>= 1) {
            if (j >= kSmallT) {                                     // partner in the same thread
                static_assert(kSmallM == 4, "slot pairs below");
                auto cx = [&](double &lo, double &hi, int m) {
                    const bool swap = (lo > hi) == (((tid + kSmallT * m) & k) == 0);
                    const double a = lo, b = hi;
                    lo = swap ? b : a;
                    hi = swap ? a : b;
                };
                if (j == kSmallT) {                                 // slots m and m + 1
                    cx(v[0], v[1], 0);
                    if (mcount > 2) cx(v[2], v[3], 2);
                } else {                                            // slots m and m + 2
                    cx(v[0], v[2], 0);
                    cx(v[1], v[3], 1);
                }
            } else if (j >= 64) {                                   // partner in another wave
#pragma unroll
                for (int m = 0; m < kSmallM; ++m)
                    if (m < mcount) sorted[tid + kSmallT * m] = v[m];
                __syncthreads();
#pragma unroll
                for (int m = 0; m < kSmallM; ++m)
                    if (m < mcount) {
                        const int32_t i = tid + kSmallT * m;
                        v[m] = bitonic_keep(v[m], sorted[i ^ j], i, j, k);
                    }
                __syncthreads();
            } else {                                                // partner in the same wave
#pragma unroll
                for (int m = 0; m < kSmallM; ++m)
                    if (m < mcount) {
                        const int32_t i = tid + kSmallT * m;
                        v[m] = bitonic_keep(v[m], __shfl_xor(v[m], j), i, j, k);
                    }
            }
        }
#pragma unroll
    for (int m = 0; m < kSmallM; ++m)
        if (m < mcount) sorted[tid + kSmallT * m] = v[m];
    // counts and the maximum: wave totals, then the waves in order (integer
    // sums and a maximum do not depend on the order)
    for (int off = 32; off > 0; off >>= 1) {
        cnt += __shfl_xor(cnt, off);
        top1 += __shfl_xor(top1, off);
        top5 += __shfl_xor(top5, off);
        w5 += __shfl_xor(w5, off);
        const double o = __shfl_xor(mx, off);
        mx = o > mx ? o : mx;
    }
    if ((tid & 63) == 0) {
        const int w = tid >> 6;
        wcnt[0][w] = cnt; wcnt[1][w] = top1; wcnt[2][w] = top5; wcnt[3][w] = w5;
        wmax[w] = mx;
    }
    __syncthreads();
    if (tid < 64) {
        // the sums in problem order: wave 0 loads 64 problems at a time and
        // adds them one by one from lane values broadcast as scalars (adding
        // +0.0 for an uncounted problem leaves a sum that starts at +0.0
        // unchanged)
        double sum = 0.0, rsum = 0.0;
        for (int32_t base = 0; base < P; base += 64) {
            const int32_t p = base + tid < P ? base + tid : P - 1;   // lanes past P read problem P - 1
            const bool c = base + tid < P && rank_s[p] != 0;
            const double r = c ? reg_s[p] : 0.0;
            const double y = c ? 1.0 - yb_s[p] : 0.0;
            const int n = P - base < 64 ? P - base : 64;
            for (int l = 0; l < n; ++l) {
                sum += bcast_lane(r, l);
                rsum += bcast_lane(y, l);
            }
        }
        cnt = top1 = top5 = w5 = 0;
        mx = -__builtin_inf();
#pragma unroll 1
        for (int w = 0; w < kSmallT / 64; ++w) {
            cnt += wcnt[0][w]; top1 += wcnt[1][w]; top5 += wcnt[2][w]; w5 += wcnt[3][w];
            mx = wmax[w] > mx ? wmax[w] : mx;
        }
        if (tid == 0) {
            if (cnt == 0) {
                for (int i = 0; i < 8; ++i) out[i] = __builtin_nan("");
                out[8] = 0.0;
            } else {
                const double p50 = 0.5 * (double)(cnt - 1), p95 = 0.95 * (double)(cnt - 1);
                const int64_t l50 = (int64_t)__builtin_floor(p50), l95 = (int64_t)__builtin_floor(p95);
                const int64_t h50 = l50 + 1 < cnt ? l50 + 1 : cnt - 1, h95 = l95 + 1 < cnt ? l95 + 1 : cnt - 1;
                out[0] = sum / (double)cnt;
                out[1] = interpolate(sorted[l50], sorted[h50], cnt, 0.5);
                out[2] = interpolate(sorted[l95], sorted[h95], cnt, 0.95);
                out[3] = mx;
                out[4] = (double)top1 / (double)cnt;
                out[5] = (double)top5 / (double)cnt;
                out[6] = (double)w5 / (double)cnt;
                out[7] = rsum / (double)cnt;
                out[8] = (double)cnt;
            }
        }
    }
    for (int32_t p = tid; p < P; p += kSmallT) {
        if (regret_out) regret_out[p] = reg_s[p];
        if (rank_out) rank_out[p] = rank_s[p];
        if (ybar_out) ybar_out[p] = yb_s[p];
    }
}

// ---------------------------------------------------------------------------
// Best static configuration
// ---------------------------------------------------------------------------
__global__ void k_fill_i32(int32_t *__restrict__ a, int64_t n, int32_t v)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        a[i] = v;
}

// first[p][id] = lowest local index of id in problem p's segment.
__global__ void k_static_first(const int64_t *__restrict__ seg, int32_t P, const int32_t *__restrict__ cfg,
                               int32_t n_cfg, int32_t *__restrict__ first)
{
    const int64_t R = seg[P];
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    // the wave's first row (wave-uniform): one scalar search per wave
    int64_t r_first = (int64_t)blockIdx.x * blockDim.x + __builtin_amdgcn_readfirstlane(threadIdx.x & ~63u);
    for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < R; r += stride, r_first += stride) {
        const int32_t p = segment_of_row_after(seg, P, r, r_first);
        const int32_t id = cfg[r];
        if (id < 0 || id >= n_cfg) continue;
        if (r < seg[p] || r >= seg[p + 1]) continue;
        atomicMin(&first[(int64_t)p * n_cfg + id], (int32_t)(r - seg[p]));
    }
}

__global__ __launch_bounds__(kEvalThreads) void k_static_best_time(const float *__restrict__ rt,
                                                                   const int64_t *__restrict__ seg,
                                                                   float *__restrict__ t_best)
{
    __shared__ float red[kEvalThreads];
    const int32_t p = blockIdx.x;
    const int64_t n = seg[p + 1] - seg[p];
    const float t = block_fastest(rt, seg[p], n > 0 ? n : 0, red);
    if (threadIdx.x == 0) t_best[p] = t;
}

__global__ void k_static_accumulate(const float *__restrict__ rt, const int64_t *__restrict__ seg, int32_t P,
                                    int32_t n_cfg, const int32_t *__restrict__ first,
                                    const float *__restrict__ t_best, int32_t *__restrict__ count,
                                    double *__restrict__ ysum)
{
    const int32_t id = blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= n_cfg) return;
    int32_t c = 0;
    double s = 0.0;
    // 32 problems at a time: their table entries, then their runtimes, are
    // requested together (one wave per SIMD: the loads in flight are what
    // hides the memory latency); the sum still runs in problem order.
    constexpr int kB = 32;
    for (int32_t p0 = 0; p0 < P; p0 += kB) {
        int32_t j[kB];
#pragma unroll
        for (int b = 0; b < kB; ++b) j[b] = p0 + b < P ? first[(int64_t)(p0 + b) * n_cfg + id] : INT_MAX;
        float t[kB];
#pragma unroll
        for (int b = 0; b < kB; ++b) t[b] = j[b] != INT_MAX ? rt[seg[p0 + b] + j[b]] : 0.0f;
#pragma unroll
        for (int b = 0; b < kB; ++b)
            if (j[b] != INT_MAX) {
                ++c;
                s += y_of(t_best[p0 + b], t[b]);
            }
    }
    count[id] = c;
    ysum[id] = s;
}

__global__ __launch_bounds__(1024) void k_static_argmax(const int32_t *__restrict__ count,
                                                        const double *__restrict__ ysum, int32_t n_cfg, int32_t P,
                                                        int32_t *__restrict__ best, double *__restrict__ mean_y)
{
    __shared__ double red_y[1024];
    __shared__ int32_t red_id[1024];
    int32_t bid = -1;
    double by = 0.0;
    for (int32_t id = threadIdx.x; id < n_cfg; id += 1024) {
        const int64_t c = count[id];
        if (c == 0 || 5 * c < 4 * (int64_t)P) continue;
        const double m = ysum[id] / (double)c;
        if (bid < 0 || m > by) { bid = id; by = m; }   // ids ascend within a thread
    }
    red_y[threadIdx.x] = by;
    red_id[threadIdx.x] = bid;
    __syncthreads();
    for (int s = 512; s > 0; s >>= 1) {
        if (threadIdx.x < s) {
            const int32_t o = red_id[threadIdx.x + s], m = red_id[threadIdx.x];
            const double oy = red_y[threadIdx.x + s], my = red_y[threadIdx.x];
            if (o >= 0 && (m < 0 || oy > my || (oy == my && o < m))) {
                red_id[threadIdx.x] = o;
                red_y[threadIdx.x] = oy;
            }
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const int32_t b = red_id[0];
        best[0] = b;
        best[1] = b < 0 ? 0 : count[b];
        mean_y[0] = b < 0 ? __builtin_nan("") : red_y[0];
    }
}

size_t up256(size_t v) { return (v + 255) / 256 * 256; }

constexpr size_t eval_workspace_bytes(int64_t P)
{
    return 3 * (((size_t)P * sizeof(double) + 255) / 256 * 256) + ((size_t)P * sizeof(int32_t) + 255) / 256 * 256;
}

// Scratch of hwsel_evaluate_noalloc: the per-problem regrets, y means, order
// statistics and ranks that hwsel_evaluate keeps in the caller's workspace,
// here in a device array of the library's code object (one copy per device,
// held until the process ends).  Every value a call reads is written earlier
// in that same call, so nothing has to be cleared between calls; calls that
// overlap on one device share the array and race.
constexpr size_t kNoAllocScratchBytes = eval_workspace_bytes(HWSEL_EVAL_NOALLOC_MAX_P);
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];
static_assert(kNoAllocScratchBytes == HWSEL_EVAL_NOALLOC_SCRATCH_BYTES, "scratch size as declared");

}  // namespace

size_t evaluate_workspace_bytes(int32_t P) { return eval_workspace_bytes(P); }

// Device address of this device's scratch copy, looked up (with the device
// current) on the first call on each device and kept.  In host code the
// array's own name is not a device address and is never passed to a kernel.
hipError_t evaluate_noalloc_scratch(void **ptr, size_t *bytes)
{
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void *per_device[kMaxDevices];
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!per_device[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        per_device[dev] = p;
    }
    *ptr = per_device[dev];
    *bytes = kNoAllocScratchBytes;
    return hipSuccess;
}

hipError_t launch_evaluate(const float *rt, const int64_t *seg, int32_t P, const int32_t *idx, int32_t k,
                           double *out, double *regret_out, int32_t *rank_out, double *ybar_out, void *ws,
                           hipStream_t s)
{
    uint8_t *w = static_cast<uint8_t *>(ws);
    double *regret = reinterpret_cast<double *>(w);
    double *ybar = reinterpret_cast<double *>(w + up256((size_t)P * 8));
    double *stats = reinterpret_cast<double *>(w + 2 * up256((size_t)P * 8));
    int32_t *rank = reinterpret_cast<int32_t *>(w + 3 * up256((size_t)P * 8));
    hipLaunchKernelGGL(k_eval_groups, dim3(P), dim3(kEvalThreads), 0, s, rt, seg, P, idx, k, regret, rank, ybar);
    if (P <= kSmallP) {
        hipLaunchKernelGGL(k_eval_small, dim3(1), dim3(kSmallT), 0, s, regret, rank, ybar, P, out, regret_out, rank_out,
                           ybar_out);
    } else {
        hipLaunchKernelGGL(k_eval_select, dim3(1), dim3(kSelectThreads), 0, s, regret, rank, P, stats);
        hipLaunchKernelGGL(k_eval_aggregate, dim3(1), dim3(256), 0, s, regret, rank, ybar, stats, P, out, regret_out,
                           rank_out, ybar_out);
    }
    return hipGetLastError();
}

size_t static_config_workspace_bytes(int32_t P, int32_t n_cfg)
{
    return up256((size_t)P * (size_t)n_cfg * sizeof(int32_t)) + up256((size_t)P * sizeof(float)) +
           up256((size_t)n_cfg * sizeof(int32_t)) + up256((size_t)n_cfg * sizeof(double));
}

hipError_t launch_static_config(const float *rt, const int64_t *seg, int32_t P, const int32_t *cfg, int32_t n_cfg,
                                int32_t *best, double *mean_y, void *ws, hipStream_t s)
{
    uint8_t *w = static_cast<uint8_t *>(ws);
    const size_t table = up256((size_t)P * (size_t)n_cfg * sizeof(int32_t));
    int32_t *first = reinterpret_cast<int32_t *>(w);
    float *t_best = reinterpret_cast<float *>(w + table);
    int32_t *count = reinterpret_cast<int32_t *>(w + table + up256((size_t)P * 4));
    double *ysum = reinterpret_cast<double *>(w + table + up256((size_t)P * 4) + up256((size_t)n_cfg * 4));
    hipLaunchKernelGGL(k_fill_i32, dim3(2048), dim3(256), 0, s, first, (int64_t)P * n_cfg, (int32_t)INT_MAX);
    hipLaunchKernelGGL(k_static_first, dim3(2048), dim3(256), 0, s, seg, P, cfg, n_cfg, first);
    hipLaunchKernelGGL(k_static_best_time, dim3(P), dim3(kEvalThreads), 0, s, rt, seg, t_best);
    hipLaunchKernelGGL(k_static_accumulate, dim3((n_cfg + 255) / 256), dim3(256), 0, s, rt, seg, P, n_cfg, first,
                       t_best, count, ysum);
    hipLaunchKernelGGL(k_static_argmax, dim3(1), dim3(1024), 0, s, count, ysum, n_cfg, P, best, mean_y);
    return hipGetLastError();
}

}  // namespace hwsel
