// Per-problem selection (top-k by score) and selection regret.
//
// One workgroup per problem segment.  Scores are mapped to 64-bit keys
// (order-preserving score bits << 32 | inverted local index), which makes
// every key unique: "score descending, index ascending" becomes "key
// descending" and the answer is unique.  The k best keys are found by
// rounds of a block-wide maximum restricted to keys below the previous
// winner.  A segment of up to 8,192 rows is read once into registers (32
// keys per thread) and gives its k best in k rounds; a longer one is read
// once too, tile by tile, keeping a running list of the k best: a tile's
// rounds extract only its keys above the list's k-th entry and stop at the
// first round that finds none.  The wave maximum of a 64-bit key runs on
// DPP: the high words' maximum, then the low words of the lanes that hold it.
#include "internal.hpp"

namespace hwsel {
namespace {

constexpr int kThreads = 256;

// Larger key = better score.  NaN ranks lowest, -0 equals +0.
__device__ __forceinline__ uint32_t desc_bits(float s)
{
    if (s != s) return 0u;
    uint32_t b = __float_as_uint(s);
    if ((b << 1) == 0u) b = 0u;
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Smaller key = faster runtime.  NaN ranks above +inf, -0 equals +0.
__device__ __forceinline__ uint32_t asc_bits(float t)
{
    if (t != t) return 0xffffffffu;
    uint32_t b = __float_as_uint(t);
    if ((b << 1) == 0u) b = 0u;
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

template <int CTRL, int ROW_MASK, bool ZERO_FILL>
__device__ __forceinline__ uint32_t dpp_max_u32(uint32_t v)
{
    const uint32_t w = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, 0xf, ZERO_FILL);
    return w > v ? w : v;
}

// Maximum over the wave of an unsigned 32-bit value (0 is the identity), in
// every lane: scan within rows, row broadcasts to lane 63, then readlane.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v)
{
    v = dpp_max_u32<0x111, 0xf, true>(v);
    v = dpp_max_u32<0x112, 0xf, true>(v);
    v = dpp_max_u32<0x114, 0xf, true>(v);
    v = dpp_max_u32<0x118, 0xf, true>(v);
    v = dpp_max_u32<0x142, 0xa, false>(v);
    v = dpp_max_u32<0x143, 0xc, false>(v);
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Maximum over the wave of 64-bit keys: the largest high word, then the
// largest low word among the lanes holding it.
__device__ __forceinline__ uint64_t wave_max_key(uint64_t v)
{
    const uint32_t hi = wave_max_u32((uint32_t)(v >> 32));
    const uint32_t lo = wave_max_u32((uint32_t)(v >> 32) == hi ? (uint32_t)v : 0u);
    return ((uint64_t)hi << 32) | lo;
}

// Block maximum with one barrier: the waves' maxima go to sh (a buffer the
// caller alternates between rounds, so no round overwrites one still read).
__device__ __forceinline__ uint64_t block_max_key(uint64_t v, uint64_t *sh)
{
    v = wave_max_key(v);
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
    __syncthreads();
    uint64_t r = sh[0];
#pragma unroll
    for (int w = 1; w < kThreads / 64; ++w) r = sh[w] > r ? sh[w] : r;
    return r;
}

__device__ __forceinline__ int64_t seg_len(const int64_t *seg, int32_t p)
{
    int64_t n = seg[p + 1] - seg[p];
    n = n < 0 ? 0 : n;
    return n > 0x7fffffff ? 0x7fffffff : n;
}

constexpr int kRegRows = 32;      // keys per thread held in registers: segments up to 8,192 rows

__global__ __launch_bounds__(kThreads) void k_topk(const float *__restrict__ scores,
                                                    const int64_t *__restrict__ seg, int32_t k,
                                                    int32_t *__restrict__ idx, float *__restrict__ vals)
{
    __shared__ uint64_t sh[2][kThreads / 64];
    const int32_t p = blockIdx.x;
    const int64_t base = seg[p];
    const int64_t n = seg_len(seg, p);
    const float *s = scores + base;
    auto key_of = [&](int64_t i) {
        return ((uint64_t)desc_bits(s[i]) << 32) | (uint64_t)(0xffffffffu - (uint32_t)i);
    };
    auto emit = [&](int32_t j, uint64_t best) {
        if (threadIdx.x == 0) {
            const int64_t o = (int64_t)p * k + j;
            if (best == 0) {
                idx[o] = -1;
                if (vals) vals[o] = -__builtin_inff();
            } else {
                const int32_t li = (int32_t)(0xffffffffu - (uint32_t)best);
                idx[o] = li;
                if (vals) vals[o] = s[li];
            }
        }
    };
    uint64_t prev = ~0ull;
    if (n <= (int64_t)kThreads * kRegRows) {            // block-uniform
        uint64_t key[kRegRows];
#pragma unroll
        for (int r = 0; r < kRegRows; ++r) {
            const int64_t i = threadIdx.x + (int64_t)r * kThreads;
            key[r] = i < n ? key_of(i) : 0ull;           // 0: no row (every real key is > 0)
        }
        for (int32_t j = 0; j < k; ++j) {
            uint64_t best = 0;
#pragma unroll
            for (int r = 0; r < kRegRows; ++r) best = (key[r] < prev && key[r] > best) ? key[r] : best;
            best = block_max_key(best, sh[j & 1]);
            emit(j, best);
            prev = best;
        }
    } else {
        // Longer segments are read once, in tiles of kThreads * kRegRows keys
        // held in registers.  top[0..kept) is the running list of the k best
        // keys (descending); from each tile only the keys above its k-th entry
        // (floor, 0 until k rows are kept) are extracted, largest first, and
        // the rounds stop as soon as none is left, then wave 0 merges them in
        // by rank (keys are unique, so ranks are exact).
        __shared__ uint64_t top[64], cand[64];
        __shared__ int32_t kept_s;
        if (threadIdx.x == 0) kept_s = 0;
        uint64_t floor = 0;
        int32_t kept = 0;
        for (int64_t t0 = 0; t0 < n; t0 += (int64_t)kThreads * kRegRows) {
            uint64_t key[kRegRows];
#pragma unroll
            for (int r = 0; r < kRegRows; ++r) {
                const int64_t i = t0 + threadIdx.x + (int64_t)r * kThreads;
                key[r] = i < n ? key_of(i) : 0ull;
            }
            int32_t m = 0;
            uint64_t c_prev = ~0ull;
            for (; m < k; ++m) {                          // block-uniform trip count
                uint64_t best = 0;
#pragma unroll
                for (int r = 0; r < kRegRows; ++r)
                    best = (key[r] < c_prev && key[r] > floor && key[r] > best) ? key[r] : best;
                best = block_max_key(best, sh[m & 1]);
                if (best == 0) break;
                if (threadIdx.x == 0) cand[m] = best;
                c_prev = best;
            }
            __syncthreads();
            if (threadIdx.x < 64 && m > 0) {
                // merged rank of each entry = its own index + the number of
                // entries of the other list above it
                const int lane = threadIdx.x;
                uint64_t mine_t = lane < kept ? top[lane] : 0ull, mine_c = lane < m ? cand[lane] : 0ull;
                int32_t rank_t = lane, rank_c = lane;
                for (int32_t q = 0; q < m; ++q) rank_t += cand[q] > mine_t;
                for (int32_t q = 0; q < kept; ++q) rank_c += top[q] > mine_c;
                __builtin_amdgcn_wave_barrier();
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // every lane has read both lists
                if (lane < kept && rank_t < k) top[rank_t] = mine_t;
                if (lane < m && rank_c < k) top[rank_c] = mine_c;
                if (lane == 0) kept_s = kept + m < k ? kept + m : k;
            }
            __syncthreads();
            kept = kept_s;
            if (kept == k) floor = top[k - 1];
        }
        for (int32_t j = 0; j < k; ++j) emit(j, j < kept ? top[j] : 0ull);
    }
}

// 1 - t_star / t_pick in binary64; equal runtimes (inf included) give 0 and a
// NaN runtime (a kernel that never finishes) gives 1.
__device__ __forceinline__ float regret_value(float t_star, float t_pick)
{
    if (t_pick == t_star) return 0.0f;
    if (t_pick != t_pick) return 1.0f;
    return (float)(1.0 - (double)t_star / (double)t_pick);
}

__global__ __launch_bounds__(kThreads) void k_regret(const float *__restrict__ rt,
                                                      const int64_t *__restrict__ seg,
                                                      const int32_t *__restrict__ idx, int32_t k,
                                                      float *__restrict__ r1, float *__restrict__ rk,
                                                      int32_t *__restrict__ best)
{
    __shared__ uint64_t sh[kThreads / 64];
    const int32_t p = blockIdx.x;
    const int64_t base = seg[p];
    const int64_t n = seg_len(seg, p);
    const float *t = rt + base;
    uint64_t m = ~0ull;
    for (int64_t i = threadIdx.x; i < n; i += kThreads) {
        const uint64_t key = ((uint64_t)asc_bits(t[i]) << 32) | (uint64_t)(uint32_t)i;
        m = key < m ? key : m;
    }
    m = ~block_max_key(~m, sh);                         // block minimum of the unique keys
    if (threadIdx.x != 0) return;
    if (n == 0) {
        r1[p] = __builtin_nanf("");
        if (rk) rk[p] = __builtin_nanf("");
        if (best) best[p] = -1;
        return;
    }
    const int32_t b = (int32_t)(uint32_t)m;
    const float t_star = t[b];
    const int32_t *pick = idx + (int64_t)p * k;
    const int32_t c0 = pick[0];
    r1[p] = (c0 >= 0 && c0 < n) ? regret_value(t_star, t[c0]) : __builtin_nanf("");
    if (rk) {
        uint64_t bk = ~0ull;
        for (int32_t j = 0; j < k; ++j) {
            const int32_t c = pick[j];
            if (c < 0 || c >= n) continue;
            const uint64_t key = ((uint64_t)asc_bits(t[c]) << 32) | (uint64_t)(uint32_t)c;
            bk = key < bk ? key : bk;
        }
        rk[p] = bk == ~0ull ? __builtin_nanf("") : regret_value(t_star, t[(uint32_t)bk]);
    }
    if (best) best[p] = b;
}

}  // namespace

hipError_t launch_topk(const float *scores, const int64_t *seg, int32_t P, int32_t k, int32_t *idx,
                       float *vals, hipStream_t s)
{
    hipLaunchKernelGGL(k_topk, dim3(P), dim3(kThreads), 0, s, scores, seg, k, idx, vals);
    return hipGetLastError();
}

hipError_t launch_regret(const float *rt, const int64_t *seg, int32_t P, const int32_t *idx,
                         int32_t k, float *r1, float *rk, int32_t *best, hipStream_t s)
{
    hipLaunchKernelGGL(k_regret, dim3(P), dim3(kThreads), 0, s, rt, seg, idx, k, r1, rk, best);
    return hipGetLastError();
}

}  // namespace hwsel
