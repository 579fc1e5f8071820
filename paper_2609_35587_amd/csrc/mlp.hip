// Feed-forward ranker 128 -> 512 -> 512 -> 256 -> 1 (GELU, bf16 activations,
// fp32 accumulation).
//
// Unpacked path: a row-block kernel with fp32 FMAs (any weights, no
// preparation).
//
// Packed path (weights arranged once by hwsel_mlp_pack): the hidden layers
// run on the bf16 matrix cores, v_mfma_f32_32x32x16_bf16.
//   * One persistent workgroup (8 waves) per compute unit walks tiles of
//     128 rows.  A tile's activations stay in LDS as bf16 for the whole
//     network ([row][unit], 16-byte chunks XOR-swizzled by row so that 16
//     consecutive rows at one logical chunk fall on 16 distinct 16-byte bank
//     groups); only X comes in, fetched while the previous tile's last layer
//     finishes, and one score per row goes out.
//   * Each layer is computed transposed, H_l^T = W_l * H_{l-1}^T: the A
//     operand is weights, pre-arranged into MFMA fragment order so every
//     fragment is one coalesced 1 KB load (L2-resident: 0.9 MB in all),
//     loaded into registers ahead of use (8 k-steps in the 512-unit layers,
//     4 in the last); the B operand is 16 bytes of one activation row from
//     LDS; the accumulator tile gives each lane 4 runs of 4 consecutive
//     units of one row.
//   * Waves split the output units of a layer, so every weight is read once
//     per tile; in a 512-unit layer a wave's two M-tiles share every
//     activation fragment read.  A layer's results wait in registers until
//     all waves have read the previous layer, then overwrite it in place.
//   * GELU(a) = max(a, 0) - |a| Phi(-|a|) with Phi(-x) = 2^P(x), P a fitted
//     cubic (|error| <= 8.2e-5, a twentieth of the bf16 rounding step that
//     follows at 1).
//   * The 256 -> 1 layer is a dot product folded into layer 3's epilogue,
//     reduced across lanes and waves in a fixed order.
#include "internal.hpp"

#include <math.h>

#include <utility>

namespace hwsel {
namespace {

// ---------------------------------------------------------------------------
// Shared pieces
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round fp32 to the nearest bf16 value (ties to even), kept in an fp32.
__device__ __forceinline__ float round_bf16(float v)
{
    uint32_t u = __float_as_uint(v);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return __uint_as_float((u | 0x00400000u) & 0xffff0000u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return __uint_as_float(u & 0xffff0000u);
}

__device__ __forceinline__ float gelu_exact(float a) { return 0.5f * a * (1.0f + erff(a * 0.70710678118654752f)); }

// GELU(a) = a Phi(a) = max(a, 0) - |a| Phi(-|a|), Phi the standard normal
// distribution function.  For x >= 0, log2 Phi(-x) is smooth and concave, and
// Phi(-x) = 2^P(x) with the cubic P below (fitted on [0, 5] by gelu_fit.py)
// leaves |error| <= 8.2e-5 in GELU for every finite a, a twentieth of the
// bf16 half-step (2e-3 at 1) every activation is rounded to next; past the
// fitted range P keeps falling, 2^P underflows to 0 and the result is
// max(a, 0).  Six vector instructions: three FMAs, v_exp_f32, a max and an
// FMA.
__device__ __forceinline__ float gelu_fast(float a)
{
    constexpr float c3 = -0.026309825479984283f, c2 = -0.4931514859199524f, c1 = -1.1354643106460571f,
                    c0 = -1.0017647743225098f;
    const float x = fabsf(a);
    float p = fmaf(c3, x, c2);
    p = fmaf(p, x, c1);
    p = fmaf(p, x, c0);
    // max(a, 0) as a signed-integer maximum of the bit pattern: exact for
    // every non-NaN a (a negative float, -0 included, has a negative pattern),
    // one instruction without the NaN-quieting copy fmaxf adds, and visible to
    // the compiler, which must see this first read of an accumulator to place
    // the wait states the matrix core needs before it
    const float pos = __int_as_float(max(__float_as_int(a), 0));
    return fmaf(-x, __builtin_amdgcn_exp2f(p), pos);
}

// ---------------------------------------------------------------------------
// Unpacked path
// ---------------------------------------------------------------------------
constexpr int kRows = 16;
constexpr int kThreads = 256;

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
        for (int r = 0; r < kRows; ++r) out[r][u] = round_bf16(gelu_exact(acc[r] + bu));
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
    const int r = threadIdx.x >> 4, part = threadIdx.x & 15;
    float acc = 0.0f;
    for (int j = part; j < 256; j += 16) acc = fmaf(bf16_to_f32(m.W4[j]), h3[r][j], acc);
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 16);
    if (part == 0 && row0 + r < R) scores[row0 + r] = acc + m.b4[0];
}

// ---------------------------------------------------------------------------
// Packed path
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kTile = 128;                    // rows per workgroup
constexpr int kMWaves = 8;
constexpr int kActBytes = kTile * 1024;       // 128 rows x 512 bf16 units
constexpr int kRedFloats = kTile;             // per wave: one partial score per row
constexpr int kLdsBytes = kActBytes + kMWaves * kRedFloats * 4;   // 132 KB
// fragment counts (32 units x 16 inputs each) per layer
constexpr int kFrag1 = (512 / 32) * (128 / 16);
constexpr int kFrag2 = (512 / 32) * (512 / 16);
constexpr int kFrag3 = (256 / 32) * (512 / 16);
constexpr size_t kPackedElems = (size_t)(kFrag1 + kFrag2 + kFrag3) * 512;

// Fragment (mt, ks) of a [n_out][k_in] weight matrix: lane l, element e
// holds W[32 mt + l % 32][16 ks + 8 (l / 32) + e].
__global__ __launch_bounds__(256) void k_mlp_pack(const uint16_t *__restrict__ W1, const uint16_t *__restrict__ W2,
                                                   const uint16_t *__restrict__ W3, uint16_t *__restrict__ out)
{
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= (int64_t)kPackedElems) return;
    int64_t idx = g;
    const uint16_t *W;
    int k_in;
    if (idx < (int64_t)kFrag1 * 512) {
        W = W1; k_in = 128;
    } else if ((idx -= (int64_t)kFrag1 * 512) < (int64_t)kFrag2 * 512) {
        W = W2; k_in = 512;
    } else {
        idx -= (int64_t)kFrag2 * 512;
        W = W3; k_in = 512;
    }
    const int e = (int)(idx & 7), lane = (int)((idx >> 3) & 63);
    const int64_t frag = idx >> 9;
    const int ksteps = k_in / 16;
    const int mt = (int)(frag / ksteps), ks = (int)(frag % ksteps);
    out[g] = W[(int64_t)(32 * mt + (lane & 31)) * k_in + 16 * ks + 8 * (lane >> 5) + e];
}

typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
typedef float f32x2_v __attribute__((ext_vector_type(2)));

// Two fp32 values to a pair of bf16 (round to nearest even), low half first.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_v){lo, hi}, bf16x2_v));
}

// Activation rows live in LDS unpadded; the 16-byte chunk j of row r is
// stored at chunk j ^ (r % 16) (within its aligned group of 16 chunks).  The
// 64 banks of LDS serve a 16-byte access of 16 lanes per cycle, and the 16
// lanes of such a group read or write 16 consecutive rows at the same logical
// chunk, which this places on 16 distinct 16-byte bank groups.
__device__ __forceinline__ int act_offset(int row, int row_bytes, int unit)
{
    return row * row_bytes + ((((unit >> 3) ^ row) & 15) | ((unit >> 3) & ~15)) * 16 + (unit & 7) * 2;
}

// acc[mt][nt] = init[mt] + products of the wave's two consecutive M-tiles
// (fragments at W0 and W0 + KS fragments) with 4 N-tiles: every activation
// fragment read serves two products and every weight fragment four.  The
// weight fragments are loaded straight into registers PF k-steps ahead.
template <int K_IN, int PF>
__device__ __forceinline__ void mma_block_mt2_direct(const bf16x8 *__restrict__ W0, const uint8_t *act, int row_bytes,
                                                     int lane, const f32x16 &init0, const f32x16 &init1,
                                                     f32x16 (&acc)[2][4])
{
    constexpr int KS = K_IN / 16;
    static_assert(KS % PF == 0, "k loop");
    const uint8_t *brow = act + (lane & 31) * row_bytes;
    const int sw = lane & 15, half = lane >> 5;
    const bf16x8 *w0 = W0 + lane, *w1 = W0 + KS * 64 + lane;
    bf16x8 a0[PF], a1[PF];
#pragma unroll
    for (int j = 0; j < PF; ++j) {
        a0[j] = w0[j * 64];
        a1[j] = w1[j * 64];
    }
    // keep the first PF k-steps' loads here: in a fully unrolled layer the
    // scheduler would otherwise sink each next to its first use and wait on
    // every one
    __builtin_amdgcn_sched_barrier(0);
    auto step = [&](int j, int ks, bool first) {
        const int chunk = (((2 * ks + half) ^ sw) & 15) | ((2 * ks + half) & ~15);
        bf16x8 b[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
            b[nt] = *reinterpret_cast<const bf16x8 *>(brow + nt * 32 * row_bytes + chunk * 16);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            acc[0][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[j], b[nt], first ? init0 : acc[0][nt], 0, 0, 0);
            acc[1][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[j], b[nt], first ? init1 : acc[1][nt], 0, 0, 0);
        }
        if (ks + PF < KS) {
            a0[j] = w0[(ks + PF) * 64];
            a1[j] = w1[(ks + PF) * 64];
        }
    };
#pragma unroll
    for (int j = 0; j < PF; ++j) step(j, j, j == 0);
#pragma unroll 1
    for (int ks = PF; ks < KS; ks += PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j) step(j, ks + j, false);
    }
}

// acc[nt] = init + products of one M-tile (fragments at W) with the 4
// N-tiles; weight fragments loaded straight into registers PF k-steps ahead.
template <int K_IN, int PF>
__device__ __forceinline__ void mma_block_mt1_direct(const bf16x8 *__restrict__ W, const uint8_t *act, int row_bytes,
                                                     int lane, const f32x16 &init, f32x16 (&acc)[4])
{
    constexpr int KS = K_IN / 16;
    static_assert(KS % PF == 0, "k loop");
    const uint8_t *brow = act + (lane & 31) * row_bytes;
    const int sw = lane & 15, half = lane >> 5;
    const bf16x8 *w = W + lane;
    bf16x8 a[PF];
#pragma unroll
    for (int j = 0; j < PF; ++j) a[j] = w[j * 64];
    __builtin_amdgcn_sched_barrier(0);
    auto step = [&](int j, int ks, bool first) {
        const int chunk = (((2 * ks + half) ^ sw) & 15) | ((2 * ks + half) & ~15);
        bf16x8 b[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
            b[nt] = *reinterpret_cast<const bf16x8 *>(brow + nt * 32 * row_bytes + chunk * 16);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
            acc[nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[j], b[nt], first ? init : acc[nt], 0, 0, 0);
        if (ks + PF < KS) a[j] = w[(ks + PF) * 64];
    };
#pragma unroll
    for (int j = 0; j < PF; ++j) step(j, j, j == 0);
#pragma unroll 1
    for (int ks = PF; ks < KS; ks += PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j) step(j, ks + j, false);
    }
}

// Bias of one 32-unit M-tile starting at unit u0, in accumulator layout.
__device__ __forceinline__ f32x16 bias_tile(const float *__restrict__ bias, int u0, int lane)
{
    f32x16 v;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const float4 b = *reinterpret_cast<const float4 *>(bias + u0 + 8 * g + 4 * (lane >> 5));
        v[4 * g + 0] = b.x;
        v[4 * g + 1] = b.y;
        v[4 * g + 2] = b.z;
        v[4 * g + 3] = b.w;
    }
    return v;
}

// GELU of one group (4 consecutive units of one row) of an accumulator
// tile, rounded to bf16 and packed.  Accumulator element v of a tile is unit
// 8 (v / 4) + 4 (lane / 32) + v % 4 (plus the tile's first unit) of row
// lane % 32 (plus the tile's first row).
__device__ __forceinline__ uint2 gelu_group(const f32x16 &acc, int g)
{
    return make_uint2(pack_bf16x2(gelu_fast(acc[4 * g + 0]), gelu_fast(acc[4 * g + 1])),
                      pack_bf16x2(gelu_fast(acc[4 * g + 2]), gelu_fast(acc[4 * g + 3])));
}

// A 512-unit hidden layer: each wave owns 64 units (two M-tiles) for all 128
// rows.  Results wait in registers until every wave has finished reading the
// layer input, then overwrite it in place.
template <int K_IN>
__device__ __forceinline__ void hidden512(const bf16x8 *__restrict__ Wf, const float *__restrict__ bias,
                                          uint8_t *act, int in_row_bytes, int wave, int lane)
{
    constexpr int KS = K_IN / 16;
    uint2 staged[2][4][4];
    {
        f32x16 acc[2][4];
        mma_block_mt2_direct<K_IN, 8>(Wf + (int64_t)(2 * wave) * KS * 64, act, in_row_bytes, lane,
                                      bias_tile(bias, 64 * wave, lane), bias_tile(bias, 64 * wave + 32, lane), acc);
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
                for (int nt = 0; nt < 4; ++nt) staged[mt][nt][g] = gelu_group(acc[mt][nt], g);
    }
    __syncthreads();
    // Lanes l and l + 32 hold the two halves of each 16-byte chunk; one
    // cross-half swap per register gives lane l (l < 32) chunk g = 2p and
    // lane l + 32 chunk g = 2p + 1 of the same row, stored with one 16-byte
    // write each.
    const int half = lane >> 5;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
            for (int p = 0; p < 2; ++p) {
                const uint2 x = staged[mt][nt][2 * p], y = staged[mt][nt][2 * p + 1];
                const auto sx = __builtin_amdgcn_permlane32_swap(x.x, y.x, false, false);
                const auto sy = __builtin_amdgcn_permlane32_swap(x.y, y.y, false, false);
                const int row = 32 * nt + (lane & 31);
                const int u = 64 * wave + 32 * mt + 8 * (2 * p + half);
                *reinterpret_cast<uint4 *>(act + act_offset(row, 1024, u)) = make_uint4(sx[0], sy[0], sx[1], sy[1]);
            }
    __syncthreads();
}

// X of one 128-row tile as a thread stages it: the same four columns of 8
// rows 16 apart, plus the standardisation of those columns.  All loads are
// issued together; X is read once, so its loads bypass the caches' retention
// (non-temporal) and leave L2 to the weight fragments.
constexpr int kXLoads = kTile * 32 / (64 * kMWaves);
constexpr int kXRowStep = 64 * kMWaves / 32;
static_assert(kXLoads * 64 * kMWaves == kTile * 32, "X staging covers the tile");

struct XTile {
    float4 mu, is, v[kXLoads];
};

__device__ __forceinline__ void load_x(const hwsel_mlp_t &m, const float *__restrict__ X, int64_t R, int64_t ld,
                                       int64_t row0, int tid, XTile &t)
{
    typedef float f32x4_v __attribute__((ext_vector_type(4)));
    const int r_first = tid >> 5, c4 = (tid & 31) * 4;
    t.mu = *reinterpret_cast<const float4 *>(m.mean + c4);
    t.is = *reinterpret_cast<const float4 *>(m.inv_std + c4);
#pragma unroll
    for (int i = 0; i < kXLoads; ++i) {
        // rows past R (R >= 1) read row R - 1 and are zeroed when staged: no
        // branch splits the batch of loads
        const int64_t r = row0 + r_first + kXRowStep * i;
        const f32x4_v x = __builtin_nontemporal_load(reinterpret_cast<const f32x4_v *>(X + (r < R ? r : R - 1) * ld + c4));
        t.v[i] = make_float4(x.x, x.y, x.z, x.w);
    }
}

// Standardise (fp32, two operations; NaN/inf read as 0), round to bf16 and
// write the tile's input activations.
__device__ __forceinline__ void stage_x(const XTile &t, int64_t row0, int64_t R, int tid, uint8_t *act)
{
    const int r_first = tid >> 5, c4 = (tid & 31) * 4;
#pragma unroll
    for (int i = 0; i < kXLoads; ++i) {
        const bool in = row0 + r_first + kXRowStep * i < R;
        const float4 v = t.v[i];
        const float z0 = ((in && __builtin_isfinite(v.x) ? v.x : 0.0f) - t.mu.x) * t.is.x;
        const float z1 = ((in && __builtin_isfinite(v.y) ? v.y : 0.0f) - t.mu.y) * t.is.y;
        const float z2 = ((in && __builtin_isfinite(v.z) ? v.z : 0.0f) - t.mu.z) * t.is.z;
        const float z3 = ((in && __builtin_isfinite(v.w) ? v.w : 0.0f) - t.mu.w) * t.is.w;
        *reinterpret_cast<uint2 *>(act + act_offset(r_first + kXRowStep * i, 256, c4)) =
            make_uint2(pack_bf16x2(z0, z1), pack_bf16x2(z2, z3));
    }
}

// Persistent: one workgroup per compute unit walks the tiles blockIdx.x,
// blockIdx.x + gridDim.x, ...  The next tile's X is requested as soon as the
// current tile's last weight fragment has landed, so that its trip to HBM
// overlaps the last epilogue and the row sums instead of starting the tile.
__global__ __launch_bounds__(64 * kMWaves, 1) void k_mlp_mfma(hwsel_mlp_t m, const bf16x8 *__restrict__ packed,
                                                              const float *__restrict__ X, int64_t R, int64_t ld,
                                                              float *__restrict__ scores)
{
    __shared__ __attribute__((aligned(1024))) uint8_t lds[kLdsBytes];
    uint8_t *act = lds;
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t n_tiles = (R + kTile - 1) / kTile;
    const bf16x8 *W1f = packed;
    const bf16x8 *W2f = W1f + kFrag1 * 64;
    const bf16x8 *W3f = W2f + kFrag2 * 64;
    const float b4 = m.b4[0];
    XTile xt;
    load_x(m, X, R, ld, (int64_t)blockIdx.x * kTile, (int)threadIdx.x, xt);
    // A tile's row scores are stored only after the next tile's X has
    // landed: the X wait would otherwise also wait for the stores.
    float pending = 0.0f;
    int64_t pending_row = -1;
    for (int64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
        // lane-derived addresses are recomputed per tile rather than hoisted
        // out of the loop and held through the hidden layers
        int ln = lane, tid = threadIdx.x;
        asm volatile("" : "+v"(ln), "+v"(tid));
        const int64_t row0 = tile * kTile;
        stage_x(xt, row0, R, tid, act);
        if (pending_row >= 0) scores[pending_row] = pending;
        __syncthreads();
        hidden512<128>(W1f, m.b1, act, 256, wave, ln);     // layer 1: 128 -> 512
        hidden512<512>(W2f, m.b2, act, 1024, wave, ln);    // layer 2: 512 -> 512

        // layer 3: 512 -> 256 (one M-tile of 32 units per wave, all four
        // N-tiles), GELU, bf16, then the 256 -> 1 dot product
        float part[4] = {0.f, 0.f, 0.f, 0.f};
        const f32x16 b3 = bias_tile(m.b3, 32 * wave, ln);
        // the W4 weights of the wave's 32 units
        uint2 w4[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) w4[g] = *reinterpret_cast<const uint2 *>(m.W4 + 32 * wave + 8 * g + 4 * (ln >> 5));
        {
            f32x16 acc[4];
            mma_block_mt1_direct<512, 4>(W3f + (int64_t)wave * 32 * 64, act, 1024, ln, b3, acc);
#pragma unroll
            for (int nt = 0; nt < 4; ++nt)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    // halfway through the epilogue (half the accumulators
                    // free), request the next tile's X
                    if (nt == 2 && g == 0) load_x(m, X, R, ld, (tile + gridDim.x) * kTile, tid, xt);
                    // two bf16 products and their sum with the running
                    // partial, one instruction per pair (bf16 products are
                    // exact in fp32)
                    const uint2 w = w4[g];
                    const uint2 y = gelu_group(acc[nt], g);
                    float p = part[nt];
                    p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, w.x), __builtin_bit_cast(bf16x2_v, y.x),
                                                        p, false);
                    p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, w.y), __builtin_bit_cast(bf16x2_v, y.y),
                                                        p, false);
                    part[nt] = p;
                }
        }
        // per-row partial sums: lanes l and l + 32 hold the same row
        float *red = reinterpret_cast<float *>(lds + kActBytes);      // [wave][128]
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const float other = __shfl_xor(part[nt], 32, 64);
            if (ln < 32) red[wave * kRedFloats + 32 * nt + ln] = part[nt] + other;
        }
        __syncthreads();
        pending_row = -1;
        if (threadIdx.x < kTile && row0 + threadIdx.x < R) {
            float s = 0.0f;
#pragma unroll
            for (int w = 0; w < kMWaves; ++w) s += red[w * kRedFloats + threadIdx.x];
            pending = s + b4;
            pending_row = row0 + threadIdx.x;
        }
        // the next tile writes its input over act only; red is not written
        // again before that tile's last layer, several barriers on
    }
    if (pending_row >= 0) scores[pending_row] = pending;
}

}  // namespace

hipError_t launch_mlp(const hwsel_mlp_t &m, const float *X, int64_t R, int64_t ld, float *scores,
                      hipStream_t s)
{
    const dim3 grid((unsigned)((R + kRows - 1) / kRows)), block(kThreads);
    hipLaunchKernelGGL(k_mlp_rows, grid, block, 0, s, m, X, R, ld, scores);
    return hipGetLastError();
}

size_t mlp_packed_bytes() { return kPackedElems * sizeof(uint16_t); }

hipError_t launch_mlp_pack(const hwsel_mlp_t &m, void *packed, hipStream_t s)
{
    const unsigned blocks = (unsigned)((kPackedElems + 255) / 256);
    hipLaunchKernelGGL(k_mlp_pack, dim3(blocks), dim3(256), 0, s, m.W1, m.W2, m.W3, static_cast<uint16_t *>(packed));
    return hipGetLastError();
}

hipError_t launch_mlp_packed(const hwsel_mlp_t &m, const void *packed, const float *X, int64_t R, int64_t ld,
                             float *scores, hipStream_t s)
{
    // one persistent workgroup per compute unit (160 KB of LDS each)
    int dev = 0, n_cu = 256;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n_cu < 1)
        n_cu = 256;
    const int64_t n_tiles = (R + kTile - 1) / kTile;
    const dim3 grid((unsigned)(n_tiles < n_cu ? n_tiles : n_cu)), block(64 * kMWaves);
    hipLaunchKernelGGL(k_mlp_mfma, grid, block, 0, s, m, static_cast<const bf16x8 *>(packed), X, R, ld, scores);
    return hipGetLastError();
}

}  // namespace hwsel
