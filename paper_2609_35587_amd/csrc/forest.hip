// Tree-ensemble scoring: s(x) = base + sum_t leaf_t(x).
//
// Two paths share the decision rule "left iff x < threshold (or NaN with
// the default-left flag)":
//
// Generic path (no packed model): one thread per row walks every tree from
// the root, reading node records and leaves through the caches and the row's
// fp32 features from X.  Any forest the header admits runs here.
//
// Packed path (model packed once by hwsel_forest_pack):
//   * Exact binning.  For feature f let U_f be the sorted distinct
//     thresholds the forest uses (at most 255).  With
//     b_f(x) = #{u in U_f : u <= x}, and a node testing x < U_f[j],
//     x < U_f[j]  <=>  b_f(x) <= j,
//     so the traversal compares u8 bins with u8 threshold ranks and gives the
//     same path as the fp32 compares (NaN is binned to 0 when it goes left,
//     255 when it goes right).  A pass writes the bins of every row once:
//     128 bytes per row instead of 512.
//   * Trees in LDS.  Trees are grouped into chunks of TC trees whose nodes
//     (u16 code: feature | rank << 8, heap order, stored as sibling pairs so
//     one 4-byte read fetches both children of a node) and leaves (fp32,
//     leaf l of tree t at l*TC + t) fill about 96 KB of LDS (128 KB for 16
//     trees, whose node pairs are stored twice).  The node layout gives every
//     lane of a half-wave its own LDS bank (see node_byte).
//   * Lanes.  A wave walks 64/TC rows x TC trees at a time; several such
//     groups are in flight per wave to cover LDS latency.  A level reads the
//     bin of the current node and the children pair together, then picks the
//     child's code with the compare's carry: one LDS round trip per level.
//     With 64 or 32 trees a half-wave reads the bins of one row, whose words
//     lie on distinct banks (conflict-free); with 16 trees it reads two rows.
//   * Chunk-stationary, XCD-aware persistent grid.  Each workgroup owns one
//     chunk for a whole row range; each wave owns a slice of every row tile
//     and a private LDS region for its bins, refilled without workgroup
//     barriers while the next slice is fetched into registers.  Workgroup b
//     runs on XCD b % 8; the workgroups of one XCD cover the same rows with
//     different chunks, so a tile is fetched from HBM about once per XCD and
//     re-read from that XCD's L2.
//   * Deterministic sums.  A chunk's per-row sum is a fixed DPP reduction
//     over its TC lanes, written to a per-chunk partial row; a last pass adds
//     base + partials in chunk order.
#include <algorithm>
#include <cstring>
#include <vector>

#include "internal.hpp"

namespace hwsel {
namespace {

// ---------------------------------------------------------------------------
// Generic path
// ---------------------------------------------------------------------------
struct ForestDev {
    int32_t n_trees, depth, n_features;
    uint32_t nan_left;
    float base;
    const uint8_t *feat;
    const float *thr;
    const float *leaf;
};

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

// ---------------------------------------------------------------------------
// Packed path: layout
// ---------------------------------------------------------------------------
constexpr int kBinSlots = 256;        // thresholds per feature incl. padding
// Bin table in LDS: threshold i of feature f at word
// (f / 32) * 32 * kBinSlots + 32 * i + f % 32, so the 32 features searched by
// a half-wave each stay on their own bank whatever their search positions.
__host__ __device__ constexpr int bin_table_index(int f, int i) { return (f >> 5) * 32 * kBinSlots + 32 * i + (f & 31); }
// Rows of bins per LDS tile: as many as fit next to the tree chunk, in whole
// groups per wave (more rows per wave = more walks in flight).  With 16
// trees per chunk the duplicated node tables leave 32 KB: 256 rows of 128 B.
__host__ __device__ constexpr int tile_rows(int tc) { return tc == 64 ? 384 : tc == 32 ? 448 : 256; }
__host__ __device__ constexpr int tile_stride(int tc) { return tc == 16 ? 128 : 132; }   // LDS bytes per bin row
constexpr int kWaves = 16;            // waves per traversal workgroup
constexpr int kXcds = 8;
constexpr int kSlotsPerXcd = 32;      // one workgroup per CU
constexpr int kBinThreads = 1024;

// Node codes (u16: feature | rank << 8) are stored as sibling pairs: the
// 4-byte word of pair p holds nodes 2p (low half) and 2p + 1 (high half), so
// one read fetches both children of node p (pair 0 holds the root in its high
// half).  Pair p of every tree sits in row p; each tree owns one 4-byte column
// (one LDS bank), so every lane of a half-wave reads its own bank (a gather
// from 32 lanes is served in one pass only when no two lanes hit one bank at
// different words):
//   TC = 64: rows of 256 bytes, tree t in column t (lanes t and t + 32 sit
//            in different half-waves);
//   TC = 32: rows of 128 bytes, tree t in column t;
//   TC = 16: rows of 128 bytes holding two copies of every tree, in columns
//            t and 16 + t, one for each of the two rows a half-wave walks.
__host__ __device__ constexpr int node_copies(int tc) { return tc == 16 ? 2 : 1; }
__host__ __device__ constexpr uint32_t pair_row_bytes(int tc) { return tc == 64 ? 256u : 128u; }

__host__ __device__ inline uint32_t node_byte(uint32_t n, int t, int copy, int tc)
{
    return (n >> 1) * pair_row_bytes(tc) + 4u * (uint32_t)(copy * 16 + t) + 2u * (n & 1u);
}

struct PackGeom {
    int tc, n_chunks, slots, stride;      // trees per chunk, chunks, heap slots (2^D), bin row bytes
    size_t thr_bytes, chunk_bytes, node_bytes, total;
};

// Trees per chunk: fill ~96 KB of LDS with nodes (2 B) and leaves (4 B).
int trees_per_chunk(int depth)
{
    int tc = 64;
    while (tc > 1 && (size_t)tc * ((size_t)6 << depth) > 96 * 1024) tc >>= 1;
    return tc;
}

PackGeom geometry(const hwsel_forest_t &f)
{
    PackGeom g;
    g.tc = trees_per_chunk(f.depth);
    g.n_chunks = (f.n_trees + g.tc - 1) / g.tc;
    g.slots = 1 << f.depth;
    g.stride = (f.n_features + 15) / 16 * 16;
    g.thr_bytes = (size_t)f.n_features * kBinSlots * sizeof(float);
    g.node_bytes = (size_t)g.slots * g.tc * 2 * node_copies(g.tc);
    g.chunk_bytes = g.node_bytes + (size_t)g.slots * g.tc * 4;
    g.total = 256 + g.thr_bytes + (size_t)g.n_chunks * g.chunk_bytes;
    return g;
}

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

constexpr int32_t kImageMagic = 0x48575346;   // "FSWH"
constexpr int32_t kImageVersion = 2;

ImageId image_id(const hwsel_forest_t &f, const PackGeom &g)
{
    return ImageId{kImageMagic, kImageVersion, f.n_trees, f.depth, f.n_features, g.tc, g.n_chunks};
}

// Check outputs of the packed traversal (hwsel_forest_score_checked).
struct LeafHook {
    uint64_t *hash;          // [R] or null: leaf-path fingerprint per row
    uint16_t *idx;           // [n_rows][n_trees] or null: leaf indices of rows [row0, row0 + n_rows)
    int64_t row0, n_rows;
    int32_t n_trees;
};

// 64-bit finaliser of SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): a
// bijection, so the fingerprint sum changes whenever one leaf does.
__device__ __forceinline__ uint64_t leaf_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

// Wrapping sum of a 64-bit value over the TC consecutive lanes of a group.
template <int TC>
__device__ __forceinline__ uint64_t group_sum_u64(uint64_t h)
{
#pragma unroll
    for (int o = 1; o < TC; o <<= 1) {
        const uint32_t lo = __shfl_xor((uint32_t)h, o, 64), hi = __shfl_xor((uint32_t)(h >> 32), o, 64);
        h += ((uint64_t)hi << 32) | lo;
    }
    return h;
}

__global__ void k_fill_u64(uint64_t *__restrict__ a, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        a[i] = 0;
}

// ---------------------------------------------------------------------------
// Packed path: kernels
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBinThreads, 1) void k_bin(const float *__restrict__ X, int64_t R, int64_t ld,
                                                         const void *__restrict__ packed, ImageId id, int nf,
                                                         uint32_t nan_bin, uint8_t *__restrict__ Xb, int stride)
{
    if (!image_matches(packed, id)) return;
    const float *__restrict__ U = reinterpret_cast<const float *>(static_cast<const uint8_t *>(packed) + 256);
    // thresholds as order-preserving keys; index i of feature f at
    // bin_table_index(f, i), so each searched feature stays on its own bank
    __shared__ uint32_t u[128 * kBinSlots];
    for (int e = threadIdx.x; e < nf * kBinSlots; e += kBinThreads)
        u[bin_table_index(e >> 8, e & 255)] = order_key(U[e]);
    __syncthreads();
    const int f = threadIdx.x & 127;
    // 8 row lanes per block; a wave's 64 threads share one, so the row
    // arithmetic below stays scalar
    const int sub = __builtin_amdgcn_readfirstlane(threadIdx.x >> 7);
    if (f >= stride) return;
    const uint8_t *uf = reinterpret_cast<const uint8_t *>(u + bin_table_index(f, 0));
    constexpr int kRowsPerThread = 8;                 // independent searches in flight
    const int64_t step_rows = (int64_t)gridDim.x * 8 * kRowsPerThread;
    // the next group's values are requested before this group's searches,
    // so the trip to HBM overlaps them
    // Branch-free: rows past R read row R - 1 and columns past nf read
    // column nf - 1 (R, nf >= 1); neither result is stored as such.
    const int fc = f < nf ? f : nf - 1;
    auto fetch = [&](int64_t r0, float (&x)[kRowsPerThread]) {
#pragma unroll
        for (int q = 0; q < kRowsPerThread; ++q) {
            const int64_t r = r0 + q;
            x[q] = X[(r < R ? r : R - 1) * ld + fc];
        }
    };
    float xn[kRowsPerThread];
    fetch(((int64_t)blockIdx.x * 8 + sub) * kRowsPerThread, xn);
    for (int64_t r0 = ((int64_t)blockIdx.x * 8 + sub) * kRowsPerThread; r0 < R; r0 += step_rows) {
        float x[kRowsPerThread];
        uint32_t kx1[kRowsPerThread], b[kRowsPerThread];
#pragma unroll
        for (int q = 0; q < kRowsPerThread; ++q) x[q] = xn[q];
        fetch(r0 + step_rows, xn);
#pragma unroll
        for (int q = 0; q < kRowsPerThread; ++q) {
            kx1[q] = order_key(x[q] == 0.0f ? 0.0f : x[q]) + 1u;
            b[q] = 0;
        }
        // b = #{u <= x} built from the top bit: at step k the probe is
        // threshold (b << (k + 1)) + 2^k - 1 (rows of 32 words, 128 bytes)
#pragma unroll
        for (int k = 7; k >= 0; --k) {
#pragma unroll
            for (int q = 0; q < kRowsPerThread; ++q) {
                const uint32_t key_u =
                    *reinterpret_cast<const uint32_t *>(uf + (b[q] << (k + 8)) + 128u * ((1u << k) - 1u));
                b[q] = search_step(b[q], key_u, kx1[q]);
            }
        }
#pragma unroll
        for (int q = 0; q < kRowsPerThread; ++q) {
            if (r0 + q >= R) break;
            uint32_t v = b[q];
            if (x[q] != x[q]) v = nan_bin;
            if (f >= nf) v = 0;
            Xb[(r0 + q) * stride + f] = (uint8_t)v;
        }
    }
}

// One level of a walk: node <- 2*node + (bin > rank), with rank the high
// byte of the node code.  Subtract-with-borrow leaves (bin > rank) in VCC and
// add-with-carry folds it in: two VALU instructions per visit.
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

// descend() that also takes the child's code from the children pair (low
// half for the left child, high half for the right one) with the same carry.
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

// The root's step: as descend_pair, and with the same carry also picks the
// children pair of the chosen child (p2 for node 2, p3 for node 3).
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



template <int TC, int D, bool HOOK>
__global__ __launch_bounds__(64 * kWaves, 1) void k_traverse(const void *__restrict__ packed, ImageId id,
                                                              const uint8_t *__restrict__ chunks, int n_chunks,
                                                              const uint8_t *__restrict__ Xb, int64_t R,
                                                              int stride, int groups_per_xcd,
                                                              int64_t rows_per_group, float *__restrict__ partial,
                                                              LeafHook hook)
{
    if (!image_matches(packed, id)) return;
    constexpr int NS = 1 << D;
    constexpr int NODE_B = NS * TC * 2 * node_copies(TC);
    constexpr int CHUNK_B = NODE_B + NS * TC * 4;
    constexpr int RPI = 64 / TC;                       // rows per lane group
    constexpr int kTileRows = tile_rows(TC);
    constexpr int kStride = tile_stride(TC);
    constexpr int ROWS_PER_WAVE = kTileRows / kWaves;
    constexpr int GROUPS = ROWS_PER_WAVE / RPI;
    constexpr int ILP = GROUPS % 8 == 0 ? 8 : GROUPS % 7 == 0 ? 7 : GROUPS % 6 == 0 ? 6 : 4;   // groups in flight
    constexpr int ITER = ROWS_PER_WAVE / (RPI * ILP);
    static_assert(ITER >= 1 && ITER * RPI * ILP == ROWS_PER_WAVE, "tile shape");
    static_assert(CHUNK_B + kTileRows * kStride <= 160 * 1024, "LDS");
    __shared__ __attribute__((aligned(16))) uint8_t lds[CHUNK_B + kTileRows * kStride];
    const float *leaves = reinterpret_cast<const float *>(lds + NODE_B);

    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int t = lane % TC, s = lane / TC;
    // The children pair of node n is the word at n * ROW_B + col.
    constexpr uint32_t ROW_B = pair_row_bytes(TC);
    const uint32_t col = node_byte(0, t, node_copies(TC) == 2 ? (s & 1) : 0, TC);
    const int xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds;
    const int slots = gridDim.x / kXcds;
    const int items = n_chunks * groups_per_xcd;
    // Each wave owns ROWS_PER_WAVE rows of every tile and a private LDS region
    // for their bins, which it refills on its own (no workgroup barrier
    // between tiles): its next rows are fetched into registers while it walks
    // the current ones.
    uint8_t *region = lds + CHUNK_B + wave * ROWS_PER_WAVE * kStride;
    constexpr int kVec = (ROWS_PER_WAVE * 8 + 63) / 64;   // uint4 per lane for 128-byte rows
    const int vpr = stride >> 4;                         // uint4 per bin row

    for (int item = slot; item < items; item += slots) {
        const int c = item % n_chunks, sub = item / n_chunks;
        const int64_t g = (int64_t)xcd * groups_per_xcd + sub;
        const int64_t r_begin = g * rows_per_group;
        const int64_t r_end = r_begin + rows_per_group < R ? r_begin + rows_per_group : R;
        __syncthreads();
        {   // chunk image -> LDS
            const uint4 *src = reinterpret_cast<const uint4 *>(chunks + (size_t)c * CHUNK_B);
            uint4 *dst = reinterpret_cast<uint4 *>(lds);
            for (int e = threadIdx.x; e < CHUNK_B / 16; e += 64 * kWaves) dst[e] = src[e];
        }
        __syncthreads();
        // The root's code and the children pairs of nodes 1, 2, 3 are the same
        // for every row: registers for the whole chunk.
        const uint32_t root = *reinterpret_cast<const uint16_t *>(lds + col + 2);   // high half of pair 0
        const uint32_t p1 = D >= 2 ? *reinterpret_cast<const uint32_t *>(lds + ROW_B + col) : 0u;
        const uint32_t p2 = D >= 3 ? *reinterpret_cast<const uint32_t *>(lds + 2 * ROW_B + col) : 0u;
        const uint32_t p3 = D >= 3 ? *reinterpret_cast<const uint32_t *>(lds + 3 * ROW_B + col) : 0u;
        uint4 preA[kVec], preB[kVec];
        const bool full_rows = stride == 128;              // wave-uniform
        // A lane's byte offsets within its wave's slice are the same for every
        // tile; only whole slices inside the row range skip the row guards.
        auto fetch = [&](int64_t t0, uint4 (&pre)[kVec]) {
            const int64_t w0 = t0 + wave * ROWS_PER_WAVE;
            const uint8_t *slice = Xb + w0 * stride;       // wave-uniform
            if (full_rows && w0 + ROWS_PER_WAVE <= r_end) {
                // 128-byte rows, all in range: chunk e % 8 of row e / 8
#pragma unroll
                for (int q = 0; q < kVec; ++q) {
                    const int e = lane + 64 * q;
                    if ((ROWS_PER_WAVE * 8) % 64 == 0 || e < ROWS_PER_WAVE * 8)
                        pre[q] = *reinterpret_cast<const uint4 *>(slice + (e >> 3) * 128 + 16 * (e & 7));
                }
            } else {
                const int n = (int)(r_end - w0 > 0 ? r_end - w0 : 0);   // rows of this slice left
#pragma unroll
                for (int q = 0; q < kVec; ++q) {
                    const int e = lane + 64 * q;
                    const int rr = e / vpr, w = e - rr * vpr;
                    pre[q] = (rr < ROWS_PER_WAVE && rr < n)
                                 ? *reinterpret_cast<const uint4 *>(slice + rr * stride + 16 * w)
                                 : make_uint4(0, 0, 0, 0);
                }
            }
        };
        // Two tiles in flight: a tile's bins are requested two tiles before
        // they are written to LDS, alternating between two register buffers.
        fetch(r_begin, preA);
        fetch(r_begin + kTileRows, preB);
        auto tile = [&](int64_t t0, uint4 (&pre)[kVec]) {
            const int64_t w0 = t0 + wave * ROWS_PER_WAVE;
            // The previous rows' reads have all returned (their results were
            // used), so the region can be overwritten.
            auto put = [&](int q, int rr, int w) {
                if constexpr (kStride % 16 == 0) {
                    *reinterpret_cast<uint4 *>(region + rr * kStride + 16 * w) = pre[q];
                } else {
                    uint32_t *d = reinterpret_cast<uint32_t *>(region + rr * kStride + 16 * w);
                    d[0] = pre[q].x; d[1] = pre[q].y; d[2] = pre[q].z; d[3] = pre[q].w;
                }
            };
            if (full_rows) {
#pragma unroll
                for (int q = 0; q < kVec; ++q) {
                    const int e = lane + 64 * q;
                    if ((ROWS_PER_WAVE * 8) % 64 == 0 || e < ROWS_PER_WAVE * 8) put(q, e >> 3, e & 7);
                }
            } else {
#pragma unroll
                for (int q = 0; q < kVec; ++q) {
                    const int e = lane + 64 * q;
                    const int rr = e / vpr, w = e - rr * vpr;
                    if (rr < ROWS_PER_WAVE) put(q, rr, w);
                }
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the region is written before any lane reads it
            fetch(t0 + 2 * kTileRows, pre);
            if (w0 >= r_end) return;                                 // wave-uniform: no rows left here
#pragma unroll 1
            for (int it = 0; it < ITER; ++it) {
                int node[ILP];
                uint32_t code[ILP];
                const uint8_t *rowp[ILP];
#pragma unroll
                for (int a = 0; a < ILP; ++a) {
                    rowp[a] = region + ((it * ILP + a) * RPI + s) * kStride;
                    node[a] = 1;
                    code[a] = root;
                }
                // Per level: the bin of the current node and the pair of its
                // children are read together; the compare then picks the
                // child's code from the pair, so a level waits for one LDS
                // round trip.  Levels 0 and 1 take their pairs from registers.
                uint32_t pair[ILP];
#pragma unroll
                for (int l = 0; l < D; ++l) {
                    uint32_t bin[ILP];
#pragma unroll
                    for (int a = 0; a < ILP; ++a) {
                        bin[a] = rowp[a][code[a] & 0xffu];
                        if (l >= 2 && l < D - 1)
                            pair[a] = *reinterpret_cast<const uint32_t *>(lds + (uint32_t)node[a] * ROW_B + col);
                    }
#pragma unroll
                    for (int a = 0; a < ILP; ++a) {
                        if (l == D - 1) node[a] = descend(node[a], code[a], bin[a]);
                        else if (l == 0 && D >= 3) descend_root(node[a], code[a], pair[a], bin[a], p1, p2, p3);
                        else if (l == 0) descend_pair(node[a], code[a], bin[a], p1);
                        else descend_pair(node[a], code[a], bin[a], pair[a]);
                    }
                }
                if constexpr (HOOK) {
#pragma unroll
                    for (int a = 0; a < ILP; ++a) {
                        const int64_t row = w0 + (it * ILP + a) * RPI + s;
                        const int32_t tree = c * TC + t;
                        const uint32_t leaf = (uint32_t)(node[a] - NS);
                        const bool real = row < r_end && tree < hook.n_trees;   // padding trees count for nothing
                        const uint64_t h =
                            group_sum_u64<TC>(real ? leaf_mix(((uint64_t)tree << 32) | leaf) : 0ull);
                        if (hook.hash && t == 0 && row < r_end)
                            atomicAdd(reinterpret_cast<unsigned long long *>(hook.hash + row), (unsigned long long)h);
                        if (hook.idx && real && row >= hook.row0 && row < hook.row0 + hook.n_rows)
                            hook.idx[(row - hook.row0) * hook.n_trees + tree] = (uint16_t)leaf;
                    }
                }
                // Leaves of all groups first, then the sums, then the stores
                // (one lane per row), so that nothing serialises the groups.
                float v[ILP];
#pragma unroll
                for (int a = 0; a < ILP; ++a) v[a] = leaves[(node[a] - NS) * TC + t];
                group_totals<TC, ILP>(v);
                float *out = partial + (int64_t)c * R + w0 + it * ILP * RPI + s;
                if (w0 + ROWS_PER_WAVE <= r_end) {                   // wave-uniform: every row is real
                    if (t == TC - 1) {
#pragma unroll
                        for (int a = 0; a < ILP; ++a) out[a * RPI] = v[a];
                    }
                } else if (t == TC - 1) {
#pragma unroll
                    for (int a = 0; a < ILP; ++a)
                        if (w0 + (it * ILP + a) * RPI + s < r_end) out[a * RPI] = v[a];
                }
            }
        };
        for (int64_t t0 = r_begin; t0 < r_end; t0 += 2 * kTileRows) {
            tile(t0, preA);
            if (t0 + kTileRows < r_end) tile(t0 + kTileRows, preB);
        }
    }
}

__global__ __launch_bounds__(256) void k_reduce(const void *__restrict__ packed, ImageId id,
                                                 const float *__restrict__ partial, int n_chunks, int64_t R,
                                                 float base, float *__restrict__ scores)
{
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= R) return;
    if (!image_matches(packed, id)) {
        scores[r] = __builtin_nanf("");
        return;
    }
    float acc = base;
    for (int c = 0; c < n_chunks; ++c) acc += partial[(int64_t)c * R + r];
    scores[r] = acc;
}

// Four rows per thread with 16-byte loads (R % 4 == 0, so every chunk's
// partial row starts 16-byte aligned); same chunk order per row.
__global__ __launch_bounds__(256) void k_reduce4(const void *__restrict__ packed, ImageId id,
                                                  const float *__restrict__ partial, int n_chunks, int64_t R,
                                                  float base, float *__restrict__ scores)
{
    const int64_t r = 4 * ((int64_t)blockIdx.x * blockDim.x + threadIdx.x);
    if (r >= R) return;
    if (!image_matches(packed, id)) {
        const float q = __builtin_nanf("");
        *reinterpret_cast<float4 *>(scores + r) = make_float4(q, q, q, q);
        return;
    }
    float4 acc = make_float4(base, base, base, base);
#pragma unroll 8
    for (int c = 0; c < n_chunks; ++c) {
        const float4 v = *reinterpret_cast<const float4 *>(partial + (int64_t)c * R + r);
        acc.x += v.x;
        acc.y += v.y;
        acc.z += v.z;
        acc.w += v.w;
    }
    *reinterpret_cast<float4 *>(scores + r) = acc;
}

// Row groups per XCD.  The XCD's kSlotsPerXcd workgroups take (chunk, group)
// items in turn.  With fewer chunks than workgroups: enough groups for one
// round.  Otherwise n_chunks * groups items should fill whole rounds: the
// fewest groups that leave under 0.5 % of the rounds' slots idle, else the
// one that leaves fewest, among those that still give every group at least
// four row tiles (125 chunks of a 4.9 M-row call: 11 groups, 1,375 items in
// 43 rounds of 32).
inline int groups_per_xcd(int n_chunks, int64_t R, int tile)
{
    if (n_chunks < kSlotsPerXcd) return (kSlotsPerXcd + n_chunks - 1) / n_chunks;
    const int64_t cap_rows = R / ((int64_t)kXcds * tile * 4);
    const int cap = cap_rows < 1 ? 1 : cap_rows > kSlotsPerXcd ? kSlotsPerXcd : (int)cap_rows;
    int best = 1;
    double best_idle = 1.0;
    for (int g = 1; g <= cap; ++g) {
        const int64_t items = (int64_t)n_chunks * g;
        const int64_t slots = (items + kSlotsPerXcd - 1) / kSlotsPerXcd * kSlotsPerXcd;
        const double idle = (double)(slots - items) / (double)slots;
        if (idle < 0.005) return g;
        if (idle < best_idle) best_idle = idle, best = g;
    }
    return best;
}

template <int TC, int D>
hipError_t launch_traverse_tc(const void *packed, ImageId id, const uint8_t *chunks, int n_chunks, const uint8_t *Xb,
                              int64_t R, int stride, float *partial, const LeafHook &hook, hipStream_t s)
{
    const int groups = groups_per_xcd(n_chunks, R, tile_rows(TC));
    const int64_t n_groups = (int64_t)kXcds * groups;
    int64_t per = (R + n_groups - 1) / n_groups;
    per = (per + tile_rows(TC) - 1) / tile_rows(TC) * tile_rows(TC);
    if (hook.hash || hook.idx)
        hipLaunchKernelGGL((k_traverse<TC, D, true>), dim3(kXcds * kSlotsPerXcd), dim3(64 * kWaves), 0, s, packed,
                           id, chunks, n_chunks, Xb, R, stride, groups, per, partial, hook);
    else
        hipLaunchKernelGGL((k_traverse<TC, D, false>), dim3(kXcds * kSlotsPerXcd), dim3(64 * kWaves), 0, s, packed,
                           id, chunks, n_chunks, Xb, R, stride, groups, per, partial, hook);
    return hipGetLastError();
}

hipError_t launch_traverse(int depth, const void *packed, ImageId id, const uint8_t *chunks, int n_chunks,
                           const uint8_t *Xb, int64_t R, int stride, float *partial, const LeafHook &hook,
                           hipStream_t s)
{
#define HWSEL_TRAVERSE(TC_, D_) \
    return launch_traverse_tc<TC_, D_>(packed, id, chunks, n_chunks, Xb, R, stride, partial, hook, s)
    switch (depth) {
    case 1: HWSEL_TRAVERSE(64, 1);
    case 2: HWSEL_TRAVERSE(64, 2);
    case 3: HWSEL_TRAVERSE(64, 3);
    case 4: HWSEL_TRAVERSE(64, 4);
    case 5: HWSEL_TRAVERSE(64, 5);
    case 6: HWSEL_TRAVERSE(64, 6);
    case 7: HWSEL_TRAVERSE(64, 7);
    case 8: HWSEL_TRAVERSE(64, 8);
    case 9: HWSEL_TRAVERSE(32, 9);
    case 10: HWSEL_TRAVERSE(16, 10);
    default: return hipErrorInvalidValue;
    }
#undef HWSEL_TRAVERSE
}

}  // namespace

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
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

bool packable(const hwsel_forest_t &f) { return f.depth >= 1 && f.depth <= 10 && f.n_features <= 128; }

size_t packed_bytes(const hwsel_forest_t &f) { return geometry(f).total; }

size_t packed_workspace_bytes(const hwsel_forest_t &f, int64_t R)
{
    const PackGeom g = geometry(f);
    return align256((size_t)R * g.stride) + (size_t)g.n_chunks * (size_t)R * sizeof(float);
}

// The packed image of a forest whose arrays are in host memory, written to
// img (host memory of packed_bytes(f) bytes): per-feature sorted distinct
// thresholds, then the chunks of sibling-pair codes and leaves.
PackStatus build_image(const hwsel_forest_t &f, const uint8_t *feat, const float *thr, const float *leaf,
                       uint8_t *img_out)
{
    const PackGeom g = geometry(f);
    const int64_t n_int = ((int64_t)1 << f.depth) - 1;
    const int64_t nn = n_int * f.n_trees;
    // distinct thresholds per feature
    std::vector<std::vector<float>> U(f.n_features);
    for (int64_t e = 0; e < nn; ++e) {
        if (feat[e] >= f.n_features) return PackStatus::bad_feature;
        if (thr[e] != thr[e]) return PackStatus::nan_threshold;
        U[feat[e]].push_back(thr[e] == 0.0f ? 0.0f : thr[e]);
    }
    std::vector<uint8_t> img(g.total, 0);
    float *table = reinterpret_cast<float *>(img.data() + 256);
    for (int j = 0; j < f.n_features; ++j) {
        auto &u = U[j];
        std::sort(u.begin(), u.end());
        u.erase(std::unique(u.begin(), u.end()), u.end());
        if (u.size() > 255) return PackStatus::too_many_thresholds;
        for (int k = 0; k < kBinSlots; ++k)
            table[j * kBinSlots + k] = k < (int)u.size() ? u[k] : __builtin_inff();
    }
    uint8_t *chunk0 = img.data() + 256 + g.thr_bytes;
    for (int c = 0; c < g.n_chunks; ++c) {
        uint8_t *nodes = chunk0 + (size_t)c * g.chunk_bytes;
        float *leaves = reinterpret_cast<float *>(chunk0 + (size_t)c * g.chunk_bytes + g.node_bytes);
        for (int tt = 0; tt < g.tc; ++tt) {
            const int64_t tree = (int64_t)c * g.tc + tt;
            if (tree >= f.n_trees) continue;   // padding trees: zero codes, zero leaves
            for (int64_t n = 0; n < n_int; ++n) {
                const uint8_t fj = feat[tree * n_int + n];
                float v = thr[tree * n_int + n];
                v = v == 0.0f ? 0.0f : v;
                const auto &u = U[fj];
                const int rank = (int)(std::lower_bound(u.begin(), u.end(), v) - u.begin());
                const uint16_t code = (uint16_t)(fj | (rank << 8));
                for (int copy = 0; copy < node_copies(g.tc); ++copy)
                    std::memcpy(nodes + node_byte((uint32_t)(n + 1), tt, copy, g.tc), &code, 2);
            }
            for (int64_t l = 0; l <= n_int; ++l) leaves[l * g.tc + tt] = leaf[tree * (n_int + 1) + l];
        }
    }
    const ImageId id = image_id(f, g);
    std::memcpy(img.data(), &id, sizeof id);
    std::memcpy(img_out, img.data(), g.total);
    return PackStatus::ok;
}

// Copy the forest to the host, build the image there, upload it.
PackStatus pack_forest(const hwsel_forest_t &f, void *packed, hipStream_t s)
{
    const PackGeom g = geometry(f);
    const int64_t n_int = ((int64_t)1 << f.depth) - 1;
    const int64_t nn = n_int * f.n_trees, nl = (n_int + 1) * f.n_trees;
    std::vector<uint8_t> feat(nn), img(g.total);
    std::vector<float> thr(nn), leaf(nl);
    if (hipMemcpyAsync(feat.data(), f.node_feature, nn, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipMemcpyAsync(thr.data(), f.node_threshold, nn * 4, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipMemcpyAsync(leaf.data(), f.leaf_value, nl * 4, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
        return PackStatus::hip_error;
    const PackStatus st = build_image(f, feat.data(), thr.data(), leaf.data(), img.data());
    if (st != PackStatus::ok) return st;
    if (hipMemcpyAsync(packed, img.data(), g.total, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
        return PackStatus::hip_error;
    return PackStatus::ok;
}

ImageId packed_image_id(const hwsel_forest_t &f) { return image_id(f, geometry(f)); }

int packed_bin_stride(const hwsel_forest_t &f) { return geometry(f).stride; }

uint32_t packed_nan_bin(const hwsel_forest_t &f) { return (f.flags & 1u) ? 0u : 255u; }

namespace {

hipError_t traverse_and_reduce(const hwsel_forest_t &f, const void *packed, int64_t R, float *scores,
                               void *workspace, const LeafHook &hook, hipStream_t s)
{
    const PackGeom g = geometry(f);
    const ImageId id = image_id(f, g);
    const uint8_t *chunks = static_cast<const uint8_t *>(packed) + 256 + g.thr_bytes;
    const uint8_t *Xb = static_cast<const uint8_t *>(workspace);
    float *partial = reinterpret_cast<float *>(static_cast<uint8_t *>(workspace) + align256((size_t)R * g.stride));
    hipError_t e = launch_traverse(f.depth, packed, id, chunks, g.n_chunks, Xb, R, g.stride, partial, hook, s);
    if (e != hipSuccess) return e;
    if (R % 4 == 0 && ((uintptr_t)scores & 15u) == 0)
        hipLaunchKernelGGL(k_reduce4, dim3((unsigned)((R / 4 + 255) / 256)), dim3(256), 0, s, packed, id, partial,
                           g.n_chunks, R, f.base_score, scores);
    else
        hipLaunchKernelGGL(k_reduce, dim3((unsigned)((R + 255) / 256)), dim3(256), 0, s, packed, id, partial,
                           g.n_chunks, R, f.base_score, scores);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_forest_packed(const hwsel_forest_t &f, const void *packed, const float *X, int64_t R,
                                int64_t ld, float *scores, void *workspace, hipStream_t s)
{
    return launch_forest_checked(f, packed, X, R, ld, scores, workspace, nullptr, nullptr, 0, 0, s);
}

hipError_t launch_forest_checked(const hwsel_forest_t &f, const void *packed, const float *X, int64_t R,
                                 int64_t ld, float *scores, void *workspace, uint64_t *leaf_hash,
                                 uint16_t *leaf_idx, int64_t leaf_row0, int64_t leaf_rows, hipStream_t s)
{
    const PackGeom g = geometry(f);
    uint8_t *Xb = static_cast<uint8_t *>(workspace);
    int dev = 0, n_cu = 256;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n_cu < 1)
        n_cu = 256;
    hipLaunchKernelGGL(k_bin, dim3(n_cu), dim3(kBinThreads), 0, s, X, R, ld, packed, image_id(f, g), f.n_features,
                       packed_nan_bin(f), Xb, g.stride);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (leaf_hash) {
        hipLaunchKernelGGL(k_fill_u64, dim3(1024), dim3(256), 0, s, leaf_hash, R);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const LeafHook hook{leaf_hash, leaf_idx, leaf_row0, leaf_idx ? leaf_rows : 0, f.n_trees};
    return traverse_and_reduce(f, packed, R, scores, workspace, hook, s);
}

// Traversal and reduction of bins already in the workspace.
hipError_t launch_forest_from_bins(const hwsel_forest_t &f, const void *packed, int64_t R, float *scores,
                                   void *workspace, hipStream_t s)
{
    return traverse_and_reduce(f, packed, R, scores, workspace, LeafHook{nullptr, nullptr, 0, 0, f.n_trees}, s);
}

}  // namespace hwsel
