// Internal launch interface between the C-ABI layer (api.hip) and the kernel
// translation units.  Launchers assume their arguments were checked by the
// caller and only enqueue work.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/hwsel.h"

namespace hwsel {

// Hardware descriptor as the kernels read it (plain copy of hwsel_hw_t).
struct HwDev {
    int64_t n_sm, smem_sm, smem_block, smem_rsv;
    int64_t regs_sm, regs_thread_max, blocks_sm_max, threads_sm_max;
    int64_t arch_id, llc, bw;
    int64_t peak[3];
};

struct CandsDev {
    const uint16_t *tile_m, *tile_n, *tile_k, *inst_n;
    const uint8_t *stages, *cluster_m, *cluster_n, *swizzle, *inst_m_div16, *inst_k;
    const uint8_t *kernel_sched, *epi_sched, *tile_sched;
};

hipError_t launch_features(const HwDev &hw, const hwsel_problem_t *problems, int32_t P,
                           const int64_t *seg, const CandsDev &c, int64_t R, int32_t F, float *X,
                           int64_t ld, hipStream_t s);

hipError_t launch_sample_score(const HwDev &hw, const hwsel_problem_t *problems, int32_t P, const int64_t *seg,
                               const CandsDev &c, int64_t R, float *scores, hipStream_t s);

hipError_t launch_linear(const hwsel_linear_t &lin, const float *X, int64_t R, int64_t ld, float *scores,
                         hipStream_t s);

size_t evaluate_workspace_bytes(int32_t P);
// Device address and size of this device's scratch array of the
// allocation-free evaluation (see evaluate.hip).
hipError_t evaluate_noalloc_scratch(void **ptr, size_t *bytes);
hipError_t launch_evaluate(const float *rt, const int64_t *seg, int32_t P, const int32_t *idx, int32_t k,
                           double *out, double *regret_out, int32_t *rank_out, double *ybar_out, void *ws,
                           hipStream_t s);
size_t static_config_workspace_bytes(int32_t P, int32_t n_cfg);
hipError_t launch_static_config(const float *rt, const int64_t *seg, int32_t P, const int32_t *cfg, int32_t n_cfg,
                                int32_t *best, double *mean_y, void *ws, hipStream_t s);

hipError_t launch_catalogue_mask(const HwDev &h, const hwsel_problem_t *probs, int32_t P, uint32_t flags,
                                 uint8_t *mask, int64_t *n_valid, hipStream_t s);
hipError_t launch_catalogue_compact(const uint8_t *mask, const int64_t *n_valid, int32_t P, int64_t *seg,
                                    int32_t *point, int64_t cap, hipStream_t s);
hipError_t launch_catalogue_candidates(const hwsel_problem_t *probs, int32_t P, const int64_t *seg,
                                       const int32_t *point, int64_t R, const hwsel_cands_out_t &out, hipStream_t s);

hipError_t launch_forest_score(const hwsel_forest_t &f, const float *X, int64_t R, int64_t ld,
                               float *scores, hipStream_t s);

hipError_t launch_forest_leaves(const hwsel_forest_t &f, const float *X, int64_t R, int64_t ld,
                                const int64_t *rows, int64_t n_rows, uint16_t *leaf_idx,
                                hipStream_t s);

// Packed forests (see forest.hip).
enum class PackStatus { ok, hip_error, bad_feature, nan_threshold, too_many_thresholds };

// Identity of a packed image, stored in its first 28 bytes (its threshold
// table starts at byte 256); every kernel that reads an image compares it
// with the forest the call is for first, and reads nothing more on a
// mismatch.
struct ImageId {
    int32_t magic, version, n_trees, depth, n_features, tc, n_chunks;
};

__device__ __forceinline__ bool image_matches(const void *packed, const ImageId &want)
{
    const int32_t *h = static_cast<const int32_t *>(packed);
    return h[0] == want.magic && h[1] == want.version && h[2] == want.n_trees && h[3] == want.depth &&
           h[4] == want.n_features && h[5] == want.tc && h[6] == want.n_chunks;
}

bool packable(const hwsel_forest_t &f);
size_t packed_bytes(const hwsel_forest_t &f);
size_t packed_workspace_bytes(const hwsel_forest_t &f, int64_t R);
PackStatus pack_forest(const hwsel_forest_t &f, void *packed, hipStream_t s);
PackStatus build_image(const hwsel_forest_t &f, const uint8_t *feat, const float *thr, const float *leaf,
                       uint8_t *img);
hipError_t launch_forest_packed(const hwsel_forest_t &f, const void *packed, const float *X, int64_t R,
                                int64_t ld, float *scores, void *workspace, hipStream_t s);
hipError_t launch_forest_checked(const hwsel_forest_t &f, const void *packed, const float *X, int64_t R,
                                 int64_t ld, float *scores, void *workspace, uint64_t *leaf_hash,
                                 uint16_t *leaf_idx, int64_t leaf_row0, int64_t leaf_rows, hipStream_t s);
// Pieces of the packed path for the fused selection: the threshold table and
// bin-row geometry of an image, and the traversal of bins already written to
// the start of the workspace.
ImageId packed_image_id(const hwsel_forest_t &f);
int packed_bin_stride(const hwsel_forest_t &f);
uint32_t packed_nan_bin(const hwsel_forest_t &f);
hipError_t launch_forest_from_bins(const hwsel_forest_t &f, const void *packed, int64_t R, float *scores,
                                   void *workspace, hipStream_t s);
hipError_t launch_features_bins(const HwDev &hw, const hwsel_problem_t *problems, int32_t P, const int64_t *seg,
                                const CandsDev &c, int64_t R, int32_t F, const void *packed, ImageId id, int nf,
                                uint32_t nan_bin, uint8_t *Xb, int stride, hipStream_t s);

hipError_t launch_mlp(const hwsel_mlp_t &m, const float *X, int64_t R, int64_t ld, float *scores,
                      hipStream_t s);
size_t mlp_packed_bytes();
hipError_t launch_mlp_pack(const hwsel_mlp_t &m, void *packed, hipStream_t s);
hipError_t launch_mlp_packed(const hwsel_mlp_t &m, const void *packed, const float *X, int64_t R, int64_t ld,
                             float *scores, hipStream_t s);

hipError_t launch_topk(const float *scores, const int64_t *seg, int32_t P, int32_t k, int32_t *idx,
                       float *vals, hipStream_t s);

hipError_t launch_regret(const float *rt, const int64_t *seg, int32_t P, const int32_t *idx,
                         int32_t k, float *r1, float *rk, int32_t *best, hipStream_t s);

// Order-preserving map of fp32 to uint32 (x < y <=> key(x) < key(y) for
// non-NaN values; -0 must be normalised to +0 first).
__device__ __forceinline__ uint32_t order_key(float v)
{
    const uint32_t u = __float_as_uint(v);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// One step of the bit-serial search: b <- 2 b + (key_u < kx1), i.e. + (u <= x)
// with kx1 = key(x) + 1.  Subtract-with-borrow leaves the comparison in VCC,
// add-with-carry shifts it in.
__device__ __forceinline__ uint32_t search_step(uint32_t b, uint32_t key_u, uint32_t kx1)
{
    uint32_t out;
    asm("v_sub_co_u32_e32 %0, vcc, %1, %2\n\t"
        "v_addc_co_u32_e32 %0, vcc, %3, %3, vcc"
        : "=&v"(out)
        : "v"(key_u), "v"(kx1), "v"(b)
        : "vcc");
    return out;
}

template <int CTRL, int ROW_MASK, bool ZERO_FILL>
__device__ __forceinline__ float dpp_add(float v)
{
    return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK, 0xf, ZERO_FILL));
}

// Sums over each aligned group of TC lanes (TC in {16, 32, 64}) of N
// independent values with DPP: an inclusive scan inside 16-lane rows, then
// row broadcasts.  The last lane of each group ends with the group's total,
// always in the same order.  The values advance stage by stage so that the
// dependent DPP steps of one are interleaved with the others'.
template <int TC, int N>
__device__ __forceinline__ void group_totals(float (&v)[N])
{
    static_assert(TC == 16 || TC == 32 || TC == 64, "group width");
#pragma unroll
    for (int a = 0; a < N; ++a) v[a] = dpp_add<0x111, 0xf, true>(v[a]);
#pragma unroll
    for (int a = 0; a < N; ++a) v[a] = dpp_add<0x112, 0xf, true>(v[a]);
#pragma unroll
    for (int a = 0; a < N; ++a) v[a] = dpp_add<0x114, 0xf, true>(v[a]);
#pragma unroll
    for (int a = 0; a < N; ++a) v[a] = dpp_add<0x118, 0xf, true>(v[a]);
    if constexpr (TC >= 32) {
#pragma unroll
        for (int a = 0; a < N; ++a) v[a] = dpp_add<0x142, 0xa, false>(v[a]);
    }
    if constexpr (TC >= 64) {
#pragma unroll
        for (int a = 0; a < N; ++a) v[a] = dpp_add<0x143, 0xc, false>(v[a]);
    }
}

// Workgroup barrier that orders LDS accesses only.  __syncthreads() also
// waits for every outstanding global load and store of the wave, which would
// cancel loads issued ahead of the barrier on purpose; use this one where the
// barrier protects LDS data alone.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Last segment p with seg[p] <= r (segments are [seg[p], seg[p+1])); the
// result is always in [0, P-1], whatever the offsets hold.
__device__ inline int32_t segment_of_row(const int64_t *__restrict__ seg, int32_t P, int64_t r)
{
    int32_t lo = 0, hi = P;
    while (hi - lo > 1) {
        const int32_t mid = (lo + hi) >> 1;
        if (seg[mid] <= r) lo = mid; else hi = mid;
    }
    return lo;
}

// segment_of_row for the lanes of one wave, whose rows r are consecutive and
// start at r_first (wave-uniform, r_first <= r): one search for r_first, on
// the scalar unit, then each lane steps past the segments that end at or
// before its row, usually none.  For non-decreasing offsets the result is
// segment_of_row(seg, P, r); it is in [0, P-1] whatever the offsets hold.
__device__ inline int32_t segment_of_row_after(const int64_t *__restrict__ seg, int32_t P, int64_t r, int64_t r_first)
{
    int32_t p = segment_of_row(seg, P, r_first);
    while (p + 1 < P && seg[p + 1] <= r) ++p;
    return p;
}

}  // namespace hwsel
