// Feature kernel: x = phi(p, c, h) for every (problem, candidate) row.
//
// One thread per row; a wave owns 64 consecutive rows.  The candidate record
// is read as coalesced struct-of-arrays streams (17 B/row), the problem record
// once per row from a tiny L2-resident table.  The feature row is built in
// registers, then staged through LDS 32 columns at a time so that every
// global store is a 16-byte vector store into a contiguous 128-byte row
// segment (8 rows per wave instruction).  The kernel is bound by the X write
// stream (4F bytes per row).
//
// Numeric contract (same as the definition the oracle follows):
//   integer columns  - exact int64 values, one conversion to fp32 (RNE);
//   ratio columns    - one binary64 division of two exact int64 values, then
//                      fp32 (the division is correctly rounded on gfx950);
//   composite columns- a fixed short sequence of binary64 operations;
//   log2 columns     - binary64 log2, then fp32.
// This translation unit is compiled with -ffp-contract=off so no multiply-add
// is fused behind the sequence's back.
#include "internal.hpp"

#include <math.h>

namespace hwsel {
namespace {

__device__ __forceinline__ int64_t cdiv64(int64_t a, int64_t b) { return (a + b - 1) / b; }
__device__ __forceinline__ int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }
__device__ __forceinline__ int64_t min64(int64_t a, int64_t b) { return a < b ? a : b; }
__device__ __forceinline__ float exact(int64_t v) { return (float)v; }
__device__ __forceinline__ float quot(int64_t n, int64_t d) { return (float)((double)n / (double)d); }
__device__ __forceinline__ float lg(int64_t v) { return (float)log2((double)v); }

// Knob codes.
constexpr int kWS = 0, kCoop = 2;
constexpr int eNone = 0, eTma = 1;
constexpr int tStreamK = 1;
constexpr int dFp16 = 1, dFp8 = 2, dFp32 = 3;
constexpr int lNN = 2, lNT = 3, lTT = 1;

// Analytic sampling score (section "Candidate Sampling"): the cluster-wave
// fill n_c / (W S_SM c_M c_N) times S sqrt(T_M T_N T_K), in binary64.
__device__ __forceinline__ float sampling_score(int64_t clusters, int64_t cwaves, int64_t cslots, int64_t cm,
                                                int64_t cn, int64_t st, int64_t tm, int64_t tn, int64_t tk)
{
    const double fill = (double)(clusters * st) / (double)(cwaves * cslots * cm * cn);
    return (float)(fill * sqrt((double)(tm * tn * tk)));
}

// What the feature map needs of a problem alone: its integer terms and the
// columns that depend on nothing else, computed once per problem rather than
// once per row (the same operations, so the same values).
struct ProbTerms {
    int64_t M, N, K, pk, a_bytes, b_bytes, epi_traffic, conv, gemm_flops;
    int32_t layout, dtype, eb, out_dtype;
    // columns 0-3, 43, 46, 49, 80, 81, 88, 119-123
    float lg_m, lg_n, lg_k, lg_flops, x43, x46, x49, x80, x81, x88, x119, x120, x121, x122, x123;
};

__device__ __forceinline__ ProbTerms problem_terms(const HwDev &h, const hwsel_problem_t &pb)
{
    ProbTerms t;
    const int64_t M = max64(pb.M, 1), N = max64(pb.N, 1), K = max64(pb.K, 1);
    const int dtype = pb.dtype < 2 ? pb.dtype : 2;
    const int64_t eb = dtype == dFp8 ? 1 : 2;          // input element bytes (A and B)
    const int64_t ob = 2;                              // output / C element bytes
    const int out_dtype = dtype == dFp16 ? dFp16 : 0;
    const int64_t pk = h.peak[dtype];
    t.M = M; t.N = N; t.K = K; t.pk = pk;
    t.layout = pb.layout < 3 ? pb.layout : 3;
    t.dtype = dtype; t.eb = (int32_t)eb; t.out_dtype = out_dtype;
    t.a_bytes = eb * M * K;
    t.b_bytes = eb * K * N;
    t.epi_traffic = 2 * ob * M * N;                    // D written + C read
    t.conv = out_dtype != dtype ? M * N * ob : 0;
    t.gemm_flops = 2 * M * N * K;
    t.lg_m = lg(M); t.lg_n = lg(N); t.lg_k = lg(K); t.lg_flops = lg(t.gemm_flops);
    t.x43 = quot(t.gemm_flops, t.a_bytes + t.b_bytes + t.epi_traffic);
    t.x46 = quot(t.a_bytes + t.b_bytes, h.llc);
    t.x49 = exact(t.epi_traffic);
    t.x80 = quot(pk, h.bw);
    t.x81 = (float)(((double)t.gemm_flops / (double)(t.a_bytes + t.b_bytes + t.epi_traffic)) /
                    ((double)pk / (double)h.bw));
    t.x88 = exact(t.conv);
    t.x119 = quot(t.a_bytes, h.llc);
    t.x120 = quot(t.b_bytes, h.llc);
    t.x121 = quot(ob * M * N, h.llc);
    t.x122 = quot(M, N);
    t.x123 = quot(K, max64(M, N));
    return t;
}

template <int F>
__device__ __forceinline__ void phi(const HwDev &h, const ProbTerms &pt, const CandsDev &c, int64_t r, float (&x)[F])
{
    // ---- problem ----
    const int64_t M = pt.M, N = pt.N, K = pt.K;
    const int layout = pt.layout;
    const int dtype = pt.dtype;
    const int64_t eb = pt.eb;                          // input element bytes (A and B)
    const int64_t ob = 2;                              // output / C element bytes
    const int out_dtype = pt.out_dtype;
    const int64_t pk = pt.pk;

    // ---- candidate ----
    const int64_t tm = max64(c.tile_m[r], 1), tn = max64(c.tile_n[r], 1), tk = max64(c.tile_k[r], 1);
    const int64_t in_ = max64(c.inst_n[r], 1);
    const int64_t st = max64(c.stages[r], 1);
    const int64_t cm = max64(c.cluster_m[r], 1), cn = max64(c.cluster_n[r], 1);
    const int64_t swz = c.swizzle[r];
    const int64_t im = 16 * max64(c.inst_m_div16[r], 1), ik = max64(c.inst_k[r], 1);
    const int ks = c.kernel_sched[r] < 2 ? c.kernel_sched[r] : 2;
    const int es = c.epi_sched[r] < 2 ? c.epi_sched[r] : 2;
    const int ts = c.tile_sched[r] < 1 ? c.tile_sched[r] : 1;

    // ---- schedule: warpgroups ----
    const int64_t threads = ks == kWS ? 256 : 384;     // producer + 1 or 2 consumer warpgroups
    const int64_t consumers = ks == kCoop ? 2 : 1;     // consumer warpgroups on one tile

    // ---- work decomposition ----
    const int64_t gm = cdiv64(M, tm), gn = cdiv64(N, tn), gk = cdiv64(K, tk);
    const int64_t ntile = gm * gn;

    // ---- shared memory, registers, residency ----
    const int64_t stage_bytes = (tm + tn) * tk * eb;
    const int64_t main_bytes = st * stage_bytes;
    const int64_t frag = min64(tm, 64) * min64(tn, 32) * ob;
    const int64_t epi_bytes = es == eNone ? 0 : (es == eTma ? 2 * frag : 4 * frag);
    const int64_t smem = (ks == kWS ? max64(main_bytes, epi_bytes) : main_bytes + epi_bytes) + h.smem_rsv;
    const int64_t by_smem = h.smem_sm / smem;
    const int64_t regs = min64(h.regs_thread_max, cdiv64(tm * tn, threads) + 32);
    const int64_t by_regs = h.regs_sm / (regs * threads);
    const int64_t by_arch = min64(h.blocks_sm_max, h.threads_sm_max / threads);
    const int64_t resident = min64(min64(by_smem, by_regs), by_arch);
    const bool fits = main_bytes + epi_bytes + h.smem_rsv <= h.smem_block;

    // ---- waves over resident slots ----
    const int64_t slot_count = h.n_sm * (resident > 0 ? resident : 1);
    const int64_t waves = cdiv64(ntile, slot_count);
    const int64_t wave_cap = waves * slot_count;

    // ---- clusters ----
    const int64_t clusters = cdiv64(M, cm * tm) * cdiv64(N, cn * tn);
    const int64_t cslots = max64(h.n_sm / (cm * cn), 1);
    const int64_t cwaves = cdiv64(clusters, cslots);

    // ---- bytes ----
    const int64_t a_bytes = pt.a_bytes, b_bytes = pt.b_bytes;
    const int64_t epi_traffic = pt.epi_traffic;
    const int64_t loads = gn * a_bytes + gm * b_bytes; // every tile loads its panels
    const int64_t conv = pt.conv;
    const int64_t tile_flops = 2 * tm * tn * tk;

    // ---- tier 1 ----
    x[0] = pt.lg_m; x[1] = pt.lg_n; x[2] = pt.lg_k; x[3] = pt.lg_flops;
    x[4] = exact(tm); x[5] = exact(tn); x[6] = exact(tk); x[7] = exact(st);
    x[8] = exact(cm); x[9] = exact(cn); x[10] = exact(cm * cn); x[11] = exact(swz);
    x[12] = exact(gm); x[13] = exact(gn); x[14] = exact(gk); x[15] = exact(ntile);
    x[16] = quot(gm * tm - M, M);
    x[17] = quot(gn * tn - N, N);
    x[18] = quot(gk * tk - K, K);
    x[19] = quot(ntile, h.n_sm);
    x[20] = exact(threads);
    x[21] = quot(tm * tn, threads);
    x[22] = exact(regs);
    x[23] = exact(by_regs);
    x[24] = exact(stage_bytes);
    x[25] = exact(main_bytes);
    x[26] = exact(epi_bytes);
    x[27] = exact(smem);
    x[28] = quot(smem, h.smem_sm);
    x[29] = exact(by_smem);
    x[30] = exact(by_arch);
    x[31] = exact(resident);
    x[32] = exact(fits ? 1 : 0);
    x[33] = exact(waves);
    x[34] = quot(ntile, wave_cap);
    x[35] = quot(wave_cap - ntile, wave_cap);
    x[36] = exact(clusters);
    x[37] = exact(cslots);
    x[38] = exact(cwaves);
    x[39] = quot(clusters, cwaves * cslots);
    x[40] = quot(gm, cm);
    x[41] = quot(gn, cn);
    x[42] = exact((cm > gm || cn > gn) ? 1 : 0);
    x[43] = pt.x43;
    x[44] = quot(2 * tm * tn, (tm + tn) * eb);
    x[45] = quot(loads, a_bytes + b_bytes);
    x[46] = pt.x46;
    x[47] = quot((tm + tn) * K * eb, h.llc);
    x[48] = exact(loads);
    x[49] = pt.x49;
    const double t_load = (double)(h.n_sm * stage_bytes) / (double)h.bw;
    const double t_mma = (double)(tile_flops * h.n_sm) / (double)(consumers * pk);
    x[50] = quot(h.n_sm * stage_bytes, h.bw);
    x[51] = quot(tile_flops * h.n_sm, consumers * pk);
    x[52] = quot(tile_flops * h.bw, consumers * pk * stage_bytes);
    x[53] = quot(min64(st, gk), st);
    x[54] = quot(gk, st);
    x[55] = quot(st * smem, h.smem_sm);
    x[56] = exact(tk * st);
    x[57] = exact(st * resident);
    x[58] = sampling_score(clusters, cwaves, cslots, cm, cn, st, tm, tn, tk);
    x[59] = exact(h.n_sm); x[60] = exact(h.smem_sm); x[61] = exact(h.regs_sm);
    x[62] = exact(h.llc); x[63] = exact(h.bw);

    const bool a_colmajor = layout == lNN || layout == lNT;
    const bool b_rowmajor = layout == lTT || layout == lNT;
    const bool streamk = ts == tStreamK;
    const double stage_t = t_load > t_mma ? t_load : t_mma;

    if constexpr (F > 64) {
        x[64] = exact(layout); x[65] = exact(a_colmajor); x[66] = exact(b_rowmajor);
        x[67] = exact(dtype); x[68] = exact(dFp32); x[69] = exact(out_dtype);
        x[70] = exact(eb); x[71] = exact(eb); x[72] = exact(ob);
        x[73] = exact(ks); x[74] = exact(es); x[75] = exact(ts); x[76] = exact(streamk);
        x[77] = exact(consumers); x[78] = exact(h.arch_id); x[79] = exact(pk);
        x[80] = pt.x80;
        x[81] = pt.x81;
        const bool ok_a = !a_colmajor || tk <= 256 * cn;
        const bool ok_b = !b_rowmajor || tk <= 256 * cm;
        const bool ok_coop = ks != kCoop || (tm % 128) == 0;
        const bool ok_sk = !streamk || ks == kCoop;
        x[82] = exact(ok_a); x[83] = exact(ok_b); x[84] = exact(ok_coop); x[85] = exact(ok_sk);
        x[86] = exact(tn <= 2 * M && tn <= 2 * N);
        x[87] = exact(fits && ok_a && ok_b && ok_coop && ok_sk);
        x[88] = pt.x88;
        const int64_t traffic = loads + epi_traffic + conv;
        x[89] = exact(traffic);
        x[90] = quot(traffic, h.bw);
        const int64_t padded = (gm * tm) * (gn * tn) * (gk * tk);
        x[91] = quot(2 * padded, pk);
        x[92] = quot(padded, M * N * K);
        x[93] = exact(h.smem_block - smem);
        x[94] = exact(by_smem == resident);
        x[95] = exact(by_regs == resident);
    }
    if constexpr (F > 96) {
        const int64_t per_kblock = cdiv64(tm, im) * cdiv64(tn, in_) * cdiv64(tk, ik);
        x[96] = exact(im); x[97] = exact(in_); x[98] = exact(ik);
        x[99] = exact(per_kblock); x[100] = exact(per_kblock * gk);
        x[101] = exact(cdiv64(tm, 64)); x[102] = exact(tm * tn); x[103] = exact(tm * tn * tk);
        x[104] = (float)sqrt((double)(tm * tn * tk));
        x[105] = exact(tm * K * eb); x[106] = exact(tn * K * eb);
        x[107] = exact(tm * tn * ob); x[108] = exact(4 * tm * tn);
        x[109] = exact(min64(st, gk)); x[110] = exact(max64(gk - st, 0));
        const double mainloop_t = stage_t * (double)gk;
        x[111] = (float)stage_t;
        x[112] = (float)mainloop_t;
        x[113] = (float)(mainloop_t * (double)waves);
        x[114] = exact(streamk ? ntile * gk : 0);
        x[115] = streamk ? x[35] : 0.0f;
        x[116] = exact(resident * threads);
        x[117] = quot(resident * threads, h.threads_sm_max);
        x[118] = exact(by_arch == resident);
        x[119] = pt.x119;
        x[120] = pt.x120;
        x[121] = pt.x121;
        x[122] = pt.x122;
        x[123] = pt.x123;
        x[124] = quot(clusters, cslots);
        const int64_t edge = ntile - (M / tm) * (N / tn);
        x[125] = exact(edge);
        x[126] = quot(edge, ntile);
        x[127] = lg(ntile);
    }
}

constexpr int kWaves = 4;
constexpr int kCachedProblems = 4;

// One row per thread.  The row's columns are produced 64 (or 32) at a time:
// each pass evaluates the feature map and keeps only its columns (the shared
// integer intermediates are recomputed, the per-column work is not), which
// keeps the live registers low enough for more than one wave per SIMD.  Each
// 32-column slab is transposed through LDS into 16-byte row stores.  The
// problem terms of the workgroup's first problems (usually its only one) are
// computed once, by the first threads, and read from LDS by every row; rows
// of a later problem compute their own.
template <int F>
__global__ __launch_bounds__(64 * kWaves) void k_features(HwDev h, const hwsel_problem_t *__restrict__ probs,
                                                          int32_t P, const int64_t *__restrict__ seg,
                                                          CandsDev c, int64_t R, float *__restrict__ X,
                                                          int64_t ld)
{
    __shared__ float stage[kWaves][64][33];
    __shared__ ProbTerms cached[kCachedProblems];
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t blk0 = (int64_t)blockIdx.x * kWaves * 64;            // < R
    const int64_t row0 = blk0 + wave * 64;
    const int64_t r = row0 + lane;
    const int32_t p0 = segment_of_row(seg, P, blk0);
    const int32_t p_end = segment_of_row(seg, P, min64(blk0 + 64 * kWaves, R) - 1) + 1;
    const int n_cached = p_end - p0 < kCachedProblems ? p_end - p0 : kCachedProblems;
    if ((int)threadIdx.x < n_cached) cached[threadIdx.x] = problem_terms(h, probs[p0 + threadIdx.x]);
    hwsel_problem_t pb{};
    int slot = -1;                                     // index into cached, or -1
    if (r < R) {
        // the wave's rows are consecutive: one scalar search for its first row
        const int32_t p = segment_of_row_after(seg, P, r, row0);
        if (p - p0 < n_cached) slot = p - p0;
        else pb = probs[p];
    }
    __syncthreads();
    constexpr int kPass = F % 64 == 0 ? 64 : 32;      // columns per evaluation of the map
    float xs[kPass];
#pragma unroll
    for (int ch = 0; ch < F / 32; ++ch) {
        if (ch % (kPass / 32) == 0) {
            float x[F];
            if (r < R) {
                // re-read per pass rather than held across passes
                int sl = slot;
                asm volatile("" : "+v"(sl));
                const ProbTerms pt = sl >= 0 ? cached[sl] : problem_terms(h, pb);
                phi<F>(h, pt, c, r, x);
            } else {
#pragma unroll
                for (int j = 0; j < F; ++j) x[j] = 0.0f;
            }
#pragma unroll
            for (int j = 0; j < kPass; ++j) xs[j] = x[ch * 32 + j];
        }
#pragma unroll
        for (int j = 0; j < 32; ++j) stage[wave][lane][j] = xs[(ch % (kPass / 32)) * 32 + j];
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int q = lane + 64 * i;
            const int rr = q >> 3, cc = (q & 7) * 4;
            const int64_t gr = row0 + rr;
            if (gr < R) {
                const float4 v = make_float4(stage[wave][rr][cc], stage[wave][rr][cc + 1],
                                             stage[wave][rr][cc + 2], stage[wave][rr][cc + 3]);
                *reinterpret_cast<float4 *>(X + gr * ld + ch * 32 + cc) = v;
            }
        }
        __syncthreads();
    }
}

// Sampling score alone, one row per thread.
__global__ __launch_bounds__(256) void k_sample_score(HwDev h, const hwsel_problem_t *__restrict__ probs, int32_t P,
                                                       const int64_t *__restrict__ seg, CandsDev c, int64_t R,
                                                       float *__restrict__ scores)
{
    const int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
    // the wave's first row (wave-uniform): one scalar search per wave
    const int64_t r_first = (int64_t)blockIdx.x * 256 + __builtin_amdgcn_readfirstlane(threadIdx.x & ~63u);
    if (r >= R) return;
    const hwsel_problem_t pb = probs[segment_of_row_after(seg, P, r, r_first)];
    const int64_t M = max64(pb.M, 1), N = max64(pb.N, 1);
    const int64_t tm = max64(c.tile_m[r], 1), tn = max64(c.tile_n[r], 1), tk = max64(c.tile_k[r], 1);
    const int64_t st = max64(c.stages[r], 1);
    const int64_t cm = max64(c.cluster_m[r], 1), cn = max64(c.cluster_n[r], 1);
    const int64_t clusters = cdiv64(M, cm * tm) * cdiv64(N, cn * tn);
    const int64_t cslots = max64(h.n_sm / (cm * cn), 1);
    const int64_t cwaves = cdiv64(clusters, cslots);
    scores[r] = sampling_score(clusters, cwaves, cslots, cm, cn, st, tm, tn, tk);
}

// Features straight to forest bins: the row's feature vector stays in
// registers and each of the first nf columns is binned against the forest's
// sorted thresholds (b = #{u : u <= x}, NaN to nan_bin), the same search as
// the forest's own binning pass; X is never written.  One workgroup per CU
// holds the threshold table in LDS and walks row tiles.
constexpr int kFbThreads = 512;
constexpr int kFbSlots = 256;
constexpr int kFbStride = 257;
constexpr int kFbChains = 8;

template <int F>
__global__ __launch_bounds__(kFbThreads, 1) void k_features_bins(HwDev h, const hwsel_problem_t *__restrict__ probs,
                                                                 int32_t P, const int64_t *__restrict__ seg,
                                                                 CandsDev c, int64_t R,
                                                                 const void *__restrict__ packed, ImageId id, int nf,
                                                                 uint32_t nan_bin, uint8_t *__restrict__ Xb,
                                                                 int stride)
{
    if (!image_matches(packed, id)) return;
    const float *__restrict__ U = reinterpret_cast<const float *>(static_cast<const uint8_t *>(packed) + 256);
    __shared__ float u[128 * kFbStride];
    for (int e = threadIdx.x; e < nf * kFbSlots; e += kFbThreads) u[(e >> 8) * kFbStride + (e & 255)] = U[e];
    __syncthreads();
    constexpr int kPass = F % 64 == 0 ? 64 : 32;      // columns per evaluation of the map
    // A wave's rows are consecutive: one scalar search for its first row,
    // each lane steps forward from there.
    const int wave_base = __builtin_amdgcn_readfirstlane(threadIdx.x & ~63u);
    for (int64_t rw = (int64_t)blockIdx.x * kFbThreads + wave_base; rw < R; rw += (int64_t)gridDim.x * kFbThreads) {
        const int64_t r = rw + (threadIdx.x & 63);
        if (r >= R) break;
        const int32_t p = segment_of_row_after(seg, P, r, rw);
        const hwsel_problem_t pb = probs[p];
        uint32_t word[F / 4];
#pragma unroll
        for (int q = 0; q < F / 4; ++q) word[q] = 0;
#pragma unroll
        for (int p0 = 0; p0 < F; p0 += kPass) {
            if (p0 >= nf) break;
            // an opaque copy of the row index keeps each pass's evaluation
            // separate (otherwise the passes are merged into one evaluation
            // with every column live)
            int64_t rp = r;
            asm volatile("" : "+v"(rp));
            float x[F];
            phi<F>(h, problem_terms(h, pb), c, rp, x);
            // kFbChains independent searches in flight
#pragma unroll
            for (int f0 = p0; f0 < p0 + kPass; f0 += kFbChains) {
                if (f0 < nf) {
                    uint32_t b[kFbChains];
#pragma unroll
                    for (int q = 0; q < kFbChains; ++q) b[q] = (uint32_t)(f0 + q) * kFbStride;
#pragma unroll
                    for (int step = 128; step > 0; step >>= 1)
#pragma unroll
                        for (int q = 0; q < kFbChains; ++q) b[q] += (u[b[q] + step - 1] <= x[f0 + q]) ? step : 0;
#pragma unroll
                    for (int q = 0; q < kFbChains; ++q) {
                        uint32_t v = b[q] - (uint32_t)(f0 + q) * kFbStride;
                        if (x[f0 + q] != x[f0 + q]) v = nan_bin;
                        if (f0 + q >= nf) v = 0;
                        word[(f0 + q) / 4] |= v << (8 * ((f0 + q) % 4));
                    }
                }
            }
        }
        uint8_t *dst = Xb + r * stride;
#pragma unroll
        for (int q = 0; q < F / 16; ++q)
            if (16 * q < stride)
                *reinterpret_cast<uint4 *>(dst + 16 * q) =
                    make_uint4(word[4 * q], word[4 * q + 1], word[4 * q + 2], word[4 * q + 3]);
    }
}

}  // namespace

hipError_t launch_features_bins(const HwDev &hw, const hwsel_problem_t *problems, int32_t P, const int64_t *seg,
                                const CandsDev &c, int64_t R, int32_t F, const void *packed, ImageId id, int nf,
                                uint32_t nan_bin, uint8_t *Xb, int stride, hipStream_t s)
{
    int dev = 0, n_cu = 256;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n_cu < 1)
        n_cu = 256;
    const int64_t need = (R + kFbThreads - 1) / kFbThreads;
    const unsigned blocks = (unsigned)(need < n_cu ? need : n_cu);
    if (F == 64)
        hipLaunchKernelGGL(k_features_bins<64>, dim3(blocks), dim3(kFbThreads), 0, s, hw, problems, P, seg, c, R, packed,
                           id, nf, nan_bin, Xb, stride);
    else if (F == 96)
        hipLaunchKernelGGL(k_features_bins<96>, dim3(blocks), dim3(kFbThreads), 0, s, hw, problems, P, seg, c, R, packed,
                           id, nf, nan_bin, Xb, stride);
    else
        hipLaunchKernelGGL(k_features_bins<128>, dim3(blocks), dim3(kFbThreads), 0, s, hw, problems, P, seg, c, R,
                           packed, id, nf, nan_bin, Xb, stride);
    return hipGetLastError();
}

hipError_t launch_sample_score(const HwDev &hw, const hwsel_problem_t *problems, int32_t P, const int64_t *seg,
                               const CandsDev &c, int64_t R, float *scores, hipStream_t s)
{
    hipLaunchKernelGGL(k_sample_score, dim3((unsigned)((R + 255) / 256)), dim3(256), 0, s, hw, problems, P, seg, c,
                       R, scores);
    return hipGetLastError();
}

hipError_t launch_features(const HwDev &hw, const hwsel_problem_t *problems, int32_t P,
                           const int64_t *seg, const CandsDev &c, int64_t R, int32_t F, float *X,
                           int64_t ld, hipStream_t s)
{
    const int64_t rows_per_block = 64 * kWaves;
    const dim3 grid((unsigned)((R + rows_per_block - 1) / rows_per_block));
    const dim3 block(64 * kWaves);
    if (F == 64)
        hipLaunchKernelGGL(k_features<64>, grid, block, 0, s, hw, problems, P, seg, c, R, X, ld);
    else if (F == 96)
        hipLaunchKernelGGL(k_features<96>, grid, block, 0, s, hw, problems, P, seg, c, R, X, ld);
    else
        hipLaunchKernelGGL(k_features<128>, grid, block, 0, s, hw, problems, P, seg, c, R, X, ld);
    return hipGetLastError();
}

}  // namespace hwsel
