// Backward kernels of the fused 3S operator on CDNA4 (gfx950): the extension
// the paper names as the next step, built from the same pieces as the
// forward kernel (row windows, 16x16 blocks with bitmaps, block pairs with
// row-contiguous gathers staged through LDS, 16x16x32 MFMA).
//
// With P the forward probabilities (recomputed from the stored log-sum-exp,
// so nothing of size nnz is kept between the passes) and G = dL/dO:
//   delta_i = G_i . O_i                           k_bwd_dq   (windows of A)
//   dP_ij   = G_i . V_j,  dS_ij = P_ij (dP_ij - delta_i)
//   dQ_i    = scale sum_j dS_ij K_j               k_bwd_dq
//   dV_j    = sum_i P_ij G_i                      k_bwd_dkdv (windows of A^T)
//   dK_j    = scale sum_i dS_ij Q_i               k_bwd_dkdv
// dK and dV are owned by the windows of the transposed pattern, so no
// atomics are needed and results are deterministic.
//
// kBF16 = false: Q, K, V, G are fp16; dS and P enter the products as fp16
// (RNE), like P in the forward (Table 5's scheme).  kBF16 = true: they are
// bfloat16; S and dP use the bf16 product, and dS and P enter the products
// as two bf16 terms (hi = RNE of the value, lo = RNE of the remainder), as
// P does in the bf16 forward, so about 16 significant bits survive.
// (backward.hip instantiates the fp16 kernels, backward_bf16.hip the bf16
// ones.)
#pragma once

#include "kernel_common.h"

namespace f3s {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

// 16x16x32 product of fp16 or (raw) bf16 operands.
template <bool kBF16>
__device__ __forceinline__ f4 bmma(h8 a, h8 b, f4 c)
{
    if constexpr (kBF16)
        return mfma16x16x32_bf16(a, b, c);
    else
        return mfma16x16x32(a, b, c);
}

// One stored element (fp16, or bf16 raw bits) as fp32.
template <bool kBF16>
__device__ __forceinline__ float widen(_Float16 x)
{
    if constexpr (kBF16)
        return __builtin_bit_cast(float, (uint32_t)__builtin_bit_cast(uint16_t, x) << 16);
    else
        return (float)x;
}

// x as a 16-bit product operand {hi, lo}: fp16 (RNE) in hi; for bf16,
// hi + lo with both bf16 (RNE), about 16 significant bits of x.
template <bool kBF16>
__device__ __forceinline__ h2 operand(float x)
{
    if constexpr (kBF16) {
        const __bf16 hb = (__bf16)x;
        return h2{__builtin_bit_cast(_Float16, hb),
                  __builtin_bit_cast(_Float16, (__bf16)(x - (float)hb))};
    } else {
        const _Float16 h = (_Float16)x;
        return h2{h, h};  // lo unused
    }
}

// Waves per SIMD (d >= 160: one wave, the accumulators spill into AGPRs).
template <int D> struct BwdWaves { static constexpr int value = 1; };
template <> struct BwdWaves<32> { static constexpr int value = 4; };
template <> struct BwdWaves<64> { static constexpr int value = 2; };
template <> struct BwdWaves<96> { static constexpr int value = 2; };
template <> struct BwdWaves<128> { static constexpr int value = 2; };
// The dQ pass holds fewer registers than the dK/dV pass: at d = 64 it fits
// four waves per SIMD (128 VGPRs) without spilling.
template <int D> struct BwdDqWaves { static constexpr int value = BwdWaves<D>::value; };
template <> struct BwdDqWaves<64> { static constexpr int value = 4; };

// Row-contiguous gather of the 32 rows (two blocks) of a block pair from two
// row-major fp16 matrices A and B (same rows): chunk f = lane + 64 j is row
// f / LPR, 16-byte chunk f % LPR.  `c` holds, in lanes 0..31, the row id of
// pair slot `lane` (already free of padding).
template <int D, bool kWide>
__device__ __forceinline__ void gather_pair(const _Float16 *A, const _Float16 *B, int c,
                                            int ld, int lane, h8 *sa, h8 *sb)
{
    constexpr int LPR = D / 8, NI = D / 16;
#pragma unroll
    for (int j = 0; j < NI; ++j) {
        const int f = lane + 64 * j;
        const int row = __shfl(c, f / LPR);
        if constexpr (kWide) {
            const int64_t off = (int64_t)row * ld + 8 * (f % LPR);
            sa[j] = load16(A + off);
            sb[j] = load16(B + off);
        } else {
            const uint32_t off = (uint32_t)row * (uint32_t)(2 * ld) + 16u * (f % LPR);
            sa[j] = load16_off(A, off);
            sb[j] = load16_off(B, off);
        }
    }
}

template <int D>
__device__ __forceinline__ void stage_pair(_Float16 *tile, int stride, int lane, const h8 *st)
{
    constexpr int LPR = D / 8, NI = D / 16;
#pragma unroll
    for (int j = 0; j < NI; ++j) {
        const int f = lane + 64 * j;
        *reinterpret_cast<h8 *>(&tile[(f / LPR) * stride + 8 * (f % LPR)]) = st[j];
    }
}

// Padding slots (-1) take the first slot of their block (slot 0 or 16),
// which is never padding; its bitmap bit is clear, so it contributes 0.
__device__ __forceinline__ int sanitize_slot(int ncol, int lane)
{
    const int f0 = __builtin_amdgcn_readlane(ncol, 0);
    const int f1 = __builtin_amdgcn_readlane(ncol, 16);
    return ncol < 0 ? ((lane & 16) ? f1 : f0) : ncol;
}

// dQ over the row windows of A.  Lane (i, g): query row i of the window;
// scores and dP as in the forward (S^T = K_hat Q^T, dP^T = V_hat G^T), then
// dQ^T += K_hat^T dS^T with K_hat read transposed from LDS.
template <int D, bool kWide, bool kBF16, int NW = 1>
__global__ __launch_bounds__(64 * NW)
__attribute__((amdgpu_waves_per_eu(BwdDqWaves<D>::value, 8))) void k_bwd_dq(
    const WorkItem *__restrict__ items, const int32_t *__restrict__ cols,
    const uint32_t *__restrict__ mask, const int32_t *__restrict__ win_row,
    const _Float16 *__restrict__ Q, const _Float16 *__restrict__ K,
    const _Float16 *__restrict__ V, const _Float16 *__restrict__ G,
    const float *__restrict__ O, const float *__restrict__ lse, float2 *__restrict__ stats,
    float *__restrict__ dQ, float *__restrict__ part, int32_t N, int32_t ld, int32_t h0,
    int32_t nh, float sl2, float scale, uint32_t order)
{
    constexpr int NC = D / 32, NT = D / 16, NI = D / 16;
    constexpr int LSK = D + 16;  // K tile: operand reads and transposed reads
    constexpr int LSV = D + 8;   // V tile: operand reads only
    __shared__ __attribute__((aligned(16))) _Float16 tKs[NW][32 * LSK];
    __shared__ __attribute__((aligned(16))) _Float16 tVs[NW][32 * LSV];
    // NW waves may share the work item (as in the forward): wave wv takes a
    // contiguous share of its block pairs; the partial dQ sums meet in LDS
    const int wv = NW > 1 ? (int)(threadIdx.x >> 6) : 0;
    _Float16 *const tK = tKs[wv];
    _Float16 *const tV = tVs[wv];

    const int lane = NW > 1 ? (int)(threadIdx.x & 63) : (int)threadIdx.x;
    const int i = lane & 15, g = lane >> 4;
    // window-major, or head by head when K and V exceed the caches (as in
    // the forward)
    const int n_it = gridDim.x / nh;
    const int wg = workgroup_position(order, nh);
    const int hl = (order & kOrderHead) ? wg / n_it : wg % nh;
    const int item = (order & kOrderHead) ? wg - hl * n_it : wg / nh;
    const int head = h0 + hl, H = ld / D;
    const WorkItem it = items[item];
    Q += (int64_t)head * D;
    K += (int64_t)head * D;
    V += (int64_t)head * D;
    G += (int64_t)head * D;
    O += (int64_t)head * D;
    dQ += (int64_t)head * D;
    // the window's rows (16-row windows, or those of a plan aligned to the
    // graphs of a batch); pad rows read the window's first row
    int32_t r0, nr;
    window_rows(win_row, N, it.window, &r0, &nr);
    const int row = r0 + i;
    const bool live = i < nr;
    const int rrow = live ? row : r0;
    int b0 = it.blk_begin, b1 = it.blk_end;
    if constexpr (NW > 1) {
        const int pairs = (b1 - b0 + 1) >> 1;
        const int pa = pairs * wv / NW, pb = pairs * (wv + 1) / NW;
        b1 = min(b1, b0 + 2 * pb);
        b0 = b0 + 2 * pa;
    }

    h8 q[NC], gq[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        q[c] = load16(Q + (int64_t)rrow * ld + 32 * c + 8 * g);
        gq[c] = load16(G + (int64_t)rrow * ld + 32 * c + 8 * g);
    }
    const float lse2 = lse[(int64_t)rrow * H + head] * kLog2e;
    // delta_i = G_i . O_i from the G values this lane holds and the matching
    // O values; the four lanes of a row together cover all d.  Every piece
    // of a split window writes the same value; the dK/dV pass reads it.
    float dl = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const float *orow = O + (int64_t)rrow * ld + 32 * c + 8 * g;
        const f4 o0 = *reinterpret_cast<const f4 *>(orow);
        const f4 o1 = *reinterpret_cast<const f4 *>(orow + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            dl += widen<kBF16>(gq[c][e]) * o0[e] + widen<kBF16>(gq[c][4 + e]) * o1[e];
    }
    dl += __shfl_xor(dl, 16);
    dl += __shfl_xor(dl, 32);
    // one 8-byte record per row and head for the dK/dV pass, which gathers
    // it for every attending row: (base-2 log-sum-exp, delta)
    if (g == 0 && live && wv == 0) stats[(int64_t)row * H + head] = float2{lse2, dl};

    f4 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};

    h8 kst[NI], vst[NI];
    uint32_t mwa = 0, mwb = 0;
    int ncol = 0;
    auto load_cols = [&](int b) {
        const int slot = lane & 31;
        const int blk = slot < 16 ? min(b, b1 - 1) : min(b + 1, b1 - 1);
        ncol = cols[(int64_t)kBlockCols * blk + (slot & 15)];
    };
    auto load_pair = [&](int b) {
        gather_pair<D, kWide>(K, V, sanitize_slot(ncol, lane), ld, lane, kst, vst);
        mwa = mask[(int64_t)kMaskWords * b + (lane >> 3)];
        mwb = mask[(int64_t)kMaskWords * min(b + 1, b1 - 1) + (lane >> 3)];
    };
    const int nib_shift = 4 * (lane & 7);
    auto step = [&](int b, bool prefetch) {
        stage_pair<D>(tK, LSK, lane, kst);
        stage_pair<D>(tV, LSV, lane, vst);
        tile_fence<NW>();
        f4 s0 = f4{0.f, 0.f, 0.f, 0.f}, s1 = s0, d0 = s0, d1 = s0;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const h8 ka = *reinterpret_cast<const h8 *>(&tK[i * LSK + 32 * c + 8 * g]);
            const h8 kb = *reinterpret_cast<const h8 *>(&tK[(16 + i) * LSK + 32 * c + 8 * g]);
            s0 = bmma<kBF16>(ka, q[c], s0);
            s1 = bmma<kBF16>(kb, q[c], s1);
        }
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const h8 va = *reinterpret_cast<const h8 *>(&tV[i * LSV + 32 * c + 8 * g]);
            const h8 vb = *reinterpret_cast<const h8 *>(&tV[(16 + i) * LSV + 32 * c + 8 * g]);
            d0 = bmma<kBF16>(va, gq[c], d0);
            d1 = bmma<kBF16>(vb, gq[c], d1);
        }
        const uint32_t nib0 = (mwa >> nib_shift) & 15u;
        const uint32_t nib1 = b + 1 < b1 ? (mwb >> nib_shift) & 15u : 0u;
        if (prefetch) {
            load_pair(b + 2);
            load_cols(b + 4);
        }
        h8 dsh, dsl;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float p0 = (nib0 >> r) & 1u ? __builtin_amdgcn_exp2f(s0[r] * sl2 - lse2) : 0.f;
            const float p1 = (nib1 >> r) & 1u ? __builtin_amdgcn_exp2f(s1[r] * sl2 - lse2) : 0.f;
            {
                const h2 t = operand<kBF16>(p0 * (d0[r] - dl));
                dsh[r] = t[0];
                dsl[r] = t[1];
            }
            {
                const h2 t = operand<kBF16>(p1 * (d1[r] - dl));
                dsh[4 + r] = t[0];
                dsl[4 + r] = t[1];
            }
        }
        // dQ^T += K_hat^T dS^T: transposed read of the K tile (slot order
        // 4g..4g+3 and 16+4g.. matches the dS values this lane holds)
        const _Float16 *ta = tK + (4 * g + (i >> 2)) * LSK + 4 * (i & 3);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const h8 a = cat44(lds_read_tr(ta + 16 * t), lds_read_tr(ta + 16 * LSK + 16 * t));
            acc[t] = bmma<kBF16>(a, dsh, acc[t]);
            if constexpr (kBF16) acc[t] = bmma<kBF16>(a, dsl, acc[t]);
        }
        tile_fence<NW>();
    };
    if (b0 < b1) {
        load_cols(b0);
        load_pair(b0);
        load_cols(b0 + 2);
        int b = b0;
        for (; b + 2 < b1; b += 2) step(b, true);
        step(b, false);
    }
    if constexpr (NW > 1) {
        // partial sums into the waves' own K tiles (16 x D floats fit), then
        // wave 0 adds them (lane (i, g) holds columns 16t + 4g .. +3 of row i)
        float *ot = reinterpret_cast<float *>(tK);
#pragma unroll
        for (int t = 0; t < NT; ++t)
            *reinterpret_cast<f4 *>(ot + i * D + 16 * t + 4 * g) = acc[t];
        __syncthreads();
        if (wv != 0) return;
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            const float *ow = reinterpret_cast<const float *>(tKs[w]) + i * D + 4 * g;
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[t] += *reinterpret_cast<const f4 *>(ow + 16 * t);
        }
    }
    float *out;
    if (it.slot < 0) {
        if (!live) return;
        out = dQ + (int64_t)row * ld;
    } else {
        const int64_t ps = (int64_t)it.slot * nh + hl;
        out = part + ps * kWindowRows * D + (int64_t)i * D;
    }
#pragma unroll
    for (int t = 0; t < NT; ++t)
        *reinterpret_cast<f4 *>(out + 16 * t + 4 * g) = acc[t] * scale;
}

// dK and dV over the row windows of A^T: lane (i, g) owns key i of the
// window; the compacted columns are the queries attending to it.
// S[query][key] = Q_hat K_w^T and dP = G_hat V_w^T come out with lane =
// key, 4 query slots per block, i.e. directly in the B-operand layout of
// dV^T += G_hat^T P and dK^T += Q_hat^T dS.
template <int D, bool kWide, bool kBF16, int NW = 1>
__global__ __launch_bounds__(64 * NW)
__attribute__((amdgpu_waves_per_eu(BwdWaves<D>::value, 8))) void k_bwd_dkdv(
    const WorkItem *__restrict__ items, const int32_t *__restrict__ cols,
    const uint32_t *__restrict__ mask, const _Float16 *__restrict__ Q,
    const _Float16 *__restrict__ K, const _Float16 *__restrict__ V,
    const _Float16 *__restrict__ G, const float2 *__restrict__ stats,
    float *__restrict__ dK, float *__restrict__ dV,
    float *__restrict__ part, int32_t N, int32_t ld, int32_t h0, int32_t nh, float sl2,
    float scale, uint32_t order)
{
    constexpr int NC = D / 32, NT = D / 16, NI = D / 16;
    constexpr int LS = D + 16;  // operand reads and transposed reads
    __shared__ __attribute__((aligned(16))) _Float16 tQs[NW][32 * LS];
    __shared__ __attribute__((aligned(16))) _Float16 tGs[NW][32 * LS];
    __shared__ float slses[NW][32], sdels[NW][32];
    // NW waves may share the work item (as in the forward): wave wv takes a
    // contiguous share of its block pairs; the partial dK, dV sums meet in LDS
    const int wv = NW > 1 ? (int)(threadIdx.x >> 6) : 0;
    _Float16 *const tQ = tQs[wv];
    _Float16 *const tG = tGs[wv];
    float *const slse = slses[wv];
    float *const sdel = sdels[wv];

    const int lane = NW > 1 ? (int)(threadIdx.x & 63) : (int)threadIdx.x;
    const int i = lane & 15, g = lane >> 4;
    // window-major, or head by head when K and V exceed the caches (as in
    // the forward)
    const int n_it = gridDim.x / nh;
    const int wg = workgroup_position(order, nh);
    const int hl = (order & kOrderHead) ? wg / n_it : wg % nh;
    const int item = (order & kOrderHead) ? wg - hl * n_it : wg / nh;
    const int head = h0 + hl, H = ld / D;
    const WorkItem it = items[item];
    Q += (int64_t)head * D;
    K += (int64_t)head * D;
    V += (int64_t)head * D;
    G += (int64_t)head * D;
    dK += (int64_t)head * D;
    dV += (int64_t)head * D;
    const int key = it.window * kWindowRows + i;
    const int rkey = min(key, N - 1);
    int b0 = it.blk_begin, b1 = it.blk_end;
    if constexpr (NW > 1) {
        const int pairs = (b1 - b0 + 1) >> 1;
        const int pa = pairs * wv / NW, pb = pairs * (wv + 1) / NW;
        b1 = min(b1, b0 + 2 * pb);
        b0 = b0 + 2 * pa;
    }

    h8 kw[NC], vw[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        kw[c] = load16(K + (int64_t)rkey * ld + 32 * c + 8 * g);
        vw[c] = load16(V + (int64_t)rkey * ld + 32 * c + 8 * g);
    }
    f4 ak[NT], av[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) ak[t] = av[t] = f4{0.f, 0.f, 0.f, 0.f};

    h8 qst[NI], gst[NI];
    uint32_t mwa = 0, mwb = 0;
    float lsev = 0.f, delv = 0.f;  // lanes 0..31: of pair slot `lane`
    int ncol = 0;
    auto load_cols = [&](int b) {
        const int slot = lane & 31;
        const int blk = slot < 16 ? min(b, b1 - 1) : min(b + 1, b1 - 1);
        ncol = cols[(int64_t)kBlockCols * blk + (slot & 15)];
    };
    auto load_pair = [&](int b) {
        const int c = sanitize_slot(ncol, lane);
        gather_pair<D, kWide>(Q, G, c, ld, lane, qst, gst);
        const float2 st = stats[(int64_t)c * H + head];
        lsev = st.x;
        delv = st.y;
        mwa = mask[(int64_t)kMaskWords * b + (lane >> 3)];
        mwb = mask[(int64_t)kMaskWords * min(b + 1, b1 - 1) + (lane >> 3)];
    };
    const int nib_shift = 4 * (lane & 7);
    auto step = [&](int b, bool prefetch) {
        stage_pair<D>(tQ, LS, lane, qst);
        stage_pair<D>(tG, LS, lane, gst);
        if (lane < 32) {
            slse[lane] = lsev;
            sdel[lane] = delv;
        }
        tile_fence<NW>();
        f4 s0 = f4{0.f, 0.f, 0.f, 0.f}, s1 = s0, d0 = s0, d1 = s0;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const h8 qa = *reinterpret_cast<const h8 *>(&tQ[i * LS + 32 * c + 8 * g]);
            const h8 qb = *reinterpret_cast<const h8 *>(&tQ[(16 + i) * LS + 32 * c + 8 * g]);
            s0 = bmma<kBF16>(qa, kw[c], s0);
            s1 = bmma<kBF16>(qb, kw[c], s1);
        }
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const h8 ga = *reinterpret_cast<const h8 *>(&tG[i * LS + 32 * c + 8 * g]);
            const h8 gb = *reinterpret_cast<const h8 *>(&tG[(16 + i) * LS + 32 * c + 8 * g]);
            d0 = bmma<kBF16>(ga, vw[c], d0);
            d1 = bmma<kBF16>(gb, vw[c], d1);
        }
        const uint32_t nib0 = (mwa >> nib_shift) & 15u;
        const uint32_t nib1 = b + 1 < b1 ? (mwb >> nib_shift) & 15u : 0u;
        f4 l0, l1, e0, e1;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            l0[r] = slse[4 * g + r];
            l1[r] = slse[16 + 4 * g + r];
            e0[r] = sdel[4 * g + r];
            e1[r] = sdel[16 + 4 * g + r];
        }
        if (prefetch) {
            load_pair(b + 2);
            load_cols(b + 4);
        }
        h8 ph, pl, dsh, dsl;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float p0 = (nib0 >> r) & 1u ? __builtin_amdgcn_exp2f(s0[r] * sl2 - l0[r]) : 0.f;
            const float p1 = (nib1 >> r) & 1u ? __builtin_amdgcn_exp2f(s1[r] * sl2 - l1[r]) : 0.f;
            {
                const h2 t = operand<kBF16>(p0);
                ph[r] = t[0];
                pl[r] = t[1];
            }
            {
                const h2 t = operand<kBF16>(p1);
                ph[4 + r] = t[0];
                pl[4 + r] = t[1];
            }
            {
                const h2 t = operand<kBF16>(p0 * (d0[r] - e0[r]));
                dsh[r] = t[0];
                dsl[r] = t[1];
            }
            {
                const h2 t = operand<kBF16>(p1 * (d1[r] - e1[r]));
                dsh[4 + r] = t[0];
                dsl[4 + r] = t[1];
            }
        }
        const int toff = (4 * g + (i >> 2)) * LS + 4 * (i & 3);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const h8 a = cat44(lds_read_tr(tG + toff + 16 * t),
                               lds_read_tr(tG + toff + 16 * LS + 16 * t));
            av[t] = bmma<kBF16>(a, ph, av[t]);
            if constexpr (kBF16) av[t] = bmma<kBF16>(a, pl, av[t]);
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const h8 a = cat44(lds_read_tr(tQ + toff + 16 * t),
                               lds_read_tr(tQ + toff + 16 * LS + 16 * t));
            ak[t] = bmma<kBF16>(a, dsh, ak[t]);
            if constexpr (kBF16) ak[t] = bmma<kBF16>(a, dsl, ak[t]);
        }
        tile_fence<NW>();
    };
    if (b0 < b1) {
        load_cols(b0);
        load_pair(b0);
        load_cols(b0 + 2);
        int b = b0;
        for (; b + 2 < b1; b += 2) step(b, true);
        step(b, false);
    }
    if constexpr (NW > 1) {
        // partial sums into the waves' own Q and G tiles (16 x D floats each
        // fit), then wave 0 adds them
        float *okt = reinterpret_cast<float *>(tQ);
        float *ovt = reinterpret_cast<float *>(tG);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            *reinterpret_cast<f4 *>(okt + i * D + 16 * t + 4 * g) = ak[t];
            *reinterpret_cast<f4 *>(ovt + i * D + 16 * t + 4 * g) = av[t];
        }
        __syncthreads();
        if (wv != 0) return;
#pragma unroll
        for (int t = 0; t < NT; ++t) ak[t] = av[t] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            const float *kw_ = reinterpret_cast<const float *>(tQs[w]) + i * D + 4 * g;
            const float *vw_ = reinterpret_cast<const float *>(tGs[w]) + i * D + 4 * g;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                ak[t] += *reinterpret_cast<const f4 *>(kw_ + 16 * t);
                av[t] += *reinterpret_cast<const f4 *>(vw_ + 16 * t);
            }
        }
    }
    float *ok, *ov;
    if (it.slot < 0) {
        if (key >= N) return;
        ok = dK + (int64_t)key * ld;
        ov = dV + (int64_t)key * ld;
    } else {
        const int64_t ps = (int64_t)it.slot * nh + hl;
        ok = part + ps * 2 * kWindowRows * D + (int64_t)i * D;
        ov = ok + kWindowRows * D;
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        *reinterpret_cast<f4 *>(ok + 16 * t + 4 * g) = ak[t] * scale;
        *reinterpret_cast<f4 *>(ov + 16 * t + 4 * g) = av[t];
    }
}

// Sum of the partials of split windows, in piece order (deterministic).
// nparts outputs per (piece, head) slot, stored back to back.
template <int D>
__global__ __launch_bounds__(256) void k_merge_sum(const int32_t *__restrict__ merges,
                                                   const int32_t *__restrict__ win_row,
                                                   const float *__restrict__ part,
                                                   float *__restrict__ out0,
                                                   float *__restrict__ out1, int32_t nparts,
                                                   int32_t N, int32_t ld, int32_t h0,
                                                   int32_t nh)
{
    const int s = blockIdx.x / nh, hl = blockIdx.x - (blockIdx.x / nh) * nh;
    const int w = merges[3 * s], first = merges[3 * s + 1], np = merges[3 * s + 2];
    const int r = threadIdx.x >> 4, q = threadIdx.x & 15;
    int32_t r0, nr;
    window_rows(win_row, N, w, &r0, &nr);
    if (r >= nr) return;
    const int row = r0 + r;
    const int64_t slot_floats = (int64_t)nparts * kWindowRows * D;
    for (int pidx = 0; pidx < nparts; ++pidx) {
        float *out = (pidx == 0 ? out0 : out1) + (int64_t)row * ld + (int64_t)(h0 + hl) * D;
        const float *src = part + ((int64_t)first * nh + hl) * slot_floats +
                           (int64_t)pidx * kWindowRows * D + (int64_t)r * D;
        for (int c4 = q; c4 < D / 4; c4 += 16) {
            // pieces summed in order; the loads of 8 pieces are issued
            // together (indices past the last piece re-read it, unused)
            f4 acc = f4{0.f, 0.f, 0.f, 0.f};
            for (int k0 = 0; k0 < np; k0 += 8) {
                f4 v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int k = min(k0 + u, np - 1);
                    v[u] = *reinterpret_cast<const f4 *>(src + k * nh * slot_floats + 4 * c4);
                }
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (k0 + u < np) acc += v[u];
            }
            *reinterpret_cast<f4 *>(out + 4 * c4) = acc;
        }
    }
}

template <int D, bool kBF16>
hipError_t launch_bwd_d(const f3s_plan_s &p, const f3s_plan_s &pt, const void *Q,
                        const void *K, const void *V, const float *O, const void *G,
                        const float *lse, float *row_stats, float *dQ, float *dK, float *dV,
                        int32_t H, float sl2, float scale, hipStream_t s)
{
    float2 *stats = reinterpret_cast<float2 *>(row_stats);
    const int32_t ld = H * D;
    const bool wide = (uint64_t)p.N * ld * 2 > 0xFFFFFFF0ull;
    const auto *q = static_cast<const _Float16 *>(Q);
    const auto *k = static_cast<const _Float16 *>(K);
    const auto *v = static_cast<const _Float16 *>(V);
    const auto *gr = static_cast<const _Float16 *>(G);
    hipError_t e = hipSuccess;
    // launch order of a group of nh heads over plan q
    const uint64_t kv_bytes = 2ull * p.N * ld * 2;
    auto order_of = [kv_bytes](const f3s_plan_s &q, int32_t nh) -> uint32_t {
        const bool head_major = head_major_order(q, nh, kv_bytes);
        return (head_major ? kOrderHead : 0u) |
               (xcd_chunks(q, nh, head_major) ? kOrderXcd : 0u);
    };
    // dQ: windows of A; partials need 16*D floats per (piece, head)
    {
        const int nw = waves_per_item(p.n_blocks, p.n_items, H,
                                      (int64_t)BwdDqWaves<D>::value * 1024);
        auto kern = nw == 4   ? (wide ? k_bwd_dq<D, true, kBF16, 4> : k_bwd_dq<D, false, kBF16, 4>)
                    : nw == 2 ? (wide ? k_bwd_dq<D, true, kBF16, 2> : k_bwd_dq<D, false, kBF16, 2>)
                              : (wide ? k_bwd_dq<D, true, kBF16> : k_bwd_dq<D, false, kBF16>);
        const int32_t group = p.n_split > 0 ? (kMaxD / D < H ? kMaxD / D : H) : H;
        for (int32_t h0 = 0; h0 < H; h0 += group) {
            const int32_t nh = H - h0 < group ? H - h0 : group;
            if (p.n_split > 0 && (int64_t)nh * D > kMaxD) return hipErrorInvalidValue;
            if (p.n_items > 0) {
                kern<<<(unsigned)((uint64_t)p.n_items * nh), 64 * nw, 0, s>>>(
                    p.items, p.cols, p.mask, p.win_row, q, k, v, gr, O, lse, stats, dQ,
                    p.part_o, p.N, ld, h0, nh, sl2, scale, order_of(p, nh));
                if ((e = hipGetLastError()) != hipSuccess) return e;
            }
            if (p.n_split > 0) {
                k_merge_sum<D><<<p.n_split * nh, 256, 0, s>>>(p.merges, p.win_row, p.part_o,
                                                             dQ, nullptr, 1, p.N, ld, h0, nh);
                if ((e = hipGetLastError()) != hipSuccess) return e;
            }
        }
    }
    // dK, dV: windows of A^T; partials need 2*16*D floats per (piece, head)
    {
        const int nw = waves_per_item(pt.n_blocks, pt.n_items, H,
                                      (int64_t)BwdWaves<D>::value * 1024);
        auto kern = nw == 4
                        ? (wide ? k_bwd_dkdv<D, true, kBF16, 4> : k_bwd_dkdv<D, false, kBF16, 4>)
                    : nw == 2
                        ? (wide ? k_bwd_dkdv<D, true, kBF16, 2> : k_bwd_dkdv<D, false, kBF16, 2>)
                        : (wide ? k_bwd_dkdv<D, true, kBF16> : k_bwd_dkdv<D, false, kBF16>);
        // the transposed plan's partial rows hold part_row floats
        const int32_t cap = pt.part_row / (2 * D);
        if (pt.n_split > 0 && cap < 1) return hipErrorInvalidValue;
        const int32_t group = pt.n_split > 0 ? (cap < H ? cap : H) : H;
        for (int32_t h0 = 0; h0 < H; h0 += group) {
            const int32_t nh = H - h0 < group ? H - h0 : group;
            if (pt.n_split > 0 && (int64_t)nh * 2 * D > pt.part_row) return hipErrorInvalidValue;
            if (pt.n_items > 0) {
                kern<<<(unsigned)((uint64_t)pt.n_items * nh), 64 * nw, 0, s>>>(
                    pt.items, pt.cols, pt.mask, q, k, v, gr, stats, dK, dV, pt.part_o,
                    pt.N, ld, h0, nh, sl2, scale, order_of(pt, nh));
                if ((e = hipGetLastError()) != hipSuccess) return e;
            }
            if (pt.n_split > 0) {
                k_merge_sum<D><<<pt.n_split * nh, 256, 0, s>>>(pt.merges, pt.win_row,
                                                              pt.part_o, dK, dV, 2, pt.N, ld,
                                                              h0, nh);
                if ((e = hipGetLastError()) != hipSuccess) return e;
            }
        }
    }
    return hipSuccess;
}

template <bool kBF16>
hipError_t launch_bwd_in(const f3s_plan_s &p, const f3s_plan_s &pt, const void *Q,
                         const void *K, const void *V, const float *O, const void *G,
                         const float *lse, float *row_stats, float *dQ, float *dK, float *dV,
                         int32_t H, int32_t d, float scale, hipStream_t s)
{
    const float sl2 = scale * kLog2e;
    switch (d) {
#define F3S_BWD_CASE(DD)                                                                 \
    case DD:                                                                             \
        return launch_bwd_d<DD, kBF16>(p, pt, Q, K, V, O, G, lse, row_stats, dQ, dK, dV, H, \
                                       sl2, scale, s);
    F3S_BWD_CASE(32)
    F3S_BWD_CASE(64)
    F3S_BWD_CASE(96)
    F3S_BWD_CASE(128)
    F3S_BWD_CASE(160)
    F3S_BWD_CASE(192)
    F3S_BWD_CASE(224)
    F3S_BWD_CASE(256)
#undef F3S_BWD_CASE
    default: return hipErrorInvalidValue;
    }
}

}  // namespace
}  // namespace f3s
