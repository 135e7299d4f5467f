// Ablation build of the fused forward: the split-row partition of a window's
// work among the waves of a workgroup (Section 3.3; the F3S_splitR variant of
// the ablation in Section 4.3), against the library's default, where the
// waves of a work item split its block pairs (split-column).  Selected by a
// plan built with F3S_SPLIT_ROW=1; fp16 inputs, fp32 output, d a multiple
// of 64, 32-bit addressing.
//
// NW waves share one work item and all walk all of its block pairs.  Wave w
// owns the feature slice [w D/NW, (w+1) D/NW):
//   scores   split-row: the wave gathers its slice of the pair's 32 K rows
//            and multiplies it with its slice of Q_i, a partial S^T over
//            D/NW of the D reduction terms; the NW partials meet in LDS
//            (one workgroup barrier per pair, double-buffered) and every
//            wave adds them up in the same order, so all waves hold the
//            same scores;
//   softmax  computed redundantly by every wave (identical values);
//   values   split-column: the wave gathers its slice of the 32 V rows and
//            accumulates the output columns of its slice only.
// No final combination is needed: each wave writes its own output columns.
// The arithmetic per element is the default kernel's except the order in
// which the score's partial sums are added, so results agree with it to
// fp32 rounding, not bit for bit.
#include "fused3s_kernel.h"

namespace f3s {
namespace {

template <int D> struct SplitRowWaves {
    static constexpr int value = (D / 32) % 4 == 0 ? 4 : 2;
};

template <int D, int NW>
__global__ __launch_bounds__(64 * NW) void k_fused3s_split_row(
    const WorkItem *__restrict__ items, const int32_t *__restrict__ cols,
    const uint32_t *__restrict__ mask, const int32_t *__restrict__ win_row,
    const _Float16 *__restrict__ Q, const _Float16 *__restrict__ K,
    const _Float16 *__restrict__ V, float *__restrict__ O, float *__restrict__ part_o,
    float *__restrict__ part_ml, float *__restrict__ lse, int32_t N, int32_t ld, int32_t h0,
    int32_t nh, float sl2, uint32_t order)
{
    constexpr int NC = D / 32;       // 32-deep chunks of the score reduction
    constexpr int NT = D / 16;       // 16-wide output tiles
    static_assert(NC % NW == 0 && NT % NW == 0, "waves must split the chunks evenly");
    constexpr int NCW = NC / NW;     // chunks of this wave's slice
    constexpr int NTW = NT / NW;     // output tiles of this wave's slice
    constexpr int DS = D / NW;       // features per wave
    constexpr int LPR = DS / 8;      // 16-byte chunks per row slice
    constexpr int NI = 32 * LPR / 64;  // chunks per lane per 32-row tile
    // Row strides of the wave's LDS tile: DS/2 + 4 dwords (4 x odd) for the
    // operand reads of K, DS/2 + 8 dwords (8 x odd) for the transposed
    // reads of V, as in the default kernel.
    constexpr int LSK = DS + 8;
    constexpr int LSV = DS + 16;
    __shared__ __attribute__((aligned(16))) _Float16 tiles[NW][32 * LSV];
    // partial scores of the pair (two blocks, 4 per lane), two buffers
    __shared__ f4 sx[2][NW][2][64];

    const int wv = (int)(threadIdx.x >> 6);
    const int lane = (int)(threadIdx.x & 63);
    _Float16 *const tile = tiles[wv];
    const int i = lane & 15;
    const int g = lane >> 4;
    const int wg = workgroup_position(order, nh);
    int item, hl;
    if (order & kOrderHead) {
        const int n_it = gridDim.x / nh;
        hl = wg / n_it;
        item = wg - hl * n_it;
    } else {
        item = wg / nh;
        hl = wg - item * nh;
    }
    const int head = h0 + hl;
    const WorkItem it = items[item];
    // this wave's feature slice of head `head`
    const int64_t fo = (int64_t)head * D + wv * DS;
    int32_t r0, nr;
    window_rows(win_row, N, it.window, &r0, &nr);
    const int row = r0 + i;
    const bool live = i < nr;
    const int b0 = it.blk_begin, b1 = it.blk_end;

    // Q_i slice: lane (i, g) holds Q[row][fo + 32c + 8g .. +7]
    h8 q[NCW];
    {
        const _Float16 *qp = Q + (int64_t)(live ? row : r0) * ld + fo + 8 * g;
#pragma unroll
        for (int c = 0; c < NCW; ++c) q[c] = load16(qp + 32 * c);
    }
    f4 o[NTW];
#pragma unroll
    for (int t = 0; t < NTW; ++t) o[t] = f4{0.f, 0.f, 0.f, 0.f};
    float m_run = -__builtin_inff();
    float l_run = 0.f;

    h8 kst[NI], vst[NI];
    uint32_t mwa = 0, mwb = 0;
    int ncol = 0;
    auto load_cols = [&](int b) {
        const int slot = lane & 31;
        const int blk = slot < 16 ? min(b, b1 - 1) : min(b + 1, b1 - 1);
        ncol = cols[(int64_t)kBlockCols * blk + (slot & 15)];
    };
    // Row slices of the pair's 32 K and V rows, spread flat over the lanes
    // (chunk f = lane + 64 j: row f / LPR, chunk f % LPR of the slice).  A
    // padding slot gathers a real column of its block (bitmap bit clear).
    auto load_pair = [&](int b) {
        const int f0 = __builtin_amdgcn_readlane(ncol, 0);
        const int f1 = __builtin_amdgcn_readlane(ncol, 16);
        const int c = ncol < 0 ? ((lane & 16) ? f1 : f0) : ncol;
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int f = lane + 64 * j;
            const int col = __shfl(c, f / LPR);
            const uint32_t off = (uint32_t)col * (uint32_t)(2 * ld) +
                                 (uint32_t)(2 * fo) + 16u * (f % LPR);
            kst[j] = load16_off(K, off);
            vst[j] = load16_off(V, off);
        }
        mwa = mask[(int64_t)kMaskWords * b + (lane >> 3)];
        mwb = mask[(int64_t)kMaskWords * min(b + 1, b1 - 1) + (lane >> 3)];
    };

    const int nib_shift = 4 * (lane & 7);
    int buf = 0;
    auto step = [&](int b, bool prefetch) {
        // ---- K row slices -> LDS, read back as MFMA A operands ----
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int f = lane + 64 * j;
            *reinterpret_cast<h8 *>(&tile[(f / LPR) * LSK + 8 * (f % LPR)]) = kst[j];
        }
        tile_fence<NW>();
        f4 s0 = f4{0.f, 0.f, 0.f, 0.f}, s1 = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NCW; ++c) {
            const _Float16 *kr = &tile[i * LSK + 32 * c + 8 * g];
            const h8 ka = *reinterpret_cast<const h8 *>(kr);
            const h8 kb = *reinterpret_cast<const h8 *>(kr + 16 * LSK);
            s0 = mfma16x16x32(ka, q[c], s0);
            s1 = mfma16x16x32(kb, q[c], s1);
        }
        // ---- this wave's partial scores -> LDS ----
        sx[buf][wv][0][lane] = s0;
        sx[buf][wv][1][lane] = s1;
        tile_fence<NW>();
        // ---- V row slices -> the same tile (stride LSV) ----
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int f = lane + 64 * j;
            *reinterpret_cast<h8 *>(&tile[(f / LPR) * LSV + 8 * (f % LPR)]) = vst[j];
        }
        const uint32_t nib0 = (mwa >> nib_shift) & 15u;
        const uint32_t nib1 = b + 1 < b1 ? (mwb >> nib_shift) & 15u : 0u;
        if (prefetch) {
            load_pair(b + 2);
            load_cols(b + 4);
        }
        // ---- the full scores: the NW partials, added in wave order (a
        //      workgroup barrier with LDS-only fences: the next pair's
        //      gathers stay in flight across it) ----
        wave_lds_fence();
        s0 = sx[buf][0][0][lane];
        s1 = sx[buf][0][1][lane];
#pragma unroll
        for (int w = 1; w < NW; ++w) {
            s0 += sx[buf][w][0][lane];
            s1 += sx[buf][w][1][lane];
        }
        buf ^= 1;
        // ---- mask + online softmax (base 2), as the default kernel ----
        float x[8];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            x[r] = masked_score(s0[r] * sl2, __builtin_amdgcn_sbfe((int)nib0, r, 1));
            x[4 + r] = masked_score(s1[r] * sl2, __builtin_amdgcn_sbfe((int)nib1, r, 1));
        }
        float mloc = x[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) mloc = fmaxf(mloc, x[e]);
        mloc = max_xor16(mloc);
        mloc = max_xor32(mloc);
        const float m_new = fmaxf(m_run, mloc);
        const float m_ref = m_new == -__builtin_inff() ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_ref);
        h8 p;
        float psum = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) p[e] = (_Float16)__builtin_amdgcn_exp2f(x[e] - m_ref);
        const h2 one = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
        for (int e = 0; e < 8; e += 2)
            psum = __builtin_amdgcn_fdot2(h2{p[e], p[e + 1]}, one, psum, false);
        l_run = l_run * alpha + psum;
        m_run = m_new;
#pragma unroll
        for (int t = 0; t < NTW; ++t) o[t] *= alpha;
        tile_fence<NW>();
        // ---- value product over this wave's output columns ----
        const _Float16 *ta = tile + (4 * g + (i >> 2)) * LSV + 4 * (i & 3);
        const _Float16 *tb = ta + 16 * LSV;
#pragma unroll
        for (int t = 0; t < NTW; ++t) {
            const h4 lo = lds_read_tr(ta + 16 * t);
            const h4 hi = lds_read_tr(tb + 16 * t);
            o[t] = mfma16x16x32(cat44(lo, hi), p, o[t]);
        }
        tile_fence<NW>();
    };

    // every wave walks the same pairs, so every wave meets every barrier
    if (b0 < b1) {
        load_cols(b0);
        load_pair(b0);
        load_cols(b0 + 2);
        int b = b0;
        for (; b + 2 < b1; b += 2) step(b, true);
        step(b, false);
    }

    float l_tot = l_run + __shfl_xor(l_run, 16);
    l_tot += __shfl_xor(l_tot, 32);
    if (it.slot < 0) {
        if (live) {
            const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
            float *op = O + (int64_t)row * ld + fo + 4 * g;
#pragma unroll
            for (int t = 0; t < NTW; ++t)
                *reinterpret_cast<f4 *>(op + 16 * t) = o[t] * inv;
            if (lse && wv == 0 && g == 0)
                lse[(int64_t)row * (ld / D) + head] =
                    l_tot > 0.f ? kLn2 * (m_run + __log2f(l_tot)) : -__builtin_inff();
        }
    } else {
        const int64_t ps = (int64_t)it.slot * nh + hl;
        float *op = part_o + ps * kWindowRows * D + i * D + wv * DS + 4 * g;
#pragma unroll
        for (int t = 0; t < NTW; ++t) *reinterpret_cast<f4 *>(op + 16 * t) = o[t];
        if (wv == 0 && g == 0) {
            part_ml[ps * 32 + i] = m_run;
            part_ml[ps * 32 + 16 + i] = l_tot;
        }
    }
}

template <int D>
hipError_t launch_split_row_d(const f3s_plan_s &p, const void *Q, const void *K,
                              const void *V, float *O, float *lse, int32_t H, float sl2,
                              hipStream_t s)
{
    constexpr int NW = SplitRowWaves<D>::value;
    const int32_t ld = H * D;
    if ((uint64_t)p.N * ld * 2 > 0xFFFFFFF0ull) return hipErrorInvalidValue;
    const int32_t group = p.n_split > 0 ? (kMaxD / D < H ? kMaxD / D : H) : H;
    for (int32_t h0 = 0; h0 < H; h0 += group) {
        const int32_t nh = H - h0 < group ? H - h0 : group;
        if (p.n_items > 0) {
            const uint64_t grid = (uint64_t)p.n_items * nh;
            if (grid > 0x7FFFFFFFull) return hipErrorInvalidConfiguration;
            const bool head_major = head_major_order(p, nh, 2ull * p.N * ld * 2);
            const uint32_t order = (head_major ? kOrderHead : 0u) |
                                   (xcd_chunks(p, nh, head_major) ? kOrderXcd : 0u);
            k_fused3s_split_row<D, NW><<<(unsigned)grid, 64 * NW, 0, s>>>(
                p.items, p.cols, p.mask, p.win_row, static_cast<const _Float16 *>(Q),
                static_cast<const _Float16 *>(K), static_cast<const _Float16 *>(V), O,
                p.part_o, p.part_ml, lse, p.N, ld, h0, nh, sl2, order);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        if (p.n_split > 0) {
            k_merge<D, false><<<p.n_split * nh, 256, 0, s>>>(p.merges, p.win_row, p.part_o,
                                                            p.part_ml, O, lse, p.N, ld, h0,
                                                            nh);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
    }
    return hipSuccess;
}

}  // namespace

hipError_t launch_fused_split_row(const f3s_plan_s &p, const void *Q, const void *K,
                                  const void *V, float *O, float *lse, int32_t H, int32_t d,
                                  float sl2, hipStream_t s)
{
    switch (d) {
    case 64: return launch_split_row_d<64>(p, Q, K, V, O, lse, H, sl2, s);
    case 128: return launch_split_row_d<128>(p, Q, K, V, O, lse, H, sl2, s);
    case 192: return launch_split_row_d<192>(p, Q, K, V, O, lse, H, sl2, s);
    case 256: return launch_split_row_d<256>(p, Q, K, V, O, lse, H, sl2, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace f3s
