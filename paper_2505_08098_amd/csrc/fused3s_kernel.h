// Fused 3S kernel for CDNA4 (gfx950): Algorithm 1 of Fused3S with the
// tensor-core tiling re-derived for 64-wide wavefronts and the 16x16x32
// matrix instructions.  Included by one source file per input storage type
// (fused3s.hip: fp16, fused3s_bf16.hip: bfloat16, fused3s_fp8.hip: fp8
// e4m3), each instantiating the
// templates for every feature size.
//
// One wavefront owns one work item (a 16-row window, or a piece of one) and
// walks its 16x16 blocks two at a time (32 compacted columns = the K depth of
// one MFMA for the value product).  Per block pair:
//
//   scores   S^T = K_hat * Q_i^T     (A = gathered K rows, read from LDS in
//                                     the operand layout; B = the window's
//                                     Q rows, in VGPRs for the whole item)
//            With S^T as the product, MFMA's accumulator layout gives every
//            lane ONE query row (lane % 16) and 4 neighbours per block, so
//            the row softmax needs only a 4-lane reduction and the
//            probabilities already sit in the B-operand layout of the next
//            product: no shuffle of P at all.
//   mask     bitmap bit clear -> score -inf (the bitmap mask of Algorithm 1)
//   softmax  online, base 2, fp32 (Section 3.5): running max m, running
//            lane-partial sum l, rescale factor alpha = 2^(m_old - m_new)
//            applied every pair (a branch around a rarely needed rescale
//            measured slower: it splits the loop body for the scheduler)
//   P        fp16 inputs: fp32 -> fp16 with round-to-nearest-even (Table 5's
//            scheme); the SAME rounded values are summed into l, so the
//            effective probabilities of a row sum to one.
//            bf16 inputs: P = P_hi + P_lo, two bfloat16 terms (hi = RNE of
//            P, lo = RNE of the exact remainder), ~16 significant bits; the
//            value product runs once per term.  A single bf16 P (8 bits)
//            would exceed the error budget of the fp16 scheme.
//   values   O_i^T += V_hat^T * P^T  (A = gathered V rows staged row-major in
//            LDS and read transposed; B = P from registers; the accumulator
//            lane layout again has lane % 16 = query row, so the alpha
//            rescale is a per-lane multiply)
//
// The gather order within a row (the reduction index of the score product)
// is permuted so each lane reads 16 contiguous bytes per load and the four
// lanes of a row cover 64 contiguous bytes: any consistent permutation of the
// reduction index leaves Q K^T unchanged (the register remapping of
// Section 3.4).  The loads of the next block pair are issued before the
// softmax and value product of the current pair (one pair in flight).
// K and V rows are gathered with row-contiguous lanes and staged through
// LDS (see the pipeline comment in the kernel).
//
// Scores and probabilities never leave registers; only O (fp32 or fp16) and,
// for split windows, the fp32 (m, l, unnormalised O) partials are written.
#pragma once

#include "kernel_common.h"

namespace f3s {
namespace {

constexpr float kLn2 = 0.6931471805599453f;

// Occupancy target (waves per SIMD) per feature size: the most waves whose
// registers fit without spilling; more resident waves = more gathers in
// flight, which is what bounds this kernel.
template <int D> struct WavesPerSimd { static constexpr int value = 1; };
template <> struct WavesPerSimd<32> { static constexpr int value = 6; };
template <> struct WavesPerSimd<64> { static constexpr int value = 4; };
template <> struct WavesPerSimd<96> { static constexpr int value = 3; };
template <> struct WavesPerSimd<128> { static constexpr int value = 2; };
template <> struct WavesPerSimd<160> { static constexpr int value = 2; };
// The bf16 variant holds the second probability term: one wave less at
// d = 32.  The narrow-gather ablation holds an address per 4-byte word: one
// wave less where it would otherwise spill (d = 64, 96, 160).
template <int D, int kIn, bool kNarrow = false>
constexpr int waves_per_simd()
{
    return WavesPerSimd<D>::value - (kIn == kInBF16 && D == 32 ? 1 : 0) -
           (kNarrow && (D == 64 || D == 96 || D == 160) ? 1 : 0);
}
// Score product for the input storage type (16-bit operands as raw bits).
template <int kIn>
__device__ __forceinline__ f4 mma_in(h8 a, h8 b, f4 c)
{
    if constexpr (kIn == kInBF16)
        return mfma16x16x32_bf16(a, b, c);
    else
        return mfma16x16x32(a, b, c);
}

// Bytes per stored element of Q, K, V.
template <int kIn> constexpr int elem_bytes() { return kIn == kInFP8 ? 1 : 2; }

// 16 stored bytes (8 fp16/bf16 elements, or 16 fp8 e4m3 elements) -> the
// compute type: unchanged for 16-bit storage; for fp8 the two fp16 halves
// (e4m3 -> fp16 is exact).
__device__ __forceinline__ void widen_fp8x16(h8 raw, h8 &lo, h8 &hi)
{
    typedef uint32_t u4 __attribute__((ext_vector_type(4)));
    const u4 w = __builtin_bit_cast(u4, raw);
    h8 out[2];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const h2 a = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w[k], 1.0f, false);
        const h2 b = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w[k], 1.0f, true);
        out[k >> 1][4 * (k & 1) + 0] = a[0];
        out[k >> 1][4 * (k & 1) + 1] = a[1];
        out[k >> 1][4 * (k & 1) + 2] = b[0];
        out[k >> 1][4 * (k & 1) + 3] = b[1];
    }
    lo = out[0];
    hi = out[1];
}

// 8 stored fp8 bytes -> 8 fp16.
__device__ __forceinline__ h8 widen_fp8x8(uint64_t raw)
{
    h8 r;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const uint32_t w = (uint32_t)(raw >> (32 * k));
        const h2 a = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 1.0f, false);
        const h2 b = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 1.0f, true);
        r[4 * k + 0] = a[0];
        r[4 * k + 1] = a[1];
        r[4 * k + 2] = b[0];
        r[4 * k + 3] = b[1];
    }
    return r;
}

// Narrow-gather staging: word cc of `w` is word (m & 3) of chunk
// (m & ~3) + cc of the row starting at `row`.
__device__ __forceinline__ void stage_words(_Float16 *row, int m, h8 w)
{
    typedef uint32_t u4v __attribute__((ext_vector_type(4)));
    const u4v words = __builtin_bit_cast(u4v, w);
    const int m0 = m & ~3, qd = m & 3;
#pragma unroll
    for (int cc = 0; cc < 4; ++cc)
        *reinterpret_cast<uint32_t *>(row + 8 * (m0 + cc) + 2 * qd) = words[cc];
}

// v where sel is all ones, -inf where sel is zero (one bit-select).
__device__ __forceinline__ float masked_score(float v, int sel)
{
    const uint32_t ninf = 0xff800000u;
    return __builtin_bit_cast(float, (__builtin_bit_cast(uint32_t, v) & (uint32_t)sel) |
                                         (ninf & ~(uint32_t)sel));
}

// Four fp32 results -> the output type at p (16-byte or 8-byte store).
template <bool kOutH>
__device__ __forceinline__ void store4(void *base, int64_t idx, f4 v)
{
    if constexpr (kOutH) {
        h4 h;
#pragma unroll
        for (int e = 0; e < 4; ++e) h[e] = (_Float16)v[e];
        *reinterpret_cast<h4 *>(static_cast<_Float16 *>(base) + idx) = h;
    } else {
        *reinterpret_cast<f4 *>(static_cast<float *>(base) + idx) = v;
    }
}

// kIn: storage type of Q, K, V (kInF16, kInBF16: 16-bit raw bits; kInFP8:
// e4m3 bytes, widened to fp16 on the way into registers / LDS, so the
// products are the fp16 ones).  kOutH: O is fp16 instead of fp32.  kWide:
// Q/K/V may exceed 4 GiB, so gathers use 64-bit addresses.  kNarrow (an
// ablation of the coalescing layout, fp16 inputs only): K and V are
// gathered in 4-byte words -- consecutive lanes of a quad read consecutive
// words of a row, each lane taking one word of each of the quad's four
// 16-byte chunks -- instead of one 16-byte chunk per lane, i.e. the access
// granularity without the register remapping of Section 3.4.  NW: waves
// per workgroup sharing one work item -- each takes a contiguous share of
// its block pairs, and the (m, l, O) partials are combined through LDS at
// the end (the paper's split-column partition of a window among warps; used
// for long windows, where one wave per window leaves the GPU with too few
// waves).  kTrace (a measurement instance): the first thread of each
// workgroup also records, after its outputs, when the workgroup started and
// ended (the 100 MHz constant clock) and on which compute unit it ran, as
// one 32-byte record per workgroup in `trace` (ordinary vector stores).
template <int D, bool kWide, int kIn, bool kOutH, bool kNarrow = false, int NW = 1,
          bool kTrace = false>
__global__ __launch_bounds__(64 * NW)
__attribute__((amdgpu_waves_per_eu(waves_per_simd<D, kIn, kNarrow>(), 8))) void k_fused3s(
    const WorkItem *__restrict__ items, const int32_t *__restrict__ cols,
    const uint32_t *__restrict__ mask, const int32_t *__restrict__ win_row,
    const void *__restrict__ Qv, const void *__restrict__ Kv, const void *__restrict__ Vv,
    void *__restrict__ O, float *__restrict__ part_o,
    float *__restrict__ part_ml, float *__restrict__ lse, int32_t N, int32_t ld,
    int32_t h0, int32_t nh, float sl2, uint32_t order, uint32_t *__restrict__ trace)
{
    uint64_t t_start = 0;
    if constexpr (kTrace) t_start = wall_clock64();
    constexpr int NC = D / 32;  // 32-deep chunks of the score reduction
    constexpr int NT = D / 16;  // 16-wide output tiles of the value product
    // One LDS tile per wave, used twice per block pair with two row strides
    // (halves).  K phase: D/2 + 4 dwords = 4 x odd, so the 16 rows read by a
    // 16-lane pass start in 16 disjoint 4-bank ranges.  V phase: D/2 + 8
    // dwords = 8 x odd, so the 8 rows of a transposed read start in disjoint
    // 8-bank ranges.
    constexpr int LSK = D + 8;
    constexpr int LSV = D + 16;
    __shared__ __attribute__((aligned(16))) _Float16 tiles[NW][32 * LSV];
    const int wv = NW > 1 ? (int)(threadIdx.x >> 6) : 0;
    _Float16 *const tile = tiles[wv];

    const int lane = NW > 1 ? (int)(threadIdx.x & 63) : (int)threadIdx.x;
    const int i = lane & 15;  // query row (accumulators) / operand row index
    const int g = lane >> 4;  // lane group: selects the reduction slots
    // Workgroups walk the work list item-major (the heads of one window back
    // to back: they share its column lists and bitmaps, and the lines of its
    // K and V rows while those stay cached) or head-major (one pass over the
    // list per head: with K and V far larger than the caches each head's
    // gathers then stream like a single head's).
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
    // Row r of head h starts at r * ld + h * D (elements) in Q, K, V and O.
    constexpr int EB = elem_bytes<kIn>();
    const char *Q = static_cast<const char *>(Qv) + (int64_t)head * D * EB;
    const char *K = static_cast<const char *>(Kv) + (int64_t)head * D * EB;
    const char *V = static_cast<const char *>(Vv) + (int64_t)head * D * EB;
    const int64_t ohead = (int64_t)head * D;
    // the window's rows: 16 from 16 w (the last window clipped at N), or
    // those of a plan aligned to the graphs of a batch
    int32_t r0, nr;
    window_rows(win_row, N, it.window, &r0, &nr);
    const int row = r0 + i;
    const bool live = i < nr;
    // this wave's blocks: whole pairs [pa, pb) of the item's pairs
    int b0 = it.blk_begin, b1 = it.blk_end;
    if constexpr (NW > 1) {
        const int pairs = (b1 - b0 + 1) >> 1;
        const int pa = pairs * wv / NW, pb = pairs * (wv + 1) / NW;
        b1 = min(b1, b0 + 2 * pb);
        b0 = b0 + 2 * pa;
    }

    // Q_i: lane (i, g) holds Q[row][32c + 8g .. +7] for each chunk c.  Pad
    // rows (past the window's last row) read its first row: their results
    // are never written and rows do not interact, so any finite values do.
    h8 q[NC];
    {
        const char *qp = Q + ((int64_t)(live ? row : r0) * ld + 8 * g) * EB;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            if constexpr (EB == 1)
                q[c] = widen_fp8x8(*reinterpret_cast<const uint64_t *>(qp + 32 * c));
            else
                q[c] = *reinterpret_cast<const h8 *>(qp + 64 * c);
        }
    }

    f4 o[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) o[t] = f4{0.f, 0.f, 0.f, 0.f};
    float m_run = -__builtin_inff();
    float l_run = 0.f;

    // Pipeline state.  The 32 K rows and 32 V rows of a block pair are
    // gathered "row-contiguous": the pair tile's 16-byte chunks are spread
    // flat over the lanes (chunk f = lane + 64 j, row f / LPR, chunk f % LPR),
    // so every 4-lane quad reads 64 contiguous bytes of ONE row; the texture
    // addresser then spends one cycle per quad instead of four (an MFMA
    // operand layout puts consecutive lanes on different rows).  The rows go
    // through LDS: K rows are read back in the MFMA A layout, V rows with
    // the transposed read.  Loads are unconditional: a padding slot (column
    // -1) or the absent second block of an odd tail gathers a real column of
    // the same block, whose bitmap bit is clear, so its probability is
    // exactly 0 and it adds 0 * (finite V) = 0.
    constexpr int LPR = D * EB / 16;  // lanes (16-byte chunks) per row
    constexpr int NI = D * EB / 32;   // chunks per lane per tile
    constexpr int CE = 16 / EB;       // elements per chunk
    h8 kst[NI], vst[NI];              // staged K and V chunks of the pair in flight
    uint32_t mwa = 0, mwb = 0;
    int ncol = 0;                // lanes 0..31: raw column of slot `lane` of the next pair

    // Raw column ids of pair (b, b+1): lane l (mod 32) takes slot l; block
    // indices clamped so reads stay inside this item (values past its end
    // are never used).
    auto load_cols = [&](int b) {
        const int slot = lane & 31;
        const int blk = slot < 16 ? min(b, b1 - 1) : min(b + 1, b1 - 1);
        ncol = cols[(int64_t)kBlockCols * blk + (slot & 15)];
    };
    // Issue the K, V and bitmap loads of pair (b, b+1).  Slots 0 and 16 are
    // never padding (the first slot of a block); the wave is fully active
    // here, so readlane sees them.
    auto load_pair = [&](int b) {
        const int f0 = __builtin_amdgcn_readlane(ncol, 0);
        const int f1 = __builtin_amdgcn_readlane(ncol, 16);
        const int c = ncol < 0 ? ((lane & 16) ? f1 : f0) : ncol;
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int f = lane + 64 * j;
            const int col = __shfl(c, f / LPR);
            if constexpr (kNarrow) {
                // word qd of chunks m0 .. m0+3 (the quad's chunks: LPR is a
                // multiple of 4, so the quad lies in one row)
                static_assert(EB == 2, "narrow gathers are defined for 16-bit inputs");
                typedef uint32_t u4v __attribute__((ext_vector_type(4)));
                const int m = f % LPR, m0 = m & ~3, qd = m & 3;
                u4v wk, wv;
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) {
                    if constexpr (kWide) {
                        const int64_t off = (int64_t)col * ld * EB + 16 * (m0 + cc) + 4 * qd;
                        wk[cc] = *reinterpret_cast<const uint32_t *>(K + off);
                        wv[cc] = *reinterpret_cast<const uint32_t *>(V + off);
                    } else {
                        const uint32_t off = (uint32_t)col * (uint32_t)(EB * ld) +
                                             16u * (m0 + cc) + 4u * qd;
                        wk[cc] = *reinterpret_cast<const uint32_t *>(K + off);
                        wv[cc] = *reinterpret_cast<const uint32_t *>(V + off);
                    }
                }
                kst[j] = __builtin_bit_cast(h8, wk);
                vst[j] = __builtin_bit_cast(h8, wv);
            } else if constexpr (kWide) {
                const int64_t off = (int64_t)col * ld * EB + 16 * (f % LPR);
                kst[j] = *reinterpret_cast<const h8 *>(K + off);
                vst[j] = *reinterpret_cast<const h8 *>(V + off);
            } else {
                // byte offset < 2^32 (checked on the host): the load takes
                // the uniform base from SGPRs and a 32-bit VGPR offset
                const uint32_t off = (uint32_t)col * (uint32_t)(EB * ld) + 16u * (f % LPR);
                kst[j] = load16_off(reinterpret_cast<const _Float16 *>(K), off);
                vst[j] = load16_off(reinterpret_cast<const _Float16 *>(V), off);
            }
        }
        mwa = mask[(int64_t)kMaskWords * b + (lane >> 3)];
        mwb = mask[(int64_t)kMaskWords * min(b + 1, b1 - 1) + (lane >> 3)];
    };

    const int nib_shift = 4 * (lane & 7);
    // One block pair: scores, mask, online softmax, value product.  With
    // `prefetch`, the loads of the pair after it are issued as soon as this
    // pair's staging registers are in LDS.
    auto step = [&](int b, bool prefetch) {
        // ---- K rows -> LDS (stride LSK), read back as MFMA A operands ----
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int f = lane + 64 * j;
            _Float16 *dst = &tile[(f / LPR) * LSK + CE * (f % LPR)];
            if constexpr (kNarrow) {
                stage_words(&tile[(f / LPR) * LSK], f % LPR, kst[j]);
            } else if constexpr (EB == 1) {
                h8 lo, hi;
                widen_fp8x16(kst[j], lo, hi);
                *reinterpret_cast<h8 *>(dst) = lo;
                *reinterpret_cast<h8 *>(dst + 8) = hi;
            } else {
                *reinterpret_cast<h8 *>(dst) = kst[j];
            }
        }
        tile_fence<NW>();
        h8 ka[NC], kb[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            ka[c] = *reinterpret_cast<const h8 *>(&tile[i * LSK + 32 * c + 8 * g]);
            kb[c] = *reinterpret_cast<const h8 *>(&tile[(16 + i) * LSK + 32 * c + 8 * g]);
        }
        // ---- scores of the two blocks (S^T: lane = row i, nbrs 4g+r) ----
        f4 s0 = f4{0.f, 0.f, 0.f, 0.f}, s1 = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            s0 = mma_in<kIn>(ka[c], q[c], s0);
            s1 = mma_in<kIn>(kb[c], q[c], s1);
        }
        tile_fence<NW>();
        // ---- V rows -> the same LDS tile (stride LSV, slot = neighbour) ----
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int f = lane + 64 * j;
            _Float16 *dst = &tile[(f / LPR) * LSV + CE * (f % LPR)];
            if constexpr (kNarrow) {
                stage_words(&tile[(f / LPR) * LSV], f % LPR, vst[j]);
            } else if constexpr (EB == 1) {
                h8 lo, hi;
                widen_fp8x16(vst[j], lo, hi);
                *reinterpret_cast<h8 *>(dst) = lo;
                *reinterpret_cast<h8 *>(dst + 8) = hi;
            } else {
                *reinterpret_cast<h8 *>(dst) = vst[j];
            }
        }
        const uint32_t nib0 = (mwa >> nib_shift) & 15u;
        // (an odd tail's absent second block re-read block b: mask it off)
        const uint32_t nib1 = b + 1 < b1 ? (mwb >> nib_shift) & 15u : 0u;
        // ---- issue the next pair's loads (staging registers are free) ----
        if (prefetch) {
            load_pair(b + 2);
            load_cols(b + 4);
        }
        // ---- mask + online softmax (base 2) ----
        // bit r of the nibble -> all-ones / zero word (signed bit-field
        // extract), then a bit-select between the score and -inf
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
        h8 p, plo;
        float psum = 0.f;
        if constexpr (kIn == kInBF16) {
            // P = hi + lo, both bfloat16; hi + lo is exact in fp32
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float pf = __builtin_amdgcn_exp2f(x[e] - m_ref);
                const __bf16 hb = (__bf16)pf;
                const float hf = (float)hb;
                const __bf16 lb = (__bf16)(pf - hf);
                p[e] = __builtin_bit_cast(_Float16, hb);
                plo[e] = __builtin_bit_cast(_Float16, lb);
                psum += hf + (float)lb;
            }
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                p[e] = (_Float16)__builtin_amdgcn_exp2f(x[e] - m_ref);
            // the sum of the rounded values, two at a time (dot with 1, 1)
            const h2 one = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
            for (int e = 0; e < 8; e += 2)
                psum = __builtin_amdgcn_fdot2(h2{p[e], p[e + 1]}, one, psum, false);
        }
        l_run = l_run * alpha + psum;
        m_run = m_new;
#pragma unroll
        for (int t = 0; t < NT; ++t) o[t] *= alpha;
        tile_fence<NW>();
        // ---- value product: A[m][slot] = V_hat[slot][16t + m] ----
        // slot order of lane group g: 4g..4g+3 (block 0), 16+4g..+3 (block 1)
        // -- the neighbours this lane's P values belong to.  Group lane s
        // addresses row 4g + s/4, columns 16t + 4(s%4).., so the transposed
        // read hands lane (m = i, g) the column 16t + m of rows 4g..4g+3.
        const _Float16 *ta = tile + (4 * g + (i >> 2)) * LSV + 4 * (i & 3);
        const _Float16 *tb = ta + 16 * LSV;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const h4 lo = lds_read_tr(ta + 16 * t);
            const h4 hi = lds_read_tr(tb + 16 * t);
            const h8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
            if constexpr (kIn == kInBF16) {
                o[t] = mfma16x16x32_bf16(a, p, o[t]);
                o[t] = mfma16x16x32_bf16(a, plo, o[t]);
            } else {
                o[t] = mfma16x16x32(a, p, o[t]);
            }
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

    // ---- finalise: full row sums, normalise, write (Algorithm 1 end) ----
    float l_tot = l_run + __shfl_xor(l_run, 16);
    l_tot += __shfl_xor(l_tot, 32);
    if constexpr (NW > 1) {
        // the waves' partial states: O (lane (i, g) holds columns 16t + 4g ..
        // +3 of row i) into the wave's own tile, which 16 x D floats fit and
        // no longer serves; then wave 0 combines them as the online softmax
        // combines blocks (a wave without blocks has m = -inf, l = 0, O = 0)
        __shared__ float s_m[NW][kWindowRows], s_l[NW][kWindowRows];
        float *ot = reinterpret_cast<float *>(tile);
#pragma unroll
        for (int t = 0; t < NT; ++t)
            *reinterpret_cast<f4 *>(ot + i * D + 16 * t + 4 * g) = o[t];
        if (g == 0) {
            s_m[wv][i] = m_run;
            s_l[wv][i] = l_tot;
        }
        __syncthreads();
        if (wv != 0) return;
        float m = -__builtin_inff();
#pragma unroll
        for (int w = 0; w < NW; ++w) m = fmaxf(m, s_m[w][i]);
        const float m_ref = m == -__builtin_inff() ? 0.f : m;
        float l = 0.f;
#pragma unroll
        for (int t = 0; t < NT; ++t) o[t] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            const float a = __builtin_amdgcn_exp2f(s_m[w][i] - m_ref);
            l += a * s_l[w][i];
            const float *ow = reinterpret_cast<const float *>(tiles[w]) + i * D + 4 * g;
#pragma unroll
            for (int t = 0; t < NT; ++t) o[t] += a * *reinterpret_cast<const f4 *>(ow + 16 * t);
        }
        m_run = m;
        l_tot = l;
    }
    if (it.slot < 0) {
        if (live) {
            const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
            const int64_t ob = (int64_t)row * ld + ohead + 4 * g;
#pragma unroll
            for (int t = 0; t < NT; ++t) store4<kOutH>(O, ob + 16 * t, o[t] * inv);
            // natural-log log-sum-exp of the row's scaled scores
            if (lse && g == 0)
                lse[(int64_t)row * (ld / D) + head] =
                    l_tot > 0.f ? kLn2 * (m_run + __log2f(l_tot)) : -__builtin_inff();
        }
    } else {
        // partial slot of (piece, head): slot * nh + head offset
        const int64_t ps = (int64_t)it.slot * nh + hl;
        float *op = part_o + ps * kWindowRows * D + i * D + 4 * g;
#pragma unroll
        for (int t = 0; t < NT; ++t) *reinterpret_cast<f4 *>(op + 16 * t) = o[t];
        if (g == 0) {
            part_ml[ps * 32 + i] = m_run;
            part_ml[ps * 32 + 16 + i] = l_tot;
        }
    }
    if constexpr (kTrace) {
        if (threadIdx.x == 0) {
            const uint64_t t_end = wall_clock64();
            // HW_ID (compute unit, shader array and engine of this wave) and
            // XCC_ID (which of the accelerator complex dies): s_getreg of
            // hardware registers 4 and 20, all 32 / the low 16 bits
            const uint32_t hw = __builtin_amdgcn_s_getreg((31 << 11) | 4);
            const uint32_t xcc = __builtin_amdgcn_s_getreg((15 << 11) | 20);
            typedef uint32_t u4t __attribute__((ext_vector_type(4)));
            u4t *rec = reinterpret_cast<u4t *>(trace + 8 * (int64_t)blockIdx.x);
            rec[0] = u4t{(uint32_t)t_start, (uint32_t)(t_start >> 32), (uint32_t)t_end,
                         (uint32_t)(t_end >> 32)};
            rec[1] = u4t{hw, xcc, (uint32_t)blockIdx.x, 0u};
        }
    }
}

// Combines the pieces of one split window in their fixed order (so the
// result is deterministic), in one online pass: with (m, l, acc) the merged
// state so far and (m_k, l_k, O_k) piece k,
//   m' = max(m, m_k),  l = 2^(m - m') l + 2^(m_k - m') l_k,
//   acc = 2^(m - m') acc + 2^(m_k - m') O_k,
// and O = acc / l at the end -- the same combination as the online softmax
// across blocks.  16 threads per row, float4 columns; the loads of kU pieces
// are issued together (independent addresses), so a window of np pieces
// costs about np / kU memory round trips.  Thread q of a row handles the
// float4 columns 4q + 64c (c < CPT) that lie inside the row.
template <int D, bool kOutH>
__global__ __launch_bounds__(256) void k_merge(const int32_t *__restrict__ merges,
                                               const int32_t *__restrict__ win_row,
                                               const float *__restrict__ part_o,
                                               const float *__restrict__ part_ml,
                                               void *__restrict__ O,
                                               float *__restrict__ lse, int32_t N,
                                               int32_t ld, int32_t h0, int32_t nh)
{
    constexpr int kU = 8;
    constexpr int CPT = (D + 63) / 64;   // float4 columns per thread (4q + 64c)
    const int s = blockIdx.x / nh, hl = blockIdx.x - (blockIdx.x / nh) * nh;
    const int w = merges[3 * s], first = merges[3 * s + 1], np = merges[3 * s + 2];
    const int r = threadIdx.x >> 4, q = threadIdx.x & 15;
    int32_t r0, nr;
    window_rows(win_row, N, w, &r0, &nr);
    if (r >= nr) return;
    const int row = r0 + r;
    // partial slot of (piece k, head) = (first + k) * nh + hl
    const float *ml = part_ml + ((int64_t)first * nh + hl) * 32;
    const int64_t mstride = (int64_t)nh * 32;
    const float *po = part_o + ((int64_t)first * nh + hl) * kWindowRows * D + r * D;
    const int64_t ostride = (int64_t)nh * kWindowRows * D;
    float m = -__builtin_inff(), l = 0.f;
    f4 acc[CPT];
#pragma unroll
    for (int c = 0; c < CPT; ++c) acc[c] = f4{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < np; k0 += kU) {
        float mk[kU], lk[kU];
        f4 ok[kU][CPT];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            // indices past the last piece re-read it (in bounds) and weigh 0
            const int k = min(k0 + u, np - 1);
            mk[u] = k0 + u < np ? ml[k * mstride + r] : -__builtin_inff();
            lk[u] = ml[k * mstride + 16 + r];
#pragma unroll
            for (int c = 0; c < CPT; ++c)
                ok[u][c] = 4 * q + 64 * c < D
                               ? *reinterpret_cast<const f4 *>(po + k * ostride + 4 * q + 64 * c)
                               : f4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const float m_new = fmaxf(m, mk[u]);
            const float m_ref = m_new == -__builtin_inff() ? 0.f : m_new;
            const float a = __builtin_amdgcn_exp2f(m - m_ref);
            const float b = __builtin_amdgcn_exp2f(mk[u] - m_ref);
            l = l * a + lk[u] * b;
#pragma unroll
            for (int c = 0; c < CPT; ++c) acc[c] = acc[c] * a + ok[u][c] * b;
            m = m_new;
        }
    }
    const float inv = l > 0.f ? 1.f / l : 0.f;
    if (lse && q == 0)
        lse[(int64_t)row * (ld / D) + h0 + hl] =
            l > 0.f ? kLn2 * (m + __log2f(l)) : -__builtin_inff();
    const int64_t orow = (int64_t)row * ld + (int64_t)(h0 + hl) * D;
#pragma unroll
    for (int c = 0; c < CPT; ++c)
        if (4 * q + 64 * c < D) store4<kOutH>(O, orow + 4 * q + 64 * c, acc[c] * inv);
}

// Heads are launched in groups whose partial results fit the plan's scratch
// (nh * D <= 256 floats per piece row); without split windows all heads go
// in one launch.
// trace (the measurement instance, fp16 -> fp32 with 32-bit addressing and
// one head only): one 32-byte record per workgroup.
template <int D, int kIn, bool kOutH, bool kNarrow = false>
hipError_t launch_d(const f3s_plan_s &p, const void *Q, const void *K,
                    const void *V, void *O, float *lse, int32_t H, float sl2,
                    hipStream_t s, uint32_t *trace = nullptr)
{
    const int32_t ld = H * D;
    const bool wide = (uint64_t)p.N * ld * elem_bytes<kIn>() > 0xFFFFFFF0ull;
    // the narrow-gather ablation keeps one wave per item
    const int nw =
        kNarrow ? 1
                : waves_per_item(p.n_blocks, p.n_items, H,
                                 (int64_t)waves_per_simd<D, kIn, kNarrow>() * 1024);
    constexpr int W2 = kNarrow ? 1 : 2, W4 = kNarrow ? 1 : 4;
    auto kern = nw == 4   ? (wide ? k_fused3s<D, true, kIn, kOutH, kNarrow, W4>
                                  : k_fused3s<D, false, kIn, kOutH, kNarrow, W4>)
                : nw == 2 ? (wide ? k_fused3s<D, true, kIn, kOutH, kNarrow, W2>
                                  : k_fused3s<D, false, kIn, kOutH, kNarrow, W2>)
                          : (wide ? k_fused3s<D, true, kIn, kOutH, kNarrow>
                                  : k_fused3s<D, false, kIn, kOutH, kNarrow>);
    if (trace) {
        if constexpr (kIn == kInF16 && !kOutH && !kNarrow) {
            if (wide || H != 1) return hipErrorInvalidValue;
            kern = nw == 4   ? k_fused3s<D, false, kIn, kOutH, false, 4, true>
                   : nw == 2 ? k_fused3s<D, false, kIn, kOutH, false, 2, true>
                             : k_fused3s<D, false, kIn, kOutH, false, 1, true>;
        } else {
            return hipErrorInvalidValue;
        }
    }
    const int32_t group = p.n_split > 0 ? (kMaxD / D < H ? kMaxD / D : H) : H;
    for (int32_t h0 = 0; h0 < H; h0 += group) {
        const int32_t nh = H - h0 < group ? H - h0 : group;
        // the plan's partial buffers hold n_pieces * kMaxD / D head slots
        if (p.n_split > 0 && (int64_t)nh * D > kMaxD) return hipErrorInvalidValue;
        if (p.n_items > 0) {
            const uint64_t grid = (uint64_t)p.n_items * nh;
            if (grid > 0x7FFFFFFFull) return hipErrorInvalidConfiguration;
            const bool head_major =
                head_major_order(p, nh, 2ull * p.N * ld * elem_bytes<kIn>());
            const uint32_t order = (head_major ? kOrderHead : 0u) |
                                   (xcd_chunks(p, nh, head_major) ? kOrderXcd : 0u);
            kern<<<(unsigned)grid, 64 * nw, 0, s>>>(p.items, p.cols, p.mask, p.win_row, Q, K,
                                               V, O, p.part_o, p.part_ml, lse, p.N, ld, h0,
                                               nh, sl2, order, trace);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        if (p.n_split > 0) {
            k_merge<D, kOutH><<<p.n_split * nh, 256, 0, s>>>(p.merges, p.win_row, p.part_o,
                                                            p.part_ml, O, lse, p.N, ld, h0,
                                                            nh);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
    }
    return hipSuccess;
}

// Dispatch over the feature size for one input storage type.
template <int kIn, bool kOutH, bool kNarrow = false>
hipError_t launch_in(const f3s_plan_s &p, const void *Q, const void *K, const void *V,
                     void *O, float *lse, int32_t H, int32_t d, float sl2, hipStream_t s,
                     uint32_t *trace = nullptr)
{
    switch (d) {
    case 32: return launch_d<32, kIn, kOutH, kNarrow>(p, Q, K, V, O, lse, H, sl2, s, trace);
    case 64: return launch_d<64, kIn, kOutH, kNarrow>(p, Q, K, V, O, lse, H, sl2, s, trace);
    case 96: return launch_d<96, kIn, kOutH, kNarrow>(p, Q, K, V, O, lse, H, sl2, s, trace);
    case 128: return launch_d<128, kIn, kOutH, kNarrow>(p, Q, K, V, O, lse, H, sl2, s, trace);
    case 160: return launch_d<160, kIn, kOutH, kNarrow>(p, Q, K, V, O, lse, H, sl2, s, trace);
    case 192: return launch_d<192, kIn, kOutH, kNarrow>(p, Q, K, V, O, lse, H, sl2, s, trace);
    case 224: return launch_d<224, kIn, kOutH, kNarrow>(p, Q, K, V, O, lse, H, sl2, s, trace);
    case 256: return launch_d<256, kIn, kOutH, kNarrow>(p, Q, K, V, O, lse, H, sl2, s, trace);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace
}  // namespace f3s
