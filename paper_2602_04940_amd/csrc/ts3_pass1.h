// Pass 1 of the Physics-Attention layer: slice logits, per-head temperature
// softmax and the tile contraction s_raw += w^T x, d += sum_i w_i (paper
// Eq. (1) and Eq. (4), Algorithm 1 tile loop).  The slice weights exist only in
// registers.
//
// Work decomposition: one workgroup per (span, head).  A span is Q consecutive
// mesh points; its four waves take 32-point blocks round-robin, each keeping a
// private M x C float32 accumulator of its head in registers (so head h's
// logits, softmax and contraction never leave the wave).  At the end the four
// wave accumulators are summed in a fixed order and written as the span's
// partial [M][C+1] (column C holds d).  Spans are folded in index order later,
// so the result is a fixed function of (x, Q) whatever the tiling.
//
// Per 32-point block and wave:
//   logits  L[p][m] = x[p][:] . W2'[:, h*M+m] + b2'   16x16x32 MFMA, A = x rows,
//           B = W2' fragments held in registers; W2' = W2 * log2(e)/tau so the
//           softmax uses exp2.  Output lane (g, m) holds points 4g+r of a 16-point tile.
//   softmax over the M slices of each point: in-lane over m-tiles, then a
//           16-lane DPP reduction (max and sum); w = exp2(L - max) / sum.
//   contraction S[m][c] += sum_p w[p][m] x[p][c]: A = w^T straight from the
//           logits output registers (slot t<4: point 4g+t, t>=4: point 16+4g+t-4),
//           B = x^T read from a per-wave LDS transpose of the block;
//           d[m] += sum_p w[p][m] via the same A against a ones operand.
#pragma once
#include "ts3_device.h"

namespace ts3 {

template <typename T, int C, int M> struct Pass1Cfg {
    static constexpr int CT = C / 16;      // 16-channel tiles
    static constexpr int MT = M / 16;      // 16-slice tiles
    static constexpr int CK = C / 32;      // K32 steps over channels
    static constexpr int WAVES = 4;
    static constexpr int XT_ROW = 36;      // LDS row (points) of the transposed block, padded
    static constexpr int XT_BYTES = WAVES * C * XT_ROW * (int)sizeof(T);
    static constexpr int RED_BYTES = WAVES * M * (C + 1) * 4;
    static constexpr int LDS_BYTES = XT_BYTES > RED_BYTES ? XT_BYTES : RED_BYTES;
};

// x       : tile base, [n_tile][C] storage elements
// n_tile  : points in this tile (tile starts on a span boundary)
// span0   : global index of the tile's first span
// Q       : points per span (multiple of 32)
// nspan   : spans in this tile (= ceil(n_tile / Q)); grid = nspan * H
// w2p     : prepared W2' fragments [H][MT][CK][64 lanes][8]
// b2s     : W2'-scaled bias [H*M]
// partials: [span][H][M][C+1] float32
template <typename T, int C, int M>
__global__ __launch_bounds__(256, 1) void k_slice_accumulate(
    const T *__restrict__ x, int64_t n_tile, int64_t span0, int32_t Q, int32_t nspan, int32_t H,
    const T *__restrict__ w2p, const float *__restrict__ b2s, float *__restrict__ partials) {
    using Cfg = Pass1Cfg<T, C, M>;
    constexpr int CT = Cfg::CT, MT = Cfg::MT, CK = Cfg::CK, XT_ROW = Cfg::XT_ROW;
    __shared__ __attribute__((aligned(16))) unsigned char lds[Cfg::LDS_BYTES];

    const int nwg = nspan * H;
    const int j = xcd_remap((int)blockIdx.x, nwg);
    const int span_local = j / H;
    const int h = j - span_local * H;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int li = lane & 15;
    const int g = lane >> 4;

    const int64_t p_begin = (int64_t)span_local * Q;
    const int64_t p_end = p_begin + Q < n_tile ? p_begin + Q : n_tile;
    const int nblk = (int)((p_end - p_begin + 31) >> 5);

    // Head h's W2' fragments and bias, resident for the whole workgroup.
    Frag<T> w2[MT][CK];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int kc = 0; kc < CK; ++kc)
            load8(w2[mt][kc], w2p + ((((size_t)h * MT + mt) * CK + kc) * 64 + lane) * 8);
    float bias[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) bias[mt] = b2s[h * M + mt * 16 + li];

    f32x4 S[MT][CT];
    f32x4 D[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        D[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) S[mt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    Frag<T> ones;
    ones8(ones);

    T *xt = reinterpret_cast<T *>(lds) + (size_t)wave * C * XT_ROW;

    for (int blk = wave; blk < nblk; blk += Cfg::WAVES) {
        const int64_t p0 = p_begin + ((int64_t)blk << 5);
        const int valid = (int)(p_end - p0 < 32 ? p_end - p0 : 32);

        // x rows of the block as logits A fragments: lane (g, li) holds
        // x[p0 + 16*pt + li][32*kc + 8*g .. +8].
        Frag<T> xa[2][CK];
#pragma unroll
        for (int pt = 0; pt < 2; ++pt) {
            const int pr = pt * 16 + li;
#pragma unroll
            for (int kc = 0; kc < CK; ++kc) {
                if (pr < valid)
                    load8(xa[pt][kc], x + (size_t)(p0 + pr) * C + kc * 32 + g * 8);
                else
                    zero8(xa[pt][kc]);
            }
        }

        // Transpose the block into LDS: xt[c][p].
        asm volatile("" ::: "memory");
#pragma unroll
        for (int pt = 0; pt < 2; ++pt)
#pragma unroll
            for (int kc = 0; kc < CK; ++kc)
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    const int c = kc * 32 + g * 8 + t;
                    if constexpr (sizeof(T) == 2) {
                        reinterpret_cast<uint16_t *>(xt)[c * XT_ROW + pt * 16 + li] = elem_bits(xa[pt][kc], t);
                    } else {
                        reinterpret_cast<float *>(xt)[c * XT_ROW + pt * 16 + li] = elem_f32(xa[pt][kc], t);
                    }
                }

        // Slice logits.
        f32x4 L[2][MT];
#pragma unroll
        for (int pt = 0; pt < 2; ++pt)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                L[pt][mt] = f32x4{bias[mt], bias[mt], bias[mt], bias[mt]};
#pragma unroll
                for (int kc = 0; kc < CK; ++kc) mma(L[pt][mt], xa[pt][kc], w2[mt][kc]);
            }

        // Softmax over the M slices of each point (point 16*pt + 4*g + r).
#pragma unroll
        for (int pt = 0; pt < 2; ++pt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float mx = L[pt][0][r];
#pragma unroll
                for (int mt = 1; mt < MT; ++mt) mx = fmaxf(mx, L[pt][mt][r]);
                mx = row16_max(mx);
                float sum = 0.f;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const float e = fast_exp2(L[pt][mt][r] - mx);
                    L[pt][mt][r] = e;
                    sum += e;
                }
                sum = row16_sum(sum);
                float inv = fast_rcp(sum);
                if (pt * 16 + g * 4 + r >= valid) inv = 0.f;  // padding points weigh nothing
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) L[pt][mt][r] *= inv;
            }

        asm volatile("" ::: "memory");
        // Contraction over the block's points.
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            Frag<T> a;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                a.set(t, L[0][mt][t]);
                a.set(t + 4, L[1][mt][t]);
            }
            mma(D[mt], a, ones);
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                Frag<T> b;
                const T *row = xt + (ct * 16 + li) * XT_ROW;
                if constexpr (sizeof(T) == 2) {
                    typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
                    const bf16x4 lo = *reinterpret_cast<const bf16x4 *>(row + g * 4);
                    const bf16x4 hi = *reinterpret_cast<const bf16x4 *>(row + 16 + g * 4);
                    b.v = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                } else {
                    const float4 lo = *reinterpret_cast<const float4 *>(row + g * 4);
                    const float4 hi = *reinterpret_cast<const float4 *>(row + 16 + g * 4);
                    b.set(0, lo.x); b.set(1, lo.y); b.set(2, lo.z); b.set(3, lo.w);
                    b.set(4, hi.x); b.set(5, hi.y); b.set(6, hi.z); b.set(7, hi.w);
                }
                mma(S[mt][ct], a, b);
            }
        }
        asm volatile("" ::: "memory");
    }

    // Fixed-order reduction of the four wave accumulators.
    __syncthreads();
    float *red = reinterpret_cast<float *>(lds);
    float *mine = red + (size_t)wave * M * (C + 1);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = mt * 16 + g * 4 + r;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) mine[m * (C + 1) + ct * 16 + li] = S[mt][ct][r];
            if (li == 0) mine[m * (C + 1) + C] = D[mt][r];
        }
    __syncthreads();
    constexpr int E = M * (C + 1);
    float *dst = partials + ((size_t)(span0 + span_local) * H + h) * E;
    for (int e = threadIdx.x; e < E; e += 256)
        dst[e] = (red[e] + red[E + e]) + (red[2 * E + e] + red[3 * E + e]);
}

}  // namespace ts3
