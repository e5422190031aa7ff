// Pass 1 of the Physics-Attention layer: slice logits, per-head temperature
// softmax and the tile contraction s_raw += w^T x, d += sum_i w_i (paper
// Eq. (1) and Eq. (4), Algorithm 1 tile loop).  The slice weights exist only in
// registers and a per-wave LDS scratch tile.
//
// Work decomposition: one workgroup per (span, head).  A span is Q consecutive
// mesh points; its four waves take 32-point blocks round-robin, each keeping a
// private M x C float32 accumulator of its head in registers, with head h's
// W2' fragments resident.  At the end the four wave accumulators are summed in
// a fixed order and written as the span's partial [M][C+1] (column C holds d).
// Spans are folded in index order later, so the result is a fixed function of
// (x, Q) whatever the tiling.
//
// Per 32-point block and wave:
//   logits  L[m][p] = W2'[:, h*M+m] . x[p] + b2'   16x16x32 MFMA, A = W2'^T
//           fragments, B = x^T from the point rows; W2' = W2 * log2(e)/tau so
//           the softmax uses exp2.  Lane (g, p) holds slices 16*mt + 4*g + r.
//   softmax over the M slices of each point: in-lane, then two cross-row swaps.
//   transpose through LDS: x rows and the normalised bf16 w rows are written
//           with 16- and 8-byte stores; ds_read_b64_tr_b16 returns them as
//           MFMA operands whose K slots hold points: slot (g, t) <-> point 8g+t.
//   contraction S[m][c] += sum_p w[p][m] x[p][c] (A = w^T, B = x) and
//           d[m] += sum_p w[p][m] (A = w^T against a ones operand).
#pragma once
#include "ts3_device.h"

namespace ts3 {

template <typename T, int C, int M> struct Pass1Cfg {
    static constexpr int CT = C / 16;      // 16-channel tiles
    static constexpr int MT = M / 16;      // 16-slice tiles
    static constexpr int CK = C / 32;      // K32 steps over channels
    static constexpr int WAVES = 4;
    // Per-wave LDS rows; a stride = 32 (mod 128) bytes keeps each transpose
    // read's four rows on distinct bank quarters.
    static constexpr int XROW = C * (int)sizeof(T) + 32;   // bytes per point row of x
    static constexpr int WROW = M * (int)sizeof(T) + 32;   // bytes per point row of w
    static constexpr int WAVE_BYTES = 32 * (XROW + WROW);
    static constexpr int XT_BYTES = WAVES * WAVE_BYTES;
    static constexpr int RED_BYTES = WAVES * M * (C + 1) * 4;
    static constexpr int LDS_BYTES = XT_BYTES > RED_BYTES ? XT_BYTES : RED_BYTES;
};

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// One 8-slot operand fragment from two transposing LDS reads.  Lane (g, j) of
// each 16-lane row points at row r0(g) + 4*half + j/4, column col0 + 4*(j%4) of
// a row-major bf16 tile (row stride `row` bytes); the result gives lane (g, i)
// column col0 + i of rows r0(g) .. r0(g)+7 in slots 0..7.
__device__ __forceinline__ void tr_frag(Frag<bf16_t> &f, const unsigned char *base, int row, int r0, int col0,
                                        int j) {
    const unsigned char *p = base + (size_t)(r0 + (j >> 2)) * row + (col0 + 4 * (j & 3)) * 2;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(p));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(p + 4 * row));
    typedef short s16x8 __attribute__((ext_vector_type(8)));
    const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    f.v = __builtin_bit_cast(bf16x8, v);
}
// fp32 tiles: the same fragment read element by element (fp32 storage is the
// parity path, not the fast one).
__device__ __forceinline__ void tr_frag(Frag<float> &f, const unsigned char *base, int row, int r0, int col0,
                                        int i) {
#pragma unroll
    for (int t = 0; t < 8; ++t) f.v[t] = *reinterpret_cast<const float *>(base + (size_t)(r0 + t) * row + (col0 + i) * 4);
}

// x       : tile base, [n_tile][C] storage elements
// n_tile  : points in this tile (tile starts on a span boundary)
// span0   : global index of the tile's first span
// Q       : points per span
// nspan   : spans in this tile (= ceil(n_tile / Q)); grid = nspan * H
// w2p     : prepared W2' fragments [H][MT][CK][64 lanes][8]
// b2s     : W2'-scaled bias [H*M]
// partials: [span][H][M][C+1] float32
template <typename T, int C, int M>
__global__ __launch_bounds__(256, 1) void k_slice_accumulate(
    const T *__restrict__ x, int64_t n_tile, int64_t span0, int32_t Q, int32_t nspan, int32_t H,
    const T *__restrict__ w2p, const float *__restrict__ b2s, float *__restrict__ partials) {
    using Cfg = Pass1Cfg<T, C, M>;
    constexpr int CT = Cfg::CT, MT = Cfg::MT, CK = Cfg::CK;
    constexpr int XROW = Cfg::XROW, WROW = Cfg::WROW;
    constexpr int KM = M >= 32 ? M / 32 : 1;
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

    // Head h's W2'^T fragments (A operand: lane row = slice) and bias, resident.
    Frag<T> w2[MT][CK];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int kc = 0; kc < CK; ++kc)
            load8(w2[mt][kc], w2p + ((((size_t)h * MT + mt) * CK + kc) * 64 + lane) * 8);
    f32x4 bias[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const float4 b = *reinterpret_cast<const float4 *>(b2s + h * M + mt * 16 + g * 4);
        bias[mt] = f32x4{b.x, b.y, b.z, b.w};
    }

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

    unsigned char *xl = lds + wave * Cfg::WAVE_BYTES;   // [32 points][XROW bytes]
    unsigned char *wl = xl + 32 * XROW;                   // [32 points][WROW bytes]

    // x rows of a block as the logits B operand: lane (g, li) holds
    // x[p0 + 16*pt + li][32*kc + 8*g .. +8] (zero past the span's end).
    auto load_x = [&](int blk, Frag<T> (&xb)[2][CK]) {
        const int64_t p0 = p_begin + ((int64_t)blk << 5);
#pragma unroll
        for (int pt = 0; pt < 2; ++pt) {
            const int64_t pr = p0 + pt * 16 + li;
#pragma unroll
            for (int kc = 0; kc < CK; ++kc) {
                if (blk < nblk && pr < p_end)
                    load8(xb[pt][kc], x + (size_t)pr * C + kc * 32 + g * 8);
                else
                    zero8(xb[pt][kc]);
            }
        }
    };

    auto process = [&](int blk, Frag<T> (&xb)[2][CK]) {
        const int64_t p0 = p_begin + ((int64_t)blk << 5);
        const int valid = (int)(p_end - p0 < 32 ? p_end - p0 : 32);
        asm volatile("" ::: "memory");
#pragma unroll
        for (int pt = 0; pt < 2; ++pt)
#pragma unroll
            for (int kc = 0; kc < CK; ++kc) {
                unsigned char *dst = xl + (pt * 16 + li) * XROW + (kc * 32 + g * 8) * (int)sizeof(T);
                if constexpr (sizeof(T) == 2) {
                    *reinterpret_cast<bf16x8 *>(dst) = xb[pt][kc].v;
                } else {
                    reinterpret_cast<float4 *>(dst)[0] = float4{xb[pt][kc].v[0], xb[pt][kc].v[1], xb[pt][kc].v[2], xb[pt][kc].v[3]};
                    reinterpret_cast<float4 *>(dst)[1] = float4{xb[pt][kc].v[4], xb[pt][kc].v[5], xb[pt][kc].v[6], xb[pt][kc].v[7]};
                }
            }

        // Slice logits [slices x points].
        auto logits = [&](f32x4 (&L)[MT][2]) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int pt = 0; pt < 2; ++pt) {
                    L[mt][pt] = bias[mt];
#pragma unroll
                    for (int kc = 0; kc < CK; ++kc) mma(L[mt][pt], w2[mt][kc], xb[pt][kc]);
                }
        };
        f32x4 L[MT][2];
        logits(L);

        // Softmax per point (lane (g, li) holds point 16*pt + li).  Fast path
        // without the max shift; a wave with any row outside the safe window
        // recomputes its logits and takes the shifted path.
        float inv[2];
        bool ok = true;
#pragma unroll
        for (int pt = 0; pt < 2; ++pt) {
            float sum = 0.f;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float e = fast_exp2(L[mt][pt][r]);
                    L[mt][pt][r] = e;
                    sum += e;
                }
            sum = xrow_sum(sum);
            ok = ok && softmax_sum_ok(sum);
            inv[pt] = fast_rcp(sum);
        }
        if (__any(!ok)) {
            logits(L);
#pragma unroll
            for (int pt = 0; pt < 2; ++pt) {
                float mx = L[0][pt][0];
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) mx = fmaxf(mx, L[mt][pt][r]);
                mx = xrow_max(mx);
                float sum = 0.f;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float e = fast_exp2(L[mt][pt][r] - mx);
                        L[mt][pt][r] = e;
                        sum += e;
                    }
                inv[pt] = fast_rcp(xrow_sum(sum));
            }
        }
#pragma unroll
        for (int pt = 0; pt < 2; ++pt)
            if (pt * 16 + li >= valid) inv[pt] = 0.f;  // padding points weigh nothing

        // Normalised w rows to LDS: lane (g, li) stores slices 16*mt + 4*g .. +3
        // of point 16*pt + li.
#pragma unroll
        for (int pt = 0; pt < 2; ++pt)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                unsigned char *dst = wl + (pt * 16 + li) * WROW + (mt * 16 + g * 4) * (int)sizeof(T);
                const float a0 = L[mt][pt][0] * inv[pt], a1 = L[mt][pt][1] * inv[pt];
                const float a2 = L[mt][pt][2] * inv[pt], a3 = L[mt][pt][3] * inv[pt];
                if constexpr (sizeof(T) == 2) {
                    typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
                    *reinterpret_cast<bf16x4 *>(dst) = bf16x4{(__bf16)a0, (__bf16)a1, (__bf16)a2, (__bf16)a3};
                } else {
                    *reinterpret_cast<float4 *>(dst) = float4{a0, a1, a2, a3};
                }
            }
        asm volatile("" ::: "memory");

        // Contraction over the block's 32 points; K slot (g, t) holds point 8g+t.
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            Frag<T> a;
            tr_frag(a, wl, WROW, 8 * g, mt * 16, li);
            mma(D[mt], a, ones);
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                Frag<T> b;
                tr_frag(b, xl, XROW, 8 * g, ct * 16, li);
                mma(S[mt][ct], a, b);
            }
        }
        asm volatile("" ::: "memory");
    };

    // Block b+4's rows load into registers while block b computes.
    Frag<T> xa[2][CK], xn[2][CK];
    load_x(wave, xn);
    for (int blk = wave; blk < nblk; blk += Cfg::WAVES) {
#pragma unroll
        for (int pt = 0; pt < 2; ++pt)
#pragma unroll
            for (int kc = 0; kc < CK; ++kc) xa[pt][kc] = xn[pt][kc];
        load_x(blk + Cfg::WAVES, xn);
        process(blk, xa);
    }
    (void)KM;

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
