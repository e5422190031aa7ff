// Pass 1 for wide point rows (bf16, C = 256): slice logits, per-head
// temperature softmax and the tile contraction s_raw += w^T x, d += sum_i w_i
// (Eq. (1) and Eq. (4), Algorithm 1 tile loop).
//
// At C = 256 one wave cannot hold both its head's W2' fragments and an M x C
// float32 accumulator, so the contraction is split by channels instead of by
// points.  One workgroup per (span, head), four waves, 128-point super-blocks
// of four 32-point blocks:
//   copy     the super-block's x rows (64 KB) arrive in one of two LDS slots
//            by direct global->LDS copies, one super-block ahead of use;
//   logits   wave v takes block v: L = W2'^T x (W2' resident, B = x rows read
//            from the slot), the max-shifted softmax over the head's M slices
//            (exp2; W2' and b2 carry log2(e)/tau), and the w rows go to the
//            block's LDS w tile (bf16);
//   contract after a barrier every wave adds all four blocks into its own
//            quarter of the channels: S[m][c] += sum_p w[p][m] x[p][c] with
//            ds_read_b64_tr_b16 operands (K slot (g, t) <-> point row 8g+t);
//            wave 0 also forms d[m] += sum_p w[p][m].
// No reduction across waves is needed; each wave writes its channels of the
// span partial [M][C+1] (column C = d).  The order of every sum is fixed by
// (x, Q), so results do not depend on the tiling.
//
// Work-group index -> (span, head) is XCD-aware: the H workgroups of one span
// run on the same XCD and read the same x rows through its L2.
#pragma once
#include "ts3_pass1.h"

namespace ts3 {

template <int C, int M> struct Pass1WideCfg {
    static constexpr int MT = M / 16, CK = C / 32;
    static constexpr int WAVES = 4;
    static constexpr int CW = C / WAVES;          // channels contracted per wave
    static constexpr int CTW = CW / 16;
    static constexpr int XROW = C * 2, WROW = M * 2;
    static constexpr int XTILE = 32 * XROW, WTILE = 32 * WROW;
    static constexpr int XSLOT = WAVES * XTILE;   // one 128-point super-block
    static constexpr int COPIES = XSLOT / 1024;   // 1 KB wave copies per super-block
    static constexpr int LDS_BYTES = 2 * XSLOT + WAVES * WTILE;
    static_assert(COPIES % WAVES == 0, "copies split evenly over the waves");
    static_assert(1024 % XROW == 0, "a 1 KB copy covers whole rows");
};

// x       : tile base, [n_tile][C] bf16
// n_tile  : points in this tile (the tile starts on a span boundary)
// span0   : global index of the tile's first span
// Q       : points per span
// nspan   : spans in this tile; grid = ceil(nspan / 8) * 8 * H (XCD groups)
// w2p     : prepared W2' fragments [H][MT][CK][64 lanes][8]
// b2s     : W2'-scaled bias [H*M]
// partials: [span][H][M][C+1] float32
template <int C, int M>
__global__ __launch_bounds__(256, 1) void k_slice_accumulate_wide(
    const bf16_t *__restrict__ x, int64_t n_tile, int64_t span0, int32_t Q, int32_t nspan, int32_t H,
    const bf16_t *__restrict__ w2p, const float *__restrict__ b2s, float *__restrict__ partials) {
    using Cfg = Pass1WideCfg<C, M>;
    constexpr int MT = Cfg::MT, CK = Cfg::CK, CTW = Cfg::CTW, CW = Cfg::CW;
    constexpr int XROW = Cfg::XROW, WROW = Cfg::WROW, XTILE = Cfg::XTILE, WTILE = Cfg::WTILE;
    constexpr int XSLOT = Cfg::XSLOT, NCH = XROW / 16, RPC = 1024 / XROW;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[Cfg::LDS_BYTES];

    // (span, head) from the XCD-aware index: workgroup j runs on XCD j % 8;
    // the H consecutive indices j / 8 of one XCD group share a span.
    const int j = (int)blockIdx.x;
    const int idx = j >> 3;
    const int h = idx % H;
    const int span_local = (idx / H) * 8 + (j & 7);
    if (span_local >= nspan) return;  // workgroup-uniform; no barrier has run

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int li = lane & 15, g = lane >> 4;
    const int64_t p_begin = (int64_t)span_local * Q;
    const int64_t p_end = p_begin + Q < n_tile ? p_begin + Q : n_tile;
    const int nsb = (int)((p_end - p_begin + 127) >> 7);
    unsigned char *const wtiles = lds + 2 * XSLOT;

    // W2'^T fragments of head h (A operand: lane row = slice) and bias.
    Frag<bf16_t> w2[MT][CK];
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
    f32x4 S[MT][CTW];
    f32x4 D[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        D[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ct = 0; ct < CTW; ++ct) S[mt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    Frag<bf16_t> ones;
    ones8(ones);
    wait_vmcnt<0>();  // the copies below are then the only loads in flight

    // Super-block i into slot sl: copy k covers super-block rows RPC*k ..
    // (block k / (32 / RPC)); lane l fills physical chunk l % NCH of its row,
    // reading the logical chunk the swizzle stores there.  Rows past the
    // span's end repeat its last point (their weights are zero).
    auto issue = [&](int i, int sl) {
        const int64_t p0 = p_begin + ((int64_t)i << 7);
        const uint32_t base = lds_addr(lds) + sl * XSLOT;
#pragma unroll
        for (int c = 0; c < Cfg::COPIES / Cfg::WAVES; ++c) {
            const int k = wave * (Cfg::COPIES / Cfg::WAVES) + c;
            const int sr = RPC * k + lane / NCH;  // row within the super-block
            const int R = sr & 31;                // row within its block
            int64_t p = p0 + sr;
            p = p < p_end ? p : p_end - 1;
            const int chunk = (lane % NCH) ^ xswz<XROW>(R);
            dma16(reinterpret_cast<const unsigned char *>(x + (size_t)p * C) + chunk * 16, base + k * 1024);
        }
    };

    issue(0, 0);
    for (int i = 0; i < nsb; ++i) {
        const int sl = i & 1;
        wait_vmcnt<0>();
        __syncthreads();  // slot sl landed for every wave; iteration i-1 is done with the w tiles and slot sl^1
        if (i + 1 < nsb) issue(i + 1, sl ^ 1);
        const unsigned char *xs = lds + sl * XSLOT;

        // Logits, softmax and w rows of block `wave`.
        {
            const unsigned char *tile = xs + wave * XTILE;
            const int64_t left = p_end - (p_begin + ((int64_t)i << 7) + 32 * wave);
            const int valid = left < 0 ? 0 : (left < 32 ? (int)left : 32);
            f32x4 L[MT][2];
#pragma unroll
            for (int pt = 0; pt < 2; ++pt) {
                const int R = prow(pt, li);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) L[mt][pt] = bias[mt];
                // all K steps' x operands first, so their LDS latency overlaps
                Frag<bf16_t> xb[CK];
#pragma unroll
                for (int kc = 0; kc < CK; ++kc)
                    xb[kc].v = *reinterpret_cast<const bf16x8 *>(tile + xoff<XROW>(R, (kc * 32 + g * 8) * 2));
#pragma unroll
                for (int kc = 0; kc < CK; ++kc)
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) mma(L[mt][pt], w2[mt][kc], xb[kc]);
            }
            unsigned char *wt = wtiles + wave * WTILE;
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
                sum = xrow_sum(sum);
                const int R = prow(pt, li);
                const float inv = R < valid ? 1.f / sum : 0.f;
                typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    *reinterpret_cast<bf16x4 *>(wt + woff<WROW>(R, (mt * 16 + g * 4) * 2)) =
                        bf16x4{(__bf16)(L[mt][pt][0] * inv), (__bf16)(L[mt][pt][1] * inv),
                               (__bf16)(L[mt][pt][2] * inv), (__bf16)(L[mt][pt][3] * inv)};
            }
        }
        __syncthreads();  // every block's w tile is written

        // This wave's channels of all four blocks.
#pragma unroll 1
        for (int b = 0; b < Cfg::WAVES; ++b) {
            const unsigned char *xt = xs + b * XTILE, *wt = wtiles + b * WTILE;
            Frag<bf16_t> a[MT];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) tr_frag<WROW>(a[mt], tr_addr<WROW, false>(wt, g, mt * 16, li));
            if (wave == 0)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) mma(D[mt], a[mt], ones);
            Frag<bf16_t> bx[CTW];  // read before the products, as above
#pragma unroll
            for (int ct = 0; ct < CTW; ++ct) tr_frag<XROW>(bx[ct], tr_addr<XROW, true>(xt, g, wave * CW + ct * 16, li));
#pragma unroll
            for (int ct = 0; ct < CTW; ++ct)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) mma(S[mt][ct], a[mt], bx[ct]);
        }
    }

    // The wave's channels of the span partial; wave 0 adds column C (d).
    float *dst = partials + ((size_t)(span0 + span_local) * H + h) * M * (C + 1);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = mt * 16 + g * 4 + r;
#pragma unroll
            for (int ct = 0; ct < CTW; ++ct) dst[(size_t)m * (C + 1) + wave * CW + ct * 16 + li] = S[mt][ct][r];
            if (wave == 0 && li == 0) dst[(size_t)m * (C + 1) + C] = D[mt][r];
        }
}

}  // namespace ts3
