// Pass 2 for wide point rows (bf16, C = 256): recompute each point's slice
// weights and decode out = sum_h w_h . Z_h (+ b3, folded into Z) (Eq. (5),
// Algorithm 1 deslice loop).
//
// At C = 256 one head's W2' and Z operands are 32 KB each, so the heads are
// streamed through LDS: 128 points per workgroup (eight waves of one 16-point
// tile, or four of two), head h's W2'^T and Z^T fragments staged in one of two LDS
// slots one head ahead of use (linear direct copies: the prepared arrays are
// already in fragment order).  Per head and wave:
//   logits  L[m][p] = W2'_h^T x_p + b2'   (A = staged W2'^T, B = x rows kept in
//           registers for the whole kernel)
//   softmax over the head's M slices (in-lane, then two cross-row swaps),
//           without the max shift while every row sum stays in the safe
//           window (else with it); the 16 x 4 outputs of two slice tiles are a B
//           fragment of the decode with K slot (g, t) <-> slice
//           32km + 16(t>>2) + 4g + (t&3), the order of the prepared Z
//   decode  out^T[c][p] += Z_h^T[c][:] . w[p][:]   (A = staged Z^T)
// Z's rows follow zchan(), so each lane stores eight consecutive channels.
#pragma once
#include "ts3_device.h"
#include "ts3_pass2.h"

namespace ts3 {

template <int C, int M, int PT = 2> struct Pass2WideCfg {
    static constexpr int MT = M / 16, CK = C / 32, CT = C / 16, KM = M / 32;
    static constexpr int PART = M * C;                 // elements of W2'_h (= of Z_h)
    static constexpr int HEAD_BYTES = 2 * PART * 2;    // bf16 W2'_h then Z_h
    static constexpr int COPIES = HEAD_BYTES / 1024;
    static constexpr int WAVES = 8 / PT;               // 128 points per workgroup
    static_assert(M % 32 == 0, "slice tiles pair into K32 steps");
    static_assert(COPIES % (2 * WAVES) == 0, "copies split evenly over the waves and halves");
};

// x: [n][C] bf16; w2p: [H][MT][CK][64][8]; zp: [H][CT][KM][64][8];
// b2s: [H*M]; out: [n][C] bf16.  PT: 16-point tiles per wave.  Grid:
// ceil(n / 128) workgroups of 512 / PT threads.
template <int C, int M, int PT>
__global__ __launch_bounds__(512 / PT, 1) void k_deslice_wide(const bf16_t *__restrict__ x, int64_t n, int32_t H,
                                                          const bf16_t *__restrict__ w2p, const float *__restrict__ b2s,
                                                          const bf16_t *__restrict__ zp, bf16_t *__restrict__ out) {
    using Cfg = Pass2WideCfg<C, M, PT>;
    constexpr int MT = Cfg::MT, CK = Cfg::CK, CT = Cfg::CT, KM = Cfg::KM;
    constexpr int HB = Cfg::HEAD_BYTES, PB = Cfg::PART * 2;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[2 * HB];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int li = lane & 15, g = lane >> 4;
    const int64_t p0 = ((int64_t)blockIdx.x * Cfg::WAVES + wave) * (16 * PT);

    // Head h's W2'^T then Z^T fragments into slot sl.
    auto issue = [&](int h, int sl) {
        const uint32_t base = lds_addr(lds) + sl * HB;
        constexpr int PER = Cfg::COPIES / Cfg::WAVES / 2;  // per half and wave
        const unsigned char *wsrc = reinterpret_cast<const unsigned char *>(w2p) + (size_t)h * PB;
        const unsigned char *zsrc = reinterpret_cast<const unsigned char *>(zp) + (size_t)h * PB;
#pragma unroll
        for (int c = 0; c < PER; ++c) {
            const int k = wave * PER + c;
            dma16(wsrc + k * 1024 + lane * 16, base + k * 1024);
            dma16(zsrc + k * 1024 + lane * 16, base + PB + k * 1024);
        }
    };
    issue(0, 0);

    // x rows of the wave's points as logits B fragments: tile pt, lane (li, g)
    // holds channels 32k + 8g .. +7 of point p0 + 16pt + li in fragment k.
    Frag<bf16_t> xb[PT][CK];
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) {
        int64_t p = p0 + 16 * pt + li;
        p = p < n ? p : n - 1;
#pragma unroll
        for (int k = 0; k < CK; ++k) load8(xb[pt][k], x + p * C + 32 * k + 8 * g);
    }
    f32x4 O[CT][PT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) O[ct][pt] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int h = 0; h < H; ++h) {
        const int sl = h & 1;
        wait_vmcnt<0>();
        __syncthreads();  // head h staged; every wave is done with head h-1's slot
        if (h + 1 < H) issue(h + 1, sl ^ 1);
        const unsigned char *wa = lds + sl * HB, *za = wa + PB;
        // Logits of head h.  A fragments are read one K step ahead of their
        // products, so LDS latency overlaps the matrix cores.
        auto logits = [&](f32x4 (&L)[MT][PT]) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const float4 b = *reinterpret_cast<const float4 *>(b2s + h * M + 16 * mt + 4 * g);
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) L[mt][pt] = f32x4{b.x, b.y, b.z, b.w};
            }
            Frag<bf16_t> a1[2][MT];
            auto read1 = [&](int kc, Frag<bf16_t>(&dst)[MT]) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    dst[mt].v = *reinterpret_cast<const bf16x8 *>(wa + ((mt * CK + kc) * 64 + lane) * 16);
            };
            read1(0, a1[0]);
#pragma unroll
            for (int kc = 0; kc < CK; ++kc) {
                if (kc + 1 < CK) read1(kc + 1, a1[(kc + 1) & 1]);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int pt = 0; pt < PT; ++pt) mma(L[mt][pt], a1[kc & 1][mt], xb[pt][kc]);
            }
        };
        f32x4 L[MT][PT];
        logits(L);
        // The decode runs with its K steps outermost: the products into one
        // accumulator are CT * PT apart (a dependent MFMA issues at half
        // rate); the Z fragment of step q+2 is read while step q's run.
        constexpr int NQ = KM * CT;
        auto zfrag = [&](int q2) { return za + (((q2 % CT) * KM + q2 / CT) * 64 + lane) * 16; };
        // Softmax without the max shift while every row sum stays in the
        // safe window; otherwise (rare) shifted, from the logits kept in L.
        f32x4 E[MT][PT];
        float inv[PT];
        bool ok = true;
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) {
            float sum = 0.f;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    E[mt][pt][r] = fast_exp2(L[mt][pt][r]);
                    sum += E[mt][pt][r];
                }
            sum = xrow_sum(sum);
            ok = ok && softmax_sum_ok(sum);
            inv[pt] = fast_rcp(sum);
        }
        if (__any(!ok)) {
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) {
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
                        E[mt][pt][r] = fast_exp2(L[mt][pt][r] - mx);
                        sum += E[mt][pt][r];
                    }
                inv[pt] = fast_rcp(xrow_sum(sum));
            }
        }
        Frag<bf16_t> wb[PT][KM];
#pragma unroll
        for (int pt = 0; pt < PT; ++pt)
#pragma unroll
            for (int km = 0; km < KM; ++km)
#pragma unroll
                for (int t = 0; t < 8; t += 2) {
                    const int mt = 2 * km + (t >> 2);
                    wb[pt][km].set2(t, E[mt][pt][t & 3] * inv[pt], E[mt][pt][(t & 3) + 1] * inv[pt]);
                }
        Frag<bf16_t> a2[4];
        a2[0].v = *reinterpret_cast<const bf16x8 *>(zfrag(0));
        a2[1].v = *reinterpret_cast<const bf16x8 *>(zfrag(1));
#pragma unroll
        for (int q2 = 0; q2 < NQ; ++q2) {
            if (q2 + 2 < NQ) a2[(q2 + 2) & 3].v = *reinterpret_cast<const bf16x8 *>(zfrag(q2 + 2));
            const int km = q2 / CT, ct = q2 % CT;
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) mma(O[ct][pt], a2[q2 & 3], wb[pt][km]);
        }
    }

    // Tiles ct = 2k, 2k+1 hold channels 32k + 8g + 4(ct & 1) + r of point p.
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) {
        const int64_t p = p0 + 16 * pt + li;
        if (p >= n) continue;
#pragma unroll
        for (int k = 0; k < CT / 2; ++k) {
            typedef __attribute__((ext_vector_type(8))) __bf16 b8;
            b8 v;
#pragma unroll
            for (int t = 0; t < 8; ++t) v[t] = (__bf16)O[2 * k + (t >> 2)][pt][t & 3];
            *reinterpret_cast<b8 *>(out + p * C + 32 * k + 8 * g) = v;
        }
    }
}

}  // namespace ts3
