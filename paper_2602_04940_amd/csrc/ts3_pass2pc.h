// Pass 2 (paper Eq. (5), Algorithm 1 deslice loop) on producer and consumer
// waves, for 16-bit storage: out[p] = sum_h sum_m softmax_m(L_h[p]) Z_h[m][:]
// (+ b3, folded into the prepared Z).
//
// 128 points per workgroup block, 32 per pair of waves sharing a SIMD:
//   wave q      (producer) keeps the x rows of its 32 points as B fragments
//               and, per head, computes the logits (A = the head's staged
//               W2'^T fragments), the softmax over the head's M slices, and
//               writes the slice weights to the pair's w tile as the decode's
//               B fragments (K slot (g, t) <-> slice 32km + 16(t>>2) + 4g +
//               (t&3), the order of the prepared Z), so no transposition;
//   wave q + 4  (consumer) decodes the previous head of the same points into
//               the 32 x C output accumulator (A = the head's staged Z
//               fragments, K steps outermost), stores a block's rows after
//               its last head, and issues the weight copies.
// Every weight fragment read from LDS feeds two MFMAs (two 16-point tiles),
// and the softmax's vector work runs beside the other wave's matrix work.
// The heads' W2' and Z parts are streamed through separate LDS slots (two
// each): step s reads W2'(s) and Z(s-1) and copies W2'(s+1) and Z(s).  Steps
// run over (block, head) pairs of a persistent workgroup's blocks, so the
// pipeline does not drain between blocks; the producer loads the next block's
// x during the current block's last head.  One barrier per step.
//
// Softmax: exp2 of the raw logits while every row sum stays in [2^-100,
// 2^100] (then it equals the shifted softmax to float32 rounding); a tile
// with a row outside the window takes the max-shifted softmax, from the
// logits kept in registers.
#pragma once
#include "ts3_device.h"
#include "ts3_pass2.h"

namespace ts3 {

template <int C, int M> struct Pass2PCCfg {
    static constexpr int MT = M / 16, CK = C / 32, CT = C / 16, KM = M / 32, PT = 2;
    static constexpr int PART = M * C;               // elements of W2'_h (= of Z_h)
    static constexpr int PB = PART * 2;              // bytes
    static constexpr int PART_COPIES = PB / 1024;
    static constexpr int HTILE = PT * KM * 64 * 16;  // bytes: a pair's w fragments
    static constexpr int LDS_BYTES = 4 * PB + 4 * 2 * HTILE;
    static constexpr int POINTS_PER_WG = 128;
    static_assert(M % 32 == 0, "slice tiles pair into K32 steps");
    static_assert(PART_COPIES % 4 == 0, "each consumer issues a quarter of a part's copies");
};

// x: [n][C] bf16; w2p: [H][MT][CK][64][8]; zp: [H][CT][KM][64][8]; b2s:
// [H*M]; out: [n][C] bf16.  Grid: at most ceil(n / 128) persistent
// workgroups of 512 threads.
template <int C, int M>
__global__ __launch_bounds__(512, 1) void k_deslice_pc(const bf16_t *__restrict__ x, int64_t n, int32_t H,
                                                       const bf16_t *__restrict__ w2p, const float *__restrict__ b2s,
                                                       const bf16_t *__restrict__ zp, bf16_t *__restrict__ out) {
    using Cfg = Pass2PCCfg<C, M>;
    using T = bf16_t;
    constexpr int MT = Cfg::MT, CK = Cfg::CK, CT = Cfg::CT, KM = Cfg::KM, PT = Cfg::PT;
    constexpr int PB = Cfg::PB, HTILE = Cfg::HTILE;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[Cfg::LDS_BYTES];
    unsigned char *const wslots = lds;           // W2'_h parts, two slots
    unsigned char *const zslots = lds + 2 * PB;  // Z_h parts, two slots

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int q = wave & 3, role = wave >> 2;
    const int li = lane & 15, g = lane >> 4;
    unsigned char *const hslots = lds + 4 * PB + q * 2 * HTILE;  // the pair's two w tiles
    const int64_t nblk = (n + Cfg::POINTS_PER_WG - 1) / Cfg::POINTS_PER_WG;
    if (n <= 0 || H <= 0 || (int64_t)blockIdx.x >= nblk) return;  // uniform over the workgroup
    const int iters = (int)((nblk - 1 - blockIdx.x) / gridDim.x + 1);  // blocks of this workgroup
    const int S = iters * H;                                          // (block, head) steps
    const int64_t pw = (int64_t)blockIdx.x * Cfg::POINTS_PER_WG + q * 32;
    const int64_t bstride = (int64_t)gridDim.x * Cfg::POINTS_PER_WG;

    if (role == 0) {
        // ---------------------------------------------------------------- producer
        // x B fragments of block i: tile pt, lane (li, g) holds channels
        // 32k + 8g .. +7 of point p0 + 16pt + li (rows past n repeat row n-1:
        // finite data whose outputs are never stored).
        auto load_x = [&](int i, Frag<T> (&xf)[PT][CK]) {
            const int64_t p0 = pw + (int64_t)i * bstride;
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) {
                int64_t p = p0 + 16 * pt + li;
                p = p < n ? p : n - 1;
#pragma unroll
                for (int kc = 0; kc < CK; ++kc) load8(xf[pt][kc], x + p * C + 32 * kc + 8 * g);
            }
        };
        Frag<T> xA[PT][CK], xB[PT][CK];
        load_x(0, xA);
        wait_vmcnt<0>();
        __syncthreads();  // W2'(0) staged (the consumers' copies)
        int s = 0;
        // Block i's heads with its x in xc; the next block's x goes to xn.
        auto block = [&](int i, Frag<T> (&xc)[PT][CK], Frag<T> (&xn)[PT][CK]) {
            for (int h = 0; h < H; ++h, ++s) {
                const unsigned char *wa = wslots + (s & 1) * PB;
                f32x4 L[MT][PT];
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const float4 b = *reinterpret_cast<const float4 *>(b2s + h * M + 16 * mt + 4 * g);
#pragma unroll
                    for (int pt = 0; pt < PT; ++pt) L[mt][pt] = f32x4{b.x, b.y, b.z, b.w};
                }
                // A fragments are read one K step ahead of their products.
                Frag<T> a1[2][MT];
                auto read1 = [&](int kc, Frag<T>(&dst)[MT]) {
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
                        dst[mt].v = *reinterpret_cast<const bf16x8 *>(wa + ((mt * CK + kc) * 64 + lane) * 16);
                };
                read1(0, a1[0]);
                __builtin_amdgcn_s_setprio(2);  // the logits first on the matrix core; the decode fills the softmax
#pragma unroll
                for (int kc = 0; kc < CK; ++kc) {
                    if (kc + 1 < CK) read1(kc + 1, a1[(kc + 1) & 1]);
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                        for (int pt = 0; pt < PT; ++pt) mma(L[mt][pt], a1[kc & 1][mt], xc[pt][kc]);
                }
                __builtin_amdgcn_s_setprio(0);
                // The next block's x, at the block's last head: loads retire in
                // order, so earlier it would hold up every later bias load.
                if (h == H - 1 && i + 1 < iters) load_x(i + 1, xn);
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
                // The decode's B fragments, in fragment order.
                unsigned char *wt = hslots + (s & 1) * HTILE;
#pragma unroll
                for (int pt = 0; pt < PT; ++pt)
#pragma unroll
                    for (int km = 0; km < KM; ++km) {
                        Frag<T> wf;
#pragma unroll
                        for (int t = 0; t < 8; t += 2) {
                            const int mt = 2 * km + (t >> 2);
                            wf.set2(t, E[mt][pt][t & 3] * inv[pt], E[mt][pt][(t & 3) + 1] * inv[pt]);
                        }
                        *reinterpret_cast<bf16x8 *>(wt + ((pt * KM + km) * 64 + lane) * 16) = wf.v;
                    }
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                __syncthreads();  // w(s) written; W2'(s+1) and Z(s) staged
            }
        };
        for (int i = 0; i < iters; i += 2) {
            block(i, xA, xB);
            if (i + 1 < iters) block(i + 1, xB, xA);
        }
        __syncthreads();  // the consumers' last step
    } else {
        // ---------------------------------------------------------------- consumer
        // A consumer's quarter of part `half` (0: W2', 1: Z) of head h into slot sl.
        auto issue_part = [&](int h, int half, int sl) {
            const unsigned char *src =
                reinterpret_cast<const unsigned char *>(half == 0 ? w2p : zp) + (size_t)h * PB;
            const uint32_t base = lds_addr(lds) + (half * 2 + sl) * PB;
#pragma unroll
            for (int c = 0; c < Cfg::PART_COPIES / 4; ++c) {
                const int k = q * (Cfg::PART_COPIES / 4) + c;
                dma16(src + k * 1024 + lane * 16, base + k * 1024);
            }
        };
        f32x4 O[CT][PT];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) O[ct][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
        issue_part(0, 0, 0);
        wait_vmcnt<0>();
        __syncthreads();  // W2'(0) staged
        int hs = 0, hn = H > 1 ? 1 : 0;  // heads of steps s and s+1
        int64_t pdec = pw;               // first point of the block decoded at step s (its step s-1)
        int hprev = -1;                  // head of step s-1
#pragma unroll 1
        for (int s = 0; s <= S; ++s) {
            if (s + 1 < S) issue_part(hn, 0, (s + 1) & 1);
            if (s < S) issue_part(hs, 1, s & 1);
            if (s > 0) {
                // Decode of step s-1, K steps outermost: the products into one
                // accumulator are CT * PT apart (a dependent MFMA issues at
                // half rate); the Z fragment of step q2+2 is read while step
                // q2's products run.
                const unsigned char *za = zslots + ((s - 1) & 1) * PB;
                const unsigned char *wt = hslots + ((s - 1) & 1) * HTILE;
                Frag<T> wb[PT][KM];
#pragma unroll
                for (int pt = 0; pt < PT; ++pt)
#pragma unroll
                    for (int km = 0; km < KM; ++km)
                        wb[pt][km].v = *reinterpret_cast<const bf16x8 *>(wt + ((pt * KM + km) * 64 + lane) * 16);
                constexpr int NQ = KM * CT;
                auto zfrag = [&](int q2) { return za + (((q2 % CT) * KM + q2 / CT) * 64 + lane) * 16; };
                Frag<T> a2[4];
                a2[0].v = *reinterpret_cast<const bf16x8 *>(zfrag(0));
                a2[1].v = *reinterpret_cast<const bf16x8 *>(zfrag(1));
#pragma unroll
                for (int q2 = 0; q2 < NQ; ++q2) {
                    if (q2 + 2 < NQ) a2[(q2 + 2) & 3].v = *reinterpret_cast<const bf16x8 *>(zfrag(q2 + 2));
                    const int km = q2 / CT, ct = q2 % CT;
#pragma unroll
                    for (int pt = 0; pt < PT; ++pt) mma(O[ct][pt], a2[q2 & 3], wb[pt][km]);
                }
                if (hprev == H - 1) {
                    // the block's last head: its rows are complete
                    store_rows<T, CT, PT, C>(O, out, pdec, n, g, li);
#pragma unroll
                    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
                        for (int pt = 0; pt < PT; ++pt) O[ct][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
                    pdec += bstride;
                }
            }
            wait_vmcnt<0>();  // this wave's copies of the step landed (and its stores left)
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            __syncthreads();
            hprev = hs;
            hs = hn;
            hn = hn + 1 < H ? hn + 1 : 0;
        }
    }
}

}  // namespace ts3
