// Pass 2 in the slice-state form, for 16-bit storage and head width 16
// (H = C / 16).  Eq. (5) decodes with the cached Z_h = s'_h W3_h, at H*M*C
// products per point.  By associativity the same output is
//     out[p] = sum_h (w_h[p] s'_h) W3_h + b3 = u[p] W3 + b3,
// u[p] = [w_0[p] s'_0, ..., w_{H-1}[p] s'_{H-1}] (H*dh = C values): the
// slice weights contract with the attended slice states (M*dh per head), and
// one C x C product with Linear3 follows, M*C + C*C instead of H*M*C
// products per point (90,112 instead of 131,072 with the logits at C = 128,
// M = 64, H = 8).  This is the order of Eq. (2), the form the paper's faster
// deslice reorders; the fused kernel keeps u in registers, so neither order
// stores anything per point.
//
// A wave decodes 32 points (two 16-point tiles) over all heads:
//   logits  L[m][p] = W2'[:, h*M+m] . x[p] + b2'  (A = W2'^T fragments from
//           LDS, B = x^T from registers), softmax over m in registers;
//   u_h     U[j][p] = sum_m s'_h[m][j] w[m][p]  (A = s'_h^T fragments whose K
//           slots follow the logits' register order, B = w from registers);
//           lane (g, p) holds j = 4g + r, so two heads' U registers are the
//           B fragment of one K step of the last product, unchanged;
//   out     O[c][p] = b3[c] + sum_k W3[k][c] u[k][p]  once per block (A = W3^T
//           fragments, streamed from global memory/L2).
// W2', s'^T and the slice bias stay in LDS for the whole launch: no barrier
// after the prologue, and the only per-block global traffic is x, the W3
// fragments and the stores.
//
// Softmax: as in the other decoders, exp2 of the raw logits while each row
// sum stays in [2^-100, 2^100]; blocks with a row outside the window are
// redone with the max-shifted softmax from global-memory operands.
#pragma once
#include "ts3_device.h"
#include "ts3_pass2.h"
#include "ts3_small.h"  // store_elem

#include <type_traits>

namespace ts3 {

template <int I, int N, typename F> __device__ __forceinline__ void static_for(F &&f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<I + 1, N>(f);
    }
}

template <int C, int M> struct Pass2SFCfg {
    static constexpr int DH = 16, H = C / DH;
    static constexpr int CT = C / 16, MT = M / 16, CK = C / 32, KM = M / 32, PT = 2, WAVES = 8;
    static constexpr int POINTS_PER_WG = WAVES * 16 * PT;
    static constexpr int W2_BYTES = H * MT * CK * 1024;  // W2'^T fragments, all heads
    static constexpr int SF_BYTES = H * KM * 1024;       // s'^T fragments, all heads
    static constexpr int B2_BYTES = H * M * 4;           // b2' = b2 * log2(e) / tau
    static constexpr int B3_BYTES = C * 4 <= 1024 ? 1024 : C * 4;
    // the small operands first, so that their LDS addresses stay within the
    // 64 KB reach of an instruction's immediate offset from one base
    static constexpr int B2_AT = 0, B3_AT = (B2_BYTES + 1023) / 1024 * 1024, SF_AT = B3_AT + B3_BYTES,
                         W2_AT = SF_AT + SF_BYTES;
    static constexpr int LDS_BYTES = W2_AT + W2_BYTES;
    static_assert(W2_AT % 1024 == 0, "W2' fragments 1 KB aligned");
    static constexpr int NXLOAD = PT * CK;  // x fragments of a wave block: one per head
    static constexpr int NW3 = CK * CT;     // W3^T fragments (K steps outermost)
    static constexpr int W3_AHEAD = 8;      // W3^T fragments in flight
    static_assert(M % 32 == 0 && C % 32 == 0, "slice and channel tiles pair into K32 steps");
    static_assert(H % 2 == 0, "two heads' u fill one K32 step of the Linear3 product");
    static_assert(NXLOAD == H, "one x fragment of the next block per head");
    static_assert(LDS_BYTES <= 160 * 1024, "resident operands exceed LDS");
};

// s'^T in u-product operand order [H][KM][64][8]: lane l, slot t holds
// s'[h][32*km + 16*(t>>2) + 4*(l>>4) + (t&3)][l & 15] (dh = 16).
template <typename T>
__global__ void k_prep_sf(const float *__restrict__ s1, int H, int M, T *__restrict__ sf) {
    const int KM = M / 32;
    const int64_t total = (int64_t)H * KM * 64 * 8;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int t = (int)(i & 7), lane = (int)((i >> 3) & 63);
        const int64_t r = i >> 9;
        const int km = (int)(r % KM), h = (int)(r / KM);
        const int m = km * 32 + (t >> 2) * 16 + (lane >> 4) * 4 + (t & 3);
        store_elem(sf + i, s1[((int64_t)h * M + m) * 16 + (lane & 15)]);
    }
}

// W3^T in out-product operand order [CK][CT][64][8]: lane l, slot t of K step
// kk holds W3[16*(2kk + (t>>2)) + 4*(l>>4) + (t&3)][zchan(ct, l & 15)], the
// row of head 2kk + (t>>2), head dimension 4*(l>>4) + (t&3) (dh = 16).
template <typename T>
__global__ void k_prep_w3f(const float *__restrict__ W3, int C, T *__restrict__ w3f) {
    const int CT = C / 16, CK = C / 32;
    const int64_t total = (int64_t)CK * CT * 64 * 8;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int t = (int)(i & 7), lane = (int)((i >> 3) & 63);
        const int64_t r = i >> 9;
        const int ct = (int)(r % CT), kk = (int)(r / CT);
        const int k = 16 * (2 * kk + (t >> 2)) + 4 * (lane >> 4) + (t & 3);
        store_elem(w3f + i, W3[(int64_t)k * C + zchan(ct, lane & 15)]);
    }
}

// One 16-point tile from global-memory operands with the max-shifted softmax
// (the fallback for blocks whose exp2 sums left the window).
template <int C, int M>
__device__ void deslice_tile_global_sf(const bf16_t *__restrict__ x, int64_t n, int64_t p0,
                                       const bf16_t *__restrict__ w2p, const float *__restrict__ b2s,
                                       const bf16_t *__restrict__ sf, const bf16_t *__restrict__ w3f,
                                       const float *__restrict__ b3, bf16_t *__restrict__ out, int lane) {
    using Cfg = Pass2SFCfg<C, M>;
    using T = bf16_t;
    constexpr int H = Cfg::H, CT = Cfg::CT, MT = Cfg::MT, CK = Cfg::CK, KM = Cfg::KM;
    const int li = lane & 15, g = lane >> 4;
    Frag<T> xb[1][CK];
    {
        const int64_t p = p0 + li;
#pragma unroll
        for (int kc = 0; kc < CK; ++kc) {
            if (p < n) load8(xb[0][kc], x + (size_t)p * C + kc * 32 + g * 8);
            else zero8(xb[0][kc]);
        }
    }
    Frag<T> ub[CK][1];
    f32x4 Uprev{0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
    for (int h = 0; h < H; ++h) {
        f32x4 L[MT][1];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const float4 bb = *reinterpret_cast<const float4 *>(b2s + h * M + mt * 16 + g * 4);
            L[mt][0] = f32x4{bb.x, bb.y, bb.z, bb.w};
#pragma unroll
            for (int kc = 0; kc < CK; ++kc) {
                Frag<T> a;
                load8(a, w2p + ((((size_t)h * MT + mt) * CK + kc) * 64 + lane) * 8);
                mma(L[mt][0], a, xb[0][kc]);
            }
        }
        Frag<T> wf[1][KM];
        softmax_shifted<T, MT, 1, KM>(L, wf);
        f32x4 U{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int km = 0; km < KM; ++km) {
            Frag<T> a;
            load8(a, sf + (((size_t)h * KM + km) * 64 + lane) * 8);
            mma(U, a, wf[0][km]);
        }
        if (h & 1) {
            Frag<T> f;
            f.set2(0, Uprev[0], Uprev[1]);
            f.set2(2, Uprev[2], Uprev[3]);
            f.set2(4, U[0], U[1]);
            f.set2(6, U[2], U[3]);
            // h is a loop variable: select the K step by value (CK <= 8)
#pragma unroll
            for (int kk = 0; kk < CK; ++kk)
                if (kk == (h >> 1)) ub[kk][0] = f;
        } else {
            Uprev = U;
        }
    }
    f32x4 O[CT][1];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
        const float4 bb = *reinterpret_cast<const float4 *>(b3 + zchan(ct, 4 * g));
        O[ct][0] = f32x4{bb.x, bb.y, bb.z, bb.w};
    }
#pragma unroll
    for (int kk = 0; kk < CK; ++kk)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            Frag<T> a;
            load8(a, w3f + (((size_t)kk * CT + ct) * 64 + lane) * 8);
            mma(O[ct][0], a, ub[kk][0]);
        }
    store_rows<T, CT, 1, C>(O, out, p0, n, g, li);
}

// x: [n][C] bf16; w2p: [H][MT][CK][64][8]; b2s: [H*M]; sf: [H][KM][64][8];
// w3f: [CK][CT][64][8]; b3: [C] float32; out: [n][C] bf16.  Grid: at most
// ceil(n / 256) persistent workgroups of 512 threads, each with at most
// P2_MAX_ITERS blocks.
template <int C, int M>
__global__ __launch_bounds__(512, 1) void k_deslice_sf(const bf16_t *__restrict__ x, int64_t n,
                                                       const bf16_t *__restrict__ w2p,
                                                       const float *__restrict__ b2s,
                                                       const bf16_t *__restrict__ sf,
                                                       const bf16_t *__restrict__ w3f,
                                                       const float *__restrict__ b3, bf16_t *__restrict__ out) {
    using Cfg = Pass2SFCfg<C, M>;
    using T = bf16_t;
    constexpr int H = Cfg::H, CT = Cfg::CT, MT = Cfg::MT, CK = Cfg::CK, KM = Cfg::KM, PT = Cfg::PT;
    constexpr int WAVES = Cfg::WAVES, NW3 = Cfg::NW3, AHEAD = Cfg::W3_AHEAD;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[Cfg::LDS_BYTES];
    const T *const sfl = reinterpret_cast<const T *>(lds + Cfg::SF_AT);
    float *const b2l = reinterpret_cast<float *>(lds + Cfg::B2_AT);
    float *const b3l = reinterpret_cast<float *>(lds + Cfg::B3_AT);

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int li = lane & 15, g = lane >> 4;
    const int64_t nblk = (n + Cfg::POINTS_PER_WG - 1) / Cfg::POINTS_PER_WG;
    if (n <= 0 || (int64_t)blockIdx.x >= nblk) return;  // uniform over the workgroup
    const int iters = (int)((nblk - 1 - blockIdx.x) / gridDim.x + 1);  // <= P2_MAX_ITERS (host)

    {   // resident operands: W2' by direct copies, the small ones through registers
        const unsigned char *src = reinterpret_cast<const unsigned char *>(w2p);
        for (int b = wave * 64; b < Cfg::W2_BYTES / 16; b += WAVES * 64)
            dma16(src + (b + lane) * 16, lds_addr(lds + Cfg::W2_AT + b * 16));
        const uint4 *s4 = reinterpret_cast<const uint4 *>(sf);
        uint4 *d4 = reinterpret_cast<uint4 *>(lds + Cfg::SF_AT);
        for (int i = threadIdx.x; i < Cfg::SF_BYTES / 16; i += 64 * WAVES) d4[i] = s4[i];
        for (int i = threadIdx.x; i < H * M; i += 64 * WAVES) b2l[i] = b2s[i];
        for (int i = threadIdx.x; i < C; i += 64 * WAVES) b3l[i] = b3[i];
    }

    // Fragment j = (pt, kc) of the B operand x^T of the wave block at p0: lane
    // (g, li) holds x[p0 + 16*pt + li][32*kc + 8*g .. +8]; rows past the end
    // read the last row (finite data whose outputs are never stored).
    auto load_xfrag = [&](int64_t p0, int j, Frag<T> (&xf)[PT][CK]) {
        const int pt = j / CK, kc = j % CK;
        const int64_t p = p0 + pt * 16 + li;
        const int64_t pc = p < n ? p : n - 1;
        load8(xf[pt][kc], x + (size_t)pc * C + kc * 32 + g * 8);
    };
    const int64_t pw = (int64_t)blockIdx.x * Cfg::POINTS_PER_WG + wave * (16 * PT);
    const int64_t bstride = (int64_t)gridDim.x * Cfg::POINTS_PER_WG;
    Frag<T> xb[PT][CK];
#pragma unroll
    for (int j = 0; j < Cfg::NXLOAD; ++j) load_xfrag(pw, j, xb);
    // The first block's x is waited for here, where the compiler sees it:
    // otherwise its wait for these loads would sit at the top of the block
    // loop and hold every later block until the previous block's stores retire.
#pragma unroll
    for (int pt = 0; pt < PT; ++pt)
#pragma unroll
        for (int kc = 0; kc < CK; ++kc) asm volatile("" : "+v"(xb[pt][kc].v));
    wait_vmcnt<0>();  // this wave's direct copies (the compiler does not count them)
    __syncthreads();  // every wave's copies and LDS stores visible
    uint64_t failed = 0;  // bit i: block i left the fast path
    f32x4 O[CT][PT];
    Frag<T> ones;
    ones8(ones);

    for (int i = 0; i < iters; ++i) {
        const int64_t p0 = pw + (int64_t)i * bstride;
        bool ok = true;
        Frag<T> ub[CK][PT];  // u of head pairs: the B fragments of the Linear3 product
        f32x4 Uprev[PT];
#pragma unroll
        for (int h = 0; h < H; ++h) {
            f32x4 L[MT][PT];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const f32x4 b = *reinterpret_cast<const f32x4 *>(b2l + h * M + mt * 16 + g * 4);
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) L[mt][pt] = b;
            }
            Frag<T> sa[KM];
#pragma unroll
            for (int km = 0; km < KM; ++km) sa[km].v = *reinterpret_cast<const bf16x8 *>(sfl + ((h * KM + km) * 64 + lane) * 8);
            // Slice tiles outermost: the exp2 of tile mt-1 rides between tile
            // mt's MFMAs; the W2' fragment of step i+2 is read while step i's
            // MFMAs run.
            auto exp_at = [&](int mt, int e) {
                const int pt = e / 4, r = e % 4;
                float v = fast_exp2(L[mt][pt][r]);
                asm volatile("" : "+v"(v));
                L[mt][pt][r] = v;
            };
            {
                constexpr int NSTEP = MT * CK, DIST = 2, EPS = (4 * PT) / CK;
                static_assert((4 * PT) % CK == 0, "exp2 spread evenly over a tile's K steps");
                // The head's fragments from one base register plus immediate
                // offsets; the base is opaque to the compiler, which would
                // otherwise hold one address register per fragment of the launch.
                uint32_t hoff = (uint32_t)(h * MT * CK * 1024 + lane * 16);
                asm volatile("" : "+v"(hoff));
                auto w2frag = [&](int s, Frag<T> &f) {
                    f.v = *reinterpret_cast<const bf16x8 *>(lds + Cfg::W2_AT + hoff + s * 1024);
                };
                Frag<T> a[4];
#pragma unroll
                for (int s = 0; s < DIST; ++s) w2frag(s, a[s]);
#pragma unroll
                for (int s = 0; s < NSTEP; ++s) {
                    const int mt = s / CK, kc = s % CK;
                    __builtin_amdgcn_sched_barrier(0);
                    if (s + DIST < NSTEP) w2frag(s + DIST, a[(s + DIST) & 3]);
#pragma unroll
                    for (int pt = 0; pt < PT; ++pt) mma(L[mt][pt], a[s & 3], xb[pt][kc]);
                    if (mt > 0)
#pragma unroll
                        for (int e = kc * EPS; e < (kc + 1) * EPS; ++e) exp_at(mt - 1, e);
                    if (s + DIST < NSTEP) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
#pragma unroll
                    for (int q = 0; q < PT || q < EPS; ++q) {
                        if (q < PT) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                        if (mt > 0 && q < EPS) __builtin_amdgcn_sched_group_barrier(0x400, 1, 0);
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int e = 0; e < 4 * PT; ++e) exp_at(MT - 1, e);
            }
            // The unnormalised exp2 terms e go into the products: u_h is
            // linear in the weights, so u_h = (s'_h^T e) / sum(e), and the row
            // sums come from the same products with an all-ones A operand
            // (every output row of that tile is the sum over the slices).
            // Both sums use the same bf16-rounded e, so the weights that u
            // averages with sum to one exactly.
            Frag<T> wf[PT][KM];
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) pack_weights<T, MT, PT, KM>(L, pt, 1.0f, wf);
            bool okk = true;
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) {
                f32x4 U{0.f, 0.f, 0.f, 0.f}, S{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int km = 0; km < KM; ++km) {
                    mma(U, sa[km], wf[pt][km]);
                    mma(S, ones, wf[pt][km]);
                }
                okk = okk && softmax_sum_ok(S[0]);
                const float inv = fast_rcp(S[0]);
#pragma unroll
                for (int r = 0; r < 4; ++r) U[r] *= inv;
                if (h & 1) {
                    ub[h >> 1][pt].set2(0, Uprev[pt][0], Uprev[pt][1]);
                    ub[h >> 1][pt].set2(2, Uprev[pt][2], Uprev[pt][3]);
                    ub[h >> 1][pt].set2(4, U[0], U[1]);
                    ub[h >> 1][pt].set2(6, U[2], U[3]);
                } else {
                    Uprev[pt] = U;
                }
            }
            ok = !__any(!okk) && ok;
        }
        // out = b3 + u W3: W3^T fragments streamed from global memory (L2),
        // K steps outermost so that consecutive MFMAs are independent.
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            const f32x4 b = *reinterpret_cast<const f32x4 *>(b3l + zchan(ct, 4 * g));
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) O[ct][pt] = b;
        }
        {
            // the kernel argument as the scalar base plus a 32-bit offset, so
            // the loads need no per-fragment 64-bit address registers
            // AHEAD fragments in flight, and the next block's x issued right
            // after the last fragment, so that no fragment's wait covers it
            // (in the last block x is reloaded anyway, clamped rows).  Each
            // load is the scalar base (the kernel argument) plus a 32-bit
            // lane offset plus an immediate, four fragments per offset.
            const unsigned char *w3b = reinterpret_cast<const unsigned char *>(w3f);
            const uint32_t voff = (uint32_t)lane * 16u;
            auto w3frag = [&](int q, Frag<T> &f) {
                f.v = *reinterpret_cast<const bf16x8 *>(w3b + (uint32_t)(voff + 4096u * (q / 4)) + (q % 4) * 1024);
            };
            Frag<T> a[AHEAD];
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int q = 0; q < AHEAD; ++q) w3frag(q, a[q]);
            static_for<0, NW3>([&](auto qc) {
                constexpr int q = decltype(qc)::value, kk = q / CT, ct = q % CT;
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) mma(O[ct][pt], a[q % AHEAD], ub[kk][pt]);
                __builtin_amdgcn_sched_barrier(0);
                if constexpr (q + AHEAD < NW3) w3frag(q + AHEAD, a[q % AHEAD]);
                if constexpr (q + AHEAD == NW3 - 1) {
#pragma unroll
                    for (int j = 0; j < Cfg::NXLOAD; ++j) load_xfrag(p0 + bstride, j, xb);
                }
                __builtin_amdgcn_sched_barrier(0);
            });
        }
        if (!ok) failed |= 1ull << i;
        // The same stores for every block (one path through the loop, so the
        // compiler's waits at its top need not allow for a block without
        // them): a row past the end computed the last row's x, so it writes
        // the last row's values to the last row.  A block that left the fast
        // path is rewritten below.
#pragma unroll
        for (int k = 0; k < CT / 2; ++k)
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) {
                const f32x4 &u = O[2 * k][pt], &v = O[2 * k + 1][pt];
                const int64_t p = p0 + pt * 16 + li;
                *reinterpret_cast<bf16x8 *>(out + (size_t)(p < n ? p : n - 1) * C + 32 * k + 8 * g) =
                    bf16x8{(__bf16)u[0], (__bf16)u[1], (__bf16)u[2], (__bf16)u[3],
                           (__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
            }
    }
    // Rare: blocks whose exp2 sums left the safe window, redone from
    // global-memory operands with the max-shifted softmax, 16 points at a time.
    while (failed) {
        const int i = __builtin_ctzll(failed);
        failed &= failed - 1;
#pragma unroll 1
        for (int pt = 0; pt < PT; ++pt)
            deslice_tile_global_sf<C, M>(x, n, pw + (int64_t)i * bstride + 16 * pt, w2p, b2s, sf, w3f, b3, out,
                                         lane);
    }
}

}  // namespace ts3
