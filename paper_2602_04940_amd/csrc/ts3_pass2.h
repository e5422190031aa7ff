// Pass 2 of the Physics-Attention layer: full-mesh decoding against the cached
// state (paper Eq. (5), Algorithm 1 deslice loop).  The slice weights are
// recomputed from x and never stored:
//     out[p] = sum_h sum_m softmax_m(L_h[p]) Z[h][m][:] + b3.
//
// A wave decodes a block of 16*PT points over all heads, so the sum over heads
// stays in its accumulator registers.  Per head:
//   logits  L[m][p] = W2'[:, h*M+m] . x[p] + b2'  16x16x32 MFMA with A = W2'^T
//           fragments, B = x^T (the wave's point rows, loaded once per block).
//           Output lane (g, p) holds slices 4g+r of each 16-slice tile, so the
//           softmax over m is an in-lane pass plus two cross-row swaps.
//   deslice out[c][p] += Z[h]^T[c][m] . w[m][p]: A = prepared Z fragments
//           whose K slots follow the logits' register order, B = w straight
//           from registers.
// Output channels: row i of channel tile ct of the Z fragments is channel
// zchan(ct, i), so that output lane (g, p) of tiles 2k and 2k+1 holds the
// eight consecutive channels 32k + 8g .. +7 of point p (one 16-byte store).
#pragma once
#include <type_traits>

#include "ts3_device.h"

namespace ts3 {

__host__ __device__ __forceinline__ int zchan(int ct, int i) {
    return 32 * (ct >> 1) + 8 * (i >> 2) + 4 * (ct & 1) + (i & 3);
}

// Softmax over one head's M slices for the wave's points, logits laid out
// [slices x points] (lane (g, p) holds slices 16*mt + 4*g + r of point p):
// w is written as the B operand of the deslice contraction, K slot (g, t) of
// step km holding slice 32*km + 16*(t>>2) + 4*g + (t&3).
template <typename T, int MT, int PT, int KM>
__device__ __forceinline__ void pack_weights(const f32x4 (&E)[MT][PT], int pt, float inv, Frag<T> (&wf)[PT][KM]) {
#pragma unroll
    for (int km = 0; km < KM; ++km)
#pragma unroll
        for (int t = 0; t < 8; t += 2) {
            const int mt = 2 * km + (t >> 2);
            if (mt < MT)
                wf[pt][km].set2(t, E[mt][pt][t & 3] * inv, E[mt][pt][(t & 3) + 1] * inv);
            else
                wf[pt][km].set2(t, 0.f, 0.f);
        }
}

template <typename T, int MT, int PT, int KM>
__device__ __forceinline__ void softmax_shifted(f32x4 (&L)[MT][PT], Frag<T> (&wf)[PT][KM]) {
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
                const float e = fast_exp2(L[mt][pt][r] - mx);
                L[mt][pt][r] = e;
                sum += e;
            }
        pack_weights<T, MT, PT, KM>(L, pt, fast_rcp(xrow_sum(sum)), wf);
    }
}

// out rows of one wave block (b3 is folded into the prepared Z): lane (g, li)
// writes channels 32k + 8g .. +7 of point p0 + 16*pt + li from tiles 2k and 2k+1.
template <typename T, int CT, int PT, int C>
__device__ __forceinline__ void store_rows(const f32x4 (&O)[CT][PT], T *__restrict__ out, int64_t p0, int64_t n,
                                           int g, int li) {
#pragma unroll
    for (int k = 0; k < CT / 2; ++k) {
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) {
            const int64_t p = p0 + pt * 16 + li;
            if (p >= n) continue;
            const f32x4 &u = O[2 * k][pt], &v = O[2 * k + 1][pt];
            T *dst = out + (size_t)p * C + 32 * k + 8 * g;
            if constexpr (sizeof(T) == 2) {
                *reinterpret_cast<bf16x8 *>(dst) = bf16x8{(__bf16)u[0], (__bf16)u[1], (__bf16)u[2], (__bf16)u[3],
                                                          (__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
            } else {
                reinterpret_cast<float4 *>(dst)[0] = float4{u[0], u[1], u[2], u[3]};
                reinterpret_cast<float4 *>(dst)[1] = float4{v[0], v[1], v[2], v[3]};
            }
        }
    }
}

// One wave block decoded from global-memory fragments with the max-shifted
// softmax: the generic kernel's body, and the rare fallback of the staged one.
template <typename T, int C, int M, int PT>
__device__ void deslice_block_global(const T *__restrict__ x, int64_t n, int64_t p0, int32_t H,
                                     const T *__restrict__ w2p, const float *__restrict__ b2s,
                                     const T *__restrict__ zp, T *__restrict__ out, int lane) {
    constexpr int CT = C / 16, MT = M / 16, CK = C / 32, KM = M >= 32 ? M / 32 : 1;
    const int li = lane & 15, g = lane >> 4;
    // B operand x^T: lane (g, li) holds x[p0 + 16*pt + li][32*kc + 8*g .. +8].
    Frag<T> xb[PT][CK];
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) {
        const int64_t p = p0 + pt * 16 + li;
#pragma unroll
        for (int kc = 0; kc < CK; ++kc) {
            if (p < n)
                load8(xb[pt][kc], x + (size_t)p * C + kc * 32 + g * 8);
            else
                zero8(xb[pt][kc]);
        }
    }
    f32x4 O[CT][PT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) O[ct][pt] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int h = 0; h < H; ++h) {
        f32x4 L[MT][PT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const float4 bb = *reinterpret_cast<const float4 *>(b2s + h * M + mt * 16 + g * 4);
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) L[mt][pt] = f32x4{bb.x, bb.y, bb.z, bb.w};
#pragma unroll
            for (int kc = 0; kc < CK; ++kc) {
                Frag<T> a;
                load8(a, w2p + ((((size_t)h * MT + mt) * CK + kc) * 64 + lane) * 8);
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) mma(L[mt][pt], a, xb[pt][kc]);
            }
        }
        Frag<T> wf[PT][KM];
        softmax_shifted<T, MT, PT, KM>(L, wf);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int km = 0; km < KM; ++km) {
                Frag<T> a;
                load8(a, zp + ((((size_t)h * CT + ct) * KM + km) * 64 + lane) * 8);
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) mma(O[ct][pt], a, wf[pt][km]);
            }
    }
    store_rows<T, CT, PT, C>(O, out, p0, n, g, li);
}

template <typename T, int C, int M> struct Pass2Cfg {
    static constexpr int PT = sizeof(T) == 2 ? 4 : 2;  // 16-point tiles per wave block
    static constexpr int WAVES = 4;
    static constexpr int POINTS_PER_WG = WAVES * 16 * PT;
};

// Generic decoding kernel (fp32 storage, and shapes whose weights do not fit
// the staged kernel's LDS): every fragment comes from global memory.
// x   : [n][C] storage elements; out: [n][C]
// w2p : prepared W2' fragments [H][MT][CK][64][8] (also the A = W2'^T layout)
// b2s : scaled bias [H*M]
// zp  : prepared Z fragments [H][CT][KM][64][8], b3/H folded in
template <typename T, int C, int M>
__global__ __launch_bounds__(256, 1) void k_deslice(const T *__restrict__ x, int64_t n, int32_t H,
                                                    const T *__restrict__ w2p,
                                                    const float *__restrict__ b2s,
                                                    const T *__restrict__ zp, T *__restrict__ out) {
    using Cfg = Pass2Cfg<T, C, M>;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t p0 = ((int64_t)blockIdx.x * Cfg::WAVES + wave) * (16 * Cfg::PT);
    if (p0 >= n) return;
    deslice_block_global<T, C, M, Cfg::PT>(x, n, p0, H, w2p, b2s, zp, out, lane);
}

// Staged decoding kernel for 16-bit storage: eight waves (two per SIMD, so one
// wave's vector-ALU work issues while the other waits) of 32 points each.
// LDS holds every head's W2' fragments (H*M*C elements, 128 KB for C=128,
// H*M=512) and two Z stages of one head each; head h+1's Z is copied by the
// workgroup (direct global->LDS) while head h is decoded, so each head costs
// one barrier.  The bias b2' of head h+1 is loaded into registers during head
// h, and the next block's x is loaded during the current block, a fragment or
// two per head into a second register set, so no block boundary waits on
// memory.  Persistent workgroups stride over 256-point blocks (at most
// P2_MAX_ITERS per launch); every wave runs every block and barrier (tail
// points are masked), so barriers never diverge.  A block whose softmax left
// the unshifted path's safe window is stored anyway and redone after the main
// loop (recorded in a wave-uniform bit mask), which keeps the slow path's
// registers out of the main loop.
constexpr int P2_MAX_ITERS = 64;

template <typename T, int C, int M> struct Pass2W8Cfg {
    static constexpr int CT = C / 16, MT = M / 16, CK = C / 32, KM = M >= 32 ? M / 32 : 1;
    static constexpr int WAVES = 8;
    static constexpr int PT = 2;
    static constexpr int POINTS_PER_WG = WAVES * 16 * PT;
    static constexpr int ZFRAGS = CT * KM;           // 1 KB fragments per head
    static constexpr int STAGE_ELEMS = ZFRAGS * 512;
    static constexpr int NSTORE = (CT / 2) * PT;     // output stores per full wave block
    static constexpr int NXLOAD = PT * CK;           // x loads per wave block
    static size_t lds_bytes(int H) {
        return ((size_t)H * MT * CK * 512 + 2 * (size_t)STAGE_ELEMS) * sizeof(T);
    }
};

template <typename T, int C, int M>
__global__ __launch_bounds__(512, 1) void k_deslice_w8(const T *__restrict__ x, int64_t n, int32_t H,
                                                       const T *__restrict__ w2p,
                                                       const float *__restrict__ b2s,
                                                       const T *__restrict__ zp, T *__restrict__ out) {
    static_assert(sizeof(T) == 2, "the staged decoder is written for 16-bit storage");
    using Cfg = Pass2W8Cfg<T, C, M>;
    constexpr int CT = Cfg::CT, MT = Cfg::MT, CK = Cfg::CK, KM = Cfg::KM, PT = Cfg::PT;
    constexpr int ZFRAGS = Cfg::ZFRAGS, WAVES = Cfg::WAVES, NSTORE = Cfg::NSTORE, NXLOAD = Cfg::NXLOAD;
    extern __shared__ __attribute__((aligned(1024))) unsigned char lds_raw[];
    T *const w2l = reinterpret_cast<T *>(lds_raw);
    T *const zs = w2l + (size_t)H * MT * CK * 512;  // two stages of STAGE_ELEMS
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int li = lane & 15;
    const int g = lane >> 4;
    const int64_t nblk = (n + Cfg::POINTS_PER_WG - 1) / Cfg::POINTS_PER_WG;
    if (n <= 0 || H <= 0 || (int64_t)blockIdx.x >= nblk) return;  // uniform over the workgroup
    const int iters = (int)((nblk - 1 - blockIdx.x) / gridDim.x + 1);  // <= P2_MAX_ITERS (host)

    {   // every head's W2' fragments, once: direct copies, all in flight
        const int64_t total16 = (int64_t)H * MT * CK * 64;  // 16-byte pieces (a multiple of 64)
        const unsigned char *src = reinterpret_cast<const unsigned char *>(w2p);
        for (int64_t b = (int64_t)wave * 64; b < total16; b += WAVES * 64)
            dma16(src + (b + lane) * 16, lds_addr(lds_raw + b * 16));
    }

    // Head h's Z fragments into stage s: wave w copies fragments w, w+8, ...
    // (a wave-uniform count of copies).
    auto stage_z = [&](int h, int s) {
        T *dst = zs + (size_t)s * Cfg::STAGE_ELEMS;
        for (int f = wave; f < ZFRAGS; f += WAVES)
            dma16(zp + ((size_t)h * ZFRAGS + f) * 512 + lane * 8, lds_addr(dst + f * 512));
    };
    auto load_bias = [&](int h, f32x4 (&b)[MT]) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const float4 v = *reinterpret_cast<const float4 *>(b2s + h * M + mt * 16 + g * 4);
            b[mt] = f32x4{v.x, v.y, v.z, v.w};
        }
    };
    // Fragment j = (pt, kc) of the B operand x^T of the wave block at p0: lane
    // (g, li) holds x[p0 + 16*pt + li][32*kc + 8*g .. +8].  Rows past the end
    // read the last row (finite data; a point's outputs depend only on its own
    // row, and padding rows are never stored).
    auto load_xfrag = [&](int64_t p0, int j, Frag<T> (&xf)[PT][CK]) {
        const int pt = j / CK, kc = j % CK;
        const int64_t p = p0 + pt * 16 + li;
        const int64_t pc = p < n ? p : n - 1;
        load8(xf[pt][kc], x + (size_t)pc * C + kc * 32 + g * 8);
    };
    // The next block's x fragments are spread over heads 0..H-2 (all at head 0
    // when H == 1): fragment j goes with head xhead(j).
    auto xhead = [&](int j) { return H > 1 ? j * (H - 1) / NXLOAD : 0; };

    const int64_t pw = (int64_t)blockIdx.x * Cfg::POINTS_PER_WG + wave * (16 * PT);
    const int64_t bstride = (int64_t)gridDim.x * Cfg::POINTS_PER_WG;
    Frag<T> xA[PT][CK], xB[PT][CK];
    f32x4 bias[MT];
#pragma unroll
    for (int j = 0; j < NXLOAD; ++j) load_xfrag(pw, j, xA);
    load_bias(0, bias);
    stage_z(0, 0);
    wait_vmcnt<0>();
    int stage = 0;
    uint64_t failed = 0;  // bit i: block i left the fast path
    f32x4 O[CT][PT];
    // Block i with its x in xb; the next block's x goes to xn.  Returns false
    // after the workgroup's last block (left unstored).  The two register
    // sets swap roles from block to block (the loop below is unrolled by
    // two), so no copy writes over the registers that the stores read.
    auto block = [&](int i, Frag<T> (&xb)[PT][CK], Frag<T> (&xn)[PT][CK]) -> bool {
        const int64_t p0 = pw + (int64_t)i * bstride;
        const bool has_next = i + 1 < iters;
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) O[ct][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
        bool ok = true;
        // One head of the block.  Head 0 is a separate call, so that the
        // compiler's wait analysis sees the block start on its own: there the
        // bias and the Z copies were retired before the previous block's
        // stores, which stay in flight; at later heads this wave's Z_h copies
        // and bias (issued during head h-1) are waited for here.
        auto head = [&](int h, auto first) {
            if constexpr (decltype(first)::value) wait_vmcnt<NSTORE>();
            else wait_vmcnt<0>();
            __syncthreads();  // every copy of Z_h landed; stage s^1 is no longer read
            f32x4 L[MT][PT];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) L[mt][pt] = bias[mt];
            const int cur = stage;
            // Slice tiles outermost: the exp2 of tile mt-1 (and their running
            // row sums) ride between tile mt's MFMAs, where the transcendental
            // unit runs beside the matrix core; the W2' fragment of step i+2
            // is read while step i's MFMAs run.  The sums keep the order
            // tile, then r, of the plain softmax.
            float esum[PT];
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) esum[pt] = 0.f;
            auto exp_at = [&](int mt, int e) {
                const int pt = e / 4, r = e % 4;
                float v = fast_exp2(L[mt][pt][r]);
                asm volatile("" : "+v"(v));
                L[mt][pt][r] = v;
                esum[pt] += v;
            };
            {
                constexpr int NSTEP = MT * CK, DIST = 2, EPS = (4 * PT) / CK;
                static_assert((4 * PT) % CK == 0, "exp2 spread evenly over a tile's K steps");
                const T *wh = w2l + (size_t)h * MT * CK * 512 + lane * 8;
                Frag<T> a[4];
#pragma unroll
                for (int i = 0; i < DIST; ++i) load8(a[i], wh + i * 512);
#pragma unroll
                for (int i = 0; i < NSTEP; ++i) {
                    const int mt = i / CK, kc = i % CK;
                    __builtin_amdgcn_sched_barrier(0);
                    if (i + DIST < NSTEP) load8(a[(i + DIST) & 3], wh + (i + DIST) * 512);
#pragma unroll
                    for (int pt = 0; pt < PT; ++pt) mma(L[mt][pt], a[i & 3], xb[pt][kc]);
                    if (mt > 0)
#pragma unroll
                        for (int e = kc * EPS; e < (kc + 1) * EPS; ++e) exp_at(mt - 1, e);
                    if (i + DIST < NSTEP) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
#pragma unroll
                    for (int q = 0; q < PT || q < EPS; ++q) {
                        if (q < PT) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                        if (mt > 0 && q < EPS) __builtin_amdgcn_sched_group_barrier(0x400, 1, 0);
                    }
                    // This head's share of the next block's x, after the first tile.
                    if (i == CK - 1 && has_next) {
                        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                        for (int j = 0; j < NXLOAD; ++j)
                            if (xhead(j) == h) load_xfrag(p0 + bstride, j, xn);
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int e = 0; e < 4 * PT; ++e) exp_at(MT - 1, e);
            }
            // The next head's Z copies and bias (or head 0's of the next
            // block), after the logits rather than at the barrier, where every
            // wave would queue them at once.
            if (h + 1 < H || has_next) {
                const int hn = h + 1 < H ? h + 1 : 0;
                stage_z(hn, stage ^ 1);
                load_bias(hn, bias);
                stage ^= 1;
            }
            Frag<T> wf[PT][KM];
            {   // the rest of the fast-path softmax: row sums across the four rows
                bool okk = true;
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) {
                    const float sm = xrow_sum(esum[pt]);
                    okk = okk && softmax_sum_ok(sm);
                    pack_weights<T, MT, PT, KM>(L, pt, fast_rcp(sm), wf);
                }
                ok = !__any(!okk) && ok;
            }
            // Decode with the K steps outermost: the MFMAs into one output
            // accumulator are CT steps apart, so the matrix core always has
            // independent work (on gfx950 an MFMA that depends on the one
            // before it issues at half rate); the Z fragment of step q+2 is
            // read while step q's MFMAs run.
            {
                const T *zl = zs + (size_t)cur * Cfg::STAGE_ELEMS + lane * 8;
                constexpr int NQ = KM * CT, DZ = 2;
                auto zfrag = [&](int q) { return zl + ((q % CT) * KM + q / CT) * 512; };
                Frag<T> a[4];
#pragma unroll
                for (int q = 0; q < DZ; ++q) load8(a[q], zfrag(q));
#pragma unroll
                for (int q = 0; q < NQ; ++q) {
                    const int km = q / CT, ct = q % CT;
                    __builtin_amdgcn_sched_barrier(0);
                    if (q + DZ < NQ) load8(a[(q + DZ) & 3], zfrag(q + DZ));
#pragma unroll
                    for (int pt = 0; pt < PT; ++pt) mma(O[ct][pt], a[q & 3], wf[pt][km]);
                    if (q + DZ < NQ) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, PT, 0);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        head(0, std::true_type{});
        for (int h = 1; h < H; ++h) head(h, std::false_type{});
        if (!ok) failed |= 1ull << i;
        if (!has_next) return false;
        // Next block's x, its first Z copies and its first bias have all had
        // at least part of a head to arrive; with them retired before the
        // stores, nothing later has to wait for the stores.
        wait_vmcnt<0>();
        // Every block but a workgroup's last is full: exactly NSTORE stores,
        // unconditionally (a failed block is rewritten below).
#pragma unroll
        for (int k = 0; k < CT / 2; ++k)
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) {
                const f32x4 &u = O[2 * k][pt], &v = O[2 * k + 1][pt];
                *reinterpret_cast<bf16x8 *>(out + (size_t)(p0 + pt * 16 + li) * C + 32 * k + 8 * g) =
                    bf16x8{(__bf16)u[0], (__bf16)u[1], (__bf16)u[2], (__bf16)u[3],
                           (__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
            }
        return true;
    };
    for (int i = 0;; i += 2) {
        if (!block(i, xA, xB)) break;
        if (!block(i + 1, xB, xA)) break;
    }
    // The workgroup's last block (possibly partial): masked stores.
    if (!((failed >> (iters - 1)) & 1)) store_rows<T, CT, PT, C>(O, out, pw + (int64_t)(iters - 1) * bstride, n, g, li);
    wait_vmcnt<0>();
    // Rare: blocks whose exp2 sums left the safe window, redone from
    // global-memory fragments with the max-shifted softmax, 16 points at a
    // time (no barriers).
    while (failed) {
        const int i = __builtin_ctzll(failed);
        failed &= failed - 1;
#pragma unroll 1
        for (int pt = 0; pt < PT; ++pt)
            deslice_block_global<T, C, M, 1>(x, n, pw + (int64_t)i * bstride + 16 * pt, H, w2p, b2s, zp, out, lane);
    }
}

}  // namespace ts3
