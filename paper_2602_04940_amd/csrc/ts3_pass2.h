// Pass 2 of the Physics-Attention layer: full-mesh decoding against the cached
// state (paper Eq. (5), Algorithm 1 deslice loop).  The slice weights are
// recomputed from x and never stored:
//     out[p] = sum_h sum_m softmax_m(L_h[p]) Z[h][m][:] + b3.
//
// Work decomposition: each wave decodes a block of 16*PT points over all
// heads, so the sum over heads stays in its accumulator registers.
// Per head:
//   logits  L[m][p] = W2'[:, h*M+m] . x[p] + b2'  16x16x32 MFMA with A = W2'^T
//           fragments, B = x^T (the wave's point rows, loaded once per block).
//           Output lane (g, p) holds slices 4g+r of each 16-slice tile, so the
//           softmax over m is an in-lane pass plus two cross-row swaps.
//   deslice out[c][p] += Z[h]^T[c][m] . w[m][p]: A = prepared Z fragments
//           whose K slots follow the logits' register order, B = w straight
//           from registers.
#pragma once
#include <type_traits>

#include "ts3_device.h"

namespace ts3 {

template <typename T, int C, int M> struct Pass2Cfg {
    static constexpr int CT = C / 16;
    static constexpr int MT = M / 16;
    static constexpr int CK = C / 32;
    static constexpr int KM = M >= 32 ? M / 32 : 1;  // K32 steps over slices (M=16 pads half a step)
    static constexpr int PT = sizeof(T) == 2 ? 4 : 2;  // 16-point tiles per wave block
    static constexpr int WAVES = 4;
    static constexpr int POINTS_PER_WG = WAVES * 16 * PT;
};

// x   : [n][C] storage elements; out: [n][C]
// w2p : prepared W2' fragments [H][MT][CK][64][8] (also the A = W2'^T layout)
// b2s : scaled bias [H*M]
// zp  : prepared Z fragments [H][CT][KM][64][8]
// b3  : [C] float32
template <typename T, int C, int M>
__global__ __launch_bounds__(256, 1) void k_deslice(const T *__restrict__ x, int64_t n, int32_t H,
                                                    const T *__restrict__ w2p,
                                                    const float *__restrict__ b2s,
                                                    const T *__restrict__ zp,
                                                    const float *__restrict__ b3, T *__restrict__ out) {
    using Cfg = Pass2Cfg<T, C, M>;
    constexpr int CT = Cfg::CT, MT = Cfg::MT, CK = Cfg::CK, KM = Cfg::KM, PT = Cfg::PT;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int li = lane & 15;
    const int g = lane >> 4;
    const int64_t p0 = ((int64_t)blockIdx.x * Cfg::WAVES + wave) * (16 * PT);
    if (p0 >= n) return;

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

        // Softmax over the head's M slices for point 16*pt + li.
        Frag<T> wf[PT][KM];
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
            const float inv = fast_rcp(xrow_sum(sum));
#pragma unroll
            for (int km = 0; km < KM; ++km)
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    const int mt = 2 * km + (t >> 2);
                    wf[pt][km].set(t, mt < MT ? L[mt][pt][t & 3] * inv : 0.f);
                }
        }

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

    // Store: lane (g, li) holds out[p0 + 16*pt + li][16*ct + 4*g + r].
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
        const float4 bb = *reinterpret_cast<const float4 *>(b3 + ct * 16 + g * 4);
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) {
            const int64_t p = p0 + pt * 16 + li;
            if (p >= n) continue;
            const float v0 = O[ct][pt][0] + bb.x, v1 = O[ct][pt][1] + bb.y;
            const float v2 = O[ct][pt][2] + bb.z, v3 = O[ct][pt][3] + bb.w;
            T *dst = out + (size_t)p * C + ct * 16 + g * 4;
            if constexpr (sizeof(T) == 2) {
                typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
                *reinterpret_cast<bf16x4 *>(dst) = bf16x4{(__bf16)v0, (__bf16)v1, (__bf16)v2, (__bf16)v3};
            } else {
                *reinterpret_cast<float4 *>(dst) = float4{v0, v1, v2, v3};
            }
        }
    }
}

}  // namespace ts3

namespace ts3 {

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

// Fast path: exp2 of the logits without a shift.  Returns false (wave-uniform)
// if any row's sum falls outside the safe window; L then holds exp2 values.
template <typename T, int MT, int PT, int KM>
__device__ __forceinline__ bool softmax_unshifted(f32x4 (&L)[MT][PT], Frag<T> (&wf)[PT][KM]) {
    bool ok = true;
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) {
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
        pack_weights<T, MT, PT, KM>(L, pt, fast_rcp(sum), wf);
    }
    return !__any(!ok);
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

// Pass 2 with the prepared W2' fragments of every head and the scaled bias
// resident in LDS (H*M*C storage elements + H*M floats; 130 KB for C=128,
// H*M=512 in bf16), and each head's Z fragments (16 KB) staged into LDS with
// direct global->LDS loads shared by the workgroup's four waves.  Persistent
// workgroups stride over 256-point blocks (64 per wave, 1 wave per SIMD).
// Per head h: [barrier; stage Z_h] [logits_h] [softmax_h] [barrier]
// [deslice_h].  Every wave runs every block and barrier (tail points are
// masked), so barriers never diverge.
template <typename T, int C, int M> struct Pass2LdsCfg {
    using Base = Pass2Cfg<T, C, M>;
    static constexpr int ZFRAGS = Base::CT * Base::KM;            // 1 KB fragments per head
    static constexpr int Z_STAGE_ELEMS = ZFRAGS * 64 * 8;
    static_assert(ZFRAGS % 4 == 0, "Z fragments split evenly over four waves");
    static size_t lds_bytes(int H) {
        return (size_t)H * Base::MT * Base::CK * 512 * sizeof(T) + (size_t)H * M * 4 +
               (size_t)Z_STAGE_ELEMS * sizeof(T);
    }
};

template <typename T, int C, int M>
__global__ __launch_bounds__(256, 1) void k_deslice_lds(const T *__restrict__ x, int64_t n, int32_t H,
                                                        const T *__restrict__ w2p,
                                                        const float *__restrict__ b2s,
                                                        const T *__restrict__ zp,
                                                        const float *__restrict__ b3, T *__restrict__ out) {
    using Cfg = Pass2Cfg<T, C, M>;
    using LCfg = Pass2LdsCfg<T, C, M>;
    constexpr int CT = Cfg::CT, MT = Cfg::MT, CK = Cfg::CK, KM = Cfg::KM, PT = Cfg::PT;
    constexpr int ZFRAGS = LCfg::ZFRAGS;
    extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];
    T *w2l = reinterpret_cast<T *>(lds_raw);
    const int64_t w2_elems = (int64_t)H * MT * CK * 64 * 8;
    float *b2l = reinterpret_cast<float *>(w2l + w2_elems);
    T *zl = reinterpret_cast<T *>(b2l + H * M);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int li = lane & 15;
    const int g = lane >> 4;

    {   // stage every head's W2' fragments and the scaled bias once
        const int64_t total16 = w2_elems * (int64_t)sizeof(T) / 16;
        const uint4 *src = reinterpret_cast<const uint4 *>(w2p);
        uint4 *dst = reinterpret_cast<uint4 *>(w2l);
        for (int64_t i = threadIdx.x; i < total16; i += 256) dst[i] = src[i];
        for (int i = threadIdx.x; i < H * M; i += 256) b2l[i] = b2s[i];
    }
    __syncthreads();

    // Wave w copies Z fragments w, w+4, ... of head h into the stage (1 KB each).
    auto stage_z = [&](int h) {
#pragma unroll
        for (int i = 0; i < ZFRAGS / 4; ++i) {
            const int f = wave + 4 * i;
            __builtin_amdgcn_global_load_lds(
                (const void *)(zp + ((size_t)h * ZFRAGS + f) * 512 + lane * 8),
                (__attribute__((address_space(3))) void *)(zl + f * 512), 16, 0, 0);
        }
    };

    const int64_t nblk = (n + Cfg::POINTS_PER_WG - 1) / Cfg::POINTS_PER_WG;

    // B operand x^T of one block: lane (g, li) holds x[p0 + 16*pt + li][32*kc + 8*g .. +8].
    auto load_x = [&](int64_t blk, Frag<T> (&xb)[PT][CK]) {
        const int64_t p0 = (blk * Cfg::WAVES + wave) * (16 * PT);
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) {
            const int64_t p = p0 + pt * 16 + li;
#pragma unroll
            for (int kc = 0; kc < CK; ++kc) {
                if (blk < nblk && p < n)
                    load8(xb[pt][kc], x + (size_t)p * C + kc * 32 + g * 8);
                else
                    zero8(xb[pt][kc]);
            }
        }
    };

    // x of the next block is loaded during the current block's last head, so
    // its latency (and the whole device's burst of block loads) overlaps compute.
    Frag<T> xb[PT][CK], xnext[PT][CK];
    load_x(blockIdx.x, xnext);
    for (int64_t blk = blockIdx.x; blk < nblk; blk += gridDim.x) {
        const int64_t p0 = (blk * Cfg::WAVES + wave) * (16 * PT);
#pragma unroll
        for (int pt = 0; pt < PT; ++pt)
#pragma unroll
            for (int kc = 0; kc < CK; ++kc) xb[pt][kc] = xnext[pt][kc];

        f32x4 O[CT][PT];

        auto logits = [&](int h, f32x4 (&L)[MT][PT]) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const float4 bb = *reinterpret_cast<const float4 *>(b2l + h * M + mt * 16 + g * 4);
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) L[mt][pt] = f32x4{bb.x, bb.y, bb.z, bb.w};
#pragma unroll
                for (int kc = 0; kc < CK; ++kc) {
                    Frag<T> a;
                    load8(a, w2l + ((((size_t)h * MT + mt) * CK + kc) * 64 + lane) * 8);
#pragma unroll
                    for (int pt = 0; pt < PT; ++pt) mma(L[mt][pt], a, xb[pt][kc]);
                }
            }
        };
        // out += Z_h^T . w_h with Z_h in the LDS stage.
        auto deslice_head = [&](const Frag<T> (&wf)[PT][KM]) {
#pragma unroll
            for (int ct = 0; ct < CT; ++ct)
#pragma unroll
                for (int km = 0; km < KM; ++km) {
                    Frag<T> a;
                    load8(a, zl + ((ct * KM + km) * 64 + lane) * 8);
#pragma unroll
                    for (int pt = 0; pt < PT; ++pt) mma(O[ct][pt], a, wf[pt][km]);
                }
        };

        // All heads of the block.  Per head: [barrier; stage Z_h] [logits_h]
        // [softmax_h] [wait; barrier] [deslice_h].  SHIFTED selects the
        // max-shifted softmax; the unshifted pass reports whether every row of
        // this wave was in the safe window.  PREFETCH loads the next block's x
        // once the last head's logits no longer need this block's.
        auto run_heads = [&](auto shifted, bool prefetch) -> bool {
#pragma unroll
            for (int ct = 0; ct < CT; ++ct)
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) O[ct][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
            bool ok = true;
            for (int hh = 0; hh < H; ++hh) {
                __syncthreads();  // every wave is done reading the stage
                stage_z(hh);
                f32x4 L[MT][PT];
                logits(hh, L);
                if (prefetch && hh == H - 1) load_x(blk + gridDim.x, xnext);
                Frag<T> wf[PT][KM];
                if constexpr (decltype(shifted)::value)
                    softmax_shifted<T, MT, PT, KM>(L, wf);
                else
                    ok = softmax_unshifted<T, MT, PT, KM>(L, wf) && ok;
                __builtin_amdgcn_s_waitcnt(0);  // this wave's stage loads have landed
                __syncthreads();                // ... and every other wave's
                deslice_head(wf);
            }
            return ok;
        };
        // Workgroup-uniform fallback: if any wave saw a row outside the safe
        // window, all waves redo the block with the max-shifted softmax.
        const bool ok = run_heads(std::false_type{}, true);
        if (__syncthreads_or(!ok)) {
            load_x(blk, xb);
            run_heads(std::true_type{}, false);
            load_x(blk + gridDim.x, xnext);
        }

#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            const float4 bb = *reinterpret_cast<const float4 *>(b3 + ct * 16 + g * 4);
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) {
                const int64_t p = p0 + pt * 16 + li;
                if (p >= n) continue;
                const float v0 = O[ct][pt][0] + bb.x, v1 = O[ct][pt][1] + bb.y;
                const float v2 = O[ct][pt][2] + bb.z, v3 = O[ct][pt][3] + bb.w;
                T *dst = out + (size_t)p * C + ct * 16 + g * 4;
                if constexpr (sizeof(T) == 2) {
                    typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
                    *reinterpret_cast<bf16x4 *>(dst) = bf16x4{(__bf16)v0, (__bf16)v1, (__bf16)v2, (__bf16)v3};
                } else {
                    *reinterpret_cast<float4 *>(dst) = float4{v0, v1, v2, v3};
                }
            }
        }
    }
}

}  // namespace ts3
