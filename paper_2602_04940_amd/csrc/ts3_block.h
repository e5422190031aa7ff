// Kernels of the pre-norm Transolver block around the Physics-Attention layer
// (the model context of section 3; 8 blocks in the paper's Table 7):
//
//   y   = x + PA(LN1(x))
//   out = y + W_b^T GELU(W_a^T LN2(y) + b_a) + b_b
//
// bf16 activations [N][C] between kernels, float32 arithmetic inside, bf16
// matrix-core operands with float32 accumulation.
//
//   k_layernorm     LN1 of the first block (later blocks get theirs from the
//                   previous block's feed-forward epilogue).
//   k_prep_mlp      W_a (bf16) and W_b (f16) as matrix-core fragments, chunked
//                   by 64 hidden units: [F/64][W_a^T part | W_b part], 64*C
//                   elements each, so one linear copy stages a chunk.
//   k_mlp_residual_pc  one kernel for the rest of the block: y = x + PA
//                   output, LN2, both feed-forward products with GELU (its
//                   tanh form in half precision, gelu2_f16) between them, the
//                   residual, and optionally the next block's LN1.
//
// k_mlp_residual_pc: 128 points per workgroup, 32 per pair of waves sharing a
// SIMD.  The producer keeps LN2(y) of its points as B fragments (K = channels)
// in registers; the hidden layer is walked in 64-unit chunks staged in LDS:
//   GEMM1  H^T[f][p] = W_a^T[f][:] . LN2(y)[p][:] + b_a[f]   (A = staged W_a^T)
//   GELU   on packed halves; the 16 x 4 outputs of two hidden tiles are
//          exactly a B fragment of the second product (K slot (g, t) <->
//          hidden unit 32km + 16(t>>2) + 4g + (t&3)), handed to the consumer
//          through LDS in that fragment order;
//   GEMM2  out^T[c][p] += W_b^T[c][:] . h[p][:]   (consumer; A = staged W_b,
//          f16 x f16) into the 32 x C output accumulator.
// Output rows of W_b's fragments follow zchan(), so a lane ends up holding the
// eight consecutive channels 32k + 8g .. +7 of its point: the same channels
// it loads for the residual, which keeps the next LayerNorm in registers.
#pragma once
#include "ts3_device.h"
#include "ts3_pass2.h"  // zchan

namespace ts3 {

constexpr float BLOCK_LN_EPS = 1e-5f;

// GELU(x) = x Phi(x) of two values, evaluated on packed halves with the
// tanh form of Hendrycks and Gimpel: Phi(x) ~ (1 + tanh(sqrt(2/pi) (x +
// 0.044715 x^3))) / 2 = 1 / (1 + exp(-2 sqrt(2/pi) (x + 0.044715 x^3))), so
// GELU(x) ~ x / (1 + 2^u) with u = -x (K1 + K2 x^2), K1 = 2 sqrt(2/pi) / ln 2,
// K2 = 0.044715 K1: four packed operations, two exp2 and two reciprocals per
// pair.  The form differs from x Phi(x) by at most 4.7e-4 (absolute); in half
// precision (every operation rounded to f16) the RMS absolute error over
// N(0, 1.5^2) inputs is 4.7e-4 and the worst 3.8e-3 (the f16 rounding of x near
// 8).  The tails need no care: for very negative x, 2^u overflows to infinity
// and the reciprocal gives 0; for large x, 2^u underflows and GELU(x) = x.
// Returns the pair as the f16 B-operand slots of the second product.
__device__ __forceinline__ f16x2 gelu2_f16(float a, float b) {
    const f16x2 x{(_Float16)a, (_Float16)b};
    const f16x2 u = x * ((x * x) * (_Float16)-0.10294280f + (_Float16)-2.30220819f);
    const f16x2 d = __builtin_elementwise_exp2(u) + (_Float16)1.0f;
    f16x2 r;
    r[0] = __builtin_amdgcn_rcph(d[0]);
    r[1] = __builtin_amdgcn_rcph(d[1]);
    return x * r;
}

__device__ __forceinline__ void unpack8(const uint4 &u, float (&v)[8]) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = __uint_as_float(w[i] << 16);
        v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}
__device__ __forceinline__ uint4 pack8(const float (&v)[8]) {
    typedef __attribute__((ext_vector_type(8))) __bf16 b8;
    b8 b;
#pragma unroll
    for (int i = 0; i < 8; ++i) b[i] = (__bf16)v[i];
    return __builtin_bit_cast(uint4, b);
}

// LayerNorm over C channels of bf16 rows; C/8 lanes per row, 8 channels each.
template <int C>
__global__ __launch_bounds__(256) void k_layernorm(const bf16_t *__restrict__ x, int64_t n,
                                                   const float *__restrict__ gam, const float *__restrict__ bet,
                                                   bf16_t *__restrict__ out) {
    constexpr int LPR = C / 8, RPW = 64 / LPR;
    const int lane = threadIdx.x & 63, sub = lane / LPR, cl = lane % LPR;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
    float gv[8], bv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        gv[i] = gam[8 * cl + i];
        bv[i] = bet[8 * cl + i];
    }
    for (int64_t r0 = ((int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) * RPW; r0 < n;
         r0 += waves * RPW) {
        const int64_t row = r0 + sub;
        const int64_t rc = row < n ? row : n - 1;
        float v[8];
        unpack8(*reinterpret_cast<const uint4 *>(x + rc * C + 8 * cl), v);
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) s += v[i];
#pragma unroll
        for (int m = 1; m < LPR; m <<= 1) s += __shfl_xor(s, m);
        const float mean = s * (1.f / C);
        float q = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            v[i] -= mean;
            q += v[i] * v[i];
        }
#pragma unroll
        for (int m = 1; m < LPR; m <<= 1) q += __shfl_xor(q, m);
        const float rstd = 1.f / sqrtf(q * (1.f / C) + BLOCK_LN_EPS);
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = v[i] * rstd * gv[i] + bv[i];
        if (row < n) *reinterpret_cast<uint4 *>(out + row * C + 8 * cl) = pack8(v);
    }
}

template <int C> struct MlpCfg {
    static constexpr int FC = 64, KM = FC / 32, CK = C / 32;
    static constexpr int PART = 64 * C;                 // elements of each half of a chunk
};

// Fragments of chunk j (hidden units 64j .. 64j+63):
//   W_a^T part, index ((ht*CK + kc)*64 + l)*8 + t:
//       W_a[c = 32kc + 8(l>>4) + t][f = 64j + 16ht + (l&15)]
//   W_b part,   index ((ct*KM + km)*64 + l)*8 + t:
//       W_b[f = 64j + 32km + 16(t>>2) + 4(l>>4) + (t&3)][c = zchan(ct, l&15)]
template <int C>
__global__ void k_prep_mlp(const float *__restrict__ Wa, const float *__restrict__ Wb, int F,
                           bf16_t *__restrict__ frag) {
    using Cfg = MlpCfg<C>;
    const int64_t total = (int64_t)(F / Cfg::FC) * 2 * Cfg::PART;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t j = i / (2 * Cfg::PART);
        const int e = (int)(i % (2 * Cfg::PART));
        const int t = e & 7, l = (e >> 3) & 63, r = e >> 9;
        float v;
        if (e < Cfg::PART) {
            const int kc = r % Cfg::CK, ht = r / Cfg::CK;
            const int c = 32 * kc + 8 * (l >> 4) + t;
            const int64_t f = 64 * j + 16 * ht + (l & 15);
            v = Wa[(int64_t)c * F + f];
        } else {
            const int r2 = r - Cfg::PART / 512;
            const int km = r2 % Cfg::KM, ct = r2 / Cfg::KM;
            const int64_t f = 64 * j + 32 * km + 16 * (t >> 2) + 4 * (l >> 4) + (t & 3);
            const int c = zchan(ct, l & 15);
            frag[i].bits = __builtin_bit_cast(uint16_t, (_Float16)Wb[f * C + c]);  // f16: the second product
            continue;
        }
        frag[i].bits = __builtin_bit_cast(uint16_t, (__bf16)v);
    }
}

// x, pa  : [n][C] bf16, the block input and its Physics-Attention output
// ln2_*  : LN2 affine [C]; frag: k_prep_mlp output; ba [F], bb [C]
// lnn_*  : the next block's LN1 affine, or NULL (then xn is not written)
// xo     : [n][C] bf16 block output (may alias x: the producer reads x before
//          the first barrier, the consumer writes xo after the last); xn: LN1
//          of xo for the next block (may alias nothing that is read here)
// grid   : ceil(n / 128) workgroups of 512 threads
//
// Producer and consumer waves, two per SIMD (one of each), 32 points per
// pair, 128 points per workgroup:
//   wave q      (producer) keeps LN2(y) of the pair's 32 points as B fragments
//               and, per 64-unit chunk j, runs GEMM1 and the GELU, writing h
//               (the f16 B fragments of GEMM2, in fragment order) to the
//               pair's h tile;
//   wave q + 4  (consumer) runs GEMM2 of chunk j-1 from that h tile into the
//               32 x C output accumulator, issues the weight copies, and at
//               the end writes the block output (and the next LN1).
// Every weight fragment read from LDS then feeds two MFMAs (two 16-point
// tiles), half the LDS traffic per point of the eight-wave kernel, and the
// GELU's vector work runs beside the other wave's matrix work.  W_a^T and W_b
// halves of a chunk are staged in separate slots (two each): step j reads
// W_a(j) and W_b(j-1) and copies W_a(j+1) and W_b(j).  One barrier per step;
// NCHUNK + 1 steps.  LDS: 4 x 64C bf16 weight slots + 2 x 4 KB h tiles per
// pair (160 KB at C = 256).
template <int C> struct MlpPCCfg {
    static constexpr int FC = 64, HT = FC / 16, KM = FC / 32, CK = C / 32, CT = C / 16, PT = 2;
    static constexpr int PART = 64 * C;                 // elements of each half of a chunk
    static constexpr int PART_BYTES = PART * 2;
    static constexpr int PART_COPIES = PART_BYTES / 1024;
    static constexpr int HTILE = PT * KM * 64 * 16;      // bytes: a pair's h fragments
    static constexpr int LDS_BYTES = 4 * PART_BYTES + 4 * 2 * HTILE;
    static_assert(PART_COPIES % 4 == 0, "each consumer issues a quarter of a part's copies");
};

template <int C, int F>
__global__ __launch_bounds__(512, 1) void k_mlp_residual_pc(
    const bf16_t *x, const bf16_t *__restrict__ pa, int64_t n, const float *__restrict__ ln2_g,
    const float *__restrict__ ln2_b, const bf16_t *__restrict__ frag, const float *__restrict__ ba,
    const float *__restrict__ bb, const float *__restrict__ lnn_g, const float *__restrict__ lnn_b, bf16_t *xo,
    bf16_t *__restrict__ xn) {
    using Cfg = MlpPCCfg<C>;
    constexpr int CK = Cfg::CK, CT = Cfg::CT, HT = Cfg::HT, KM = Cfg::KM, PT = Cfg::PT;
    constexpr int NCHUNK = F / Cfg::FC, PB = Cfg::PART_BYTES, HTILE = Cfg::HTILE;
    static_assert(F % Cfg::FC == 0, "hidden width in 64-unit chunks");
    __shared__ __attribute__((aligned(1024))) unsigned char lds[Cfg::LDS_BYTES];
    unsigned char *const wa_slots = lds;               // W_a^T parts, two slots
    unsigned char *const wb_slots = lds + 2 * PB;      // W_b parts, two slots

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int q = wave & 3, role = wave >> 2;
    const int li = lane & 15, g = lane >> 4;
    const int64_t p0 = (int64_t)blockIdx.x * 128 + q * 32;
    unsigned char *const hslots = lds + 4 * PB + q * 2 * HTILE;  // the pair's two h tiles

    // A consumer's quarter of part `half` (0: W_a^T, 1: W_b) of chunk j into slot sl.
    auto issue_part = [&](int j, int half, int sl) {
        const unsigned char *src = reinterpret_cast<const unsigned char *>(frag) + ((size_t)(2 * j + half)) * PB;
        const uint32_t base = lds_addr(lds) + (half * 2 + sl) * PB;
#pragma unroll
        for (int c = 0; c < Cfg::PART_COPIES / 4; ++c) {
            const int k = q * (Cfg::PART_COPIES / 4) + c;
            dma16(src + k * 1024 + lane * 16, base + k * 1024);
        }
    };

    if (role == 0) {
        // ---------------------------------------------------------------- producer
        // y = x + pa and LN2(y) as B fragments: tile pt, lane (li, g) holds
        // point p0 + 16pt + li, channels 32k + 8g .. +7 in slot t of fragment k.
        Frag<bf16_t> yb[PT][CK];
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) {
            int64_t p = p0 + 16 * pt + li;
            p = p < n ? p : n - 1;
            float y[CK][8];
            float s = 0.f;
#pragma unroll
            for (int k = 0; k < CK; ++k) {
                float a[8], b[8];
                unpack8(*reinterpret_cast<const uint4 *>(x + p * C + 32 * k + 8 * g), a);
                unpack8(*reinterpret_cast<const uint4 *>(pa + p * C + 32 * k + 8 * g), b);
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    y[k][t] = a[t] + b[t];
                    s += y[k][t];
                }
            }
            const float mean = xrow_sum(s) * (1.f / C);
            float qq = 0.f;
#pragma unroll
            for (int k = 0; k < CK; ++k)
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    y[k][t] -= mean;
                    qq += y[k][t] * y[k][t];
                }
            const float rstd = 1.f / sqrtf(xrow_sum(qq) * (1.f / C) + BLOCK_LN_EPS);
#pragma unroll
            for (int k = 0; k < CK; ++k) {
                const float4 g0 = *reinterpret_cast<const float4 *>(ln2_g + 32 * k + 8 * g);
                const float4 g1 = *reinterpret_cast<const float4 *>(ln2_g + 32 * k + 8 * g + 4);
                const float4 b0 = *reinterpret_cast<const float4 *>(ln2_b + 32 * k + 8 * g);
                const float4 b1 = *reinterpret_cast<const float4 *>(ln2_b + 32 * k + 8 * g + 4);
                const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
                const float bbv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
                for (int t = 0; t < 8; t += 2)
                    yb[pt][k].set2(t, y[k][t] * rstd * gg[t] + bbv[t], y[k][t + 1] * rstd * gg[t + 1] + bbv[t + 1]);
            }
        }
        wait_vmcnt<0>();
        __syncthreads();  // W_a(0) staged (the consumers' copies)
#pragma unroll 1
        for (int j = 0; j <= NCHUNK; ++j) {
            if (j < NCHUNK) {
                const unsigned char *wa = wa_slots + (j & 1) * PB;
                f32x4 Hh[HT][PT];
#pragma unroll
                for (int ht = 0; ht < HT; ++ht) {
                    const float4 b = *reinterpret_cast<const float4 *>(ba + 64 * j + 16 * ht + 4 * g);
#pragma unroll
                    for (int pt = 0; pt < PT; ++pt) Hh[ht][pt] = f32x4{b.x, b.y, b.z, b.w};
                }
                // A fragments are read one K step ahead of their products.
                Frag<bf16_t> a1[2][HT];
                auto read1 = [&](int kc, Frag<bf16_t>(&dst)[HT]) {
#pragma unroll
                    for (int ht = 0; ht < HT; ++ht)
                        dst[ht].v = *reinterpret_cast<const bf16x8 *>(wa + ((ht * CK + kc) * 64 + lane) * 16);
                };
                read1(0, a1[0]);
                __builtin_amdgcn_s_setprio(2);  // GEMM1 first on the matrix core; GEMM2 fills the GELU
#pragma unroll
                for (int kc = 0; kc < CK; ++kc) {
                    if (kc + 1 < CK) read1(kc + 1, a1[(kc + 1) & 1]);
#pragma unroll
                    for (int ht = 0; ht < HT; ++ht)
#pragma unroll
                        for (int pt = 0; pt < PT; ++pt) mma(Hh[ht][pt], a1[kc & 1][ht], yb[pt][kc]);
                }
                __builtin_amdgcn_s_setprio(0);
                // GELU into the f16 B fragments of GEMM2, stored in fragment order.
                unsigned char *ht_out = hslots + (j & 1) * HTILE;
#pragma unroll
                for (int pt = 0; pt < PT; ++pt)
#pragma unroll
                    for (int km = 0; km < KM; ++km) {
                        u32x4 u;
#pragma unroll
                        for (int t = 0; t < 8; t += 2) {
                            const int ht = 2 * km + (t >> 2);
                            u[t >> 1] =
                                __builtin_bit_cast(uint32_t, gelu2_f16(Hh[ht][pt][t & 3], Hh[ht][pt][(t & 3) + 1]));
                        }
                        *reinterpret_cast<u32x4 *>(ht_out + ((pt * KM + km) * 64 + lane) * 16) = u;
                    }
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            __syncthreads();  // h(j) written; W_a(j+1) and W_b(j) staged
        }
    } else {
        // ---------------------------------------------------------------- consumer
        f32x4 Z[CT][PT];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) Z[ct][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
        issue_part(0, 0, 0);
        wait_vmcnt<0>();
        __syncthreads();  // W_a(0) staged
#pragma unroll 1
        for (int j = 0; j <= NCHUNK; ++j) {
            if (j + 1 < NCHUNK) issue_part(j + 1, 0, (j + 1) & 1);
            if (j < NCHUNK) issue_part(j, 1, j & 1);
            if (j > 0) {
                // GEMM2 of chunk j-1: the W_b fragment of channel tile ct+1 is
                // read while tile ct's products run.
                const unsigned char *wb = wb_slots + ((j - 1) & 1) * PB;
                const unsigned char *hin = hslots + ((j - 1) & 1) * HTILE;
                Frag<f16_t> hb[PT][KM];
#pragma unroll
                for (int pt = 0; pt < PT; ++pt)
#pragma unroll
                    for (int km = 0; km < KM; ++km)
                        hb[pt][km].v = *reinterpret_cast<const f16x8 *>(hin + ((pt * KM + km) * 64 + lane) * 16);
                // K steps outermost: the two products into one accumulator are
                // CT * PT apart (a dependent MFMA issues at half rate); the
                // fragment of step q+2 is read while step q's products run.
                constexpr int NQ = KM * CT;
                auto bfrag = [&](int q2) { return wb + (((q2 % CT) * KM + q2 / CT) * 64 + lane) * 16; };
                Frag<f16_t> a2[4];
                a2[0].v = *reinterpret_cast<const f16x8 *>(bfrag(0));
                a2[1].v = *reinterpret_cast<const f16x8 *>(bfrag(1));
#pragma unroll
                for (int q2 = 0; q2 < NQ; ++q2) {
                    if (q2 + 2 < NQ) a2[(q2 + 2) & 3].v = *reinterpret_cast<const f16x8 *>(bfrag(q2 + 2));
                    const int km = q2 / CT, ct = q2 % CT;
#pragma unroll
                    for (int pt = 0; pt < PT; ++pt) mma(Z[ct][pt], a2[q2 & 3], hb[pt][km]);
                }
            }
            wait_vmcnt<0>();  // this wave's copies of the step landed
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            __syncthreads();
        }

        // out = x + pa + z + bb; lane (li, g) of tile pt holds channels
        // 32k + 8g + 4h + r in Z[2k + h][pt][r].
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) {
            const int64_t p = p0 + 16 * pt + li;
            const int64_t pc = p < n ? p : n - 1;
            float o[CK][8];
#pragma unroll
            for (int k = 0; k < CK; ++k) {
                float a[8], b[8];
                unpack8(*reinterpret_cast<const uint4 *>(x + pc * C + 32 * k + 8 * g), a);
                unpack8(*reinterpret_cast<const uint4 *>(pa + pc * C + 32 * k + 8 * g), b);
                const float4 c0 = *reinterpret_cast<const float4 *>(bb + 32 * k + 8 * g);
                const float4 c1 = *reinterpret_cast<const float4 *>(bb + 32 * k + 8 * g + 4);
                const float cb[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
#pragma unroll
                for (int t = 0; t < 8; ++t) o[k][t] = (a[t] + b[t]) + (Z[2 * k + (t >> 2)][pt][t & 3] + cb[t]);
            }
            if (lnn_g) {  // uniform
                // the next block's LN1 of the rounded output
                float sr = 0.f;
#pragma unroll
                for (int k = 0; k < CK; ++k)
#pragma unroll
                    for (int t = 0; t < 8; ++t) {
                        o[k][t] = (float)(__bf16)o[k][t];
                        sr += o[k][t];
                    }
                const float mean = xrow_sum(sr) * (1.f / C);
                float qq = 0.f;
#pragma unroll
                for (int k = 0; k < CK; ++k)
#pragma unroll
                    for (int t = 0; t < 8; ++t) qq += (o[k][t] - mean) * (o[k][t] - mean);
                const float rstd = 1.f / sqrtf(xrow_sum(qq) * (1.f / C) + BLOCK_LN_EPS);
#pragma unroll
                for (int k = 0; k < CK; ++k) {
                    float v[8];
#pragma unroll
                    for (int t = 0; t < 8; ++t)
                        v[t] = (o[k][t] - mean) * rstd * lnn_g[32 * k + 8 * g + t] + lnn_b[32 * k + 8 * g + t];
                    if (p < n) *reinterpret_cast<uint4 *>(xn + p * C + 32 * k + 8 * g) = pack8(v);
                }
            }
            if (p < n)
#pragma unroll
                for (int k = 0; k < CK; ++k) *reinterpret_cast<uint4 *>(xo + p * C + 32 * k + 8 * g) = pack8(o[k]);
        }
    }
}

}  // namespace ts3
