// Pass 1 in the projected form, for 16-bit storage, C = 128 and head width
// 16 (H = 8): per span and head the kernel accumulates
//     t[m][j] = sum_p w[p][m] (x[p] W1)[h*16 + j]   and   d[m] = sum_p w[p][m],
// the slice sums of the projected features of Eq. (2) (x_proj = x W1; the bias
// b1 is added once the sums are divided by d), instead of the M x C sums of
// the raw features that Linear1 then maps (Eq. (4), Algorithm 1).  By
// linearity both give the same physical states s = t / d + b1; the projected
// sums take 2*(H*M*dh + C*C) products per point (with the remainder terms
// below) where the raw ones take H*M*C (49,152 against 65,536 at C = 128,
// M = 64), and a span's partial shrinks from M*(C+1) to M*(dh+1) floats per
// head.
//
// The producer/consumer split is that of k_slice_accumulate_pc, with three
// block streams instead of two: a workgroup of 12 waves serves a span and two
// heads, each head's blocks in three interleaved streams (blocks s, s+3, ...),
// one producer and one consumer wave per (stream, head).  Three waves per SIMD
// (154 registers each fit the 168 that allows) give each SIMD's matrix core a
// third instruction stream while the others wait on their dependencies:
// measured 23.3 -> 21.1 ms per 100M-point layer against two streams.  Per
// 32-point block:
//   producer: the logits (A = W2'^T resident, B = x^T from LDS), exp2 of
//             them, and the row sums S[p] = sum_m e[p][m] from MFMAs with an
//             all-ones A operand on the packed e (no vector row sums); it
//             writes e (unnormalised, bf16) to the pair's w tile and 1/S[p]
//             (zero for padding rows) to the pair's scale row;
//   consumer: xw[p][j] = x[p] . W1[:, h*16 + j] (A = the same x fragments as
//             the producer's logits, B = W1 fragments resident), then
//             t += e^T (xw / S) and d += e^T (1 / S) (A = e^T from transposing
//             LDS reads).  The rows of xw in its output registers are the K
//             slots of the contraction's B operand, so no transposition.
// The normalisation 1/S thus costs 8 multiplies per consumer step instead of
// 32 per producer step; both contractions use the same bf16 e.
//
// Precision.  The raw form rounds each weight once and multiplies exact
// stored features; here W1 and the projected rows would be rounded as well,
// systematic errors of 2^-9 that the token attention can amplify when the
// slice tokens are large.  So W1 enters as two bfloat16 parts (rounded value
// and rounded remainder, two products into the same float32 accumulators) and
// each projected row xw / S as two parts (two products into t): the state
// then matches the raw form's accuracy for 8 extra products per point and
// head.
#pragma once
#include "ts3_pass1.h"

namespace ts3 {

constexpr int PCP_THREADS = 768;  // 12 waves: 3 block streams x 2 heads x 2 roles

template <int C, int M> struct Pass1PCPCfg {
    using T = bf16_t;
    static constexpr int STREAMS = 3, PAIRS = 2 * STREAMS, WAVES = 2 * PAIRS;
    static_assert(WAVES * 64 == PCP_THREADS, "the launch bound assumes this workgroup size");
    static constexpr int MT = M / 16;  // 16-slice tiles of a head
    static constexpr int CT = C / 16, CK = C / 32;
    static constexpr int XROW = C * 2, XTILE = 32 * XROW;
    static constexpr int WROW = M * 2, WTILE = 32 * WROW;
    static constexpr int NSX = 4, NSW = 2, AHEAD = 3;
    static constexpr int ROWS_PER_LOAD = 1024 / XROW, LOADS = 32 / ROWS_PER_LOAD;
    // Each head's two waves issue four of the stream's eight 1 KB copies of a
    // block: the producer P_LOADS of them (none), the consumer the rest.
    static constexpr int HEAD_LOADS = LOADS / 2, P_LOADS = 0, C_LOADS = HEAD_LOADS - P_LOADS;
    static constexpr int X_BYTES = STREAMS * NSX * XTILE;
    static constexpr int W_BYTES = PAIRS * NSW * WTILE;
    static constexpr int DH = 16, E = M * (DH + 1);  // a head's partial: t and d
    static constexpr int RED_BYTES = PAIRS * E * 4;
    static constexpr int V_BYTES = PAIRS * NSW * 32 * 4;  // 1/S per point, per pair and w slot
    static constexpr int PIPE_BYTES = X_BYTES + W_BYTES + V_BYTES;
    static constexpr int LDS_BYTES = PIPE_BYTES > RED_BYTES ? PIPE_BYTES : RED_BYTES;
    static_assert(ROWS_PER_LOAD == 4 && HEAD_LOADS == 4, "copies split as whole 1 KB pieces");
    static_assert(CK == 4 && CT == 8 && MT <= 4, "the address sets are written for C = 128, M <= 64");
};

// W1 in the consumer's B-operand order, as two bfloat16 parts whose sum is
// W1 to about 2^-17 relative: w1p[0][H][CK][64][8] the rounded values,
// w1p[1][...] the rounded remainders.  Lane l, slot t holds
// W1[32*kc + 8*(l>>4) + t][h*16 + (l&15)] (head width 16).
__global__ void k_prep_w1(const float *__restrict__ W1, int C, int H, bf16_t *__restrict__ w1p) {
    const int CK = C / 32;
    const int64_t total = (int64_t)H * CK * 64 * 8;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int t = (int)(i & 7), lane = (int)((i >> 3) & 63);
        const int64_t r = i >> 9;
        const int kc = (int)(r % CK), h = (int)(r / CK);
        const float w = W1[(int64_t)(kc * 32 + (lane >> 4) * 8 + t) * C + h * 16 + (lane & 15)];
        const __bf16 hi = (__bf16)w;
        reinterpret_cast<__bf16 *>(w1p)[i] = hi;
        reinterpret_cast<__bf16 *>(w1p)[total + i] = (__bf16)(w - (float)hi);
    }
}

// Arguments as k_slice_accumulate (H = C / 16, even) plus w1p; partials are
// [span][H][M][17] (t then d).  Grid nspan * H / 2, PCP_THREADS threads.
template <int C, int M>
__global__ __launch_bounds__(PCP_THREADS, 1) void k_slice_accumulate_pcp(
    const bf16_t *__restrict__ x, int64_t n_tile, int64_t span0, int32_t Q, int32_t nspan, int32_t H,
    const bf16_t *__restrict__ w2p, const float *__restrict__ b2s, const bf16_t *__restrict__ w1p,
    float *__restrict__ partials) {
    using Cfg = Pass1PCPCfg<C, M>;
    using T = bf16_t;
    constexpr int MT = Cfg::MT, CT = Cfg::CT, CK = Cfg::CK, KMS = (Cfg::MT + 1) / 2;
    constexpr int NSX = Cfg::NSX, NSW = Cfg::NSW, AHEAD = Cfg::AHEAD;
    constexpr int XROW = Cfg::XROW, WROW = Cfg::WROW, XTILE = Cfg::XTILE, WTILE = Cfg::WTILE, DH = Cfg::DH;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[Cfg::LDS_BYTES];

    const int HP = H / 2;
    const int nwg = nspan * HP;
    const int jwg = xcd_remap((int)blockIdx.x, nwg);  // a span's head pairs share an XCD (and its L2)
    const int span_local = jwg / HP;
    const int hp = jwg - span_local * HP;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    constexpr int NST = Cfg::STREAMS, NPAIR = Cfg::PAIRS;
    const int pair = wave % NPAIR, role = wave / NPAIR;  // role 0: logits and softmax, 1: contraction
    const int stream = pair % NST, hsel = pair / NST;
    const int h = 2 * hp + hsel;
    const int li = lane & 15, g = lane >> 4;

    const int64_t p_begin = (int64_t)span_local * Q;
    const int64_t p_end = p_begin + Q < n_tile ? p_begin + Q : n_tile;
    const int nrows = (int)(p_end - p_begin);  // <= Q <= 2^30
    const int nblk = (nrows + 31) >> 5;
    const int nit = (nblk + NST - 1) / NST;  // block steps, the same for every wave

    unsigned char *const xring = lds + stream * NSX * XTILE;
    unsigned char *const wring = lds + Cfg::X_BYTES + pair * NSW * WTILE;
    float *const vring = reinterpret_cast<float *>(lds + Cfg::X_BYTES + Cfg::W_BYTES) + pair * NSW * 32;
    const uint32_t xring_lds = lds_addr(xring);

    // This wave's share of block j of its stream (mesh block stream + 3j) into
    // x slot SL: copies i = 4*hsel + I0 .. 4*hsel + I0 + NL - 1 (the producer's
    // first, then the consumer's); rows past the span's end repeat its last
    // row.  Row offsets within the span are 32-bit.
    constexpr int NCH = XROW / 16;
    auto copy_off = [&](int i) {
        const int R = i * Cfg::ROWS_PER_LOAD + lane / NCH;
        return (uint32_t)(R * XROW + (((lane % NCH) ^ xswz<XROW>(R)) << 4));
    };
    auto issue_x = [&](int j, auto slot, auto rl) {
        constexpr int SL = decltype(slot)::value, RL = decltype(rl)::value;
        constexpr int NL = RL == 0 ? Cfg::P_LOADS : Cfg::C_LOADS, I0 = RL == 0 ? 0 : Cfg::P_LOADS;
        if constexpr (NL == 0) return;
        const int r0 = (stream + NST * j) << 5;
        const uint32_t dst = xring_lds + SL * XTILE;
        if (__builtin_expect(r0 + 32 <= nrows, 1)) {
            const void *base = x + (p_begin + r0) * C;
#pragma unroll
            for (int kk = 0; kk < NL; ++kk) {
                const int i = 4 * hsel + I0 + kk;
                dma16s<0>(copy_off(i), base, dst + i * 1024);
            }
        } else {
#pragma unroll
            for (int kk = 0; kk < NL; ++kk) {
                const int i = 4 * hsel + I0 + kk;
                const int R = i * Cfg::ROWS_PER_LOAD + lane / NCH;
                const int ch = (lane % NCH) ^ xswz<XROW>(R);
                const int r = r0 + R < nrows ? r0 + R : nrows - 1;
                dma16(reinterpret_cast<const unsigned char *>(x + (size_t)(p_begin + r) * C) + ch * 16, dst + i * 1024);
            }
        }
    };
    auto block_valid = [&](int j) {
        const int left = nrows - ((stream + NST * j) << 5);
        return left <= 0 ? 0 : left < 32 ? left : 32;
    };

    // Shared start of both roles (each role runs it after its own loads):
    // zero "block -1" (x slot NSX-1, w slot NSW-1 and its scales), so the
    // first contraction adds nothing, and copy blocks 0..2.
    auto prologue = [&](auto rl) {
        constexpr int NL = decltype(rl)::value == 0 ? Cfg::P_LOADS : Cfg::C_LOADS;
        wait_vmcnt<0>();  // the ring's wait counts assume only its own copies are in flight
        uint4 *zx = reinterpret_cast<uint4 *>(xring + (NSX - 1) * XTILE);
        uint4 *zw = reinterpret_cast<uint4 *>(wring + (NSW - 1) * WTILE);
        const int sidx = hsel * 2 + role;  // 0..3 within the stream
        for (int i = sidx * 64 + lane; i < XTILE / 16; i += 256) zx[i] = uint4{0u, 0u, 0u, 0u};
        for (int i = role * 64 + lane; i < WTILE / 16; i += 128) zw[i] = uint4{0u, 0u, 0u, 0u};
        if (role == 0 && lane < 32) vring[(NSW - 1) * 32 + lane] = 0.f;
        issue_x(0, ic<0>{}, rl);
        issue_x(1, ic<1>{}, rl);
        issue_x(2, ic<2>{}, rl);
        wait_vmcnt<2 * NL>();        // this wave's copies of block 0
        __syncthreads();             // everyone's copies of block 0 and the zero tiles visible
    };
    static_assert(NSX == 4 && NSW == 2 && AHEAD == 3, "the unrolled loops below assume these ring depths");

    const uint32_t xbase = (uint32_t)(stream * NSX * XTILE);
    const uint32_t wbase = (uint32_t)(Cfg::X_BYTES + pair * NSW * WTILE);
    // The end of every step: this wave's copies of block j+1 have landed
    // (those of block j+2 may not have); the barrier makes every wave's copies
    // of block j+1 visible, with block j's w rows; then the copies of block
    // j + AHEAD go into the slot block j-1 released.
    auto end_step = [&](int j, auto prev, auto rl) {
        wait_vmcnt<decltype(rl)::value == 0 ? Cfg::P_LOADS : Cfg::C_LOADS>();
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __syncthreads();
        issue_x(j + AHEAD, prev, rl);
    };
    // Steps j .. j+3 use x slots 0..3 and w slots 0, 1, 0, 1.
    auto run_steps = [&](auto &&step) {
        int j = 0;
        for (; j + 4 <= nit; j += 4) {
            step(j, ic<0>{}, ic<0>{});
            step(j + 1, ic<1>{}, ic<1>{});
            step(j + 2, ic<2>{}, ic<0>{});
            step(j + 3, ic<3>{}, ic<1>{});
        }
        if (j < nit) step(j, ic<0>{}, ic<0>{});
        if (j + 1 < nit) step(j + 1, ic<1>{}, ic<1>{});
        if (j + 2 < nit) step(j + 2, ic<2>{}, ic<0>{});
        wait_vmcnt<0>();
    };

    float *red = reinterpret_cast<float *>(lds);
    if (role == 0) {
        // ---------------------------------------------------------------- producer
        Frag<T> w2[MT][CK];  // head h's W2'^T fragments (all slices) and bias, resident
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
        Frag<T> ones;
        ones8(ones);
        prologue(ic<0>{});
        // x-row addresses of point tile pt (rows prow(pt, .)) at K step kc, and
        // the w-row addresses of point tile pt at slice tile mt, held in registers.
        uint32_t xl00 = xbase + xoff<XROW>(prow(0, li), 16 * g), xl10 = xbase + xoff<XROW>(prow(1, li), 16 * g);
        uint32_t xl01 = xl00 ^ (1 << 6), xl02 = xl00 ^ (2 << 6), xl03 = xl00 ^ (3 << 6);
        uint32_t xl11 = xl10 ^ (1 << 6), xl12 = xl10 ^ (2 << 6), xl13 = xl10 ^ (3 << 6);
        auto xl_at = [&](int pt, int kc) {
            return pt == 0 ? (kc == 0 ? xl00 : kc == 1 ? xl01 : kc == 2 ? xl02 : xl03)
                           : (kc == 0 ? xl10 : kc == 1 ? xl11 : kc == 2 ? xl12 : xl13);
        };
        uint32_t ws00 = wbase + woff<WROW>(prow(0, li), 8 * g), ws10 = wbase + woff<WROW>(prow(1, li), 8 * g);
        uint32_t ws01 = ws00 ^ (1 << 5), ws02 = ws00 ^ (2 << 5), ws03 = ws00 ^ (3 << 5);
        uint32_t ws11 = ws10 ^ (1 << 5), ws12 = ws10 ^ (2 << 5), ws13 = ws10 ^ (3 << 5);
        auto ws_at = [&](int pt, int mt) {
            return pt == 0 ? (mt == 0 ? ws00 : mt == 1 ? ws01 : mt == 2 ? ws02 : ws03)
                           : (mt == 0 ? ws10 : mt == 1 ? ws11 : mt == 2 ? ws12 : ws13);
        };
        // The x fragments of step kc+1 are read while step kc's MFMAs run.
        auto logits = [&](auto slot, f32x4 (&L)[MT][2]) {
            constexpr int SL = decltype(slot)::value;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) L[mt][0] = L[mt][1] = bias[mt];
            Frag<T> xb[2][2];
#pragma unroll
            for (int pt = 0; pt < 2; ++pt) xb[0][pt].v = *reinterpret_cast<const bf16x8 *>(lds + xl_at(pt, 0) + SL * XTILE);
#pragma unroll
            for (int kc = 0; kc < CK; ++kc) {
                __builtin_amdgcn_sched_barrier(0);
                if (kc + 1 < CK)
#pragma unroll
                    for (int pt = 0; pt < 2; ++pt)
                        xb[(kc + 1) & 1][pt].v = *reinterpret_cast<const bf16x8 *>(lds + xl_at(pt, kc + 1) + SL * XTILE);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int pt = 0; pt < 2; ++pt) mma(L[mt][pt], w2[mt][kc], xb[kc & 1][pt]);
                if (kc + 1 < CK) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, MT * 2, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        };
        auto step = [&](int j, auto slot, auto wslot) {
            constexpr int SL = decltype(slot)::value, SW = decltype(wslot)::value;
            constexpr int PREV = (SL + NSX - 1) % NSX;
            asm volatile("" : "+v"(xl00), "+v"(xl01), "+v"(xl02), "+v"(xl03), "+v"(xl10), "+v"(xl11), "+v"(xl12),
                         "+v"(xl13));
            asm volatile("" : "+v"(ws00), "+v"(ws01), "+v"(ws02), "+v"(ws03), "+v"(ws10), "+v"(ws11), "+v"(ws12),
                         "+v"(ws13));
            const int valid = block_valid(j);
            f32x4 L[MT][2];
            // The producer's logits MFMAs go first on the SIMD's matrix core
            // (the consumer's contraction fills the softmax that follows):
            // measured 2% faster than equal priorities.
            __builtin_amdgcn_s_setprio(2);
            logits(slot, L);
            __builtin_amdgcn_s_setprio(0);
            // exp2 of the raw logits, packed to bf16 as the B operand of the
            // row-sum products (K slot (g, t) <-> slice 32km + 16(t>>2) + 4g +
            // (t&3)); the same packed pairs are the w-tile rows.
            auto pack_e = [&](Frag<T> (&ef)[2][KMS]) {
#pragma unroll
                for (int pt = 0; pt < 2; ++pt)
#pragma unroll
                    for (int km = 0; km < KMS; ++km)
#pragma unroll
                        for (int t = 0; t < 8; t += 2) {
                            const int mt = 2 * km + (t >> 2);
                            if (mt < MT) ef[pt][km].set2(t, L[mt][pt][t & 3], L[mt][pt][(t & 3) + 1]);
                            else ef[pt][km].set2(t, 0.f, 0.f);
                        }
            };
            auto row_sums = [&](const Frag<T> (&ef)[2][KMS], float (&S)[2]) {
#pragma unroll
                for (int pt = 0; pt < 2; ++pt) {
                    f32x4 acc{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int km = 0; km < KMS; ++km) mma(acc, ones, ef[pt][km]);
                    S[pt] = acc[0];  // every row of the all-ones product is the sum
                }
            };
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int pt = 0; pt < 2; ++pt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) L[mt][pt][r] = fast_exp2(L[mt][pt][r]);
            Frag<T> ef[2][KMS];
            pack_e(ef);
            float S[2];
            row_sums(ef, S);
            if (__any(!(softmax_sum_ok(S[0]) && softmax_sum_ok(S[1])))) {
                // Rare: a row's exp2 sum left the safe window; redo the block's
                // rows with the max shift.
                logits(slot, L);
#pragma unroll
                for (int pt = 0; pt < 2; ++pt) {
                    float mx = L[0][pt][0];
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                        for (int r = 0; r < 4; ++r) mx = fmaxf(mx, L[mt][pt][r]);
                    mx = xrow_max(mx);
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                        for (int r = 0; r < 4; ++r) L[mt][pt][r] = fast_exp2(L[mt][pt][r] - mx);
                }
                pack_e(ef);
                row_sums(ef, S);
            }
            typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
            typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
#pragma unroll
            for (int pt = 0; pt < 2; ++pt) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    // slots 4(mt&1) .. +3 of K step mt>>1 hold this tile's four values
                    const u32x4_t w = __builtin_bit_cast(u32x4_t, ef[pt][mt >> 1].v);
                    const uint2 half = (mt & 1) ? uint2{w[2], w[3]} : uint2{w[0], w[1]};
                    *reinterpret_cast<uint2 *>(lds + ws_at(pt, mt) + SW * WTILE) = half;
                }
                // 1/S per point (zero for padding rows: they weigh nothing)
                if (g == 0) vring[SW * 32 + pt * 16 + li] = prow(pt, li) < valid ? fast_rcp(S[pt]) : 0.f;
            }
            end_step(j, ic<PREV>{}, ic<0>{});
        };
        run_steps(step);
        __syncthreads();  // the pipeline's LDS becomes the reduction buffer
        __syncthreads();  // the consumers' accumulators are in it
    } else {
        // ---------------------------------------------------------------- consumer
        prologue(ic<1>{});
        f32x4 Tt[MT], Dd[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) Tt[mt] = Dd[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
        Frag<T> w1[CK], w1l[CK];  // head h's W1 fragments (B operand of x W1) and remainders, resident
#pragma unroll
        for (int kc = 0; kc < CK; ++kc) {
            load8(w1[kc], w1p + (((size_t)h * CK + kc) * 64 + lane) * 8);
            load8(w1l[kc], w1p + (((size_t)(H + h) * CK + kc) * 64 + lane) * 8);
        }
        // x-row addresses of point tile pt at K step kc (the producer's logits
        // operands, here the A operand of x W1) and the e^T addresses of slice
        // tile mt, held in registers.
        uint32_t xl00 = xbase + xoff<XROW>(prow(0, li), 16 * g), xl10 = xbase + xoff<XROW>(prow(1, li), 16 * g);
        uint32_t xl01 = xl00 ^ (1 << 6), xl02 = xl00 ^ (2 << 6), xl03 = xl00 ^ (3 << 6);
        uint32_t xl11 = xl10 ^ (1 << 6), xl12 = xl10 ^ (2 << 6), xl13 = xl10 ^ (3 << 6);
        auto xl_at = [&](int pt, int kc) {
            return pt == 0 ? (kc == 0 ? xl00 : kc == 1 ? xl01 : kc == 2 ? xl02 : xl03)
                           : (kc == 0 ? xl10 : kc == 1 ? xl11 : kc == 2 ? xl12 : xl13);
        };
        uint32_t wa0 = wbase + woff<WROW>(8 * g + (li >> 2), 8 * (li & 3));
        uint32_t wa1 = wa0 ^ (1 << 5), wa2 = wa0 ^ (2 << 5), wa3 = wa0 ^ (3 << 5);
        auto wa_at = [&](int mt) { return mt == 0 ? wa0 : mt == 1 ? wa1 : mt == 2 ? wa2 : wa3; };
        // Contraction of the block in x slot sl and w slot sw (constants in the
        // loop, so the slot offsets become immediates; the last block's are
        // run-time values, one code path instead of one per slot).  K slot
        // (g, t) of both contraction operands is block row 8g + t, the point
        // (t >> 2, 4g + (t & 3)) of the producer's tiles.
        auto contract = [&](int sl, int sw) {
            Frag<T> a[MT];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) tr_frag<WROW>(a[mt], lds + wa_at(mt) + sw * WTILE);
            f32x4 xw[2];
#pragma unroll
            for (int pt = 0; pt < 2; ++pt) xw[pt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < CK; ++kc)
#pragma unroll
                for (int pt = 0; pt < 2; ++pt) {
                    Frag<T> xa;
                    xa.v = *reinterpret_cast<const bf16x8 *>(lds + xl_at(pt, kc) + sl * XTILE);
                    mma(xw[pt], xa, w1[kc]);  // lane (g, i): points (pt, 4g + r), column i
                    mma(xw[pt], xa, w1l[kc]);
                }
            const f32x4 v0 = *reinterpret_cast<const f32x4 *>(vring + sw * 32 + 4 * g);
            const f32x4 v1 = *reinterpret_cast<const f32x4 *>(vring + sw * 32 + 16 + 4 * g);
            // xw / S (its rounded value and rounded remainder) and 1 / S, in K-slot order
            const float y[8] = {xw[0][0] * v0[0], xw[0][1] * v0[1], xw[0][2] * v0[2], xw[0][3] * v0[3],
                                xw[1][0] * v1[0], xw[1][1] * v1[1], xw[1][2] * v1[2], xw[1][3] * v1[3]};
            Frag<T> bt, btl, bd;
#pragma unroll
            for (int t = 0; t < 8; t += 2) bt.set2(t, y[t], y[t + 1]);
            const u32x4 hb = __builtin_bit_cast(u32x4, bt.v);
#pragma unroll
            for (int t = 0; t < 8; t += 2)
                btl.set2(t, y[t] - __uint_as_float(hb[t >> 1] << 16),
                         y[t + 1] - __uint_as_float(hb[t >> 1] & 0xffff0000u));
            bd.set2(0, v0[0], v0[1]);
            bd.set2(2, v0[2], v0[3]);
            bd.set2(4, v1[0], v1[1]);
            bd.set2(6, v1[2], v1[3]);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                mma(Tt[mt], a[mt], bt);
                mma(Tt[mt], a[mt], btl);
                mma(Dd[mt], a[mt], bd);
            }
            __builtin_amdgcn_sched_barrier(0);
        };
        auto step = [&](int j, auto slot, auto wslot) {
            constexpr int SL = decltype(slot)::value, SW = decltype(wslot)::value;
            constexpr int PREV = (SL + NSX - 1) % NSX, PREVW = (SW + NSW - 1) % NSW;
            asm volatile("" : "+v"(xl00), "+v"(xl01), "+v"(xl02), "+v"(xl03), "+v"(xl10), "+v"(xl11), "+v"(xl12),
                         "+v"(xl13));
            asm volatile("" : "+v"(wa0), "+v"(wa1), "+v"(wa2), "+v"(wa3));
            contract(PREV, PREVW);  // block j-1
            end_step(j, ic<PREV>{}, ic<1>{});
        };
        run_steps(step);
        {   // the last block (slots 3 and 1 if there was none)
            const int last = (nit + NSX - 1) % NSX;
            contract(last, last & 1);
        }
        __syncthreads();  // the pipeline's LDS becomes the reduction buffer
        float *mine = red + (size_t)pair * Cfg::E;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = mt * 16 + g * 4 + r;
                mine[m * (DH + 1) + li] = Tt[mt][r];
                if (li == 0) mine[m * (DH + 1) + DH] = Dd[mt][r];
            }
        __syncthreads();
    }

    // Fixed-order reduction: head h0 + hh is the sum of its streams' pairs in
    // stream order.
    constexpr int E = Cfg::E;
    for (int e = threadIdx.x; e < 2 * E; e += Cfg::WAVES * 64) {
        const int hh = e / E, er = e - hh * E;
        const float *src = red + (size_t)(NST * hh) * E + er;
        float acc = src[0];
#pragma unroll
        for (int q = 1; q < NST; ++q) acc += src[q * E];
        partials[((size_t)(span0 + span_local) * H + 2 * hp + hh) * (size_t)E + er] = acc;
    }
}

}  // namespace ts3
