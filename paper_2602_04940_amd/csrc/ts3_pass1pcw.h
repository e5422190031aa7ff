// Pass 1 for wide rows (bf16, C = 256) on eight waves, two heads per
// workgroup, with the two waves of each SIMD in different roles: the
// computation of k_slice_accumulate (paper Eq. (1) and Eq. (4), Algorithm 1
// tile loop).
//
// At C = 256 a head's W2'^T fragments take 128 VGPRs and its M x C float32
// accumulator 256, so each head gets four waves.  One workgroup per (span,
// head pair h0 = 2hp, h1 = 2hp + 1); wave w works on head h0 + ((w & 3) >> 1)
// and part w & 1:
//   w < 4  (producer) computes the logits of point tile `part` (16 of the 32
//          points) of block j (A = the head's W2'^T fragments, resident; B =
//          x rows from LDS), their softmax over the head's M slices, and
//          writes the tile's w rows to the head's w tile;
//   w >= 4 (consumer) contracts block j-1 for channel half `part`:
//          S[m][c] += sum_p w[p][m] x[p][c] over all M slices and the block's
//          32 points (operands from ds_read_b64_tr_b16), with d[m] += sum_p
//          w[p][m] on part 0, and issues a quarter of the x copies.
// Waves w and w + 4 share a SIMD, so every SIMD holds one producer and one
// consumer with about the same number of MFMAs per block (32, and 32 or 36):
// one wave's softmax runs beside the other's matrix work.  The consumers own
// disjoint parts of the span partial, so no reduction across waves is needed.
//
// A block's 16 KB of rows reach the LDS ring (four slots) by direct
// global->LDS copies issued three blocks ahead.  Each consumer waits for its
// own copies of block j+1 before the barrier that ends step j, which makes
// all of them visible for step j+1.  The w tiles have two slots per head
// (block j's are written in step j and read in step j+1).  Rows are unpadded
// and XOR-swizzled as in the other pass-1 kernels.  The order of every sum is
// fixed by (x, Q), so results do not depend on the tiling.  H is even: the
// one supported wide shape (M = 64) has H in {4, 8, 16}, since the token side
// needs dh <= 64.
#pragma once
#include "ts3_pass1.h"

namespace ts3 {

template <int C, int M> struct Pass1PCWCfg {
    static constexpr int WAVES = 8;
    static constexpr int MT = M / 16, CT = C / 16, CK = C / 32;
    static constexpr int CTH = CT / 2;                       // channel tiles per consumer
    static constexpr int XROW = C * 2, XTILE = 32 * XROW;    // 16 KB per 32-point block
    static constexpr int WROW = M * 2, WTILE = 32 * WROW;
    static constexpr int NSX = 4, NSW = 2, AHEAD = 3;
    static constexpr int ROWS_PER_LOAD = 1024 / XROW;        // rows per 1 KB copy
    static constexpr int LOADS = 32 / ROWS_PER_LOAD;         // copies per block
    static constexpr int C_LOADS = LOADS / 4;                // per consumer
    static constexpr int X_BYTES = NSX * XTILE;
    static constexpr int W_BYTES = 2 * NSW * WTILE;          // two heads
    static constexpr int LDS_BYTES = X_BYTES + W_BYTES;
    static_assert(C == 256 && ROWS_PER_LOAD == 2 && C_LOADS == 4, "written for 512-byte rows");
    static_assert(M % 16 == 0 && MT <= 4, "at most four 16-slice tiles per head");
};

// Arguments as k_slice_accumulate (H even); grid nspan * H / 2, 512 threads.
template <int C, int M>
__global__ __launch_bounds__(512, 1) void k_slice_accumulate_pcw(
    const bf16_t *__restrict__ x, int64_t n_tile, int64_t span0, int32_t Q, int32_t nspan, int32_t H,
    const bf16_t *__restrict__ w2p, const float *__restrict__ b2s, float *__restrict__ partials) {
    using Cfg = Pass1PCWCfg<C, M>;
    using T = bf16_t;
    constexpr int MT = Cfg::MT, CK = Cfg::CK, CTH = Cfg::CTH;
    constexpr int NSX = Cfg::NSX, NSW = Cfg::NSW, AHEAD = Cfg::AHEAD;
    constexpr int XROW = Cfg::XROW, WROW = Cfg::WROW, XTILE = Cfg::XTILE, WTILE = Cfg::WTILE;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[Cfg::LDS_BYTES];

    const int HP = H / 2;
    const int nwg = nspan * HP;
    const int jwg = xcd_remap((int)blockIdx.x, nwg);  // a span's head pairs share an XCD (and its L2)
    const int span_local = jwg / HP;
    const int hp = jwg - span_local * HP;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int q = wave & 3, role = wave >> 2;  // role 0: logits and softmax, 1: contraction
    const int hsel = q >> 1, part = q & 1;
    const int h = 2 * hp + hsel;
    const int li = lane & 15, g = lane >> 4;

    const int64_t p_begin = (int64_t)span_local * Q;
    const int64_t p_end = p_begin + Q < n_tile ? p_begin + Q : n_tile;
    const int nrows = (int)(p_end - p_begin);  // <= Q <= 2^30
    const int nit = (nrows + 31) >> 5;        // blocks, the same for every wave

    unsigned char *const xring = lds;
    unsigned char *const wring = lds + Cfg::X_BYTES + hsel * NSW * WTILE;
    const uint32_t xring_lds = lds_addr(xring);

    // Consumer q's quarter of block j's copies into x slot SL: copies 4q ..
    // 4q+3, each two rows; rows past the span's end repeat its last row.
    constexpr int NCH = XROW / 16;
    auto issue_x = [&](int j, auto slot) {
        constexpr int SL = decltype(slot)::value;
        const int r0 = j << 5;
        const uint32_t dst = xring_lds + SL * XTILE;
        if (__builtin_expect(r0 + 32 <= nrows, 1)) {
            const void *base = x + (p_begin + r0) * C;
#pragma unroll
            for (int kk = 0; kk < Cfg::C_LOADS; ++kk) {
                const int i = Cfg::C_LOADS * q + kk;
                const int R = i * Cfg::ROWS_PER_LOAD + lane / NCH;
                dma16s<0>((uint32_t)(R * XROW + (((lane % NCH) ^ xswz<XROW>(R)) << 4)), base, dst + i * 1024);
            }
        } else {
#pragma unroll
            for (int kk = 0; kk < Cfg::C_LOADS; ++kk) {
                const int i = Cfg::C_LOADS * q + kk;
                const int R = i * Cfg::ROWS_PER_LOAD + lane / NCH;
                const int ch = (lane % NCH) ^ xswz<XROW>(R);
                const int r = r0 + R < nrows ? r0 + R : nrows - 1;
                dma16(reinterpret_cast<const unsigned char *>(x + (size_t)(p_begin + r) * C) + ch * 16, dst + i * 1024);
            }
        }
    };
    auto block_valid = [&](int j) {
        const int left = nrows - (j << 5);
        return left <= 0 ? 0 : left < 32 ? left : 32;
    };

    // Shared start of both roles (each role runs it after its own loads):
    // zero "block -1" (x slot NSX-1 and both heads' w slot NSW-1), so the first
    // contraction adds nothing, and copy blocks 0..2.
    auto prologue = [&](auto rl) {
        constexpr bool CONS = decltype(rl)::value == 1;
        wait_vmcnt<0>();  // the ring's wait counts assume only its own copies are in flight
        uint4 *zx = reinterpret_cast<uint4 *>(xring + (NSX - 1) * XTILE);
        for (int i = wave * 64 + lane; i < XTILE / 16; i += 512) zx[i] = uint4{0u, 0u, 0u, 0u};
        uint4 *zw = reinterpret_cast<uint4 *>(wring + (NSW - 1) * WTILE);
        for (int i = (role * 2 + part) * 64 + lane; i < WTILE / 16; i += 256) zw[i] = uint4{0u, 0u, 0u, 0u};
        if constexpr (CONS) {
            issue_x(0, ic<0>{});
            issue_x(1, ic<1>{});
            issue_x(2, ic<2>{});
            wait_vmcnt<2 * Cfg::C_LOADS>();  // this wave's copies of block 0
        }
        __syncthreads();  // everyone's copies of block 0 and the zero tiles visible
    };
    static_assert(NSX == 4 && NSW == 2 && AHEAD == 3, "the unrolled loops below assume these ring depths");

    // The end of every step: this wave's copies of block j+1 have landed
    // (those of block j+2 may not have); the barrier makes every wave's copies
    // of block j+1 visible, with block j's w rows; then the copies of block
    // j + AHEAD go into the slot block j-1 released.
    auto end_step = [&](int j, auto prev, auto rl) {
        constexpr bool CONS = decltype(rl)::value == 1;
        if constexpr (CONS) wait_vmcnt<Cfg::C_LOADS>();
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __syncthreads();
        // (Issued past the last block too, as clamped rows, so that every
        // step's wait count is the same.)
        if constexpr (CONS) issue_x(j + AHEAD, prev);
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

    const int R = prow(part, li);  // this lane's point row in the producer's tile
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
        prologue(ic<0>{});
        // The x fragment of step kc+1 is read while step kc's MFMAs run.
        auto logits = [&](auto slot, f32x4 (&L)[MT]) {
            constexpr int SL = decltype(slot)::value;
            const unsigned char *xt = lds + SL * XTILE;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) L[mt] = bias[mt];
            Frag<T> xb[2];
            xb[0].v = *reinterpret_cast<const bf16x8 *>(xt + xoff<XROW>(R, (g * 8) * 2));
#pragma unroll
            for (int kc = 0; kc < CK; ++kc) {
                __builtin_amdgcn_sched_barrier(0);
                if (kc + 1 < CK)
                    xb[(kc + 1) & 1].v = *reinterpret_cast<const bf16x8 *>(xt + xoff<XROW>(R, ((kc + 1) * 32 + g * 8) * 2));
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) mma(L[mt], w2[mt][kc], xb[kc & 1]);
                if (kc + 1 < CK) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, MT, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        };
        auto step = [&](int j, auto slot, auto wslot) {
            constexpr int SL = decltype(slot)::value, SW = decltype(wslot)::value;
            constexpr int PREV = (SL + NSX - 1) % NSX;
            {
                const int valid = block_valid(j);
                f32x4 L[MT];
                // The producer's logits MFMAs go first on the SIMD's matrix
                // core; the consumer's contraction fills the softmax after it.
                __builtin_amdgcn_s_setprio(2);
                logits(slot, L);
                __builtin_amdgcn_s_setprio(0);
                float sum = 0.f;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float e = fast_exp2(L[mt][r]);
                        L[mt][r] = e;
                        sum += e;
                    }
                sum = xrow_sum(sum);
                float inv = R < valid ? fast_rcp(sum) : 0.f;  // padding points weigh nothing
                if (__any(!softmax_sum_ok(sum))) {
                    // Rare: a row's exp2 sum left the safe window; redo the
                    // tile's rows with the max shift.
                    logits(slot, L);
                    float mx = L[0][0];
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                        for (int r = 0; r < 4; ++r) mx = fmaxf(mx, L[mt][r]);
                    mx = xrow_max(mx);
                    float s2 = 0.f;
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const float e = fast_exp2(L[mt][r] - mx);
                            L[mt][r] = e;
                            s2 += e;
                        }
                    inv = R < valid ? fast_rcp(xrow_sum(s2)) : 0.f;
                }
                typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
                unsigned char *wt = wring + SW * WTILE;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    *reinterpret_cast<bf16x4 *>(wt + woff<WROW>(R, (mt * 16 + g * 4) * 2)) =
                        bf16x4{(__bf16)(L[mt][0] * inv), (__bf16)(L[mt][1] * inv), (__bf16)(L[mt][2] * inv),
                               (__bf16)(L[mt][3] * inv)};
            }
            end_step(j, ic<PREV>{}, ic<0>{});
        };
        run_steps(step);
    } else {
        // ---------------------------------------------------------------- consumer
        prologue(ic<1>{});
        f32x4 S[MT][CTH];
        f32x4 D[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            D[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ct = 0; ct < CTH; ++ct) S[mt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        Frag<T> ones;
        ones8(ones);
        const int c0 = part * (C / 2);
        // Contraction of the block in x slot sl and w slot sw (constants in
        // the loop; the last block's are run-time values); the xT fragment of
        // channel tile ct+1 is read while tile ct's MFMAs run.
        auto contract = [&](int sl, int sw) {
            const unsigned char *xt = lds + sl * XTILE, *wt = wring + sw * WTILE;
            Frag<T> a[MT], b;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) tr_frag<WROW>(a[mt], tr_addr<WROW, false>(wt, g, mt * 16, li));
            tr_frag<XROW>(b, tr_addr<XROW, true>(xt, g, c0, li));
            __builtin_amdgcn_sched_barrier(0);
            if (part == 0)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) mma(D[mt], a[mt], ones);
#pragma unroll
            for (int ct = 0; ct < CTH; ++ct) {
                Frag<T> bn;
                if (ct + 1 < CTH) tr_frag<XROW>(bn, tr_addr<XROW, true>(xt, g, c0 + (ct + 1) * 16, li));
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) mma(S[mt][ct], a[mt], b);
                b = bn;
            }
            __builtin_amdgcn_sched_barrier(0);
        };
        auto step = [&](int j, auto slot, auto wslot) {
            constexpr int SL = decltype(slot)::value, SW = decltype(wslot)::value;
            constexpr int PREV = (SL + NSX - 1) % NSX, PREVW = (SW + NSW - 1) % NSW;
            contract(PREV, PREVW);  // block j-1
            end_step(j, ic<PREV>{}, ic<1>{});
        };
        run_steps(step);
        {
            // the last block (slots 3 and 1 if there was none)
            const int last = (nit + NSX - 1) % NSX;
            contract(last, last & 1);
            // This consumer's channels of the span partial; part 0 adds column C (d).
            float *dst = partials + ((size_t)(span0 + span_local) * H + h) * M * (C + 1);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int m = mt * 16 + g * 4 + r;
#pragma unroll
                    for (int ct = 0; ct < CTH; ++ct) dst[(size_t)m * (C + 1) + c0 + ct * 16 + li] = S[mt][ct][r];
                    if (part == 0 && li == 0) dst[(size_t)m * (C + 1) + C] = D[mt][r];
                }
        }
    }
}

}  // namespace ts3
