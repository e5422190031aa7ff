// Pass 1 on eight waves, two heads per workgroup, with the two waves of each
// SIMD in different roles, for 16-bit storage, C = 128 and M >= 32: the
// computation of k_slice_accumulate (paper Eq. (1) and Eq. (4), Algorithm 1
// tile loop).
//
// One workgroup per (span, head pair h0 = 2hp, h1 = 2hp + 1).  Pair q (waves
// q and q+4, which share a SIMD) works on head h0 + (q >> 1) and on block
// stream q & 1 (the span's 32-point blocks 0, 2, 4, ... or 1, 3, 5, ...), so
// each stream's blocks serve one pair of each head and every x row is copied
// into LDS once for two heads.  Within a pair the work is split by kind:
//   wave q   (producer) computes the logits of all 32 points of block j (A =
//            W2'^T fragments resident in registers, B = x^T from LDS), their
//            softmax over the head's M slices, and writes the w rows to the
//            pair's w tile;
//   wave q+4 (consumer) contracts block j-1 over all M slices:
//            S[m][c] += sum_p w[p][m] x[p][c] and d[m] += sum_p w[p][m],
//            operands from ds_read_b64_tr_b16, and issues the x copies.
// One wave of the SIMD then runs matrix-core work while the other runs the
// softmax's vector work, instead of both running the same phase at once (as
// they did when each wave took half the rows of both phases: 1 ms slower per
// layer at 100M points).
//
// A block's 8 KB of rows reach the stream's LDS ring (four slots) by direct
// global->LDS copies issued three blocks ahead; the consumers issue all eight
// 1 KB copies (giving the producer half of its head's copies measured 1 ms
// slower per layer: it is the longer of the two waves).  Each consumer waits
// for its own copies of block j+1 before the barrier that ends step j, which
// makes all of them visible for step j+1.  The w tiles have two slots (block
// j's are written in step j and read in step j+1).  Tile rows are unpadded and
// XOR-swizzled for the LDS access phases (no bank conflicts); every tile
// address is a register plus an immediate offset.  The two streams'
// accumulators of a head are summed in a fixed order at the end, and every
// tiling of a shape sums a span the same way (tiled and untiled runs agree
// bitwise).
//
// Measured alternatives: interleaving the producer's exp2 with its logits
// MFMAs (slice tiles outermost) changed nothing; running the producer one
// block behind (softmax of block j-1, then logits of block j, beside the
// contraction of block j-2, on a six-slot ring) was 0.5 ms slower per layer.
#pragma once
#include "ts3_pass1.h"

namespace ts3 {

template <int C, int M> struct Pass1PCCfg {
    using T = bf16_t;
    static constexpr int WAVES = 8, PAIRS = 4, STREAMS = 2;
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
    static constexpr int RED_BYTES = PAIRS * M * (C + 1) * 4;
    static constexpr int PIPE_BYTES = X_BYTES + W_BYTES;
    static constexpr int LDS_BYTES = PIPE_BYTES > RED_BYTES ? PIPE_BYTES : RED_BYTES;
    static_assert(ROWS_PER_LOAD == 4 && HEAD_LOADS == 4, "copies split as whole 1 KB pieces");
    static_assert(CK == 4 && CT == 8 && MT <= 4, "the address sets are written for C = 128, M <= 64");
};

// Arguments as k_slice_accumulate (H even); grid nspan * H / 2, 512 threads.
template <int C, int M>
__global__ __launch_bounds__(512, 1) void k_slice_accumulate_pc(
    const bf16_t *__restrict__ x, int64_t n_tile, int64_t span0, int32_t Q, int32_t nspan, int32_t H,
    const bf16_t *__restrict__ w2p, const float *__restrict__ b2s, float *__restrict__ partials) {
    using Cfg = Pass1PCCfg<C, M>;
    using T = bf16_t;
    constexpr int MT = Cfg::MT, CT = Cfg::CT, CK = Cfg::CK;
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
    const int pair = wave & 3, role = wave >> 2;  // role 0: logits and softmax, 1: contraction
    const int stream = pair & 1, hsel = pair >> 1;
    const int h = 2 * hp + hsel;
    const int li = lane & 15, g = lane >> 4;

    const int64_t p_begin = (int64_t)span_local * Q;
    const int64_t p_end = p_begin + Q < n_tile ? p_begin + Q : n_tile;
    const int nrows = (int)(p_end - p_begin);  // <= Q <= 2^30
    const int nblk = (nrows + 31) >> 5;
    const int nit = (nblk + 1) >> 1;  // block steps, the same for every wave

    unsigned char *const xring = lds + stream * NSX * XTILE;
    unsigned char *const wring = lds + Cfg::X_BYTES + pair * NSW * WTILE;
    const uint32_t xring_lds = lds_addr(xring);

    // This wave's share of block j of its stream (mesh block stream + 2j) into
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
        const int r0 = (stream + 2 * j) << 5;
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
        const int left = nrows - ((stream + 2 * j) << 5);
        return left <= 0 ? 0 : left < 32 ? left : 32;
    };

    // Shared start of both roles (each role runs it after its own loads):
    // zero "block -1" (x slot NSX-1, w slot NSW-1), so the first contraction
    // adds nothing, and copy blocks 0..2.
    auto prologue = [&](auto rl) {
        constexpr int NL = decltype(rl)::value == 0 ? Cfg::P_LOADS : Cfg::C_LOADS;
        wait_vmcnt<0>();  // the ring's wait counts assume only its own copies are in flight
        uint4 *zx = reinterpret_cast<uint4 *>(xring + (NSX - 1) * XTILE);
        uint4 *zw = reinterpret_cast<uint4 *>(wring + (NSW - 1) * WTILE);
        const int sidx = hsel * 2 + role;  // 0..3 within the stream
        for (int i = sidx * 64 + lane; i < XTILE / 16; i += 256) zx[i] = uint4{0u, 0u, 0u, 0u};
        for (int i = role * 64 + lane; i < WTILE / 16; i += 128) zw[i] = uint4{0u, 0u, 0u, 0u};
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
                inv[pt] = prow(pt, li) < valid ? fast_rcp(sum) : 0.f;  // padding points weigh nothing
            }
            if (__any(!ok)) {
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
                    float s2 = 0.f;
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const float e = fast_exp2(L[mt][pt][r] - mx);
                            L[mt][pt][r] = e;
                            s2 += e;
                        }
                    inv[pt] = prow(pt, li) < valid ? fast_rcp(xrow_sum(s2)) : 0.f;
                }
            }
            typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
#pragma unroll
            for (int pt = 0; pt < 2; ++pt)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    *reinterpret_cast<bf16x4 *>(lds + ws_at(pt, mt) + SW * WTILE) =
                        bf16x4{(__bf16)(L[mt][pt][0] * inv[pt]), (__bf16)(L[mt][pt][1] * inv[pt]),
                               (__bf16)(L[mt][pt][2] * inv[pt]), (__bf16)(L[mt][pt][3] * inv[pt])};
            end_step(j, ic<PREV>{}, ic<0>{});
        };
        run_steps(step);
        __syncthreads();  // the pipeline's LDS becomes the reduction buffer
        __syncthreads();  // the consumers' accumulators are in it
    } else {
        // ---------------------------------------------------------------- consumer
        prologue(ic<1>{});
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
        // xT fragment addresses of channel tile ct and wT fragment addresses of
        // slice tile mt, held in registers.
        uint32_t xt0 = xbase + xoff<XROW>(8 * g + (li >> 2), 8 * (li & 3));
        uint32_t xt1 = xt0 ^ (1 << 5), xt2 = xt0 ^ (2 << 5), xt3 = xt0 ^ (3 << 5), xt4 = xt0 ^ (4 << 5),
                 xt5 = xt0 ^ (5 << 5), xt6 = xt0 ^ (6 << 5), xt7 = xt0 ^ (7 << 5);
        auto xt_at = [&](int ct) {
            return ct == 0 ? xt0 : ct == 1 ? xt1 : ct == 2 ? xt2 : ct == 3 ? xt3 : ct == 4 ? xt4 : ct == 5 ? xt5 : ct == 6 ? xt6 : xt7;
        };
        uint32_t wa0 = wbase + woff<WROW>(8 * g + (li >> 2), 8 * (li & 3));
        uint32_t wa1 = wa0 ^ (1 << 5), wa2 = wa0 ^ (2 << 5), wa3 = wa0 ^ (3 << 5);
        auto wa_at = [&](int mt) { return mt == 0 ? wa0 : mt == 1 ? wa1 : mt == 2 ? wa2 : wa3; };
        // Contraction of the block in x slot SL and w slot SW; the xT fragment
        // of channel tile ct+1 is read while tile ct's MFMAs run.
        // Contraction of the block in x slot sl and w slot sw (constants in the
        // loop, so the slot offsets become immediates; the last block's are
        // run-time values, one code path instead of one per slot).
        auto contract = [&](int sl, int sw) {
            Frag<T> a[MT], b;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) tr_frag<WROW>(a[mt], lds + wa_at(mt) + sw * WTILE);
            tr_frag<XROW>(b, lds + xt_at(0) + sl * XTILE);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) mma(D[mt], a[mt], ones);
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                Frag<T> bn;
                if (ct + 1 < CT) tr_frag<XROW>(bn, lds + xt_at(ct + 1) + sl * XTILE);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) mma(S[mt][ct], a[mt], b);
                b = bn;
            }
            __builtin_amdgcn_sched_barrier(0);
        };
        auto step = [&](int j, auto slot, auto wslot) {
            constexpr int SL = decltype(slot)::value, SW = decltype(wslot)::value;
            constexpr int PREV = (SL + NSX - 1) % NSX, PREVW = (SW + NSW - 1) % NSW;
            asm volatile("" : "+v"(xt0), "+v"(xt1), "+v"(xt2), "+v"(xt3), "+v"(xt4), "+v"(xt5), "+v"(xt6), "+v"(xt7));
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
        float *mine = red + (size_t)pair * M * (C + 1);
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
    }

    // Fixed-order reduction: head h0 + hh is stream 0's pair plus stream 1's.
    constexpr int E = M * (C + 1);
    for (int e = threadIdx.x; e < 2 * E; e += 512) {
        const int hh = e / E, er = e - hh * E;
        const float *src = red + (size_t)(2 * hh) * E + er;
        partials[((size_t)(span0 + span_local) * H + 2 * hp + hh) * (size_t)E + er] = src[0] + src[E];
    }
}

}  // namespace ts3
