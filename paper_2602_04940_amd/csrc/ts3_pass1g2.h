// Pass 1 on eight waves with two heads per workgroup, for 16-bit storage,
// C = 128 and M >= 32: the computation of k_slice_accumulate (paper Eq. (1)
// and Eq. (4), Algorithm 1 tile loop), with each x row copied into LDS once
// for two heads instead of once per head.
//
// One workgroup per (span, head pair h0 = 2hp, h1 = 2hp + 1).  Wave pair q
// (waves q and q+4) works on head h0 + (q >> 1) and on block stream q & 1:
// pairs 0 and 2 take the span's 32-point blocks 0, 2, 4, ..., pairs 1 and 3
// the blocks 1, 3, 5, ..., so each stream's blocks are shared by one pair of
// each head.  Within a pair, wave q + 4*hf
//   computes the logits and softmax of the block's rows prow(hf, .) (its 16
//            points) over all M slices of its head (A = W2'^T fragments
//            resident in registers, B = x^T from LDS) and writes their w rows
//            to the pair's w tile;
//   contracts slices hf*M/2 .. hf*M/2 + M/2 - 1 over all 32 points of the
//            previous block: S_own[m][c] += sum_p w[p][m] x[p][c] and d_own[m]
//            += sum_p w[p][m], operands from ds_read_b64_tr_b16.
// The rows prow(hf, .) of a block are four 1 KB copies; the hf-waves of the
// stream's two pairs issue two each, so a wave's logits read rows copied by
// another wave.  Copies go three blocks ahead into a stream ring of four x
// slots, and each wave waits for its own copies of block j+1 before the
// barrier that ends step j, which makes them visible for step j+1.  The two
// heads' accumulators are summed over their two pairs in a fixed order at the
// end and written as two span partials [M][C+1].
#pragma once
#include "ts3_pass1.h"

namespace ts3 {

template <int C, int M> struct Pass1G2Cfg {
    using T = bf16_t;
    static constexpr int WAVES = 8, PAIRS = 4, STREAMS = 2;
    static constexpr int MT = M / 16;             // 16-slice tiles of a head
    static constexpr int MH = M / 2;              // slices contracted per wave
    static constexpr int MTH = MH / 16;
    static constexpr int CT = C / 16, CK = C / 32;
    static constexpr int XROW = C * 2, XTILE = 32 * XROW;
    static constexpr int WROW = M * 2, WTILE = 32 * WROW;
    // x slots per stream and w tiles per pair.  Block j's copies are issued at
    // the end of step j-3 into the slot of block j-4, released by step j-3's
    // barrier (block j-4's contraction runs in step j-3); block j's w tile is
    // read in step j+1, before step j+2 rewrites its slot.
    static constexpr int NSX = 4, NSW = 2, AHEAD = 3;
    static constexpr int ROWS_PER_LOAD = 1024 / XROW, LOADS = 32 / ROWS_PER_LOAD;
    static constexpr int MY_LOADS = LOADS / 4;    // copies per wave per block
    static constexpr int X_BYTES = STREAMS * NSX * XTILE;
    static constexpr int W_BYTES = PAIRS * NSW * WTILE;
    static constexpr int RED_BYTES = WAVES * MH * (C + 1) * 4;
    static constexpr int PIPE_BYTES = X_BYTES + W_BYTES;
    static constexpr int LDS_BYTES = PIPE_BYTES > RED_BYTES ? PIPE_BYTES : RED_BYTES;
    static_assert(MH % 16 == 0, "each wave contracts whole 16-slice tiles");
    // A 1 KB copy holds rows 4i .. 4i+3 at C = 128; the rows of point tile hf
    // (row bit 2 = hf) are the copies i = 2k + hf.
    static_assert(ROWS_PER_LOAD == 4 && MY_LOADS == 2, "copies split as whole 1 KB pieces");
};

// Arguments as k_slice_accumulate (H even); grid nspan * H / 2, 512 threads.
template <int C, int M>
__global__ __launch_bounds__(512, 1) void k_slice_accumulate_g2(
    const bf16_t *__restrict__ x, int64_t n_tile, int64_t span0, int32_t Q, int32_t nspan, int32_t H,
    const bf16_t *__restrict__ w2p, const float *__restrict__ b2s, float *__restrict__ partials) {
    using Cfg = Pass1G2Cfg<C, M>;
    using T = bf16_t;
    constexpr int MT = Cfg::MT, MTH = Cfg::MTH, CT = Cfg::CT, CK = Cfg::CK, MH = Cfg::MH;
    constexpr int NSX = Cfg::NSX, NSW = Cfg::NSW, AHEAD = Cfg::AHEAD, MY_LOADS = Cfg::MY_LOADS;
    constexpr int XROW = Cfg::XROW, WROW = Cfg::WROW, XTILE = Cfg::XTILE, WTILE = Cfg::WTILE;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[Cfg::LDS_BYTES];

    const int HP = H / 2;
    const int nwg = nspan * HP;
    const int jwg = xcd_remap((int)blockIdx.x, nwg);  // a span's head pairs share an XCD (and its L2)
    const int span_local = jwg / HP;
    const int hp = jwg - span_local * HP;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int pair = wave & 3, hf = wave >> 2;
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
    // x slot SL: copies i = 2k + hf for k = 2*hsel, 2*hsel + 1; lane mapping
    // and rows past the span's end as in k_slice_accumulate.
    constexpr int NCH = XROW / 16;
    auto copy_off = [&](int i) {
        const int R = i * Cfg::ROWS_PER_LOAD + lane / NCH;
        return (uint32_t)(R * XROW + (((lane % NCH) ^ xswz<XROW>(R)) << 4));
    };
    // Row offsets within the span are 32-bit; only the global base is 64-bit.
    auto issue_x = [&](int j, auto slot) {
        constexpr int SL = decltype(slot)::value;
        const int r0 = (stream + 2 * j) << 5;
        const uint32_t dst = xring_lds + SL * XTILE;
        if (__builtin_expect(r0 + 32 <= nrows, 1)) {
            const void *base = x + (p_begin + r0) * C;
#pragma unroll
            for (int kk = 0; kk < MY_LOADS; ++kk) {
                const int i = 2 * (2 * hsel + kk) + hf;
                dma16s<0>(copy_off(i), base, dst + i * 1024);
            }
        } else {
#pragma unroll
            for (int kk = 0; kk < MY_LOADS; ++kk) {
                const int i = 2 * (2 * hsel + kk) + hf;
                const int R = i * Cfg::ROWS_PER_LOAD + lane / NCH;
                const int ch = (lane % NCH) ^ xswz<XROW>(R);
                const int r = r0 + R < nrows ? r0 + R : nrows - 1;
                dma16(reinterpret_cast<const unsigned char *>(x + (size_t)(p_begin + r) * C) + ch * 16, dst + i * 1024);
            }
        }
    };

    // Head h's W2'^T fragments (all slices) and bias, resident.
    Frag<T> w2[MT][CK];
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
    f32x4 S[MTH][CT];
    f32x4 D[MTH];
#pragma unroll
    for (int mt = 0; mt < MTH; ++mt) {
        D[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) S[mt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    Frag<T> ones;
    ones8(ones);
    wait_vmcnt<0>();  // the ring's wait counts assume only its own copies are in flight

    // Tile addresses as in k_slice_accumulate: (per-lane base) ^ (tile index
    // constant) + (immediate), relative to lds.  This wave's point tile is hf
    // (row bit 2), its contraction slices the tiles hf*MTH .. hf*MTH+MTH-1.
    const uint32_t xbase = (uint32_t)(stream * NSX * XTILE);
    const uint32_t wbase = (uint32_t)(Cfg::X_BYTES + pair * NSW * WTILE);
    const uint32_t xl0 = xbase + xoff<XROW>(prow(hf, li), 16 * g);
    const uint32_t xt0 = xbase + xoff<XROW>(8 * g + (li >> 2), 8 * (li & 3));
    // The x-tile addresses of every K step (logits) and channel tile
    // (contraction), computed once and held in registers: an XOR in front
    // of each read costs more than the registers.
    static_assert(CK == 4 && CT == 8, "the address sets below are written for C = 128");
    uint32_t xl1 = xl0 ^ (1 << 6), xl2 = xl0 ^ (2 << 6), xl3 = xl0 ^ (3 << 6);
    uint32_t xt1 = xt0 ^ (1 << 5), xt2 = xt0 ^ (2 << 5), xt3 = xt0 ^ (3 << 5), xt4 = xt0 ^ (4 << 5),
             xt5 = xt0 ^ (5 << 5), xt6 = xt0 ^ (6 << 5), xt7 = xt0 ^ (7 << 5);
    uint32_t xl0v = xl0, xt0v = xt0;
    auto xl_at = [&](int kc) { return kc == 0 ? xl0v : kc == 1 ? xl1 : kc == 2 ? xl2 : xl3; };
    auto xt_at = [&](int ct) {
        return ct == 0 ? xt0v : ct == 1 ? xt1 : ct == 2 ? xt2 : ct == 3 ? xt3 : ct == 4 ? xt4 : ct == 5 ? xt5 : ct == 6 ? xt6 : xt7;
    };
    uint32_t wt0 = wbase + woff<WROW>(8 * g + (li >> 2), 8 * (li & 3));
    uint32_t ws0 = wbase + woff<WROW>(prow(hf, li), 8 * g);

    // The x fragment of step kc+1 is read while step kc's MFMAs run.
    auto logits = [&](auto slot, f32x4 (&L)[MT]) {
        constexpr int SL = decltype(slot)::value;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) L[mt] = bias[mt];
        Frag<T> xb[2];
        xb[0].v = *reinterpret_cast<const bf16x8 *>(lds + xl_at(0) + SL * XTILE);
#pragma unroll
        for (int kc = 0; kc < CK; ++kc) {
            __builtin_amdgcn_sched_barrier(0);
            if (kc + 1 < CK)
                xb[(kc + 1) & 1].v = *reinterpret_cast<const bf16x8 *>(lds + xl_at(kc + 1) + SL * XTILE);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) mma(L[mt], w2[mt][kc], xb[kc & 1]);
            if (kc + 1 < CK) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, MT, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    auto read_a = [&](auto wslot, Frag<T> (&a)[MTH]) {
        constexpr int SW = decltype(wslot)::value;
#pragma unroll
        for (int mt = 0; mt < MTH; ++mt)
            tr_frag<WROW>(a[mt], lds + (wt0 ^ ((hf * MTH + mt) << 5)) + SW * WTILE);
    };
    auto read_b = [&](auto slot, int ct, Frag<T> &b) {
        constexpr int SL = decltype(slot)::value;
        tr_frag<XROW>(b, lds + xt_at(ct) + SL * XTILE);
    };
    auto contract = [&](auto slot, auto wslot) {
        Frag<T> a[MTH], b;
        read_a(wslot, a);
#pragma unroll
        for (int mt = 0; mt < MTH; ++mt) mma(D[mt], a[mt], ones);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            read_b(slot, ct, b);
#pragma unroll
            for (int mt = 0; mt < MTH; ++mt) mma(S[mt][ct], a[mt], b);
        }
    };
    auto store_w = [&](auto wslot, const f32x4 (&E)[MT], float inv) {
        constexpr int SW = decltype(wslot)::value;
        typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            *reinterpret_cast<bf16x4 *>(lds + (ws0 ^ (mt << 5)) + SW * WTILE) =
                bf16x4{(__bf16)(E[mt][0] * inv), (__bf16)(E[mt][1] * inv), (__bf16)(E[mt][2] * inv),
                       (__bf16)(E[mt][3] * inv)};
    };
    auto block_valid = [&](int j) {
        const int left = nrows - ((stream + 2 * j) << 5);
        return left <= 0 ? 0 : left < 32 ? left : 32;
    };

    // Step j (block j of the stream, x slot SL = j % NSX, w slot SW = j % NSW):
    // this wave's logits and softmax (16 points, all slices) beside the
    // previous block's contraction (its slices, 32 points), the w rows, the
    // wait for its copies of block j+1, one barrier, then the copies of block
    // j + AHEAD into the slot the previous block released.
    auto step = [&](int j, auto slot, auto wslot) {
        constexpr int SL = decltype(slot)::value, SW = decltype(wslot)::value;
        constexpr int PREV = (SL + NSX - 1) % NSX, PREVW = (SW + NSW - 1) % NSW;
        asm volatile("" : "+v"(xl0v), "+v"(xl1), "+v"(xl2), "+v"(xl3), "+v"(wt0), "+v"(ws0));
        asm volatile("" : "+v"(xt0v), "+v"(xt1), "+v"(xt2), "+v"(xt3), "+v"(xt4), "+v"(xt5), "+v"(xt6), "+v"(xt7));
        const bool row_valid = prow(hf, li) < block_valid(j);
        Frag<T> a[MTH], b;
        read_a(ic<PREVW>{}, a);
        read_b(ic<PREV>{}, 0, b);
        f32x4 L[MT];
        logits(slot, L);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int mt = 0; mt < MTH; ++mt) mma(D[mt], a[mt], ones);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            Frag<T> bn;
            if (ct + 1 < CT) read_b(ic<PREV>{}, ct + 1, bn);
#pragma unroll
            for (int mt = 0; mt < MTH; ++mt) mma(S[mt][ct], a[mt], b);
            b = bn;
        }
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
        const bool ok = softmax_sum_ok(sum);
        float inv = row_valid ? fast_rcp(sum) : 0.f;  // padding points weigh nothing
        interleave_chain<0, MTH * (CT + 1), 3, MTH - 1, MTH, 2, 0>();
        __builtin_amdgcn_sched_barrier(0);
        if (__any(!ok)) {
            // Rare: a row's exp2 sum left the safe window; redo this wave's
            // rows with the max shift.
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
            inv = row_valid ? fast_rcp(xrow_sum(s2)) : 0.f;
        }
        store_w(wslot, L, inv);
        // This wave's copies of block j+1 have landed (those of block j+2 may
        // not have); the barrier makes every wave's copies of block j+1
        // visible, with this block's w rows and the partner's.
        wait_vmcnt<MY_LOADS>();
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __syncthreads();  // block j-1's x slot is no longer read
        issue_x(j + AHEAD, ic<PREV>{});
    };

    // "Block -1" (x slot NSX-1, w slot NSW-1) holds zeros so the first
    // contraction adds nothing: the stream's four waves of each point half and
    // pair clear the tiles between them.
    {
        uint4 *zx = reinterpret_cast<uint4 *>(xring + (NSX - 1) * XTILE);
        uint4 *zw = reinterpret_cast<uint4 *>(wring + (NSW - 1) * WTILE);
        const int sidx = hsel * 2 + hf;  // 0..3 within the stream
        for (int i = sidx * 64 + lane; i < XTILE / 16; i += 256) zx[i] = uint4{0u, 0u, 0u, 0u};
        for (int i = hf * 64 + lane; i < WTILE / 16; i += 128) zw[i] = uint4{0u, 0u, 0u, 0u};
    }
    static_assert(NSX == 4 && NSW == 2 && AHEAD == 3, "the unrolled loop below assumes these ring depths");
    issue_x(0, ic<0>{});
    issue_x(1, ic<1>{});
    issue_x(2, ic<2>{});
    wait_vmcnt<2 * MY_LOADS>();  // this wave's copies of block 0
    __syncthreads();             // everyone's copies of block 0 and the zero tiles visible
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
    switch ((nit + NSX - 1) % NSX) {  // the last block (slots 3 and 1 if there was none)
        case 0: contract(ic<0>{}, ic<0>{}); break;
        case 1: contract(ic<1>{}, ic<1>{}); break;
        case 2: contract(ic<2>{}, ic<0>{}); break;
        default: contract(ic<3>{}, ic<1>{}); break;
    }

    // Fixed-order reduction: head h0 + hh is the sum of pairs 2hh and 2hh+1,
    // per slice half.
    __syncthreads();
    float *red = reinterpret_cast<float *>(lds);
    float *mine = red + (size_t)wave * MH * (C + 1);
#pragma unroll
    for (int mt = 0; mt < MTH; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = mt * 16 + g * 4 + r;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) mine[m * (C + 1) + ct * 16 + li] = S[mt][ct][r];
            if (li == 0) mine[m * (C + 1) + C] = D[mt][r];
        }
    __syncthreads();
    constexpr int EH = MH * (C + 1);  // one slice half's elements
    for (int e = threadIdx.x; e < 4 * EH; e += 512) {
        const int hh = e / (2 * EH), er = e - hh * 2 * EH;
        const int half = er / EH, r = er - half * EH;
        const float *src = red + (size_t)(2 * hh + 4 * half) * EH + r;
        partials[((size_t)(span0 + span_local) * H + 2 * hp + hh) * (size_t)(M * (C + 1)) + er] = src[0] + src[EH];
    }
}

}  // namespace ts3
