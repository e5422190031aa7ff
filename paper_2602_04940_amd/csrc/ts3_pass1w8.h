// Pass 1 on eight waves (two per SIMD) for 16-bit storage and M >= 32: the
// same computation as k_slice_accumulate (paper Eq. (1) and Eq. (4),
// Algorithm 1 tile loop), split so that a wave holds only half of a head's
// accumulator and the vector-ALU work of two waves issues on each SIMD.
//
// One workgroup per (span, head).  Waves q and q+4 form pair q and take the
// same 32-point blocks (q, q+4, q+8, ... of the span).  Wave q+4*hf
//   copies x rows prow(hf, .) of each block (its 16 points) into the pair's
//            LDS ring and computes their logits and softmax over all M slices
//            (A = W2'^T fragments, B = x^T from LDS), writing their w rows to
//            the pair's w tile;
//   contracts slices hf*M/2 .. hf*M/2 + M/2 - 1 over all 32 points of the
//            previous block: S_own[m][c] += sum_p w[p][m] x[p][c], d_own[m] +=
//            sum_p w[p][m], with operands from ds_read_b64_tr_b16.
// One barrier per block makes the partner's w rows and x rows visible before
// the contraction and frees the previous block's slots for the next copies.
// The four pairs' accumulators are summed in a fixed order at the end and
// written as the span's partial [M][C+1], as in the four-wave kernel.
#pragma once
#include "ts3_pass1.h"

namespace ts3 {

template <int C, int M> struct Pass1W8Cfg {
    using T = bf16_t;
    static constexpr int WAVES = 8, PAIRS = 4;
    static constexpr int MT = M / 16;             // 16-slice tiles of the head
    static constexpr int MH = M / 2;              // slices contracted per wave
    static constexpr int MTH = MH / 16;
    static constexpr int CT = C / 16, CK = C / 32;
    static constexpr int XROW = C * 2, XTILE = 32 * XROW;
    static constexpr int WROW = M * 2, WTILE = 32 * WROW;
    static constexpr int NS = 3;                  // x ring depth and w tiles per pair
    static constexpr int ROWS_PER_LOAD = 1024 / XROW, LOADS = 32 / ROWS_PER_LOAD;
    static constexpr int MY_LOADS = LOADS / 2;    // copies per wave per block
    static constexpr int X_BYTES = PAIRS * NS * XTILE;
    static constexpr int W_BYTES = PAIRS * NS * WTILE;
    static constexpr int RED_BYTES = WAVES * MH * (C + 1) * 4;
    static constexpr int PIPE_BYTES = X_BYTES + W_BYTES;
    static constexpr int LDS_BYTES = PIPE_BYTES > RED_BYTES ? PIPE_BYTES : RED_BYTES;
    static_assert(MH % 16 == 0, "each wave contracts whole 16-slice tiles");
    // A 1 KB copy holds rows 4i .. 4i+3 (C = 128) or 8i .. 8i+7 (C = 64); the
    // rows of point tile hf (row bit 2 = hf) are whole copies only at C = 128.
    static_assert(ROWS_PER_LOAD == 4, "a wave's rows must be whole 1 KB copies");
};

// Arguments as k_slice_accumulate; 512 threads per workgroup.
template <int C, int M>
__global__ __launch_bounds__(512, 1) void k_slice_accumulate_w8(
    const bf16_t *__restrict__ x, int64_t n_tile, int64_t span0, int32_t Q, int32_t nspan, int32_t H,
    const bf16_t *__restrict__ w2p, const float *__restrict__ b2s, float *__restrict__ partials) {
    using Cfg = Pass1W8Cfg<C, M>;
    using T = bf16_t;
    constexpr int MT = Cfg::MT, MTH = Cfg::MTH, CT = Cfg::CT, CK = Cfg::CK, MH = Cfg::MH, NS = Cfg::NS;
    constexpr int XROW = Cfg::XROW, WROW = Cfg::WROW, XTILE = Cfg::XTILE, WTILE = Cfg::WTILE;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[Cfg::LDS_BYTES];

    const int nwg = nspan * H;
    const int jwg = xcd_remap((int)blockIdx.x, nwg);
    const int span_local = jwg / H;
    const int h = jwg - span_local * H;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int pair = wave & 3, hf = wave >> 2;
    const int li = lane & 15, g = lane >> 4;

    const int64_t p_begin = (int64_t)span_local * Q;
    const int64_t p_end = p_begin + Q < n_tile ? p_begin + Q : n_tile;
    const int nblk = (int)((p_end - p_begin + 31) >> 5);
    const int nit = (nblk + Cfg::PAIRS - 1) / Cfg::PAIRS;  // block iterations, the same for every wave

    unsigned char *const xring = lds + pair * NS * XTILE;
    unsigned char *const wring = lds + Cfg::X_BYTES + pair * NS * WTILE;
    const uint32_t xring_lds = lds_addr(xring);

    // This wave's rows of block j of the pair (mesh block pair + 4j) into x
    // slot SL: copies hf, hf+2, ... (rows prow(hf, .)); lane mapping and the
    // handling of rows past the span's end as in k_slice_accumulate.
    constexpr int NCH = XROW / 16;
    auto copy_off = [&](int i) {
        const int R = i * Cfg::ROWS_PER_LOAD + lane / NCH;
        return (uint32_t)(R * XROW + (((lane % NCH) ^ xswz<XROW>(R)) << 4));
    };
    auto issue_x = [&](int j, auto slot) {
        constexpr int SL = decltype(slot)::value;
        const int64_t p0 = p_begin + ((int64_t)(pair + Cfg::PAIRS * j) << 5);
        const uint32_t dst = xring_lds + SL * XTILE;
        if (p0 + 32 <= p_end) {
            const void *base = x + p0 * C;
#pragma unroll
            for (int k = 0; k < Cfg::MY_LOADS; ++k) {
                const int i = 2 * k + hf;
                dma16s<0>(copy_off(i), base, dst + i * 1024);
            }
        } else {
#pragma unroll
            for (int k = 0; k < Cfg::MY_LOADS; ++k) {
                const int i = 2 * k + hf;
                const int R = i * Cfg::ROWS_PER_LOAD + lane / NCH;
                const int kk = (lane % NCH) ^ xswz<XROW>(R);
                int64_t p = p0 + R;
                p = p < p_end ? p : p_end - 1;
                dma16(reinterpret_cast<const unsigned char *>(x + (size_t)p * C) + kk * 16, dst + i * 1024);
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
    const uint32_t xbase = (uint32_t)(pair * NS * XTILE);
    const uint32_t wbase = (uint32_t)(Cfg::X_BYTES + pair * NS * WTILE);
    uint32_t xl0 = xbase + xoff<XROW>(prow(hf, li), 16 * g);
    uint32_t xt0 = xbase + xoff<XROW>(8 * g + (li >> 2), 8 * (li & 3));
    uint32_t wt0 = wbase + woff<WROW>(8 * g + (li >> 2), 8 * (li & 3));
    uint32_t ws0 = wbase + woff<WROW>(prow(hf, li), 8 * g);

    // The x fragment of step kc+1 is read while step kc's MFMAs run.
    auto logits = [&](auto slot, f32x4 (&L)[MT]) {
        constexpr int SL = decltype(slot)::value;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) L[mt] = bias[mt];
        Frag<T> xb[2];
        xb[0].v = *reinterpret_cast<const bf16x8 *>(lds + xl0 + SL * XTILE);
#pragma unroll
        for (int kc = 0; kc < CK; ++kc) {
            __builtin_amdgcn_sched_barrier(0);
            if (kc + 1 < CK)
                xb[(kc + 1) & 1].v = *reinterpret_cast<const bf16x8 *>(lds + (xl0 ^ ((kc + 1) << 6)) + SL * XTILE);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) mma(L[mt], w2[mt][kc], xb[kc & 1]);
            if (kc + 1 < CK) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, MT, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    auto read_a = [&](auto slot, Frag<T> (&a)[MTH]) {
        constexpr int SL = decltype(slot)::value;
#pragma unroll
        for (int mt = 0; mt < MTH; ++mt)
            tr_frag<WROW>(a[mt], lds + (wt0 ^ ((hf * MTH + mt) << 5)) + SL * WTILE);
    };
    auto read_b = [&](auto slot, int ct, Frag<T> &b) {
        constexpr int SL = decltype(slot)::value;
        tr_frag<XROW>(b, lds + (xt0 ^ (ct << 5)) + SL * XTILE);
    };
    auto contract = [&](auto slot) {
        Frag<T> a[MTH], b;
        read_a(slot, a);
#pragma unroll
        for (int mt = 0; mt < MTH; ++mt) mma(D[mt], a[mt], ones);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            read_b(slot, ct, b);
#pragma unroll
            for (int mt = 0; mt < MTH; ++mt) mma(S[mt][ct], a[mt], b);
        }
    };
    auto store_w = [&](auto slot, const f32x4 (&E)[MT], float inv) {
        constexpr int SL = decltype(slot)::value;
        typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            *reinterpret_cast<bf16x4 *>(lds + (ws0 ^ (mt << 5)) + SL * WTILE) =
                bf16x4{(__bf16)(E[mt][0] * inv), (__bf16)(E[mt][1] * inv), (__bf16)(E[mt][2] * inv),
                       (__bf16)(E[mt][3] * inv)};
    };
    auto block_valid = [&](int j) {
        const int64_t left = p_end - (p_begin + ((int64_t)(pair + Cfg::PAIRS * j) << 5));
        return (int)(left <= 0 ? 0 : left < 32 ? left : 32);
    };

    // Block j in slot SL = j % NS: this wave's logits and softmax (16 points,
    // all slices) beside the previous block's contraction (its slices, 32
    // points), the w rows, one barrier, then the copy of block j + 2 into the
    // freed slot.
    auto step = [&](int j, auto slot) {
        constexpr int SL = decltype(slot)::value;
        constexpr int PREV = (SL + NS - 1) % NS;
        asm volatile("" : "+v"(xl0), "+v"(xt0), "+v"(wt0), "+v"(ws0));
        const bool row_valid = prow(hf, li) < block_valid(j);
        Frag<T> a[MTH], b;
        read_a(ic<PREV>{}, a);
        read_b(ic<PREV>{}, 0, b);
        wait_vmcnt<(NS - 2) * Cfg::MY_LOADS>();  // this wave's rows of block j have landed
        asm volatile("" ::: "memory");
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
        store_w(slot, L, inv);
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __syncthreads();  // partner's rows and w of block j visible; block j-1's slots are free
        issue_x(j + NS - 1, ic<PREV>{});
    };

    // "Block -1" (slot NS-1) holds zeros so the first contraction adds nothing;
    // each wave clears the half of the pair's tiles it also writes later.
    {
        uint4 *zx = reinterpret_cast<uint4 *>(xring + (NS - 1) * XTILE);
        uint4 *zw = reinterpret_cast<uint4 *>(wring + (NS - 1) * WTILE);
        for (int i = hf * 64 + lane; i < XTILE / 16; i += 128) zx[i] = uint4{0u, 0u, 0u, 0u};
        for (int i = hf * 64 + lane; i < WTILE / 16; i += 128) zw[i] = uint4{0u, 0u, 0u, 0u};
    }
    __syncthreads();
    static_assert(NS == 3, "the unrolled loop below assumes a ring of three");
    issue_x(0, ic<0>{});
    issue_x(1, ic<1>{});
    int j = 0;
    for (; j + 3 <= nit; j += 3) {
        step(j, ic<0>{});
        step(j + 1, ic<1>{});
        step(j + 2, ic<2>{});
    }
    if (j < nit) step(j, ic<0>{});
    if (j + 1 < nit) step(j + 1, ic<1>{});
    wait_vmcnt<0>();
    switch ((nit + NS - 1) % NS) {  // the last block (slot 2 if there was none)
        case 0: contract(ic<0>{}); break;
        case 1: contract(ic<1>{}); break;
        default: contract(ic<2>{}); break;
    }

    // Fixed-order reduction over the four pairs, per slice half.
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
    constexpr int EH = MH * (C + 1);  // one half's elements
    float *dst = partials + ((size_t)(span0 + span_local) * H + h) * (size_t)(M * (C + 1));
    for (int e = threadIdx.x; e < 2 * EH; e += 512) {
        const int half = e / EH, r = e - half * EH;
        const float *src = red + (size_t)(4 * half) * EH + r;
        dst[e] = (src[0] + src[EH]) + (src[2 * EH] + src[3 * EH]);
    }
}

}  // namespace ts3
