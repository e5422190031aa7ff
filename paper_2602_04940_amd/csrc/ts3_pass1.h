// Pass 1 of the Physics-Attention layer: slice logits, per-head temperature
// softmax and the tile contraction s_raw += w^T x, d += sum_i w_i (paper
// Eq. (1) and Eq. (4), Algorithm 1 tile loop).  The slice weights exist only in
// registers and a per-wave LDS scratch tile.
//
// Work decomposition: one workgroup per (span, head).  A span is Q consecutive
// mesh points; its four waves take 32-point blocks round-robin, each keeping a
// private M x C float32 accumulator of its head in registers, with head h's
// W2' fragments resident.  At the end the four wave accumulators are summed in
// a fixed order and written as the span's partial [M][C+1] (column C holds d).
// Spans are folded in index order later, so the result is a fixed function of
// (x, Q) whatever the tiling.
//
// Per 32-point block and wave:
//   x rows   arrive in a per-wave LDS ring by direct global->LDS loads, NX-1
//            blocks ahead of use; they never pass through registers.
//   logits   L[m][p] = W2'[:, h*M+m] . x[p] + b2'   16x16x32 MFMA, A = W2'^T
//            fragments, B = x^T read from the ring; W2' = W2 * log2(e)/tau so
//            the softmax uses exp2.  Lane (g, p) holds slices 16*mt + 4*g + r.
//   softmax  over the M slices of each point: in-lane, then two cross-row swaps.
//   w rows   normalised and written to a per-wave LDS tile (two tiles, so
//            block b's softmax can run while block b-1 is contracted).
//   contract S[m][c] += sum_p w[p][m] x[p][c] (A = w^T, B = x) and
//            d[m] += sum_p w[p][m] (A = w^T against a ones operand), with
//            ds_read_b64_tr_b16 giving operands whose K slots hold points:
//            slot (g, t) <-> point 8g+t.
// With bf16 storage block b-1's contraction (matrix cores) is interleaved with
// block b's softmax (vector ALU); fp32 storage, the parity path, runs the
// steps of a block back to back.
#pragma once
#include "ts3_device.h"

namespace ts3 {

template <typename T, int C, int M> struct Pass1Cfg {
    static constexpr int CT = C / 16;      // 16-channel tiles
    static constexpr int MT = M / 16;      // 16-slice tiles
    static constexpr int CK = C / 32;      // K32 steps over channels
    static constexpr int WAVES = 4;
    static constexpr bool PIPE = sizeof(T) == 2;
    static constexpr int XROW = C * (int)sizeof(T);    // bytes per point row of x
    static constexpr int WROW = M * (int)sizeof(T);    // bytes per point row of w
    static constexpr int XTILE = 32 * XROW;
    static constexpr int WTILE = 32 * WROW;
    static constexpr int NX = PIPE ? 3 : 1;            // x ring depth
    static constexpr int NW = PIPE ? 2 : 1;            // w tiles
    static constexpr int ROWS_PER_LOAD = 1024 / XROW;  // rows per 1 KB wave load
    static constexpr int LOADS = 32 / ROWS_PER_LOAD;   // wave loads per block
    static constexpr int WAVE_BYTES = NX * XTILE + NW * WTILE;
    static constexpr int XT_BYTES = WAVES * WAVE_BYTES;
    static constexpr int RED_BYTES = WAVES * M * (C + 1) * 4;
    static constexpr int LDS_BYTES = XT_BYTES > RED_BYTES ? XT_BYTES : RED_BYTES;
    static_assert(ROWS_PER_LOAD * XROW == 1024, "x rows must tile a 1 KB load");
};

// Bank-conflict-free placement inside unpadded tile rows.
// x rows (16-byte chunks): chunk k of row R sits at k ^ xswz(R).  Each group of
// eight consecutive rows sees all eight values mod 8, so 8-lane phases of
// 16-byte accesses to consecutive rows hit distinct banks, and a 16-lane
// transpose read (rows 8g+q, q < 4, two chunks) sees 2q in bits 1-2.
template <int ROWB> __device__ __forceinline__ int xswz(int R) {
    constexpr int NCH = ROWB / 16;
    const int f = (2 * (R & 3)) ^ ((R >> 2) & 1) ^ (NCH >= 16 ? ((R >> 3) & 1) << 3 : 0);
    return f & (NCH - 1);
}
template <int ROWB> __device__ __forceinline__ int xoff(int R, int byte) {
    return R * ROWB + (((byte >> 4) ^ xswz<ROWB>(R)) << 4) + (byte & 15);
}
// w rows (8-byte slots): slot s of row R sits at s ^ wswz(R), chosen per row
// width so that the sixteen rows of an 8-byte store phase and the four rows x
// four slots of a transpose read cover distinct banks.
template <int ROWB> __device__ __forceinline__ int wswz(int R) {
    constexpr int NS = ROWB / 8;
    if constexpr (NS >= 16) return ((R & 3) << 2) | ((R >> 2) & 3);
    else if constexpr (NS == 8) return (((R >> 1) & 1) << 2) | ((R >> 2) & 3);
    else return ((R >> 2) & 3) & (NS - 1);
}
template <int ROWB> __device__ __forceinline__ int woff(int R, int byte) {
    return R * ROWB + (((byte >> 3) ^ wswz<ROWB>(R)) << 3) + (byte & 7);
}

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// One 8-slot operand fragment from two transposing LDS reads.  Lane (g, j) of
// each 16-lane row reads row 8g + 4*half + j/4, columns col0 + 4*(j%4) .. +3 of
// a tile; the result gives lane (g, i) column col0 + i of rows 8g .. 8g+7 in
// slots 0..7.  OFF maps (row, logical byte) to the tile's swizzled offset.
template <int ROWB, bool XT>
__device__ __forceinline__ void tr_frag(Frag<bf16_t> &f, const unsigned char *base, int g, int col0, int j) {
    const int r = 8 * g + (j >> 2);
    const int byte = (col0 + 4 * (j & 3)) * 2;
    const int o0 = XT ? xoff<ROWB>(r, byte) : woff<ROWB>(r, byte);
    const int o1 = XT ? xoff<ROWB>(r + 4, byte) : woff<ROWB>(r + 4, byte);
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(base + o0));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(base + o1));
    typedef short s16x8 __attribute__((ext_vector_type(8)));
    const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    f.v = __builtin_bit_cast(bf16x8, v);
}
// fp32 tiles: the same fragment read element by element (fp32 storage is the
// parity path, not the fast one).
template <int ROWB, bool XT>
__device__ __forceinline__ void tr_frag(Frag<float> &f, const unsigned char *base, int g, int col0, int i) {
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const int o = XT ? xoff<ROWB>(8 * g + t, (col0 + i) * 4) : woff<ROWB>(8 * g + t, (col0 + i) * 4);
        f.v[t] = *reinterpret_cast<const float *>(base + o);
    }
}

// x       : tile base, [n_tile][C] storage elements
// n_tile  : points in this tile (tile starts on a span boundary)
// span0   : global index of the tile's first span
// Q       : points per span
// nspan   : spans in this tile (= ceil(n_tile / Q)); grid = nspan * H
// w2p     : prepared W2' fragments [H][MT][CK][64 lanes][8]
// b2s     : W2'-scaled bias [H*M]
// partials: [span][H][M][C+1] float32
template <typename T, int C, int M>
__global__ __launch_bounds__(256, 1) void k_slice_accumulate(
    const T *__restrict__ x, int64_t n_tile, int64_t span0, int32_t Q, int32_t nspan, int32_t H,
    const T *__restrict__ w2p, const float *__restrict__ b2s, float *__restrict__ partials) {
    using Cfg = Pass1Cfg<T, C, M>;
    constexpr int CT = Cfg::CT, MT = Cfg::MT, CK = Cfg::CK;
    constexpr int XROW = Cfg::XROW, WROW = Cfg::WROW, NX = Cfg::NX, NW = Cfg::NW;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[Cfg::LDS_BYTES];

    const int nwg = nspan * H;
    const int jwg = xcd_remap((int)blockIdx.x, nwg);
    const int span_local = jwg / H;
    const int h = jwg - span_local * H;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int li = lane & 15;
    const int g = lane >> 4;

    const int64_t p_begin = (int64_t)span_local * Q;
    const int64_t p_end = p_begin + Q < n_tile ? p_begin + Q : n_tile;
    const int nblk = (int)((p_end - p_begin + 31) >> 5);
    const int nmine = nblk > wave ? (nblk - wave + Cfg::WAVES - 1) / Cfg::WAVES : 0;

    unsigned char *wave_lds = lds + wave * Cfg::WAVE_BYTES;
    auto xslot = [&](int j) { return wave_lds + (j % NX) * Cfg::XTILE; };
    auto wslot = [&](int j) { return wave_lds + NX * Cfg::XTILE + (j % NW) * Cfg::WTILE; };

    // Block j of this wave (mesh block wave + 4j) into x slot j % NX.  Lane l of
    // load i fills physical chunk l % NCH of row i*ROWS_PER_LOAD + l / NCH, so it
    // reads the logical chunk stored there.  Rows past the span's end repeat
    // its last point (finite data that the zero weights of padding points
    // cancel exactly), which also keeps every wave's load count uniform.
    auto issue_x = [&](int j) {
        constexpr int NCH = XROW / 16;
        unsigned char *slot = xslot(j);
        const int64_t p0 = p_begin + ((int64_t)(wave + Cfg::WAVES * j) << 5);
#pragma unroll
        for (int i = 0; i < Cfg::LOADS; ++i) {
            const int R = i * Cfg::ROWS_PER_LOAD + lane / NCH;
            const int k = (lane % NCH) ^ xswz<XROW>(R);
            int64_t p = p0 + R;
            p = p < p_end ? p : p_end - 1;
            const unsigned char *src = reinterpret_cast<const unsigned char *>(x + (size_t)p * C) + k * 16;
            dma16(src, lds_addr(slot + i * 1024));
        }
    };

    // Head h's W2'^T fragments (A operand: lane row = slice) and bias, resident.
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
    // Settle the loads above before the x ring starts: the ring's counts
    // assume its own copies are the only memory operations in flight.
    wait_vmcnt<0>();

    // Logits B operand from x slot j: lane (g, li) holds point 16*pt + li,
    // channels 32*kc + 8*g .. +8.
    auto read_x = [&](int j, Frag<T> (&xb)[2][CK]) {
        const unsigned char *src = xslot(j);
#pragma unroll
        for (int pt = 0; pt < 2; ++pt)
#pragma unroll
            for (int kc = 0; kc < CK; ++kc) {
                const int R = pt * 16 + li, byte = (kc * 32 + g * 8) * (int)sizeof(T);
                if constexpr (sizeof(T) == 2) {
                    xb[pt][kc].v = *reinterpret_cast<const bf16x8 *>(src + xoff<XROW>(R, byte));
                } else {
                    const float4 a = *reinterpret_cast<const float4 *>(src + xoff<XROW>(R, byte));
                    const float4 b = *reinterpret_cast<const float4 *>(src + xoff<XROW>(R, byte + 16));
                    xb[pt][kc].v[0] = a.x; xb[pt][kc].v[1] = a.y; xb[pt][kc].v[2] = a.z; xb[pt][kc].v[3] = a.w;
                    xb[pt][kc].v[4] = b.x; xb[pt][kc].v[5] = b.y; xb[pt][kc].v[6] = b.z; xb[pt][kc].v[7] = b.w;
                }
            }
    };
    auto logits = [&](const Frag<T> (&xb)[2][CK], f32x4 (&L)[MT][2]) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int pt = 0; pt < 2; ++pt) {
                L[mt][pt] = bias[mt];
#pragma unroll
                for (int kc = 0; kc < CK; ++kc) mma(L[mt][pt], w2[mt][kc], xb[pt][kc]);
            }
    };
    // S += w^T x, d += sum_p w for block j (x slot j % NX, w tile j % NW).
    auto contract = [&](int j) {
        const unsigned char *xt = xslot(j), *wt = wslot(j);
        Frag<T> a[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) tr_frag<WROW, false>(a[mt], wt, g, mt * 16, li);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) mma(D[mt], a[mt], ones);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            Frag<T> b;
            tr_frag<XROW, true>(b, xt, g, ct * 16, li);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) mma(S[mt][ct], a[mt], b);
        }
    };
    // exp2 of the logits in place; per point the reciprocal row sum (zero for
    // padding points).  Returns false if a row left the unshifted window.
    auto softmax_fast = [&](f32x4 (&L)[MT][2], float (&inv)[2], int valid) {
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
            inv[pt] = (pt * 16 + li < valid) ? fast_rcp(sum) : 0.f;
        }
        return ok;
    };
    auto softmax_shifted = [&](f32x4 (&L)[MT][2], float (&inv)[2], int valid) {
#pragma unroll
        for (int pt = 0; pt < 2; ++pt) {
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
            inv[pt] = (pt * 16 + li < valid) ? fast_rcp(xrow_sum(sum)) : 0.f;
        }
    };
    // Normalised w rows into w tile j % NW: lane (g, li) stores slices
    // 16*mt + 4*g .. +3 of point 16*pt + li.
    auto store_w = [&](int j, const f32x4 (&E)[MT][2], const float (&inv)[2]) {
        unsigned char *dst = wslot(j);
#pragma unroll
        for (int pt = 0; pt < 2; ++pt)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const int R = pt * 16 + li, byte = (mt * 16 + g * 4) * (int)sizeof(T);
                const float a0 = E[mt][pt][0] * inv[pt], a1 = E[mt][pt][1] * inv[pt];
                const float a2 = E[mt][pt][2] * inv[pt], a3 = E[mt][pt][3] * inv[pt];
                if constexpr (sizeof(T) == 2) {
                    typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
                    *reinterpret_cast<bf16x4 *>(dst + woff<WROW>(R, byte)) =
                        bf16x4{(__bf16)a0, (__bf16)a1, (__bf16)a2, (__bf16)a3};
                } else {
                    *reinterpret_cast<float2 *>(dst + woff<WROW>(R, byte)) = float2{a0, a1};
                    *reinterpret_cast<float2 *>(dst + woff<WROW>(R, byte + 8)) = float2{a2, a3};
                }
            }
    };
    auto block_valid = [&](int j) {
        const int64_t left = p_end - (p_begin + ((int64_t)(wave + Cfg::WAVES * j) << 5));
        return (int)(left < 32 ? left : 32);
    };

    if constexpr (Cfg::PIPE) {
        // The tiles of "block -1" hold zeros, so the first iteration's
        // contraction of the previous block adds exactly nothing.
        {
            uint4 *zx = reinterpret_cast<uint4 *>(xslot(NX - 1));
            uint4 *zw = reinterpret_cast<uint4 *>(wslot(NW - 1));
            for (int i = lane; i < Cfg::XTILE / 16; i += 64) zx[i] = uint4{0u, 0u, 0u, 0u};
            for (int i = lane; i < Cfg::WTILE / 16; i += 64) zw[i] = uint4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int j = 0; j < NX - 1; ++j) issue_x(j);
        for (int j = 0; j < nmine; ++j) {
            const int valid = block_valid(j);
            wait_vmcnt<(NX - 2) * Cfg::LOADS>();  // block j's rows have landed
            asm volatile("" ::: "memory");
            Frag<T> xb[2][CK];
            read_x(j, xb);
            f32x4 L[MT][2];
            logits(xb, L);
            __builtin_amdgcn_sched_barrier(0);
            // Block j-1's contraction (matrix cores) interleaved with block j's
            // softmax and w rows (vector ALU).
            contract(j - 1 + NX * NW);
            float inv[2];
            const bool ok = softmax_fast(L, inv, valid);
            store_w(j, L, inv);
            interleave_mfma_valu<MT * (CT + 1), 4, 2>();
            __builtin_amdgcn_sched_barrier(0);
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            issue_x(j - 1 + NX);  // block j-1's x slot is free again
            if (__any(!ok)) {
                // Rare: some row's exp2 sum left the safe window; redo the
                // block with the max shift.
                read_x(j, xb);
                logits(xb, L);
                softmax_shifted(L, inv, valid);
                store_w(j, L, inv);
            }
            asm volatile("" ::: "memory");
        }
        wait_vmcnt<0>();
        contract(nmine - 1 + NX * NW);  // the last block
    } else {
        for (int j = 0; j < nmine; ++j) {
            const int valid = block_valid(j);
            issue_x(j);
            wait_vmcnt<0>();
            asm volatile("" ::: "memory");
            Frag<T> xb[2][CK];
            read_x(j, xb);
            f32x4 L[MT][2];
            logits(xb, L);
            float inv[2];
            if (__any(!softmax_fast(L, inv, valid))) {
                logits(xb, L);
                softmax_shifted(L, inv, valid);
            }
            store_w(j, L, inv);
            asm volatile("" ::: "memory");
            contract(j);
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        }
    }

    // Fixed-order reduction of the four wave accumulators.
    __syncthreads();
    float *red = reinterpret_cast<float *>(lds);
    float *mine = red + (size_t)wave * M * (C + 1);
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
    constexpr int E = M * (C + 1);
    float *dst = partials + ((size_t)(span0 + span_local) * H + h) * E;
    for (int e = threadIdx.x; e < E; e += 256)
        dst[e] = (red[e] + red[E + e]) + (red[2 * E + e] + red[3 * E + e]);
}

}  // namespace ts3
