// Backward of the Physics-Attention layer for float32 storage, with the slice
// weights recomputed tile by tile instead of stored: the paper trains with
// every tile's slice computation checkpointed (section 3.2, "Geometry slice
// tiling", and the Checkpoint steps of Algorithm 1).  Given the output
// gradient g = dL/dx_out:
//
//   k_bw_head   per (span, head): recompute w; partial dZ[m][:] =
//               sum_p w[p][m] g_p (and sum_p w in column C)
//   k_bw_token  per head: back through Linear3, the attention among the
//               head's M tokens, Linear1 and the normalisation: ds_raw, dd
//               and the token-side weight gradients
//   k_bw_dx     per wave block of 16-point tiles, over all heads: recompute
//               w; dw = g.Z + x.ds_raw + dd; dz = (1/tau) w (dw - sum_m w dw);
//               dx = sum_h dz W2_h^T + w ds_raw_h; dz is stored
//   k_bw_dw2    per (span, head): partial dW2^T[m][:] = sum_p dz[p][m] x_p
//               and db2 = sum_p dz, from the stored dz
//
// Span partials are folded in index order by the forward's fold kernels, so
// every gradient is a fixed function of the inputs (any tiling, any run).
// Contractions use the 16x16x4 float32 MFMA through the fragment helpers of
// ts3_device.h (lane (row, g), slot t); A fragments are read from L2-resident
// arrays, transposes go through per-wave LDS tiles.
#pragma once
#include "ts3_device.h"

namespace ts3 {

// Row-major [rows][K] float32 array -> A (or B) fragment whose lane row r and
// slot (g, t) hold element [r][k0 + 8g + t]: 8 consecutive floats.
__device__ __forceinline__ void frag_row(Frag<float> &f, const float *row_k0, int g) {
    load8(f, row_k0 + 8 * g);
}

// Pack a [slices x points] register tile (lane (p, g) holds slices 16mt + 4g
// + r of point p, tiles mt < MT) as the B operand of K32 step km: slot t holds
// slice 32km + 16(t>>2) + 4g + (t&3); zero past M.
template <int MT>
__device__ __forceinline__ void pack_b(const f32x4 (&E)[MT], int km, Frag<float> &f) {
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const int mt = 2 * km + (t >> 2);
        f.v[t] = mt < MT ? E[mt < MT ? mt : 0][t & 3] : 0.f;
    }
}

// A fragment for the same K order from a row-major [rows][M] array: lane row
// r, slot t holds [r][32km + 16(t>>2) + 4g + (t&3)] (zero past M).
template <int M>
__device__ __forceinline__ void frag_slices(Frag<float> &f, const float *row, int km, int g) {
    const float4 a = *reinterpret_cast<const float4 *>(row + 32 * km + 4 * g);
    f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
    if (M >= 32) {
        const float4 b = *reinterpret_cast<const float4 *>(row + 32 * km + 16 + 4 * g);
        f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
    } else {
        f.v[4] = f.v[5] = f.v[6] = f.v[7] = 0.f;
    }
}

// Max-shifted softmax over a head's M slices of one 16-point tile, in place
// (E holds exp2-scaled logits); rows of invalid points become zero.
template <int MT>
__device__ __forceinline__ void softmax_tile(f32x4 (&E)[MT], bool valid) {
    float mx = E[0][0];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) mx = fmaxf(mx, E[mt][r]);
    mx = xrow_max(mx);
    float sum = 0.f;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float e = fast_exp2(E[mt][r] - mx);
            E[mt][r] = e;
            sum += e;
        }
    const float tot = xrow_sum(sum);  // every lane takes part in the cross-row swaps
    const float inv = valid ? 1.f / tot : 0.f;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) E[mt][r] *= inv;
}

// Logits of head h for NT 16-point tiles whose x rows start at xrow[t]
// (lane row li): E[t][mt] = b2s + W2'^T x, exp2-scaled (W2' = W2 log2(e) /
// tau).  Each A fragment (read from L2) serves all NT tiles.
template <int C, int M, int NT>
__device__ __forceinline__ void logits_tiles(f32x4 (&E)[NT][M / 16], const float *w2p, const float *b2s, int h,
                                             const float *const (&xrow)[NT], int lane) {
    constexpr int MT = M / 16, CK = C / 32;
    const int g = lane >> 4;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const float4 b = *reinterpret_cast<const float4 *>(b2s + h * M + mt * 16 + g * 4);
#pragma unroll
        for (int t = 0; t < NT; ++t) E[t][mt] = f32x4{b.x, b.y, b.z, b.w};
    }
    // K steps not unrolled: each step's fragments are loaded where they are
    // used (unrolled, the compiler hoists them all and spills).
#pragma unroll 1
    for (int kc = 0; kc < CK; ++kc) {
        Frag<float> xb[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) frag_row(xb[t], xrow[t] + 32 * kc, g);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            Frag<float> a;
            load8(a, w2p + ((((size_t)h * MT + mt) * CK + kc) * 64 + lane) * 8);
#pragma unroll
            for (int t = 0; t < NT; ++t) mma(E[t][mt], a, xb[t]);
        }
    }
}

// dw[m][p] = dd[h][m] + Z[h][m] . g_p + ds_raw[h][m] . x_p, then
// dz = inv_tau * w * (dw - sum_m w dw) in place of dw (W holds w), for NT
// tiles sharing every A fragment.
template <int C, int M, int NT>
__device__ __forceinline__ void dz_tiles(f32x4 (&Dz)[NT][M / 16], const f32x4 (&W)[NT][M / 16], const float *Z,
                                         const float *dsr, const float *dd, int h, const float *const (&xrow)[NT],
                                         const float *const (&grow)[NT], float inv_tau, int lane) {
    constexpr int MT = M / 16, CK = C / 32;
    const int g = lane >> 4, li = lane & 15;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const float4 b = *reinterpret_cast<const float4 *>(dd + h * M + mt * 16 + g * 4);
#pragma unroll
        for (int t = 0; t < NT; ++t) Dz[t][mt] = f32x4{b.x, b.y, b.z, b.w};
    }
#pragma unroll 1
    for (int kc = 0; kc < CK; ++kc) {
        Frag<float> gb[NT], xb[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            frag_row(gb[t], grow[t] + 32 * kc, g);
            frag_row(xb[t], xrow[t] + 32 * kc, g);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const size_t row = ((size_t)h * M + mt * 16 + li) * C + 32 * kc;
            Frag<float> a;
            frag_row(a, Z + row, g);
#pragma unroll
            for (int t = 0; t < NT; ++t) mma(Dz[t][mt], a, gb[t]);
            frag_row(a, dsr + row, g);
#pragma unroll
            for (int t = 0; t < NT; ++t) mma(Dz[t][mt], a, xb[t]);
        }
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        float s = 0.f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) s += W[t][mt][r] * Dz[t][mt][r];
        s = xrow_sum(s);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) Dz[t][mt][r] = inv_tau * W[t][mt][r] * (Dz[t][mt][r] - s);
    }
}

// Workgroups are dispatched to the eight XCDs in turn (workgroup i to XCD
// i % 8).  The per-(span, head) kernels below give the H workgroups of a span
// consecutive places on one XCD, so they run together and read the span's
// point rows through that XCD's L2 once.  Grid: 8 * ceil(nspan / 8) * H.
constexpr int BW_XCDS = 8;
__device__ __forceinline__ bool bw_span_head(int nspan, int H, int &span_local, int &h) {
    const int xcd = (int)blockIdx.x % BW_XCDS, slot = (int)blockIdx.x / BW_XCDS;
    span_local = (slot / H) * BW_XCDS + xcd;
    h = slot % H;
    return span_local < nspan;
}

// dZ span partials: partials[span][h][m][c] = sum_p w[p][m] g[p][c] over the
// span's points, column C = sum_p w[p][m].  One workgroup per (span, head),
// eight waves, the span's points in 128-point blocks.  Wave v computes the
// slice weights of the block's 16-point tile v (the head's W2' staged in LDS
// once per workgroup) and writes them transposed to LDS, beside the block's
// transposed g rows; after a barrier every wave contracts the block for its
// own part of the output: wave v the channel tile v (K = points), waves 4 + mt
// the column sums of slice tile mt.  No wave's sum needs another's, and each
// runs over the blocks in order, so a span's partial is the same for any
// tiling.  x, gout: tile bases [n_tile][C]; the tile starts on a span
// boundary.
constexpr int BW_HEAD_PTS = 128;             // points per block: one 16-point tile per wave
constexpr int BW_HEAD_LD = BW_HEAD_PTS + 8;  // floats per transposed LDS row (bank spread)

template <int C, int M>
__global__ __launch_bounds__(512, 1) void k_bw_head(const float *__restrict__ x, const float *__restrict__ gout,
                                                    int64_t n_tile, int64_t span0, int32_t Q, int32_t nspan,
                                                    int32_t H, const float *__restrict__ w2p,
                                                    const float *__restrict__ b2s, float *__restrict__ partials) {
    constexpr int MT = M / 16, CT = C / 16, NK = BW_HEAD_PTS / 32, LD = BW_HEAD_LD;
    constexpr int GQ = C / 4, GITEMS = BW_HEAD_PTS * GQ, GPER = GITEMS / 512;
    static_assert(CT <= 8 && MT <= 4, "one channel tile per wave and one column-sum tile per wave");
    static_assert(GITEMS % 512 == 0, "every thread moves the same number of g pieces");
    __shared__ __attribute__((aligned(16))) float lds[M * C + (M + C) * LD];
    float *const w2s = lds;         // the head's W2' fragments [MT][CK][64][8]
    float *const wT = w2s + M * C;  // [M][LD]: w of the block, transposed
    float *const gT = wT + M * LD;  // [C][LD]: g rows of the block, transposed
    int span_local, h;
    if (!bw_span_head(nspan, H, span_local, h)) return;  // uniform, before any barrier
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 15, g = lane >> 4;
    const int64_t p_begin = (int64_t)span_local * Q;
    const int64_t p_end = p_begin + Q < n_tile ? p_begin + Q : n_tile;
    const int nblk = (int)((p_end - p_begin + BW_HEAD_PTS - 1) / BW_HEAD_PTS);
    const bool has_ct = wave < CT;
    const int dmt = wave - 4;  // this wave's column-sum tile, if 0 <= dmt < MT
    const bool has_d = dmt >= 0 && dmt < MT;

    {   // the head's W2' fragments (contiguous in w2p)
        const float4 *src = reinterpret_cast<const float4 *>(w2p + (size_t)h * M * C);
        for (int i = tid; i < M * C / 4; i += 512) reinterpret_cast<float4 *>(w2s)[i] = src[i];
    }
    // g piece it: point it % PTS, float4 column it / PTS (a wave's transposed
    // writes then cover consecutive points of one LDS row).  Rows past the
    // span's end are zero.
    float4 gv[GPER];
    auto load_g = [&](int b) {
        const int64_t pb = p_begin + (int64_t)b * BW_HEAD_PTS;
#pragma unroll
        for (int k = 0; k < GPER; ++k) {
            const int it = tid + 512 * k;
            const int p = it % BW_HEAD_PTS, q = it / BW_HEAD_PTS;
            gv[k] = pb + p < p_end ? *reinterpret_cast<const float4 *>(gout + (pb + p) * C + 4 * q)
                                   : float4{0.f, 0.f, 0.f, 0.f};
        }
    };
    f32x4 S[MT], D = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) S[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    Frag<float> ones;
    ones8(ones);
    if (nblk > 0) load_g(0);
    __syncthreads();  // W2' staged

    for (int b = 0; b < nblk; ++b) {
        const int64_t pb = p_begin + (int64_t)b * BW_HEAD_PTS;
        // w of tile `wave` (rows past the span's end repeat its last point
        // and get zero weight)
        f32x4 E[1][MT];
        {
            const int64_t p = pb + 16 * wave + li;
            const bool valid = p < p_end;
            const float *xr[1] = {x + (valid ? p : p_end - 1) * C};
            logits_tiles<C, M, 1>(E, w2s, b2s + (size_t)h * M, 0, xr, lane);
            softmax_tile<MT>(E[0], valid);
        }
        __syncthreads();  // every wave finished reading the previous block's tiles
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) wT[(mt * 16 + g * 4 + r) * LD + 16 * wave + li] = E[0][mt][r];
#pragma unroll
        for (int k = 0; k < GPER; ++k) {
            const int it = tid + 512 * k;
            const int p = it % BW_HEAD_PTS, q = it / BW_HEAD_PTS;
            gT[(4 * q + 0) * LD + p] = gv[k].x;
            gT[(4 * q + 1) * LD + p] = gv[k].y;
            gT[(4 * q + 2) * LD + p] = gv[k].z;
            gT[(4 * q + 3) * LD + p] = gv[k].w;
        }
        if (b + 1 < nblk) load_g(b + 1);  // lands during this block's products and the next logits
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) {
            Frag<float> a[MT];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) frag_row(a[mt], wT + (mt * 16 + li) * LD + 32 * kk, g);
            if (has_ct) {
                Frag<float> bf;
                frag_row(bf, gT + (wave * 16 + li) * LD + 32 * kk, g);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) mma(S[mt], a[mt], bf);
            }
            if (has_d) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    if (mt == dmt) mma(D, a[mt], ones);
            }
        }
    }

    // lane (li, g) of tile (mt, ct) holds m = 16mt + 4g + r, c = 16ct + li;
    // column-sum tiles hold the sums in every column.
    float *dst = partials + ((size_t)(span0 + span_local) * H + h) * (size_t)(M * (C + 1));
    if (has_ct) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) dst[(size_t)(mt * 16 + g * 4 + r) * (C + 1) + wave * 16 + li] = S[mt][r];
    }
    if (has_d && li == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[(size_t)(dmt * 16 + g * 4 + r) * (C + 1) + C] = D[r];
    }
}

// dx for wave blocks of NT 16-point tiles (four waves per workgroup): over the
// heads, recompute w and dz, then dx[p][c] += sum_m dz[p][m] W2[c][hM+m] +
// w[p][m] ds_raw[h][m][c]; every A fragment (read from L2) serves the NT
// tiles.  dsT is ds_raw transposed per head: [H][C][M].  W2 is the layer's
// (unscaled) Linear2 weight [C][H*M].  dz of every point and head is also
// written to dzs [H][n][M] (the dW2 contraction reads it there).
// Grid: ceil(n / (64 NT)) workgroups.
template <int C, int M, int NT>
__global__ __launch_bounds__(256, 1) void k_bw_dx(const float *__restrict__ x, const float *__restrict__ gout,
                                                  int64_t n, int32_t H, const float *__restrict__ w2p,
                                                  const float *__restrict__ b2s, const float *__restrict__ W2,
                                                  const float *__restrict__ Z, const float *__restrict__ dsr,
                                                  const float *__restrict__ dsT, const float *__restrict__ dd,
                                                  float inv_tau, float *__restrict__ dx, float *__restrict__ dzs) {
    constexpr int MT = M / 16, CT = C / 16, KM = M >= 32 ? M / 32 : 1;
    const int lane = threadIdx.x & 63;
    const int wave = (int)(threadIdx.x >> 6);
    const int li = lane & 15, g = lane >> 4;
    const int64_t p0 = ((int64_t)blockIdx.x * 4 + wave) * (16 * NT);
    if (p0 >= n) return;  // wave-uniform; the kernel has no barriers
    bool valid[NT];
    const float *xr[NT], *gr[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int64_t p = p0 + 16 * t + li;
        valid[t] = p < n;
        const int64_t pc = valid[t] ? p : n - 1;
        xr[t] = x + pc * C;
        gr[t] = gout + pc * C;
    }
    const int HM = H * M;

    f32x4 O[NT][CT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) O[t][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int h = 0; h < H; ++h) {
        f32x4 E[NT][MT], Dz[NT][MT];
        logits_tiles<C, M, NT>(E, w2p, b2s, h, xr, lane);
#pragma unroll
        for (int t = 0; t < NT; ++t) softmax_tile<MT>(E[t], valid[t]);
        dz_tiles<C, M, NT>(Dz, E, Z, dsr, dd, h, xr, gr, inv_tau, lane);
        // lane (li, g) holds slices 16mt + 4g .. +3 of point p0 + 16t + li
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            if (!valid[t]) continue;
            float *row = dzs + ((size_t)h * n + p0 + 16 * t + li) * M + 4 * g;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                *reinterpret_cast<float4 *>(row + 16 * mt) = float4{Dz[t][mt][0], Dz[t][mt][1], Dz[t][mt][2], Dz[t][mt][3]};
        }
#pragma unroll
        for (int km = 0; km < KM; ++km) {
            Frag<float> wf[NT], zf[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                pack_b<MT>(E[t], km, wf[t]);
                pack_b<MT>(Dz[t], km, zf[t]);
            }
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                const int c = ct * 16 + li;
                Frag<float> a;
                frag_slices<M>(a, W2 + (size_t)c * HM + h * M, km, g);
#pragma unroll
                for (int t = 0; t < NT; ++t) mma(O[t][ct], a, zf[t]);
                frag_slices<M>(a, dsT + ((size_t)h * C + c) * M, km, g);
#pragma unroll
                for (int t = 0; t < NT; ++t) mma(O[t][ct], a, wf[t]);
            }
        }
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int64_t p = p0 + 16 * t + li;
        if (!valid[t]) continue;
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
            *reinterpret_cast<float4 *>(dx + p * C + ct * 16 + g * 4) =
                float4{O[t][ct][0], O[t][ct][1], O[t][ct][2], O[t][ct][3]};
    }
}

// dW2 span partials from the stored dz: partials[span][h][m][c] = sum_p
// dz[h][p][m] x[p][c] over the span's points, column C = sum_p dz[h][p][m]
// (db2).  One workgroup per (span, head), eight waves; every wave runs every
// point of the span and owns part of the output: wave v the channel tiles ct
// = v, v+8, ... (K = points), and wave 4 + mt the column sums of slice tile mt.
// No wave's sum needs another's, and each is taken over the span's 64-point
// blocks in order, so a span's partial is the same for any tiling.  Each
// block's x and dz rows are transposed into LDS once for all eight waves
// (two stages; the next block's rows are loaded during the current block's
// products).  x: the tile's rows [n][C]; dzs: [H][n][M] for the same points.
// Grid as k_bw_head (XCD-aware).
constexpr int BW_DW2_PTS = 64;  // points per block (the K of a block's products)
constexpr int BW_DW2_LD = BW_DW2_PTS + 8;  // floats per transposed LDS row (bank spread)

template <int C, int M> struct BwDw2Cfg {
    static constexpr int XQ = C / 4, ZQ = M / 4;      // float4 per point row
    static constexpr int XITEMS = BW_DW2_PTS * XQ;    // float4 loads per block
    static constexpr int ZITEMS = BW_DW2_PTS * ZQ;
    static constexpr int XPER = (XITEMS + 511) / 512;  // per thread
    static constexpr int ZPER = (ZITEMS + 511) / 512;
    static constexpr int STAGE = (C + M) * BW_DW2_LD;  // floats: x^T [C][LD], then dz^T [M][LD]
};

template <int C, int M>
__global__ __launch_bounds__(512, 1) void k_bw_dw2(const float *__restrict__ x, const float *__restrict__ dzs,
                                                   int64_t n_tile, int64_t span0, int32_t Q, int32_t nspan,
                                                   int32_t H, float *__restrict__ partials) {
    using Cfg = BwDw2Cfg<C, M>;
    constexpr int MT = M / 16, CT = C / 16, NK = BW_DW2_PTS / 32, LD = BW_DW2_LD;
    static_assert(CT <= 8 && MT <= 4, "one channel tile per wave and one column-sum tile per wave");
    __shared__ __attribute__((aligned(16))) float lds[2 * Cfg::STAGE];
    int span_local, h;
    if (!bw_span_head(nspan, H, span_local, h)) return;  // uniform, before any barrier
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 15, g = lane >> 4;
    const int64_t p_begin = (int64_t)span_local * Q;
    const int64_t p_end = p_begin + Q < n_tile ? p_begin + Q : n_tile;
    const int nblk = (int)((p_end - p_begin + BW_DW2_PTS - 1) / BW_DW2_PTS);
    const float *dzh = dzs + (size_t)h * n_tile * M;
    const bool has_ct = wave < CT;
    const int dmt = wave - 4;  // this wave's column-sum tile, if 0 <= dmt < MT
    const bool has_d = dmt >= 0 && dmt < MT;

    // Thread item it < ITEMS: point it % PTS, float4 column it / PTS, so a
    // wave's transposed writes cover consecutive points of one LDS row.
    float4 xv[Cfg::XPER], zv[Cfg::ZPER];
    auto load = [&](int b) {
        const int64_t pb = p_begin + (int64_t)b * BW_DW2_PTS;
#pragma unroll
        for (int k = 0; k < Cfg::XPER; ++k) {
            const int it = tid + 512 * k;
            const int p = it % BW_DW2_PTS, q = it / BW_DW2_PTS;
            const bool ok = it < Cfg::XITEMS && pb + p < p_end;
            xv[k] = ok ? *reinterpret_cast<const float4 *>(x + (pb + p) * C + 4 * q) : float4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int k = 0; k < Cfg::ZPER; ++k) {
            const int it = tid + 512 * k;
            const int p = it % BW_DW2_PTS, q = it / BW_DW2_PTS;
            const bool ok = it < Cfg::ZITEMS && pb + p < p_end;
            zv[k] = ok ? *reinterpret_cast<const float4 *>(dzh + (pb + p) * M + 4 * q) : float4{0.f, 0.f, 0.f, 0.f};
        }
    };
    // Rows past the span's end are zero in both operands.
    auto store = [&](int s) {
        float *xt = lds + s * Cfg::STAGE, *zt = xt + C * LD;
#pragma unroll
        for (int k = 0; k < Cfg::XPER; ++k) {
            const int it = tid + 512 * k;
            if (it >= Cfg::XITEMS) continue;
            const int p = it % BW_DW2_PTS, q = it / BW_DW2_PTS;
            xt[(4 * q + 0) * LD + p] = xv[k].x;
            xt[(4 * q + 1) * LD + p] = xv[k].y;
            xt[(4 * q + 2) * LD + p] = xv[k].z;
            xt[(4 * q + 3) * LD + p] = xv[k].w;
        }
#pragma unroll
        for (int k = 0; k < Cfg::ZPER; ++k) {
            const int it = tid + 512 * k;
            if (it >= Cfg::ZITEMS) continue;
            const int p = it % BW_DW2_PTS, q = it / BW_DW2_PTS;
            zt[(4 * q + 0) * LD + p] = zv[k].x;
            zt[(4 * q + 1) * LD + p] = zv[k].y;
            zt[(4 * q + 2) * LD + p] = zv[k].z;
            zt[(4 * q + 3) * LD + p] = zv[k].w;
        }
    };

    f32x4 S[MT], D = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) S[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    Frag<float> ones;
    ones8(ones);

    if (nblk > 0) {
        load(0);
        store(0);
    }
    __syncthreads();
    for (int b = 0; b < nblk; ++b) {
        const int s = b & 1;
        if (b + 1 < nblk) load(b + 1);  // lands during this block's products
        const float *xt = lds + s * Cfg::STAGE, *zt = xt + C * LD;
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) {
            Frag<float> a[MT];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) frag_row(a[mt], zt + (mt * 16 + li) * LD + 32 * kk, g);
            if (has_ct) {
                Frag<float> bf;
                frag_row(bf, xt + (wave * 16 + li) * LD + 32 * kk, g);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) mma(S[mt], a[mt], bf);
            }
            if (has_d) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    if (mt == dmt) mma(D, a[mt], ones);
            }
        }
        if (b + 1 < nblk) store(s ^ 1);  // stage s^1 was last read before the previous barrier
        __syncthreads();
    }

    // partials[span][h][m][c]: lane (li, g) of tile (mt, ct) holds m = 16mt +
    // 4g + r, c = 16ct + li; column-sum tiles hold the sums in every column.
    float *dst = partials + ((size_t)(span0 + span_local) * H + h) * (size_t)(M * (C + 1));
    if (has_ct) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) dst[(size_t)(mt * 16 + g * 4 + r) * (C + 1) + wave * 16 + li] = S[mt][r];
    }
    if (has_d && li == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[(size_t)(dmt * 16 + g * 4 + r) * (C + 1) + C] = D[r];
    }
}

// Token side of the backward, one workgroup per head (256 threads):
//   Z[h] = s1[h] W3_h            -> ds1, dW3_h
//   s1 = softmax(q k^T / sqrt(dh)) v, q,k,v = s Wq,Wk,Wv  -> ds, dWq, dWk, dWv
//   s = mean W1_h + b1_h          -> dmean, dW1_h, db1_h
//   mean = s_raw / (d + eps) (0 where d + eps <= 0) -> ds_raw, dsT, dd
// and db3 = sum_m dZ[0][m] (every head's weights sum to one per point).
// Dynamic LDS: floats mean, dZ [M][C] and s, s1, q, k, v, ds1, dq, dk, dv, ds
// [M][dh] and P, dP [M][M].
__global__ __launch_bounds__(256, 1) void k_bw_token(
    const float *__restrict__ s_raw, const float *__restrict__ dsum, const float *__restrict__ s,
    const float *__restrict__ s1, const float *__restrict__ dZ, const float *__restrict__ W1,
    const float *__restrict__ Wq, const float *__restrict__ Wk, const float *__restrict__ Wv,
    const float *__restrict__ W3, int C, int H, int M, int dh, float eps, float *__restrict__ dsr,
    float *__restrict__ dsT, float *__restrict__ dd, float *__restrict__ dW1, float *__restrict__ db1,
    float *__restrict__ dWq, float *__restrict__ dWk, float *__restrict__ dWv, float *__restrict__ dW3,
    float *__restrict__ db3) {
    extern __shared__ float sm[];
    const int h = blockIdx.x, tid = threadIdx.x, nt = blockDim.x;
    const int HD = H * dh;
    float *mean = sm, *gz = mean + M * C;
    float *ss = gz + M * C, *s1s = ss + M * dh, *q = s1s + M * dh, *k = q + M * dh, *v = k + M * dh;
    float *ds1 = v + M * dh, *dq = ds1 + M * dh, *dk = dq + M * dh, *dv = dk + M * dh, *ds = dv + M * dh;
    float *P = ds + M * dh, *dP = P + M * M;
    const float scale = 1.f / sqrtf((float)dh);
    for (int i = tid; i < M * C; i += nt) {
        const int m = i / C;
        const float den = dsum[h * M + m] + eps;
        mean[i] = den > 0.f ? s_raw[(size_t)h * M * C + i] / den : 0.f;
        gz[i] = dZ[(size_t)h * M * C + i];
    }
    for (int i = tid; i < M * dh; i += nt) {
        ss[i] = s[(size_t)h * M * dh + i];
        s1s[i] = s1[(size_t)h * M * dh + i];
    }
    __syncthreads();
    // ds1 = dZ W3_h^T; dW3_h = s1^T dZ; q, k, v
    for (int i = tid; i < M * dh; i += nt) {
        const int m = i / dh, j = i % dh;
        float a = 0.f, aq = 0.f, ak = 0.f, av = 0.f;
        for (int c = 0; c < C; ++c) a += gz[m * C + c] * W3[(size_t)(h * dh + j) * C + c];
        for (int t = 0; t < dh; ++t) {
            const float sv = ss[m * dh + t];
            aq += sv * Wq[((size_t)h * dh + t) * dh + j];
            ak += sv * Wk[((size_t)h * dh + t) * dh + j];
            av += sv * Wv[((size_t)h * dh + t) * dh + j];
        }
        ds1[i] = a;
        q[i] = aq;
        k[i] = ak;
        v[i] = av;
    }
    for (int i = tid; i < dh * C; i += nt) {
        const int j = i / C, c = i % C;
        float a = 0.f;
        for (int m = 0; m < M; ++m) a += s1s[m * dh + j] * gz[m * C + c];
        dW3[(size_t)(h * dh + j) * C + c] = a;
    }
    if (h == 0)
        for (int c = tid; c < C; c += nt) {
            float a = 0.f;
            for (int m = 0; m < M; ++m) a += gz[m * C + c];
            db3[c] = a;
        }
    __syncthreads();
    // P = softmax_rows(q k^T * scale); dP = ds1 v^T
    for (int i = tid; i < M * M; i += nt) {
        const int a_ = i / M, b_ = i % M;
        float dot = 0.f, dpv = 0.f;
        for (int j = 0; j < dh; ++j) {
            dot += q[a_ * dh + j] * k[b_ * dh + j];
            dpv += ds1[a_ * dh + j] * v[b_ * dh + j];
        }
        P[i] = dot * scale;
        dP[i] = dpv;
    }
    __syncthreads();
    for (int a_ = tid; a_ < M; a_ += nt) {
        float mx = P[a_ * M];
        for (int b_ = 1; b_ < M; ++b_) mx = fmaxf(mx, P[a_ * M + b_]);
        float sum = 0.f;
        for (int b_ = 0; b_ < M; ++b_) {
            const float e = expf(P[a_ * M + b_] - mx);
            P[a_ * M + b_] = e;
            sum += e;
        }
        const float inv = 1.f / sum;
        float dot = 0.f;
        for (int b_ = 0; b_ < M; ++b_) {
            P[a_ * M + b_] *= inv;
            dot += dP[a_ * M + b_] * P[a_ * M + b_];
        }
        // dP becomes da = P (dP - rowsum(dP P))
        for (int b_ = 0; b_ < M; ++b_) dP[a_ * M + b_] = P[a_ * M + b_] * (dP[a_ * M + b_] - dot);
    }
    __syncthreads();
    // dv = P^T ds1; dq = da k * scale; dk = da^T q * scale
    for (int i = tid; i < M * dh; i += nt) {
        const int m = i / dh, j = i % dh;
        float av = 0.f, aq = 0.f, ak = 0.f;
        for (int t = 0; t < M; ++t) {
            av += P[t * M + m] * ds1[t * dh + j];
            aq += dP[m * M + t] * k[t * dh + j];
            ak += dP[t * M + m] * q[t * dh + j];
        }
        dv[i] = av;
        dq[i] = aq * scale;
        dk[i] = ak * scale;
    }
    __syncthreads();
    // dWq/dWk/dWv = s^T (dq, dk, dv); ds = dq Wq^T + dk Wk^T + dv Wv^T
    for (int i = tid; i < dh * dh; i += nt) {
        const int t = i / dh, j = i % dh;
        float aq = 0.f, ak = 0.f, av = 0.f;
        for (int m = 0; m < M; ++m) {
            const float sv = ss[m * dh + t];
            aq += sv * dq[m * dh + j];
            ak += sv * dk[m * dh + j];
            av += sv * dv[m * dh + j];
        }
        dWq[(size_t)h * dh * dh + i] = aq;
        dWk[(size_t)h * dh * dh + i] = ak;
        dWv[(size_t)h * dh * dh + i] = av;
    }
    for (int i = tid; i < M * dh; i += nt) {
        const int m = i / dh, t = i % dh;
        float a = 0.f;
        for (int j = 0; j < dh; ++j)
            a += dq[m * dh + j] * Wq[((size_t)h * dh + t) * dh + j] + dk[m * dh + j] * Wk[((size_t)h * dh + t) * dh + j] +
                 dv[m * dh + j] * Wv[((size_t)h * dh + t) * dh + j];
        ds[i] = a;
    }
    __syncthreads();
    // dW1_h = mean^T ds; db1_h = sum_m ds
    for (int i = tid; i < C * dh; i += nt) {
        const int c = i / dh, j = i % dh;
        float a = 0.f;
        for (int m = 0; m < M; ++m) a += mean[m * C + c] * ds[m * dh + j];
        dW1[(size_t)c * HD + h * dh + j] = a;
    }
    for (int j = tid; j < dh; j += nt) {
        float a = 0.f;
        for (int m = 0; m < M; ++m) a += ds[m * dh + j];
        db1[h * dh + j] = a;
    }
    // dmean = ds W1_h^T (kept in gz); ds_raw = dmean / den; dd = -sum_c dmean mean / den
    for (int i = tid; i < M * C; i += nt) {
        const int m = i / C, c = i % C;
        float a = 0.f;
        for (int j = 0; j < dh; ++j) a += ds[m * dh + j] * W1[(size_t)c * HD + h * dh + j];
        const float den = dsum[h * M + m] + eps;
        const float r = den > 0.f ? a / den : 0.f;
        gz[i] = a;
        dsr[(size_t)h * M * C + i] = r;
        dsT[((size_t)h * C + c) * M + m] = r;
    }
    __syncthreads();
    for (int m = tid; m < M; m += nt) {
        const float den = dsum[h * M + m] + eps;
        float a = 0.f;
        for (int c = 0; c < C; ++c) a += gz[m * C + c] * mean[m * C + c];
        dd[h * M + m] = den > 0.f ? -a / den : 0.f;
    }
}

// dW2[c][h*M + m] = dW2T[h][m][c].
__global__ void k_bw_transpose_w2(const float *__restrict__ dW2T, int C, int HM, float *__restrict__ dW2) {
    const int64_t total = (int64_t)C * HM;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t c = i / HM, hm = i % HM;
        dW2[i] = dW2T[hm * C + c];
    }
}

}  // namespace ts3
