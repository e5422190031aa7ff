// Small kernels of the layer: operand preparation, the ordered fold of span
// partials, and the slice-domain work (Linear1, per-head token attention,
// Linear3) that the paper moves off the points (Eq. (3), Table 2).  These touch
// O(H*M*C) data and run in microseconds.
#pragma once
#include "ts3_device.h"

namespace ts3 {

__device__ __forceinline__ void store_elem(float *p, float v) { *p = v; }
__device__ __forceinline__ void store_elem(bf16_t *p, float v) {
    *reinterpret_cast<__bf16 *>(p) = (__bf16)v;
}

// W2' = W2 * scale in MFMA fragment order [H][MT][CK][64][8]: lane l, slot t
// holds W2'[32*kc + 8*(l>>4) + t][h*M + 16*mt + (l&15)].  b2s = b2 * scale.
// scale = log2(e) / tau, so the softmax can use exp2.
template <typename T>
__global__ void k_prep_w2(const float *__restrict__ W2, const float *__restrict__ b2, float scale,
                          int C, int H, int M, T *__restrict__ w2p, float *__restrict__ b2s) {
    const int MT = M / 16, CK = C / 32, HM = H * M;
    const int64_t total = (int64_t)H * MT * CK * 64 * 8;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int t = (int)(i & 7), lane = (int)((i >> 3) & 63);
        int64_t r = i >> 9;
        const int kc = (int)(r % CK); r /= CK;
        const int mt = (int)(r % MT);
        const int h = (int)(r / MT);
        const int c = kc * 32 + (lane >> 4) * 8 + t;
        const int col = h * M + mt * 16 + (lane & 15);
        store_elem(w2p + i, W2[(int64_t)c * HM + col] * scale);
    }
    const int64_t tid = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (tid < HM) b2s[tid] = (b2 ? b2[tid] : 0.f) * scale;
}

// Z in decoding-operand order [H][CT][KM][64][8]: lane l, slot t holds
// Z[h][32*km + 16*(t>>2) + 4*(l>>4) + (t&3)][zchan(ct, l&15)] + b3[c] / H (zero
// past M).  Each head's slice weights sum to one (Eq. (1)), so the H heads of
// the deslice add b3 exactly once per point and pass 2 needs no bias pass.
template <typename T>
__global__ void k_prep_z(const float *__restrict__ Z, const float *__restrict__ b3, int C, int H, int M,
                         T *__restrict__ zp) {
    const int CT = C / 16, KM = M >= 32 ? M / 32 : 1;
    const float bscale = 1.f / (float)H;
    const int64_t total = (int64_t)H * CT * KM * 64 * 8;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int t = (int)(i & 7), lane = (int)((i >> 3) & 63);
        int64_t r = i >> 9;
        const int km = (int)(r % KM); r /= KM;
        const int ct = (int)(r % CT);
        const int h = (int)(r / CT);
        const int m = km * 32 + (t >> 2) * 16 + (lane >> 4) * 4 + (t & 3);
        const int c = zchan(ct, lane & 15);
        store_elem(zp + i, m < M ? Z[((int64_t)h * M + m) * C + c] + b3[c] * bscale : 0.f);
    }
}

// Zero the partials of spans that no tile wrote, so the fold sees zeros there.
__global__ void k_zero(float *__restrict__ p, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0.f;
}

// Ordered fold of span partials (Eq. (4) sum over tiles): element e of
// [H][M][C+1] is summed over spans 0..nspan-1 in two fixed levels (runs of
// FOLD spans, then the runs in order), giving the same bits for any tiling.
constexpr int FOLD = 64;
// T is the fold's accumulator: float, or double (the partials are added in
// float64 and rounded once at the end); runs hold T.
template <typename T>
__global__ void k_fold_runs(const float *__restrict__ partials, int64_t E, int64_t nspan, T *__restrict__ runs) {
    const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const int64_t run = blockIdx.y;
    if (e >= E) return;
    const int64_t s0 = run * FOLD;
    const int64_t s1 = s0 + FOLD < nspan ? s0 + FOLD : nspan;
    T acc = 0;
    for (int64_t s = s0; s < s1; ++s) acc += (T)partials[s * E + e];
    runs[run * E + e] = acc;
}

// The same fold taken one tile at a time: the tile's spans [g0, g0 + ns)
// (partials[0 .. ns) of this launch) are added to the runs they fall in.  A
// run starting inside the tile starts from zero, one begun by an earlier tile
// continues from its stored sum; each run is thus the same sequential sum,
// in span order, as k_fold_runs forms, and holds the same bits.
template <typename T>
__global__ void k_fold_runs_tile(const float *__restrict__ partials, int64_t E, int64_t g0, int64_t ns,
                                 T *__restrict__ runs) {
    const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const int64_t run = g0 / FOLD + blockIdx.y;
    if (e >= E) return;
    const int64_t r0 = run * FOLD;
    const int64_t s0 = r0 > g0 ? r0 : g0;
    const int64_t s1 = r0 + FOLD < g0 + ns ? r0 + FOLD : g0 + ns;
    T acc = s0 == r0 ? (T)0 : runs[run * E + e];
    for (int64_t s = s0; s < s1; ++s) acc += (T)partials[(s - g0) * E + e];
    runs[run * E + e] = acc;
}

template <typename T>
__global__ void k_fold_final(const T *__restrict__ runs, int64_t E, int64_t nrun, int C, float *__restrict__ s_raw,
                             float *__restrict__ dsum) {
    const int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (e >= E) return;
    T acc = 0;
    for (int64_t r = 0; r < nrun; ++r) acc += runs[r * E + e];
    const int64_t hm = e / (C + 1);
    const int c = (int)(e - hm * (C + 1));
    if (c < C)
        s_raw[hm * C + c] = (float)acc;
    else
        dsum[hm] = (float)acc;
}

// s[h][m][j] = (d^-1 s_raw)[h][m][:] . W1[:, h*dh + j] + b1[h*dh + j]; one
// workgroup of one wave per slice token (grid H*M), a lane per output column.
// The mean is taken before Linear1 (the physical state of Appendix A.4); an
// empty slice (d + eps <= 0) has mean zero.  The mean is formed where it is
// used (s_raw rows stay in L2), so no shape needs LDS.  Each output is one
// sequential sum over c, so the launch shape does not change its rounding.
__global__ void k_finalize(const float *__restrict__ s_raw, const float *__restrict__ dsum,
                           const float *__restrict__ W1, const float *__restrict__ b1, int C, int H,
                           int M, int dh, float eps, float *__restrict__ s) {
    const int hm = blockIdx.x;  // h * M + m
    const int h = hm / M;
    const int HD = H * dh;
    const float den = dsum[hm] + eps;
    const float *row = s_raw + (int64_t)hm * C;
    for (int jj = threadIdx.x; jj < dh; jj += blockDim.x) {
        const int col = h * dh + jj;
        float acc = b1 ? b1[col] : 0.f;
#pragma unroll 8
        for (int c = 0; c < C; ++c) {
            const float mean = den > 0.f ? row[c] / den : 0.f;
            acc = fmaf(mean, W1[(int64_t)c * HD + col], acc);
        }
        s[(int64_t)hm * dh + jj] = acc;
    }
}

// Projected form (head width 16): t_raw [H][M][16] already holds
// sum_i w_i (x_i W1_h), so s = t_raw / (d + eps) + b1, zero mean for an
// empty slice as above.
__global__ void k_finalize_proj(const float *__restrict__ t_raw, const float *__restrict__ dsum,
                                const float *__restrict__ b1, int H, int M, float eps, float *__restrict__ s) {
    const int h = blockIdx.x;
    for (int i = threadIdx.x; i < M * 16; i += blockDim.x) {
        const int m = i >> 4, col = h * 16 + (i & 15);
        const float den = dsum[h * M + m] + eps;
        const float v = t_raw[((int64_t)h * M + m) * 16 + (i & 15)];
        s[((int64_t)h * M + m) * 16 + (i & 15)] = (den > 0.f ? v / den : 0.f) + (b1 ? b1[col] : 0.f);
    }
}

// Per-head attention among the M slice tokens, then Linear3 without bias:
// q,k,v = s Wq[h], s Wk[h], s Wv[h]; A = softmax(q k^T / sqrt(dh)); s1 = A v;
// Z[h][m][c] = s1[m][:] . W3[h*dh .. h*dh+dh-1][c].  Grid (H, ZB): the ZB
// workgroups of a head each run its attention (the same arithmetic, so the
// same s1) and write Z for their C / ZB columns; the first also writes s1.
__global__ void k_attention(const float *__restrict__ s, const float *__restrict__ Wq,
                            const float *__restrict__ Wk, const float *__restrict__ Wv,
                            const float *__restrict__ W3, int C, int H, int M, int dh,
                            float *__restrict__ s1, float *__restrict__ Z) {
    extern __shared__ float sm[];
    const int h = blockIdx.x;
    float *ss = sm;             // [M][dh]
    float *q = ss + M * dh;     // [M][dh]
    float *k = q + M * dh;
    float *v = k + M * dh;
    float *A = v + M * dh;      // [M][M]
    float *o = A + M * M;       // [M][dh]
    const int n = M * dh;
    for (int i = threadIdx.x; i < n; i += blockDim.x) ss[i] = s[(int64_t)h * n + i];
    __syncthreads();
    const float *wq = Wq + (int64_t)h * dh * dh, *wk = Wk + (int64_t)h * dh * dh,
                *wv = Wv + (int64_t)h * dh * dh;
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
        const int m = i / dh, jj = i - m * dh;
        float aq = 0.f, ak = 0.f, av = 0.f;
        for (int u = 0; u < dh; ++u) {
            const float x = ss[m * dh + u];
            aq = fmaf(x, wq[u * dh + jj], aq);
            ak = fmaf(x, wk[u * dh + jj], ak);
            av = fmaf(x, wv[u * dh + jj], av);
        }
        q[i] = aq; k[i] = ak; v[i] = av;
    }
    __syncthreads();
    const float scale = 1.0f / sqrtf((float)dh);
    for (int i = threadIdx.x; i < M * M; i += blockDim.x) {
        const int a = i / M, b = i - a * M;
        float acc = 0.f;
        for (int u = 0; u < dh; ++u) acc = fmaf(q[a * dh + u], k[b * dh + u], acc);
        A[i] = acc * scale;
    }
    __syncthreads();
    for (int a = threadIdx.x; a < M; a += blockDim.x) {
        float mx = A[a * M];
        for (int b = 1; b < M; ++b) mx = fmaxf(mx, A[a * M + b]);
        float sum = 0.f;
        for (int b = 0; b < M; ++b) {
            const float e = expf(A[a * M + b] - mx);
            A[a * M + b] = e;
            sum += e;
        }
        for (int b = 0; b < M; ++b) A[a * M + b] /= sum;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
        const int a = i / dh, jj = i - a * dh;
        float acc = 0.f;
        for (int b = 0; b < M; ++b) acc = fmaf(A[a * M + b], v[b * dh + jj], acc);
        o[i] = acc;
        if (blockIdx.y == 0) s1[(int64_t)h * n + i] = acc;
    }
    __syncthreads();
    const int CB = C / (int)gridDim.y, c0 = (int)blockIdx.y * CB;
    for (int i = threadIdx.x; i < M * CB; i += blockDim.x) {
        const int m = i / CB, c = c0 + (i - m * CB);
        float acc = 0.f;
        for (int u = 0; u < dh; ++u) acc = fmaf(o[m * dh + u], W3[(int64_t)(h * dh + u) * C + c], acc);
        Z[((int64_t)h * M + m) * C + c] = acc;
    }
}

}  // namespace ts3
