// Runtime-shape kernels: the layer for any C and M that are multiples of 16
// (C <= 512, M <= 256) without a tuned kernel, in plain vector arithmetic
// with float32 accumulation.  The same computation as the tuned passes (paper
// Eq. (1), Eq. (4) and Eq. (5), Algorithm 1), with the same span partials and
// ordered fold, so results are tiling-independent in the same way; these are
// the correct-but-slow path for unusual shapes.
//
// Operand layouts (written by k_prep_w2_rt and k_prep_z_rt, storage type T):
//   w2r[h*M + m][c] = W2[c][h*M + m] * log2(e) / tau
//   zr [h*M + m][c] = Z[h][m][c] + b3[c] / H
#pragma once
#include "ts3_small.h"  // store_elem

namespace ts3 {

constexpr int RT_MAX_C = 512, RT_MAX_M = 256, RT_PTS = 16;

template <typename T>
__global__ void k_prep_w2_rt(const float *__restrict__ W2, const float *__restrict__ b2, float scale, int C, int H,
                             int M, T *__restrict__ w2r, float *__restrict__ b2s) {
    const int HM = H * M;
    const int64_t total = (int64_t)HM * C;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t hm = i / C;
        const int c = (int)(i - hm * C);
        store_elem(w2r + i, W2[(int64_t)c * HM + hm] * scale);
    }
    const int64_t tid = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (tid < HM) b2s[tid] = (b2 ? b2[tid] : 0.f) * scale;
}

template <typename T>
__global__ void k_prep_z_rt(const float *__restrict__ Z, const float *__restrict__ b3, int C, int H, int M,
                            T *__restrict__ zr) {
    const float bscale = 1.f / (float)H;
    const int64_t total = (int64_t)H * M * C;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int c = (int)(i % C);
        store_elem(zr + i, Z[i] + b3[c] * bscale);
    }
}

// Logits of RT_PTS points (rows xs[p][0..C)) for slice m = threadIdx.x < M
// of head h, then the max-shifted softmax over the head's M slices, one point
// per thread of the first RT_PTS; ws[p][m] holds the weights (zero for points
// p >= np).  Ends with a barrier.
template <typename T>
__device__ void rt_weights(const float *xs, float *ws, int np, int h, int C, int M, const T *__restrict__ w2r,
                           const float *__restrict__ b2s) {
    const int m = threadIdx.x;
    if (m < M) {
        float a[RT_PTS];
        const float b = b2s[h * M + m];
#pragma unroll
        for (int p = 0; p < RT_PTS; ++p) a[p] = b;
        const T *wr = w2r + ((int64_t)h * M + m) * C;
        for (int c = 0; c < C; ++c) {
            const float w = to_f32(wr[c]);
#pragma unroll
            for (int p = 0; p < RT_PTS; ++p) a[p] = fmaf(xs[p * C + c], w, a[p]);
        }
#pragma unroll
        for (int p = 0; p < RT_PTS; ++p) ws[p * M + m] = a[p];
    }
    __syncthreads();
    if (threadIdx.x < RT_PTS) {
        const int p = threadIdx.x;
        float *row = ws + p * M;
        if (p < np) {
            float mx = row[0];
            for (int k = 1; k < M; ++k) mx = fmaxf(mx, row[k]);
            float sum = 0.f;
            for (int k = 0; k < M; ++k) {
                const float e = exp2f(row[k] - mx);
                row[k] = e;
                sum += e;
            }
            const float inv = 1.f / sum;
            for (int k = 0; k < M; ++k) row[k] *= inv;
        } else {
            for (int k = 0; k < M; ++k) row[k] = 0.f;
        }
    }
    __syncthreads();
}

// Pass 1: partials[span][h][m][c] = sum over the span's points of w[p][m]
// x[p][c] for the workgroup's 64 channels c, column C = sum_p w[p][m] (chunk
// 0).  Grid: nspan * H * ceil(C / 64) workgroups of 256 threads; dynamic LDS
// RT_PTS * (C + M) floats.  Each sum runs over the span's points in order.
template <typename T>
__global__ __launch_bounds__(256) void k_slice_accumulate_rt(const T *__restrict__ x, int64_t n_tile, int64_t span0,
                                                             int32_t Q, int32_t H, int C, int M,
                                                             const T *__restrict__ w2r, const float *__restrict__ b2s,
                                                             float *__restrict__ partials) {
    extern __shared__ float sm[];
    float *xs = sm;             // [RT_PTS][C]
    float *ws = sm + RT_PTS * C;  // [RT_PTS][M]
    const int nchunk = (C + 63) / 64;
    int bid = blockIdx.x;
    const int chunk = bid % nchunk;
    bid /= nchunk;
    const int h = bid % H, span_local = bid / H;
    const int tid = threadIdx.x;
    const int64_t p_begin = (int64_t)span_local * Q;
    const int64_t p_end = p_begin + Q < n_tile ? p_begin + Q : n_tile;
    const int c0 = chunk * 64, cw = C - c0 < 64 ? C - c0 : 64;
    const int ne = M * cw;  // accumulated elements (m, c) of this workgroup, <= 64 per thread
    float acc[64];
#pragma unroll
    for (int k = 0; k < 64; ++k) acc[k] = 0.f;
    float dacc = 0.f;
    for (int64_t pb = p_begin; pb < p_end; pb += RT_PTS) {
        const int np = p_end - pb < RT_PTS ? (int)(p_end - pb) : RT_PTS;
        __syncthreads();  // the previous block's xs and ws are no longer read
        for (int i = tid; i < RT_PTS * C; i += 256) {
            const int p = i / C, c = i - p * C;
            xs[i] = p < np ? to_f32(x[(pb + p) * C + c]) : 0.f;
        }
        __syncthreads();
        rt_weights<T>(xs, ws, np, h, C, M, w2r, b2s);
#pragma unroll
        for (int k = 0; k < 64; ++k) {
            const int e = tid + 256 * k;
            if (e < ne) {
                const int m = e / cw, c = e - m * cw;
                float a = acc[k];
#pragma unroll
                for (int p = 0; p < RT_PTS; ++p) a = fmaf(ws[p * M + m], xs[p * C + c0 + c], a);
                acc[k] = a;
            }
        }
        if (chunk == 0 && tid < M)
#pragma unroll
            for (int p = 0; p < RT_PTS; ++p) dacc += ws[p * M + tid];
    }
    float *dst = partials + ((size_t)(span0 + span_local) * H + h) * (size_t)M * (C + 1);
#pragma unroll
    for (int k = 0; k < 64; ++k) {
        const int e = tid + 256 * k;
        if (e < ne) {
            const int m = e / cw, c = e - m * cw;
            dst[(size_t)m * (C + 1) + c0 + c] = acc[k];
        }
    }
    if (chunk == 0 && tid < M) dst[(size_t)tid * (C + 1) + C] = dacc;
}

// Pass 2: out[p][c] = sum_h sum_m w_h[p][m] zr[h*M + m][c] for RT_PTS points
// per workgroup (256 threads; dynamic LDS RT_PTS * (C + M) floats).
template <typename T>
__global__ __launch_bounds__(256) void k_deslice_rt(const T *__restrict__ x, int64_t n, int32_t H, int C, int M,
                                                    const T *__restrict__ w2r, const float *__restrict__ b2s,
                                                    const T *__restrict__ zr, T *__restrict__ out) {
    extern __shared__ float sm[];
    float *xs = sm;
    float *ws = sm + RT_PTS * C;
    const int tid = threadIdx.x;
    const int64_t p0 = (int64_t)blockIdx.x * RT_PTS;
    const int np = n - p0 < RT_PTS ? (int)(n - p0) : RT_PTS;
    for (int i = tid; i < RT_PTS * C; i += 256) {
        const int p = i / C, c = i - p * C;
        xs[i] = p < np ? to_f32(x[(p0 + p) * C + c]) : 0.f;
    }
    __syncthreads();
    const int ne = RT_PTS * C;  // output elements (p, c), <= 32 per thread
    float acc[RT_MAX_C * RT_PTS / 256];
#pragma unroll
    for (int k = 0; k < RT_MAX_C * RT_PTS / 256; ++k) acc[k] = 0.f;
    for (int h = 0; h < H; ++h) {
        rt_weights<T>(xs, ws, np, h, C, M, w2r, b2s);
#pragma unroll
        for (int k = 0; k < RT_MAX_C * RT_PTS / 256; ++k) {
            const int e = tid + 256 * k;
            if (e < ne) {
                const int p = e / C, c = e - p * C;
                const T *zc = zr + (int64_t)h * M * C + c;
                float a = acc[k];
                for (int m = 0; m < M; ++m) a = fmaf(ws[p * M + m], to_f32(zc[(int64_t)m * C]), a);
                acc[k] = a;
            }
        }
        __syncthreads();  // ws is rewritten by the next head
    }
#pragma unroll
    for (int k = 0; k < RT_MAX_C * RT_PTS / 256; ++k) {
        const int e = tid + 256 * k;
        if (e < ne) {
            const int p = e / C, c = e - p * C;
            if (p < np) store_elem(out + (p0 + p) * C + c, acc[k]);
        }
    }
}

}  // namespace ts3
