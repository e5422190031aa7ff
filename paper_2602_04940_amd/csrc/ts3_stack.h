// Host side of the Transolver block stack: L pre-norm blocks, each a
// Physics-Attention layer (its own ts3_state, so every block's physical state
// stays cached) followed by the feed-forward network of ts3_block.h.  Included
// once, at the end of ts3.hip: it uses the layer entry points and the error
// helpers defined there.
#pragma once
#include "ts3_block.h"

struct ts3_stack {
    ts3_desc desc{};
    int32_t L = 0, F = 0;
    std::vector<ts3_state *> layers;
    bf16_t *xn = nullptr;    // LN1 of the current block's input [max_points][C]
    bf16_t *pa = nullptr;    // Physics-Attention output [max_points][C]
    bf16_t *frag = nullptr;  // feed-forward fragments, one block's worth
    int64_t bytes = 0;
};

namespace {

struct StackKernels {
    void (*ln)(const bf16_t *, int64_t, const float *, const float *, bf16_t *, hipStream_t);
    void (*prep)(const float *, const float *, int, bf16_t *, hipStream_t);
    void (*mlp)(const bf16_t *, const bf16_t *, int64_t, const float *, const float *, const bf16_t *,
                const float *, const float *, const float *, const float *, bf16_t *, bf16_t *, hipStream_t);
};

template <int C> void launch_ln(const bf16_t *x, int64_t n, const float *g, const float *b, bf16_t *out,
                                hipStream_t st) {
    const int64_t rows_per_wg = 4 * (64 / (C / 8));
    const unsigned grid = (unsigned)std::min<int64_t>((n + rows_per_wg - 1) / rows_per_wg, 8192);
    hipLaunchKernelGGL(k_layernorm<C>, dim3(grid), dim3(256), 0, st, x, n, g, b, out);
}
template <int C> void launch_prep(const float *Wa, const float *Wb, int F, bf16_t *frag, hipStream_t st) {
    hipLaunchKernelGGL(k_prep_mlp<C>, dim3(1024), dim3(256), 0, st, Wa, Wb, F, frag);
}
template <int C, int F>
void launch_mlp(const bf16_t *x, const bf16_t *pa, int64_t n, const float *l2g, const float *l2b,
                const bf16_t *frag, const float *ba, const float *bb, const float *lng, const float *lnb, bf16_t *xo,
                bf16_t *xn, hipStream_t st) {
    hipLaunchKernelGGL((k_mlp_residual_pc<C, F>), dim3((unsigned)((n + 127) / 128)), dim3(512), 0, st, x, pa, n,
                       l2g, l2b, frag, ba, bb, lng, lnb, xo, xn);
}

bool find_stack_kernels(int C, int F, StackKernels *k) {
    if (C == 128 && F == 512) {
        *k = StackKernels{&launch_ln<128>, &launch_prep<128>, &launch_mlp<128, 512>};
        return true;
    }
    if (C == 256 && F == 1024) {
        *k = StackKernels{&launch_ln<256>, &launch_prep<256>, &launch_mlp<256, 1024>};
        return true;
    }
    return false;
}

ts3_status check_block(const ts3_block_weights *b) {
    if (!b->ln1_g || !b->ln1_b || !b->ln2_g || !b->ln2_b || !b->Wa || !b->ba || !b->Wb || !b->bb)
        return fail(TS3_ERR_INVALID_ARG, "a LayerNorm or feed-forward pointer of a block is NULL");
    return TS3_OK;
}

// LN1 of block 0 into xn, then per block: attention output into pa, and the
// feed-forward kernel writing the block output over x and the next LN1 into
// xn.  `attend(l)` runs block l's Physics-Attention from xn into pa.
template <typename Attend>
ts3_status run_blocks(ts3_stack *s, const ts3_block_weights *blocks, bf16_t *x, int64_t n, hipStream_t hs,
                      Attend attend) {
    StackKernels k{};
    find_stack_kernels(s->desc.C, s->F, &k);
    for (int l = 0; l < s->L; ++l) {
        ts3_status st = check_block(&blocks[l]);
        if (st != TS3_OK) return st;
    }
    k.ln(x, n, blocks[0].ln1_g, blocks[0].ln1_b, s->xn, hs);
    LAUNCH_CHECK("layernorm");
    for (int l = 0; l < s->L; ++l) {
        ts3_status st = attend(l);
        if (st != TS3_OK) return st;
        const ts3_block_weights &b = blocks[l];
        k.prep(b.Wa, b.Wb, s->F, s->frag, hs);
        LAUNCH_CHECK("feed-forward fragments");
        const bool next = l + 1 < s->L;
        k.mlp(x, s->pa, n, b.ln2_g, b.ln2_b, s->frag, b.ba, b.bb, next ? blocks[l + 1].ln1_g : nullptr,
              next ? blocks[l + 1].ln1_b : nullptr, x, s->xn, hs);
        LAUNCH_CHECK("feed-forward");
    }
    return TS3_OK;
}

}  // namespace

extern "C" {

ts3_status ts3_stack_create(const ts3_desc *desc, int32_t n_blocks, int32_t hidden, ts3_stack **out) {
    if (!desc || !out) return fail(TS3_ERR_INVALID_ARG, "NULL argument");
    *out = nullptr;
    if (n_blocks < 1 || n_blocks > 1024) return fail(TS3_ERR_INVALID_ARG, "1 <= n_blocks <= 1024 required");
    if (desc->io_dtype != TS3_BF16) return fail(TS3_ERR_UNSUPPORTED, "the block stack stores bf16 activations");
    StackKernels k{};
    if (!find_stack_kernels(desc->C, hidden, &k))
        return fail(TS3_ERR_UNSUPPORTED, "no feed-forward kernel for C=%d, hidden=%d (supported: (128, 512), "
                    "(256, 1024))", desc->C, hidden);
    ts3_status s = check_desc(desc);
    if (s != TS3_OK) return s;
    ts3_stack *st = new (std::nothrow) ts3_stack();
    if (!st) return fail(TS3_ERR_OUT_OF_MEMORY, "host allocation failed");
    st->desc = *desc;
    st->L = n_blocks;
    st->F = hidden;
    for (int l = 0; l < n_blocks; ++l) {
        ts3_state *ls = nullptr;
        s = ts3_state_create(desc, &ls);
        if (s != TS3_OK) {
            ts3_stack_free(st);
            return s;
        }
        st->layers.push_back(ls);
        st->bytes += ls->bytes;
    }
    const int64_t act = std::max<int64_t>(desc->max_points, 1) * desc->C * 2;
    struct Req {
        void **p;
        int64_t bytes;
    } reqs[] = {{(void **)&st->xn, act}, {(void **)&st->pa, act}, {(void **)&st->frag, (int64_t)2 * hidden * desc->C * 2}};
    for (auto &r : reqs) {
        hipError_t e = hipMalloc(r.p, (size_t)r.bytes);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            ts3_stack_free(st);
            return fail(e == hipErrorOutOfMemory ? TS3_ERR_OUT_OF_MEMORY : TS3_ERR_HIP, "hipMalloc(%lld bytes): %s",
                        (long long)r.bytes, hipGetErrorString(e));
        }
        st->bytes += r.bytes;
    }
    *out = st;
    return TS3_OK;
}

ts3_status ts3_stack_free(ts3_stack *s) {
    if (!s) return TS3_OK;
    for (ts3_state *l : s->layers) ts3_state_free(l);
    (void)hipFree(s->xn);
    (void)hipFree(s->pa);
    (void)hipFree(s->frag);
    delete s;
    return TS3_OK;
}

ts3_status ts3_stack_bytes(const ts3_stack *s, int64_t *bytes) {
    if (!s || !bytes) return fail(TS3_ERR_INVALID_ARG, "NULL argument");
    *bytes = s->bytes;
    return TS3_OK;
}

ts3_status ts3_stack_layer(ts3_stack *s, int32_t l, ts3_state **layer) {
    if (!s || !layer) return fail(TS3_ERR_INVALID_ARG, "NULL argument");
    if (l < 0 || l >= s->L) return fail(TS3_ERR_INVALID_ARG, "block %d of %d", l, s->L);
    *layer = s->layers[(size_t)l];
    return TS3_OK;
}

ts3_status ts3_stack_forward(ts3_stack *s, const ts3_block_weights *blocks, void *x, int64_t N, int64_t tile,
                             int64_t chunk, void *stream) {
    if (!s || !blocks) return fail(TS3_ERR_INVALID_ARG, "NULL argument");
    if (N <= 0 || N > s->desc.max_points) return fail(TS3_ERR_INVALID_ARG, "0 < N <= max_points required");
    if (!x || ((uintptr_t)x & 15)) return fail(TS3_ERR_INVALID_ARG, "x must be a 16-byte aligned device pointer");
    hipStream_t hs = (hipStream_t)stream;
    bf16_t *xb = (bf16_t *)x;
    return run_blocks(s, blocks, xb, N, hs, [&](int l) {
        return ts3_layer_forward(s->layers[(size_t)l], &blocks[l].pa, s->xn, N, tile, chunk, s->pa, stream);
    });
}

ts3_status ts3_stack_decode(ts3_stack *s, const ts3_block_weights *blocks, void *q, int64_t n, int64_t chunk,
                            void *stream) {
    if (!s || !blocks) return fail(TS3_ERR_INVALID_ARG, "NULL argument");
    if (n < 0 || n > s->desc.max_points) return fail(TS3_ERR_INVALID_ARG, "0 <= n <= max_points required");
    if (n == 0) return TS3_OK;
    if (!q || ((uintptr_t)q & 15)) return fail(TS3_ERR_INVALID_ARG, "q must be a 16-byte aligned device pointer");
    if (chunk <= 0) return fail(TS3_ERR_INVALID_ARG, "chunk > 0 required");
    for (ts3_state *l : s->layers)
        if (l->phase != PH_ATTEND) return fail(TS3_ERR_BAD_STATE, "every block needs its cached state");
    const int64_t C = s->desc.C;
    bf16_t *qb = (bf16_t *)q;
    return run_blocks(s, blocks, qb, n, (hipStream_t)stream, [&](int l) {
        for (int64_t c0 = 0; c0 < n; c0 += chunk) {
            const int64_t m = std::min(chunk, n - c0);
            ts3_status st = ts3_deslice(s->layers[(size_t)l], &blocks[l].pa, s->xn + c0 * C, m, s->pa + c0 * C, stream);
            if (st != TS3_OK) return st;
        }
        return TS3_OK;
    });
}

ts3_status ts3_stack_feedforward(ts3_stack *s, const ts3_block_weights *blocks, int32_t l, void *x, const void *pa,
                                 int64_t n, void *xn_next, void *stream) {
    if (!s || !blocks) return fail(TS3_ERR_INVALID_ARG, "NULL argument");
    if (l < 0 || l >= s->L) return fail(TS3_ERR_INVALID_ARG, "block %d of %d", l, s->L);
    if (n < 0 || n > s->desc.max_points) return fail(TS3_ERR_INVALID_ARG, "0 <= n <= max_points required");
    if (n == 0) return TS3_OK;
    if (!x || !pa || ((uintptr_t)x & 15) || ((uintptr_t)pa & 15) || ((uintptr_t)xn_next & 15))
        return fail(TS3_ERR_INVALID_ARG, "x, pa (and xn_next) must be 16-byte aligned device pointers");
    ts3_status st = check_block(&blocks[l]);
    if (st != TS3_OK) return st;
    const bool next = xn_next && l + 1 < s->L;
    if (next) {
        st = check_block(&blocks[l + 1]);
        if (st != TS3_OK) return st;
    }
    StackKernels k{};
    find_stack_kernels(s->desc.C, s->F, &k);
    hipStream_t hs = (hipStream_t)stream;
    const ts3_block_weights &b = blocks[l];
    k.prep(b.Wa, b.Wb, s->F, s->frag, hs);
    LAUNCH_CHECK("feed-forward fragments");
    k.mlp((const bf16_t *)x, (const bf16_t *)pa, n, b.ln2_g, b.ln2_b, s->frag, b.ba, b.bb,
          next ? blocks[l + 1].ln1_g : nullptr, next ? blocks[l + 1].ln1_b : nullptr, (bf16_t *)x, (bf16_t *)xn_next,
          hs);
    LAUNCH_CHECK("feed-forward");
    return TS3_OK;
}

}  // extern "C"
