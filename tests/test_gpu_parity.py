"""GPU parity: the HIP path through the C ABI against the float64 oracle.

Bars: float32 storage -> normwise max relative error <= 1e-4; bfloat16
storage with float32 accumulation -> relative L2 <= 2e-2.  Tiled and untiled
runs, tile order, and reruns must agree bitwise.
"""
import math

import numpy as np
import pytest

import oracle
from gpu_helpers import (assert_bf16_close, assert_state_close, banner, match_sums, normwise, rel_l2, state_of,
                         sums_key, to_device, to_host)
from ts3_synth import WORKLOADS, make_weights
from ts3_synth.workloads import small_features

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-4
BF16_TOL = 2e-2


def _torch():
    import torch
    return torch


def _layer(C, H, M, dtype, tau=0.5, Q=1024, max_points=1 << 16, eps=0.0):
    from paper_2602_04940_amd import PhysicsAttention
    return PhysicsAttention(C, H, M, C // H, tau, dtype, group_span=Q, max_points=max_points, eps=eps)


def _weights(W):
    from paper_2602_04940_amd import LayerWeights
    return LayerWeights(W)


def _state(layer):
    return state_of(layer)


def _run(x64, W, C, H, M, dtype, tau, tile, chunk, Q, eps=0.0):
    torch = _torch()
    x = to_device(x64, dtype)
    lw = _weights(W)
    with _layer(C, H, M, dtype, tau, Q, max(len(x64), 1), eps) as layer:
        out = layer.forward(lw, x, tile=tile, chunk=chunk)
        torch.cuda.synchronize()
        return to_host(out), _state(layer), out


# ------------------------------------------------------------ named workloads

def test_fp32_ellipsoid_4k_layer_and_state():
    wl = WORKLOADS["ellipsoid_4k_fp32"]
    banner(f"{wl.name}: N={wl.N} C={wl.C} H={wl.H} M={wl.M} fp32")
    x = small_features(wl, wl.N)
    W = make_weights(wl.C, wl.H, wl.M, wl.dh, seed=0)
    got, st, _ = _run(x, W, wl.C, wl.H, wl.M, "fp32", wl.tau, tile=wl.tile, chunk=wl.chunk, Q=1024)
    ref_st = match_sums(st, oracle.build_state(x, W, wl.H, wl.M, 1 / wl.tau), x, W, wl.H, wl.M, 1 / wl.tau)
    for k in (sums_key(st), "d", "s", "s1", "Z"):
        assert normwise(st[k], ref_st[k]) <= FP32_TOL, k
    ref = oracle.layer_forward_fast(x, W, wl.H, wl.M, 1 / wl.tau)
    err = normwise(got, ref)
    print(f"normwise max rel err {err:.3e}")
    assert err <= FP32_TOL


@pytest.fixture(scope="module")
def ellipsoid_1m():
    wl = WORKLOADS["ellipsoid_1m_bf16"]
    banner(f"{wl.name}: generating inputs")
    x = small_features(wl, wl.N)
    W = make_weights(wl.C, wl.H, wl.M, wl.dh, seed=0)
    banner(f"{wl.name}: oracle pass 1")
    st = oracle.build_state(x, W, wl.H, wl.M, 1 / wl.tau, tile=wl.tile)
    banner(f"{wl.name}: oracle pass 2")
    ref = np.concatenate([oracle.deslice(x[c:c + wl.chunk], W["W2"], W["b2"], st["Z"], W["b3"], wl.H, wl.M,
                                         1 / wl.tau) for c in range(0, wl.N, wl.chunk)])
    return wl, x, W, ref, st


def test_bf16_ellipsoid_1m_tiled_matches_oracle_and_untiled_bitwise(ellipsoid_1m):
    torch = _torch()
    wl, x, W, ref, ref_st = ellipsoid_1m
    banner(f"{wl.name}: N={wl.N} tile={wl.tile} Q={wl.group_span} bf16")
    got, st, out_t = _run(x, W, wl.C, wl.H, wl.M, "bf16", wl.tau, wl.tile, wl.chunk, wl.group_span)
    match_sums(st, ref_st, x, W, wl.H, wl.M, 1 / wl.tau, wl.tile)
    assert_bf16_close(got, ref, "out", BF16_TOL)
    assert_state_close(st, ref_st, "state", BF16_TOL)
    one_tile = -(-wl.N // wl.group_span) * wl.group_span
    got1, st1, out_1 = _run(x, W, wl.C, wl.H, wl.M, "bf16", wl.tau, one_tile, wl.N, wl.group_span)
    assert np.array_equal(st1["Z"], st["Z"]) and np.array_equal(st1[sums_key(st)], st[sums_key(st)])
    assert torch.equal(out_1, out_t)


# ------------------------------------------------------------ shape sweep

SHAPES = [(64, 4, 16), (64, 4, 32), (64, 1, 32), (128, 8, 16), (128, 8, 32), (128, 8, 64), (128, 2, 64),
          (128, 1, 32)]


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("C,H,M", SHAPES)
def test_shapes_ragged_tiles_random_biases(C, H, M, dtype):
    N, Q, tile, chunk = 1000, 128, 384, 333
    banner(f"shape C={C} H={H} M={M} {dtype} N={N} tile={tile} Q={Q}")
    rng = np.random.default_rng(C * 1000 + H * 10 + M)
    x = rng.standard_normal((N, C))
    if dtype == "bf16":
        from ts3_synth import round_bf16
        x = round_bf16(x)
    else:
        x = x.astype(np.float32).astype(np.float64)
    W = make_weights(C, H, M, C // H, seed=3, bias_seed=4)
    got, st, _ = _run(x, W, C, H, M, dtype, 0.5, tile, chunk, Q)
    ref = oracle.layer_forward_fast(x, W, H, M, 2.0)
    ref_st = match_sums(st, oracle.build_state(x, W, H, M, 2.0), x, W, H, M, 2.0)
    if dtype == "fp32":
        assert normwise(got, ref) <= FP32_TOL
        for k in (sums_key(st), "d", "Z"):
            assert normwise(st[k], ref_st[k]) <= FP32_TOL, k
    else:
        assert_bf16_close(got, ref, "out", BF16_TOL)
        assert_state_close(st, ref_st, "state", BF16_TOL)


@pytest.mark.parametrize("C,H,M", [(256, 8, 64), (256, 4, 64)])
def test_wide_rows_bf16_ragged_spans_random_biases(C, H, M):
    """C = 256 (the car-surface stack's width): pass 1 with two producer and
    two consumer waves per head; spans of 12 blocks of 32 points, the last
    span ragged."""
    N, Q, tile, chunk = 2000, 384, 768, 333
    banner(f"wide shape C={C} H={H} M={M} bf16 N={N} tile={tile} Q={Q}")
    from ts3_synth import round_bf16
    rng = np.random.default_rng(C * 1000 + H * 10 + M)
    x = round_bf16(rng.standard_normal((N, C)))
    W = make_weights(C, H, M, C // H, seed=3, bias_seed=4)
    got, st, _ = _run(x, W, C, H, M, "bf16", 0.5, tile, chunk, Q)
    ref = oracle.layer_forward_fast(x, W, H, M, 2.0)
    ref_st = match_sums(st, oracle.build_state(x, W, H, M, 2.0), x, W, H, M, 2.0)
    assert_bf16_close(got, ref, "out", BF16_TOL)
    assert_state_close(st, ref_st, "state", BF16_TOL)
    got1, st1, _ = _run(x, W, C, H, M, "bf16", 0.5, 2304, N, Q)
    assert np.array_equal(got1, got)
    for k in (sums_key(st), "d", "Z"):
        assert np.array_equal(st1[k], st[k]), k


RT_SHAPES = [(192, 4, 48, "fp32"), (192, 4, 48, "bf16"), (256, 8, 64, "fp32"), (128, 8, 128, "bf16"),
             (96, 6, 16, "fp32"), (512, 8, 16, "bf16"), (48, 1, 80, "fp32")]


@pytest.mark.parametrize("C,H,M,dtype", RT_SHAPES)
def test_runtime_shape_kernels_ragged_tiles(C, H, M, dtype):
    """Shapes without a tuned kernel (any C, M that are multiples of 16):
    the runtime-shape vector kernels, ragged spans and chunks, tiled and
    untiled runs bitwise equal."""
    N, Q, tile, chunk = 1000, 160, 480, 333
    banner(f"runtime shape C={C} H={H} M={M} {dtype} N={N} tile={tile} Q={Q}")
    rng = np.random.default_rng(C * 1000 + H * 10 + M + 7)
    x = rng.standard_normal((N, C))
    if dtype == "bf16":
        from ts3_synth import round_bf16
        x = round_bf16(x)
    else:
        x = x.astype(np.float32).astype(np.float64)
    W = make_weights(C, H, M, C // H, seed=5, bias_seed=6)
    got, st, _ = _run(x, W, C, H, M, dtype, 0.5, tile, chunk, Q)
    ref = oracle.layer_forward_fast(x, W, H, M, 2.0)
    ref_st = match_sums(st, oracle.build_state(x, W, H, M, 2.0), x, W, H, M, 2.0)
    if dtype == "fp32":
        assert normwise(got, ref) <= FP32_TOL
        for k in (sums_key(st), "d", "Z"):
            assert normwise(st[k], ref_st[k]) <= FP32_TOL, k
    else:
        assert_bf16_close(got, ref, "out", BF16_TOL)
        assert_state_close(st, ref_st, "state", BF16_TOL)
    got1, st1, _ = _run(x, W, C, H, M, dtype, 0.5, 1120, N, Q)
    assert np.array_equal(got1, got)
    for k in (sums_key(st), "d", "Z"):
        assert np.array_equal(st1[k], st[k]), k


@pytest.mark.parametrize("Q", [64, 96, 100, 160])
def test_bf16_two_head_workgroups_odd_block_counts(Q):
    """Pass 1 with two heads per workgroup and the span's 32-point blocks in
    three interleaved streams: Q = 64 gives two blocks (the third stream has
    none), Q = 96 one block per stream, Q = 100 four blocks (the last of 4
    points; two streams end on a step with no points), Q = 160 five blocks.
    States match the oracle and tiled runs match an untiled one bitwise."""
    C, H, M, N = 128, 8, 64, 4100
    banner(f"two-head pass 1, Q={Q}, N={N}")
    rng = np.random.default_rng(Q)
    from ts3_synth import round_bf16
    x = round_bf16(rng.standard_normal((N, C)))
    W = make_weights(C, H, M, C // H, seed=7, bias_seed=8)
    got, st, out_t = _run(x, W, C, H, M, "bf16", 0.5, 10 * Q, 1000, Q)
    ref = oracle.layer_forward_fast(x, W, H, M, 2.0)
    ref_st = match_sums(st, oracle.build_state(x, W, H, M, 2.0), x, W, H, M, 2.0)
    assert_bf16_close(got, ref, "out", BF16_TOL)
    assert_state_close(st, ref_st, "state", BF16_TOL)
    one_tile = -(-N // Q) * Q
    got1, st1, out_1 = _run(x, W, C, H, M, "bf16", 0.5, one_tile, N, Q)
    for k in (sums_key(st), "d", "Z"):
        assert np.array_equal(st1[k], st[k]), k
    assert np.array_equal(got1, got)


# ------------------------------------------------------------ special cases

@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_infinite_temperature_gives_mean_pool(dtype):
    C, H, M, N = 64, 4, 32, 777
    banner(f"1/tau=0 {dtype}")
    rng = np.random.default_rng(1)
    from ts3_synth import round_storage
    x = round_storage(rng.standard_normal((N, C)), dtype)
    W = make_weights(C, H, M, C // H, seed=5, bias_seed=6)
    got, st, _ = _run(x, W, C, H, M, dtype, math.inf, 256, 500, 128)
    ref = oracle.layer_forward_fast(x, W, H, M, 0.0)
    if dtype == "fp32":
        assert normwise(got, ref) <= FP32_TOL
    else:
        assert_bf16_close(got, ref, "out", BF16_TOL)
    np.testing.assert_allclose(st["d"], N / M, rtol=1e-5 if dtype == "fp32" else 1e-2)


def test_one_hot_slices_fp32():
    C, H, M, N = 64, 4, 16, 1024
    banner("one-hot slices fp32")
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3 * N, C)).astype(np.float32).astype(np.float64)
    W = make_weights(C, H, M, C // H, seed=7)
    # keep points whose two largest logits differ by > 0.05 in every head (weights are one-hot)
    lg = np.sort((x @ W["W2"].astype(np.float64)).reshape(-1, H, M), axis=2)
    x = x[((lg[:, :, -1] - lg[:, :, -2]) > 0.05).all(axis=1)][:N]
    assert len(x) == N
    got, st, _ = _run(x, W, C, H, M, "fp32", 1.0 / 200.0, 512, 512, 256)
    ref_st = oracle.build_state(x, W, H, M, 200.0)
    assert normwise(st[sums_key(st)], ref_st[sums_key(st)]) <= FP32_TOL
    assert normwise(st["d"], ref_st["d"]) <= FP32_TOL
    ref = oracle.layer_forward_fast(x, W, H, M, 200.0)
    assert normwise(got, ref) <= FP32_TOL


@pytest.mark.parametrize("C,Q", [(128, 512), (256, 384)])
def test_bf16_shifted_softmax_fallback_mixed_with_fast_path(C, Q):
    """bf16 at the benchmark shape (and at the stack's width C = 256) with a
    region of points whose logits overflow exp2 (sums outside [2^-100,
    2^100]): the blocks holding them take the max-shifted path in both
    passes, the others the unshifted one."""
    H, M, N = 8, 64, 6000
    banner(f"bf16 softmax fallback mixed with the fast path, C={C}")
    from ts3_synth import round_bf16
    rng = np.random.default_rng(21)
    W = make_weights(C, H, M, C // H, seed=5, bias_seed=6)
    W2 = W["W2"].astype(np.float64)
    it = 2.0
    x = rng.standard_normal((N, C))
    # points lo..hi-1 point along one W2 column per head, scaled so that each
    # head's largest logit exceeds 2^130 in exp2 units (the unshifted sum
    # overflows); candidates whose weights are not one-hot by a wide margin
    # (top two logits under 24 exp2 units apart) are dropped
    lo, hi = 2100, 2900
    cols = rng.integers(0, M, size=(2000, H)) + np.arange(H) * M
    cand = round_bf16(300.0 * W2[:, cols].sum(axis=2).T + 0.1 * rng.standard_normal((2000, C)))
    lgc = np.sort((cand @ W2).reshape(-1, H, M), axis=2) * it / np.log(2.0)
    good = ((lgc[:, :, -1] - lgc[:, :, -2]).min(axis=1) > 24) & (lgc[:, :, -1].max(axis=1) > 130)
    assert good.sum() >= hi - lo
    x[lo:hi] = cand[good][:hi - lo]
    x = round_bf16(x)
    lg = (x @ W2) * it / np.log(2.0)
    assert np.abs(lg[:lo]).max() < 40 and np.abs(lg[hi:]).max() < 40   # fast-path rows elsewhere
    got, st, _ = _run(x, W, C, H, M, "bf16", 1 / it, 3 * Q if C == 128 else 4 * Q, 1000, Q)
    ref = oracle.layer_forward_fast(x, W, H, M, it)
    ref_st = match_sums(st, oracle.build_state(x, W, H, M, it), x, W, H, M, it)
    assert_bf16_close(got, ref, "out", BF16_TOL)
    assert_state_close(st, ref_st, "state", BF16_TOL)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_permuted_and_duplicated_points(dtype):
    torch = _torch()
    C, H, M, N = 128, 8, 32, 640
    banner(f"permutation/duplication {dtype}")
    rng = np.random.default_rng(3)
    from ts3_synth import round_storage
    x = round_storage(rng.standard_normal((N, C)), dtype)
    W = make_weights(C, H, M, C // H, seed=8)
    got, st, _ = _run(x, W, C, H, M, dtype, 0.5, 640, 640, 64)
    perm = rng.permutation(N)
    got_p, st_p, _ = _run(x[perm], W, C, H, M, dtype, 0.5, 640, 640, 64)
    got_d, st_d, _ = _run(np.concatenate([x, x]), W, C, H, M, dtype, 0.5, 1280, 1280, 64)
    f = normwise if dtype == "fp32" else rel_l2
    tol = FP32_TOL if dtype == "fp32" else BF16_TOL
    assert f(got_p, got[perm]) <= tol
    assert f(st_p["Z"], st["Z"]) <= tol
    assert f(st_d["Z"], st["Z"]) <= tol
    assert f(got_d, np.concatenate([got, got])) <= tol


def test_empty_mesh_and_empty_chunks():
    torch = _torch()
    C, H, M = 64, 4, 16
    banner("empty mesh")
    W = make_weights(C, H, M, C // H, seed=9, bias_seed=10)
    lw = _weights(W)
    with _layer(C, H, M, "fp32", Q=64, max_points=64) as layer:
        x = torch.empty((0, C), device="cuda", dtype=torch.float32)
        layer.forward(lw, x, tile=64, chunk=64)
        st = _state(layer)
        ref_st = oracle.build_state(np.zeros((0, C)), W, H, M, 2.0)
        for k in ("s", "s1", "Z"):
            assert normwise(st[k], ref_st[k]) <= FP32_TOL, k
        y = layer.deslice(lw, x)
        assert y.shape == (0, C)


# ------------------------------------------------------------ determinism

def test_rerun_and_reverse_tile_order_are_bitwise_identical():
    torch = _torch()
    C, H, M, N, Q = 128, 8, 64, 5000, 256
    banner("determinism bf16 C=128 M=64")
    rng = np.random.default_rng(4)
    from ts3_synth import round_bf16
    x64 = round_bf16(rng.standard_normal((N, C)))
    W = make_weights(C, H, M, C // H, seed=11)
    lw = _weights(W)
    x = to_device(x64, "bf16")
    with _layer(C, H, M, "bf16", Q=Q, max_points=N) as layer:
        out_a = layer.forward(lw, x, tile=1024, chunk=999).clone()
        Za = layer.get(4)
        out_b = layer.forward(lw, x, tile=1024, chunk=4096).clone()
        layer.reset()
        starts = list(range(0, N, 512))[::-1]
        for t0 in starts:
            layer.accumulate(lw, x[t0:t0 + 512], t0)
        layer.finalize(lw)
        layer.attention(lw)
        out_c = layer.deslice(lw, x)
        Zc = layer.get(4)
    torch.cuda.synchronize()
    assert torch.equal(out_a, out_b) and torch.equal(out_a, out_c)
    assert np.array_equal(Za, Zc)


# ------------------------------------------------------------ pass 2 alone

@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_deslice_with_injected_state(dtype):
    torch = _torch()
    C, H, M, N = 128, 8, 64, 3001
    banner(f"deslice with injected Z {dtype}")
    rng = np.random.default_rng(5)
    from ts3_synth import round_storage
    x64 = round_storage(rng.standard_normal((N, C)), dtype)
    W = make_weights(C, H, M, C // H, seed=12, bias_seed=13)
    Z = rng.standard_normal((H, M, C)) * 0.3
    b3 = rng.standard_normal(C) * 0.1
    lw = _weights(W)
    with _layer(C, H, M, dtype, Q=128, max_points=N) as layer:
        layer.set_state(lw, Z.astype(np.float32), b3.astype(np.float32))
        out = layer.deslice(lw, to_device(x64, dtype))
        torch.cuda.synchronize()
    ref = oracle.deslice(x64, W["W2"], W["b2"], Z.astype(np.float32), b3.astype(np.float32), H, M, 2.0)
    got = to_host(out)
    if dtype == "fp32":
        assert normwise(got, ref) <= FP32_TOL
    else:
        assert_bf16_close(got, ref, "out", BF16_TOL)


# ------------------------------------------------------------ error paths

def test_call_order_and_argument_errors():
    torch = _torch()
    from paper_2602_04940_amd import _lib as L
    C, H, M = 64, 4, 16
    banner("error paths")
    W = make_weights(C, H, M, C // H, seed=14)
    lw = _weights(W)
    lw2 = _weights(W)  # same values, different W2 pointer
    x = torch.zeros((256, C), device="cuda", dtype=torch.float32)

    def status(fn):
        try:
            fn()
        except L.TS3Error as e:
            return e.status
        return L.TS3_OK

    with _layer(C, H, M, "fp32", Q=64, max_points=512) as layer:
        assert status(lambda: layer.deslice(lw, x)) == L.TS3_ERR_BAD_STATE
        assert status(lambda: layer.attention(lw)) == L.TS3_ERR_BAD_STATE
        assert status(lambda: layer.accumulate(lw, x[:64], 32)) == L.TS3_ERR_INVALID_ARG   # misaligned
        assert status(lambda: layer.accumulate(lw, x, 320)) == L.TS3_ERR_INVALID_ARG       # past max_points
        assert status(lambda: layer.accumulate(lw, x[:128], 0)) == L.TS3_OK
        assert status(lambda: layer.accumulate(lw, x[:64], 64)) == L.TS3_ERR_INVALID_ARG   # overlap
        assert status(lambda: layer.accumulate(lw2, x[:64], 128)) == L.TS3_ERR_INVALID_ARG  # other W2
        assert status(lambda: layer.accumulate(lw, x[:40], 192)) == L.TS3_OK              # ragged last
        assert status(lambda: layer.accumulate(lw, x[:64], 256)) == L.TS3_ERR_INVALID_ARG  # past the ragged end
        assert status(lambda: layer.accumulate(lw, x[:64], 128)) == L.TS3_OK              # before it: fine
        layer.finalize(lw)
        assert status(lambda: layer.accumulate(lw, x[:64], 128)) == L.TS3_ERR_BAD_STATE
        layer.attention(lw)
        assert status(lambda: layer.deslice(lw2, x)) == L.TS3_ERR_INVALID_ARG
        assert status(lambda: layer.deslice(lw, x)) == L.TS3_OK
        torch.cuda.synchronize()
    from paper_2602_04940_amd import PhysicsAttention
    with pytest.raises(L.TS3Error) as e:
        PhysicsAttention(C, H, M, C // H, 0.5, "fp32", group_span=32, max_points=10 ** 9)  # ~0.5 TB
    assert e.value.status == L.TS3_ERR_OUT_OF_MEMORY


def test_projected_state_reports_its_sums():
    """bfloat16 storage, C = 128, head width 16, M a multiple of 32: pass 1
    sums projected rows and the state exposes t_raw, not s_raw; float32
    storage and wider heads keep the unprojected sums."""
    from paper_2602_04940_amd import _lib as L
    banner("projected-state buffers")
    for (C, H, M, dtype, proj) in [(128, 8, 64, "bf16", True), (128, 8, 32, "bf16", True),
                                   (128, 8, 64, "fp32", False), (128, 2, 64, "bf16", False),
                                   (128, 8, 16, "bf16", False), (64, 4, 32, "bf16", False)]:
        with _layer(C, H, M, dtype, Q=128, max_points=256) as layer:
            assert layer.projected() == proj, (C, H, M, dtype)
            hidden = L.TS3_S_RAW if proj else L.TS3_T_RAW
            try:
                layer.get(hidden)
                raise AssertionError("no error")
            except L.TS3Error as e:
                assert e.status == L.TS3_ERR_UNSUPPORTED, (C, H, M, dtype, e.status)


@pytest.mark.parametrize("dtype,eps", [("fp32", 0.0), ("fp32", 0.5), ("bf16", 0.0), ("bf16", 0.5)])
def test_empty_slices_and_eps(dtype, eps):
    """One-hot slice weights (1/tau = 20000, every point's top two logits at
    least 0.05 apart in every head, so the other weights underflow to zero in
    float32 and float64 alike), and every fourth slice's bias lowered by 5 so
    that no point reaches it: those slices have d = 0 and s = b1 exactly
    (reading 7); eps > 0 divides by d + eps.  bf16 at C = 128 with head width
    16 runs the projected pass 1; both passes take the shifted softmax (the
    exp2 sums overflow)."""
    C, H, M, N = 128, 8, 64, 1500
    banner(f"empty slices, eps={eps}, {dtype}")
    rng = np.random.default_rng(61)
    from ts3_synth import round_storage
    W = make_weights(C, H, M, C // H, seed=21, bias_seed=22)
    b2 = W["b2"].copy().reshape(H, M)
    b2[:, ::4] -= 5.0
    W["b2"] = b2.reshape(-1)
    cand = round_storage(rng.standard_normal((8 * N, C)), dtype)
    lg = np.sort((cand @ W["W2"].astype(np.float64) + W["b2"]).reshape(-1, H, M), axis=2)
    x = cand[((lg[:, :, -1] - lg[:, :, -2]) > 0.05).all(axis=1)][:N]
    assert len(x) == N
    it = 20000.0
    got, st, _ = _run(x, W, C, H, M, dtype, 1.0 / it, 512, 700, 256, eps=eps)
    ref_st = match_sums(st, oracle.build_state(x, W, H, M, it, eps=eps), x, W, H, M, it)
    ref = oracle.layer_forward_fast(x, W, H, M, it, eps=eps)
    empty = ref_st["d"] == 0
    print(f"{int(empty.sum())} of {H * M} slices empty", flush=True)
    assert empty.sum() >= 8 and (~empty).sum() >= 8
    assert (st["d"][empty] == 0).all()
    b1 = W["b1"].astype(np.float32).reshape(H, 1, C // H)
    assert np.array_equal(st["s"][empty], np.broadcast_to(b1, st["s"].shape)[empty])
    if dtype == "fp32":
        for k in (sums_key(st), "d", "s", "Z"):
            assert normwise(st[k], ref_st[k]) <= FP32_TOL, k
        assert normwise(got, ref) <= FP32_TOL
    else:
        assert_state_close(st, ref_st, "state", BF16_TOL)
        assert_bf16_close(st["s"].reshape(H * M, -1), ref_st["s"].reshape(H * M, -1), "state s", BF16_TOL, block=M)
        assert_bf16_close(got, ref, "out", BF16_TOL)
