"""GPU parity of the layer backward (float32 storage) against the float64
backward oracle, through the C ABI.

Bar: float32 storage -> normwise max relative error <= 1e-4 for dx and for
every weight gradient; the gradients of tiled and untiled runs must agree
bitwise (span partials are folded in index order).
"""
import numpy as np
import pytest

from gpu_helpers import banner, normwise, to_device, to_host
from oracle import backward as BW
from ts3_synth import make_weights

pytestmark = pytest.mark.gpu

TOL = 1e-4
NAMES = ("dW2", "db2", "dW1", "db1", "dWq", "dWk", "dWv", "dW3", "db3")


def _torch():
    import torch
    return torch


def _layer(C, H, M, Q, N, accum="fp32"):
    from paper_2602_04940_amd import PhysicsAttention
    return PhysicsAttention(C, H, M, C // H, 0.5, "fp32", group_span=Q, max_points=N, accum=accum)


def _weights(W):
    from paper_2602_04940_amd import LayerWeights
    return LayerWeights(W)


def _gpu_backward(x64, g64, W, C, H, M, Q, tile, accum="fp32"):
    torch = _torch()
    N = len(x64)
    x, g, lw = to_device(x64, "fp32"), to_device(g64, "fp32"), _weights(W)
    with _layer(C, H, M, Q, N, accum) as layer:
        layer.forward(lw, x, tile=tile, chunk=tile)
        dx, grads = layer.backward(lw, x, g, tile=tile)
        torch.cuda.synchronize()
        return to_host(dx), {k: v.cpu().numpy().astype(np.float64) for k, v in grads.items()}


SHAPES = [(64, 4, 16), (64, 4, 32), (128, 8, 64)]


@pytest.mark.parametrize("C,H,M", SHAPES)
def test_backward_matches_oracle_ragged_tiles_random_biases(C, H, M):
    N, Q, tile = 2500, 256, 1024
    banner(f"backward fp32 C={C} H={H} M={M} N={N}")
    rng = np.random.default_rng(C + M)
    x64 = rng.standard_normal((N, C)).astype(np.float32).astype(np.float64)
    g64 = rng.standard_normal((N, C)).astype(np.float32).astype(np.float64)
    W = make_weights(C, H, M, C // H, seed=3, bias_seed=4)
    dx, grads = _gpu_backward(x64, g64, W, C, H, M, Q, tile)
    ref = BW.layer_backward(x64, {k: np.asarray(v, np.float64) for k, v in W.items()}, g64, H, M, 2.0)
    err = normwise(dx, ref["dx"])
    print(f"dx normwise {err:.2e}", flush=True)
    assert err <= TOL
    for k in NAMES:
        e = normwise(grads[k], ref[k])
        print(f"{k} normwise {e:.2e}", flush=True)
        assert e <= TOL, k


def test_backward_is_tiling_independent_and_deterministic():
    C, H, M, N, Q = 128, 8, 64, 3000, 128
    banner("backward tiling independence fp32 C=128 M=64")
    rng = np.random.default_rng(11)
    x64 = rng.standard_normal((N, C)).astype(np.float32).astype(np.float64)
    g64 = rng.standard_normal((N, C)).astype(np.float32).astype(np.float64)
    W = make_weights(C, H, M, C // H, seed=5, bias_seed=6)
    dx_a, ga = _gpu_backward(x64, g64, W, C, H, M, Q, 1024)
    dx_b, gb = _gpu_backward(x64, g64, W, C, H, M, Q, 384)
    dx_c, gc = _gpu_backward(x64, g64, W, C, H, M, Q, 1024)
    assert np.array_equal(dx_a, dx_b) and np.array_equal(dx_a, dx_c)
    for k in NAMES:
        assert np.array_equal(ga[k], gb[k]) and np.array_equal(ga[k], gc[k]), k


def test_backward_with_the_float64_fold_matches_oracle_and_is_tiling_independent():
    C, H, M, N, Q = 128, 8, 64, 3000, 128
    banner("backward with the float64 fold of span partials")
    rng = np.random.default_rng(13)
    x64 = rng.standard_normal((N, C)).astype(np.float32).astype(np.float64)
    g64 = rng.standard_normal((N, C)).astype(np.float32).astype(np.float64)
    W = make_weights(C, H, M, C // H, seed=7, bias_seed=8)
    dx_a, ga = _gpu_backward(x64, g64, W, C, H, M, Q, 1024, accum="fp64")
    dx_b, gb = _gpu_backward(x64, g64, W, C, H, M, Q, 384, accum="fp64")
    assert np.array_equal(dx_a, dx_b)
    for k in NAMES:
        assert np.array_equal(ga[k], gb[k]), k
    ref = BW.layer_backward(x64, {k: np.asarray(v, np.float64) for k, v in W.items()}, g64, H, M, 2.0)
    assert normwise(dx_a, ref["dx"]) <= TOL
    for k in NAMES:
        assert normwise(ga[k], ref[k]) <= TOL, k
