"""Pins for the Transolver-block oracle (oracle/block.py): LayerNorm, exact
GELU, the feed-forward network, the block's residual structure, and decoding
from cached per-block states."""
import math

import numpy as np
import pytest
import torch
from scipy.special import ndtr

from oracle import block as BK
from oracle import physics_attention as PA
from ts3_synth import make_block_weights


def _blocks(L=2, C=16, H=2, M=4, F=64, bias=True):
    return [{k: np.asarray(v, np.float64) for k, v in
             make_block_weights(C, H, M, C // H, F, seed=10 + l, bias_seed=(20 + l) if bias else None).items()}
            for l in range(L)]


def test_layer_norm_matches_torch_and_normalises():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((50, 24)) * 3 + 1.5
    g, b = rng.uniform(0.5, 1.5, 24), rng.uniform(-0.5, 0.5, 24)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (24,), torch.from_numpy(g), torch.from_numpy(b),
                                         eps=1e-5).numpy()
    np.testing.assert_allclose(BK.layer_norm(x, g, b), ref, rtol=1e-12, atol=1e-12)
    z = BK.layer_norm(x, np.ones(24), np.zeros(24))
    np.testing.assert_allclose(z.mean(axis=1), 0, atol=1e-12)
    np.testing.assert_allclose((z ** 2).mean(axis=1), 1 - 1e-5 / (x.var(axis=1) + 1e-5), rtol=1e-12)


def test_gelu_is_x_times_the_normal_cdf():
    x = np.linspace(-8, 8, 1601)
    np.testing.assert_allclose(BK.gelu(x), x * ndtr(x), rtol=1e-13, atol=1e-15)
    # odd part: GELU(x) - GELU(-x) = x; the standard normal CDF at 1 is 0.8413447460685429
    np.testing.assert_allclose(BK.gelu(x) - BK.gelu(-x), x, atol=1e-14)
    assert abs(BK.gelu(1.0) - 0.8413447460685429) < 1e-15
    assert BK.gelu(0.0) == 0.0


def test_mlp_matches_loops():
    rng = np.random.default_rng(1)
    N, C, F = 3, 4, 6
    x, Wa, ba = rng.standard_normal((N, C)), rng.standard_normal((C, F)), rng.standard_normal(F)
    Wb, bb = rng.standard_normal((F, C)), rng.standard_normal(C)
    out = np.zeros((N, C))
    for i in range(N):
        h = [0.0] * F
        for f in range(F):
            a = ba[f] + sum(x[i, c] * Wa[c, f] for c in range(C))
            h[f] = 0.5 * a * (1 + math.erf(a / math.sqrt(2)))
        for c in range(C):
            out[i, c] = bb[c] + sum(h[f] * Wb[f, c] for f in range(F))
    np.testing.assert_allclose(BK.mlp(x, Wa, ba, Wb, bb), out, rtol=1e-12)


def test_zero_output_weights_make_the_block_the_identity():
    B = _blocks(1)[0]
    for k in ("W3", "b3", "Wb", "bb"):
        B[k] = np.zeros_like(B[k])
    x = np.random.default_rng(2).standard_normal((40, 16))
    np.testing.assert_array_equal(BK.block_forward(x, B, 2, 4, 2.0), x)


def test_block_is_permutation_equivariant_and_tiling_independent():
    B = _blocks(1)[0]
    rng = np.random.default_rng(3)
    x = rng.standard_normal((60, 16))
    perm = rng.permutation(60)
    y = BK.block_forward(x, B, 2, 4, 2.0)
    np.testing.assert_allclose(BK.block_forward(x[perm], B, 2, 4, 2.0), y[perm], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(BK.block_forward(x, B, 2, 4, 2.0, tile=7), y, rtol=1e-11, atol=1e-12)


def test_attention_part_of_the_block_is_the_layer():
    B = _blocks(1)[0]
    B["Wb"], B["bb"] = np.zeros_like(B["Wb"]), np.zeros_like(B["bb"])
    x = np.random.default_rng(4).standard_normal((30, 16))
    xn = BK.layer_norm(x, B["ln1_g"], B["ln1_b"])
    np.testing.assert_allclose(BK.block_forward(x, B, 2, 4, 2.0) - x, PA.layer_forward_orig(xn, B, 2, 4, 2.0),
                               rtol=1e-10, atol=1e-12)


def test_decoding_from_cached_states_reproduces_the_forward():
    blocks = _blocks(3)
    x = np.random.default_rng(5).standard_normal((50, 16))
    Zs = BK.stack_states(x, blocks, 2, 4, 2.0)
    np.testing.assert_allclose(BK.stack_decode(x, blocks, Zs, 2, 4, 2.0), BK.stack_forward(x, blocks, 2, 4, 2.0),
                               rtol=1e-11, atol=1e-12)


def _mutants():
    orig_ln, orig_gelu, orig_mlp = BK.layer_norm, BK.gelu, BK.mlp

    def ln_unbiased(x, gamma, beta, eps=BK.LN_EPS):
        x = np.asarray(x, float)
        return (x - x.mean(-1, keepdims=True)) / np.sqrt(x.var(-1, ddof=1, keepdims=True) + eps) * gamma + beta

    def gelu_tanh(x):
        x = np.asarray(x, float)
        return 0.5 * x * (1 + np.tanh(math.sqrt(2 / math.pi) * (x + 0.044715 * x ** 3)))

    def mlp_no_hidden_bias(x, Wa, ba, Wb, bb):
        return orig_mlp(x, Wa, np.zeros_like(ba), Wb, bb)

    def ln_no_beta(x, gamma, beta, eps=BK.LN_EPS):
        return orig_ln(x, gamma, np.zeros_like(beta), eps)

    return {"unbiased variance": ("layer_norm", ln_unbiased), "tanh GELU": ("gelu", gelu_tanh),
            "hidden bias dropped": ("mlp", mlp_no_hidden_bias), "LayerNorm beta dropped": ("layer_norm", ln_no_beta)}


@pytest.mark.parametrize("name", sorted(_mutants()))
def test_planted_block_mistakes_are_caught(name, monkeypatch):
    fn_name, fn = _mutants()[name]
    monkeypatch.setattr(BK, fn_name, fn)
    caught = False
    try:
        test_layer_norm_matches_torch_and_normalises()
        test_gelu_is_x_times_the_normal_cdf()
        test_mlp_matches_loops()
    except AssertionError:
        caught = True
    assert caught, f"'{name}' passed the pins"
