"""Pins for the float64 backward oracle (oracle/backward.py).

The backward is pinned against the forward it differentiates, never against
itself: every gradient (of x and of each weight and bias) is compared entry
by entry with central finite differences of the float64 forward on small
problems; the tiled backward must equal the untiled one; and invariants that
hold for any input are checked (a head's logit gradients sum to zero over its
slices, because the softmax ignores a common shift; b3's gradient is the
column sum of the output gradient; with 1/tau = 0 the slice weights ignore
the logits).  Plausible mistakes planted in the oracle must fail the pins.
"""
import numpy as np
import pytest

from oracle import backward as BW
from oracle import physics_attention as PA
from ts3_synth import make_weights

PARAMS = ("W2", "b2", "W1", "b1", "Wq", "Wk", "Wv", "W3", "b3")


def _problem(N=40, C=8, H=2, M=4, seed=0):
    rng = np.random.default_rng(100 + seed)
    x = rng.standard_normal((N, C))
    W = {k: np.asarray(v, np.float64) for k, v in make_weights(C, H, M, C // H, seed=seed, bias_seed=seed + 7).items()}
    g = rng.standard_normal((N, C))
    return x, W, g, H, M


def _loss(x, W, g, H, M, inv_tau):
    return float((PA.layer_forward_fast(x, W, H, M, inv_tau) * g).sum())


def _central_differences(x, W, g, H, M, inv_tau, step=1e-5):
    """d loss / d every entry of x and of each weight, by central differences."""
    out = {}
    targets = [("dx", x)] + [("d" + k, W[k]) for k in PARAMS]
    for name, arr in targets:
        grad = np.zeros_like(arr)
        flat, gflat = arr.reshape(-1), grad.reshape(-1)
        for i in range(flat.size):
            keep = flat[i]
            flat[i] = keep + step
            up = _loss(x, W, g, H, M, inv_tau)
            flat[i] = keep - step
            down = _loss(x, W, g, H, M, inv_tau)
            flat[i] = keep
            gflat[i] = (up - down) / (2 * step)
        out[name] = grad
    return out


def _matches_fd(grads, fd, tol=2e-6):
    return all(np.allclose(grads[k], fd[k], rtol=tol, atol=tol) for k in fd)


_FD_CACHE = {}


def _fd_case(seed, inv_tau):
    key = (seed, inv_tau)
    if key not in _FD_CACHE:
        x, W, g, H, M = _problem(seed=seed)
        _FD_CACHE[key] = (x, W, g, H, M, _central_differences(x, W, g, H, M, inv_tau))
    return _FD_CACHE[key]


@pytest.mark.parametrize("seed,inv_tau", [(0, 2.0), (1, 0.7)])
def test_every_gradient_matches_central_differences(seed, inv_tau):
    x, W, g, H, M, fd = _fd_case(seed, inv_tau)
    grads = BW.layer_backward(x, W, g, H, M, inv_tau)
    for k in fd:
        np.testing.assert_allclose(grads[k], fd[k], rtol=2e-6, atol=2e-6, err_msg=k)


@pytest.mark.parametrize("tile", [7, 13, 40])
def test_tiled_backward_equals_untiled(tile):
    x, W, g, H, M = _problem(N=40, seed=2)
    ref = BW.layer_backward(x, W, g, H, M, 2.0)
    got = BW.layer_backward(x, W, g, H, M, 2.0, tile=tile)
    for k in ("dx",) + tuple("d" + p for p in PARAMS):
        np.testing.assert_allclose(got[k], ref[k], rtol=1e-12, atol=1e-13, err_msg=k)


def test_logit_gradients_sum_to_zero_over_each_head_and_b3_is_column_sum():
    x, W, g, H, M = _problem(N=64, C=16, H=4, M=8, seed=3)
    grads = BW.layer_backward(x, W, g, H, M, 2.0)
    db2 = grads["db2"].reshape(H, M)
    assert np.abs(db2.sum(axis=1)).max() <= 1e-12 * np.abs(db2).max()
    dW2 = grads["dW2"].reshape(-1, H, M)
    assert np.abs(dW2.sum(axis=2)).max() <= 1e-12 * np.abs(dW2).max()
    np.testing.assert_allclose(grads["db3"], g.sum(axis=0), rtol=0, atol=1e-13)


def test_zero_inverse_temperature_leaves_linear2_without_gradient():
    x, W, g, H, M = _problem(N=24, seed=4)
    grads = BW.layer_backward(x, W, g, H, M, 0.0)
    assert np.abs(grads["dW2"]).max() == 0.0 and np.abs(grads["db2"]).max() == 0.0
    assert np.abs(grads["dW1"]).max() > 0.0


def _mutants():
    """Plausible backward mistakes; each must make some gradient disagree with
    the central differences."""
    orig_tok, orig_dx = BW.token_backward, BW.dx_tile

    def tok_no_dd(state, dZ, W, H, eps=0.0):
        ds_raw, dd, out = orig_tok(state, dZ, W, H, eps)
        return ds_raw, np.zeros_like(dd), out

    def tok_dd_sign(state, dZ, W, H, eps=0.0):
        ds_raw, dd, out = orig_tok(state, dZ, W, H, eps)
        return ds_raw, -dd, out

    def tok_attn_transposed(state, dZ, W, H, eps=0.0):
        W2 = dict(W)
        W2["Wq"], W2["Wk"] = W["Wk"], W["Wq"]
        return orig_tok(state, dZ, W2, H, eps)

    def dx_no_slice_path(x_tile, g_tile, W2, b2, Z, ds_raw, dd, H, M, inv_tau):
        dx, dw2, db2 = orig_dx(x_tile, g_tile, W2, b2, Z, ds_raw, dd, H, M, inv_tau)
        w = PA.slice_weights(x_tile, W2, b2, H, M, inv_tau)
        return dx - np.einsum("nhm,hmc->nc", w, ds_raw), dw2, db2

    def dx_no_softmax_centering(x_tile, g_tile, W2, b2, Z, ds_raw, dd, H, M, inv_tau):
        x_tile = np.asarray(x_tile, float)
        N = len(x_tile)
        w = PA.slice_weights(x_tile, W2, b2, H, M, inv_tau)
        dw = np.einsum("nc,hmc->nhm", g_tile, Z) + np.einsum("nc,hmc->nhm", x_tile, ds_raw) + dd[None]
        dz = (inv_tau * w * dw).reshape(N, H * M)
        return dz @ np.asarray(W2, float).T + np.einsum("nhm,hmc->nc", w, ds_raw), x_tile.T @ dz, dz.sum(axis=0)

    return {"dd dropped": ("token_backward", tok_no_dd), "dd sign": ("token_backward", tok_dd_sign),
            "q and k swapped": ("token_backward", tok_attn_transposed),
            "slice path of dx dropped": ("dx_tile", dx_no_slice_path),
            "softmax backward not centred": ("dx_tile", dx_no_softmax_centering)}


@pytest.mark.parametrize("name", sorted(_mutants()))
def test_planted_backward_mistakes_are_caught(name, monkeypatch):
    fn_name, fn = _mutants()[name]
    monkeypatch.setattr(BW, fn_name, fn)
    x, W, g, H, M, fd = _fd_case(0, 2.0)
    assert not _matches_fd(BW.layer_backward(x, W, g, H, M, 2.0), fd), f"'{name}' passed the pins"
