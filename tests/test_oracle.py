"""Pins for the float64 oracle (CPU only).

Each check ties the oracle to something other than itself: a hand-worked
example, brute-force loops, closed forms, invariants the paper's equations
imply, or a library attention routine.  ``test_planted_mistakes_are_caught``
plants plausible mistakes in the oracle and requires every one to fail a pin.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import oracle.physics_attention as PA
from oracle.brute import layer_forward_loops, slice_tokens_loops
from ts3_synth import WORKLOADS, make_weights
from ts3_synth.workloads import small_features

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_case(N=24, C=8, H=2, M=3, seed=7, bias=True, scale=1.0):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((N, C)) * scale
    W = make_weights(C, H, M, C // H, seed=seed + 1, bias_seed=seed + 2 if bias else None)
    return x, W


# ------------------------------------------------------------ golden fixture

def _num(v):
    if isinstance(v, str):
        v = v.replace("ln3", repr(math.log(3.0)))
        if "*" in v:
            a, b = v.split("*")
            return float(Fraction(a)) * float(b)
        return float(Fraction(v)) if "/" in v or v.strip("-").isdigit() else float(v)
    return float(v)


def _arr(a):
    if isinstance(a, list):
        return np.array([_arr(v) for v in a])
    return _num(a)


def load_golden():
    with open(os.path.join(GOLDEN, "two_point_two_head.json")) as f:
        g = json.load(f)
    W = {k: np.asarray(_arr(g[k]), dtype=np.float32) for k in
         ("W2", "b2", "W1", "b1", "Wq", "Wk", "Wv", "W3", "b3")}
    return g, np.array(g["x"]), W


def check_golden():
    g, x, W = load_golden()
    H, M, it = g["H"], g["M"], g["inv_tau"]
    st = oracle.build_state(x, W, H, M, it)
    e = g["expect"]
    for key in ("d", "s_raw", "s", "s1", "Z"):
        np.testing.assert_allclose(st[key], _arr(e[key]), rtol=1e-6, atol=1e-7, err_msg=key)
    for out in (oracle.layer_forward_fast(x, W, H, M, it), oracle.layer_forward_orig(x, W, H, M, it)):
        np.testing.assert_allclose(out, _arr(e["out"]), rtol=1e-6, atol=1e-7)


def test_golden_two_point_two_head():
    check_golden()


# --------------------------------------------------------- brute-force loops

def check_brute():
    for (N, C, H, M, seed) in [(9, 4, 1, 3, 1), (16, 8, 2, 3, 2), (11, 6, 3, 2, 3)]:
        x, W = _rand_case(N, C, H, M, seed)
        ref = np.array(layer_forward_loops(x, W, H, M, 1.7))
        np.testing.assert_allclose(oracle.layer_forward_orig(x, W, H, M, 1.7), ref, rtol=0, atol=1e-12)
        np.testing.assert_allclose(oracle.layer_forward_fast(x, W, H, M, 1.7, tile=4, chunk=5), ref,
                                   rtol=0, atol=1e-12)


def test_brute_force_loops_match():
    check_brute()


# ------------------------------------- projected sums (Linear1 before the sum)

def check_projected():
    """State from sums taken after Linear1: the hand-worked s of the fixture,
    the loop form's slice tokens, and the closed form sum_m t[h, m] =
    (sum_i x_i) W1_h (each point's weights sum to one per head)."""
    g, x, W = load_golden()
    H, M, it = g["H"], g["M"], g["inv_tau"]
    t, d = oracle.projected_accumulate(x, W["W2"], W["b2"], W["W1"], H, M, it)
    np.testing.assert_allclose(oracle.projected_finalize(t, d, W["b1"], H), _arr(g["expect"]["s"]),
                               rtol=1e-6, atol=1e-7)
    for (N, C, H, M, seed) in [(9, 4, 1, 3, 1), (16, 8, 2, 3, 2), (11, 6, 3, 2, 3)]:
        x, W = _rand_case(N, C, H, M, seed)
        _, s_ref = slice_tokens_loops(x, W, H, M, 1.7)
        t, d = oracle.projected_accumulate(x, W["W2"], W["b2"], W["W1"], H, M, 1.7)
        np.testing.assert_allclose(oracle.projected_finalize(t, d, W["b1"], H), np.array(s_ref), rtol=0, atol=1e-12)
        dh = C // H
        col = x.sum(axis=0) @ W["W1"].astype(np.float64)
        for h in range(H):
            np.testing.assert_allclose(t[h].sum(axis=0), col[h * dh:(h + 1) * dh], rtol=0, atol=1e-12)


def test_projected_sums_give_the_same_state():
    check_projected()


def test_projected_sums_are_additive_and_empty_slices_give_b1():
    x, W = _rand_case(N=500, C=16, H=4, M=6, seed=13)
    t, d = oracle.projected_accumulate(x, W["W2"], W["b2"], W["W1"], 4, 6, 2.0)
    parts = [oracle.projected_accumulate(x[i:i + 77], W["W2"], W["b2"], W["W1"], 4, 6, 2.0)
             for i in range(0, 500, 77)]
    np.testing.assert_allclose(sum(p[0] for p in parts), t, rtol=1e-13, atol=1e-13 * np.abs(t).max())
    np.testing.assert_allclose(sum(p[1] for p in parts), d, rtol=1e-13)
    s = oracle.projected_finalize(np.zeros_like(t), np.zeros_like(d), W["b1"], 4)
    np.testing.assert_array_equal(s, np.broadcast_to(W["b1"].astype(np.float64).reshape(4, 1, 4), s.shape))


def test_projected_state_equals_raw_state_with_eps_and_empty_slices():
    """Reading 1's order with eps > 0 and with slices that no point reaches:
    the projected state t / (d + eps) + b1 equals Linear1((d + eps)^-1 s_raw)
    + b1, and an empty slice (d + eps = 0) gives b1 in both."""
    x, W = _rand_case(N=200, C=12, H=3, M=5, seed=17)
    s_raw, d = oracle.slice_accumulate(x, W["W2"], W["b2"], 3, 5, 1.3)
    t, d2 = oracle.projected_accumulate(x, W["W2"], W["b2"], W["W1"], 3, 5, 1.3)
    np.testing.assert_array_equal(d, d2)
    for eps in (0.0, 0.25, 7.0):
        np.testing.assert_allclose(oracle.projected_finalize(t, d, W["b1"], 3, eps),
                                   oracle.slice_finalize(s_raw, d, W["W1"], W["b1"], 3, eps), rtol=0, atol=1e-12)
    empty = np.zeros_like(d, dtype=bool)
    empty[0, 1] = empty[2, 4] = True
    s_raw[empty] = 0
    t[empty] = 0
    d = np.where(empty, 0.0, d)
    sp = oracle.projected_finalize(t, d, W["b1"], 3)
    sr = oracle.slice_finalize(s_raw, d, W["W1"], W["b1"], 3)
    np.testing.assert_allclose(sp, sr, rtol=0, atol=1e-12)
    b1 = W["b1"].astype(np.float64).reshape(3, 4)
    np.testing.assert_array_equal(sp[0, 1], b1[0])
    np.testing.assert_array_equal(sp[2, 4], b1[2])


# ------------------------------------------------------ invariants of Eq. (1)

def test_softmax_rows_sum_to_one_and_d_sums_to_N():
    x, W = _rand_case(N=300, C=16, H=4, M=8)
    w = oracle.slice_weights(x, W["W2"], W["b2"], 4, 8, 2.0)
    assert np.abs(w.sum(axis=2) - 1).max() <= 1e-15 * 8
    assert (w > 0).all()
    _, d = oracle.slice_accumulate(x, W["W2"], W["b2"], 4, 8, 2.0)
    np.testing.assert_allclose(d.sum(axis=1), 300, rtol=1e-14)


def test_slice_sum_over_m_is_column_sum_of_x():
    # sum_m s_raw[h, m, :] = sum_i x_i for every head (rows of w sum to one)
    x, W = _rand_case(N=200, C=12, H=3, M=5)
    s_raw, _ = oracle.slice_accumulate(x, W["W2"], W["b2"], 3, 5, 1.3)
    for h in range(3):
        np.testing.assert_allclose(s_raw[h].sum(axis=0), x.sum(axis=0), rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------- closed forms

def _mean_pool_closed_form(x, W, H):
    """M = 1 (or 1/tau = 0): every token of head h is s_h = mean(x) W1^h + b1^h,
    attention over identical tokens returns s_h Wv_h, so every point outputs
    sum_h (s_h Wv_h) W3^h + b3."""
    N, C = x.shape
    dh = C // H
    mu = x.mean(axis=0)
    W1, b1, W3 = W["W1"].astype(float), W["b1"].astype(float), W["W3"].astype(float)
    y = W["b3"].astype(float).copy()
    for h in range(H):
        sh = mu @ W1[:, h * dh:(h + 1) * dh] + b1[h * dh:(h + 1) * dh]
        y += (sh @ W["Wv"][h].astype(float)) @ W3[h * dh:(h + 1) * dh]
    return np.broadcast_to(y, (N, C))


def check_closed_forms():
    x, W = _rand_case(N=50, C=8, H=2, M=1, seed=11)
    ref = _mean_pool_closed_form(x, W, 2)
    np.testing.assert_allclose(oracle.layer_forward_fast(x, W, 2, 1, 1.0), ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(oracle.layer_forward_orig(x, W, 2, 1, 1.0), ref, rtol=0, atol=1e-12)
    x, W = _rand_case(N=50, C=8, H=2, M=6, seed=12)
    ref = _mean_pool_closed_form(x, W, 2)
    np.testing.assert_allclose(oracle.layer_forward_fast(x, W, 2, 6, 0.0, tile=7), ref, rtol=0,
                               atol=1e-12)


def test_M1_and_zero_inverse_temperature_reduce_to_mean_pool():
    check_closed_forms()


def check_one_hot():
    """With well-separated logits each point falls in one slice, and the slice
    state d^-1 s_raw is the plain mean of x over that slice's points."""
    rng = np.random.default_rng(3)
    N, C, H, M = 400, 6, 2, 4
    x = rng.standard_normal((N, C))
    W = make_weights(C, H, M, C // H, seed=4)
    # Slice logits from a random projection; a large 1/tau makes the softmax one-hot.
    logits = (x @ W["W2"].astype(float) + W["b2"]).reshape(N, H, M)
    inv_tau = 200.0
    lab = logits.argmax(axis=2)
    srt = np.sort(logits, axis=2)
    margin = (srt[:, :, -1] - srt[:, :, -2]).min()
    keep = (srt[:, :, -1] - srt[:, :, -2] > 0.2).all(axis=1)
    x, lab = x[keep], lab[keep]
    s_raw, d = oracle.slice_accumulate(x, W["W2"], W["b2"], H, M, inv_tau)
    for h in range(H):
        cnt = np.bincount(lab[:, h], minlength=M)
        for c in range(C):
            seg = np.bincount(lab[:, h], weights=x[:, c], minlength=M)
            np.testing.assert_allclose(s_raw[h, :, c] / d[h], seg / cnt, rtol=0, atol=1e-12)
        np.testing.assert_allclose(d[h], cnt, rtol=0, atol=1e-12)
    assert margin >= 0


def test_one_hot_slices_give_segment_means():
    check_one_hot()


# ------------------------------------------------ equivalences the paper claims

def check_orig_equals_fast():
    x, W = _rand_case(N=257, C=16, H=4, M=5, seed=21, bias=True)
    a = oracle.layer_forward_orig(x, W, 4, 5, 2.0)
    b = oracle.layer_forward_fast(x, W, 4, 5, 2.0)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12 * np.abs(a).max())


def test_project_then_slice_equals_slice_then_project():
    check_orig_equals_fast()


@pytest.mark.parametrize("tile", [1000, 500, 143, 64, 37])
def test_tiled_equals_untiled(tile):
    x, W = _rand_case(N=1000, C=16, H=2, M=8, seed=5)
    a = oracle.build_state(x, W, 2, 8, 2.0)
    b = oracle.build_state(x, W, 2, 8, 2.0, tile=tile)
    for k in ("s_raw", "d", "Z"):
        np.testing.assert_allclose(b[k], a[k], rtol=1e-13, atol=1e-13 * np.abs(a[k]).max())


def test_pass2_chunk_independence():
    x, W = _rand_case(N=300, C=8, H=2, M=4, seed=8)
    st = oracle.build_state(x, W, 2, 4, 2.0)
    full = oracle.deslice(x, W["W2"], W["b2"], st["Z"], W["b3"], 2, 4, 2.0)
    idx = np.random.default_rng(0).choice(300, 40, replace=False)
    part = oracle.deslice(x[idx], W["W2"], W["b2"], st["Z"], W["b3"], 2, 4, 2.0)
    np.testing.assert_array_equal(part, full[idx])


def test_permutation_equivariance_and_duplication_invariance():
    x, W = _rand_case(N=120, C=8, H=2, M=4, seed=9)
    out = oracle.layer_forward_fast(x, W, 2, 4, 2.0)
    Z = oracle.build_state(x, W, 2, 4, 2.0)["Z"]
    perm = np.random.default_rng(1).permutation(120)
    np.testing.assert_allclose(oracle.layer_forward_fast(x[perm], W, 2, 4, 2.0), out[perm],
                               rtol=1e-12, atol=1e-12)
    xx = np.concatenate([x, x])
    np.testing.assert_allclose(oracle.build_state(xx, W, 2, 4, 2.0)["Z"], Z, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.layer_forward_fast(xx, W, 2, 4, 2.0), np.concatenate([out, out]),
                               rtol=1e-12, atol=1e-12)


# ------------------------------------------------------ library attention

def check_attention_library():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(2)
    H, M, dh = 3, 7, 5
    s = rng.standard_normal((H, M, dh))
    Wq, Wk, Wv = (rng.standard_normal((H, dh, dh)) for _ in range(3))
    ours = oracle.token_attention(s, Wq, Wk, Wv)
    st = torch.from_numpy(s)
    q = torch.einsum("hmd,hde->hme", st, torch.from_numpy(Wq))
    k = torch.einsum("hmd,hde->hme", st, torch.from_numpy(Wk))
    v = torch.einsum("hmd,hde->hme", st, torch.from_numpy(Wv))
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v).numpy()
    np.testing.assert_allclose(ours, ref, rtol=1e-12, atol=1e-12)


def test_token_attention_matches_library_sdpa():
    check_attention_library()


# ------------------------------------------------------- workload inputs

def test_workload_inputs_are_deterministic_and_normalised():
    w = WORKLOADS["ellipsoid_4k_fp32"]
    a = small_features(w, 4096)
    b = small_features(w, 4096)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_allclose(a.mean(axis=1), 0, atol=1e-6)
    np.testing.assert_allclose(a.std(axis=1), 1, atol=1e-3)
    assert np.array_equal(a[:1000], small_features(w, 1000))  # prefix-stable sampler


# ------------------------------------------------------- planted mistakes

def _mutants():
    """Plausible oracle mistakes; each must be caught by some pin."""
    orig = {n: getattr(PA, n) for n in ("slice_weights", "slice_finalize", "linear3_tokens",
                                          "token_attention", "deslice", "slice_accumulate",
                                          "projected_accumulate", "projected_finalize")}

    def sw_wrong_axis(x, W2, b2, H, M, inv_tau):
        lg = (np.asarray(x, float) @ W2.astype(float) + b2).reshape(len(x), H, M) * inv_tau
        e = np.exp(lg - lg.max(axis=1, keepdims=True))
        return e / e.sum(axis=1, keepdims=True)

    def sw_tau_mult(x, W2, b2, H, M, inv_tau):
        return orig["slice_weights"](x, W2, b2, H, M, 1.0 / inv_tau if inv_tau else 0.0)

    def sw_no_bias(x, W2, b2, H, M, inv_tau):
        return orig["slice_weights"](x, W2, np.zeros_like(b2), H, M, inv_tau)

    def fin_no_b1(s_raw, d, W1, b1, H, eps=0.0):
        return orig["slice_finalize"](s_raw, d, W1, np.zeros_like(b1), H, eps)

    def fin_norm_after(s_raw, d, W1, b1, H, eps=0.0):
        C = s_raw.shape[2]
        dh = C // H
        return np.stack([(s_raw[h] @ W1[:, h * dh:(h + 1) * dh].astype(float)
                          + b1[h * dh:(h + 1) * dh]) / d[h][:, None] for h in range(H)])

    def fin_rows_of_W1(s_raw, d, W1, b1, H, eps=0.0):
        return orig["slice_finalize"](s_raw, d, np.ascontiguousarray(W1.T).reshape(W1.shape), b1, H, eps)

    def l3_cols(s1, W3):
        H, M, dh = s1.shape
        W3t = np.ascontiguousarray(np.asarray(W3, float).T)
        C = W3t.shape[0]
        return np.stack([s1[h] @ W3t.reshape(-1, C)[h * dh:(h + 1) * dh] for h in range(H)])

    def att_no_scale(s, Wq, Wk, Wv):
        dh = s.shape[2]
        return orig["token_attention"](s * dh ** 0.25, Wq, Wk, Wv / dh ** 0.25)

    def att_transposed(s, Wq, Wk, Wv):
        out = np.empty_like(np.asarray(s, float))
        for h in range(s.shape[0]):
            q, k, v = s[h] @ Wq[h], s[h] @ Wk[h], s[h] @ Wv[h]
            a = q @ k.T / np.sqrt(s.shape[2])
            a = np.exp(a - a.max(axis=0, keepdims=True))
            a = a / a.sum(axis=0, keepdims=True)
            out[h] = a.T @ v
        return out

    def des_bias_per_head(x, W2, b2, Z, b3, H, M, inv_tau):
        return orig["deslice"](x, W2, b2, Z, np.asarray(b3) * H, H, M, inv_tau)

    def acc_unweighted_d(x_tile, W2, b2, H, M, inv_tau):
        s_raw, d = orig["slice_accumulate"](x_tile, W2, b2, H, M, inv_tau)
        return s_raw, np.full_like(d, len(x_tile) / M)

    def pacc_bias_in_sum(x_tile, W2, b2, W1, H, M, inv_tau):
        t, d = orig["projected_accumulate"](x_tile, W2, b2, W1, H, M, inv_tau)
        return t + 0.5 * d[:, :, None], d

    def pacc_head_block(x_tile, W2, b2, W1, H, M, inv_tau):
        C = W1.shape[1]
        perm = np.roll(np.arange(C), C // H)  # head h meets head h-1's columns
        return orig["projected_accumulate"](x_tile, W2, b2, np.asarray(W1)[:, perm], H, M, inv_tau)

    def pfin_no_b1(t_raw, d, b1, H, eps=0.0):
        return orig["projected_finalize"](t_raw, d, np.zeros_like(b1), H, eps)

    return {
        "projected sums carry a bias": ("projected_accumulate", pacc_bias_in_sum),
        "projected with another head's W1 block": ("projected_accumulate", pacc_head_block),
        "b1 dropped from projected state": ("projected_finalize", pfin_no_b1),
        "softmax over heads": ("slice_weights", sw_wrong_axis),
        "temperature multiplied": ("slice_weights", sw_tau_mult),
        "b2 dropped": ("slice_weights", sw_no_bias),
        "b1 dropped": ("slice_finalize", fin_no_b1),
        "normalise after Linear1": ("slice_finalize", fin_norm_after),
        "W1 blocks transposed": ("slice_finalize", fin_rows_of_W1),
        "W3 blocks from columns": ("linear3_tokens", l3_cols),
        "attention scale dropped": ("token_attention", att_no_scale),
        "attention transposed": ("token_attention", att_transposed),
        "b3 added per head": ("deslice", des_bias_per_head),
        "d not the weight sum": ("slice_accumulate", acc_unweighted_d),
    }


def _pins_pass():
    checks = [check_golden, check_brute, check_closed_forms, check_one_hot, check_orig_equals_fast,
              check_attention_library, check_projected]
    for c in checks:
        try:
            c()
        except AssertionError:
            return False
    return True


def test_pins_pass_unmutated():
    assert _pins_pass()


@pytest.mark.parametrize("name", sorted(_mutants()))
def test_planted_mistakes_are_caught(name, monkeypatch):
    fn_name, fn = _mutants()[name]
    monkeypatch.setattr(PA, fn_name, fn)
    monkeypatch.setattr(oracle, fn_name, fn, raising=False)
    assert not _pins_pass(), f"planted mistake '{name}' passed every pin"


def test_pool_driver_equals_the_in_process_oracle_bitwise():
    """oracle.pool only distributes tiles and chunks: its state and decoding
    equal build_state / deslice bit for bit (same tile order, same zero start)."""
    from oracle.pool import OraclePool
    rng = np.random.default_rng(31)
    C, H, M, N, tile = 32, 2, 16, 700, 96
    x = rng.standard_normal((N, C)).astype(np.float32).astype(np.float64)
    W = make_weights(C, H, M, C // H, seed=2, bias_seed=3)
    ref = oracle.build_state(x, W, H, M, 1.7, tile=tile)
    with OraclePool(2) as pool:
        st = pool.state(x, W, H, M, 1.7, tile=tile)
        out = pool.decode(x, W["W2"], W["b2"], st["Z"], W["b3"], H, M, 1.7, chunk=250)
    for k in ("s_raw", "d", "s", "s1", "Z"):
        assert np.array_equal(st[k], ref[k]), k
    assert np.array_equal(out, oracle.deslice(x, W["W2"], W["b2"], ref["Z"], W["b3"], H, M, 1.7))
