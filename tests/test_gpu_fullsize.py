"""Parity at the benchmark's full size: the 100M-point volume mesh, C=128, H=8,
M=64, bf16, in the launch configuration bench.py times (1M-point tiles and
decode chunks, group span 15,625, tiles alternating over two streams).

The float64 oracle cannot redo pass 1 over 1e8 points in test time.  Pass 1 is
checked on outputs the oracle can compute one at a time, and through properties
that hold at any size:
  * the span partials of 16 seeded spans (15,625 points each, anywhere in the
    mesh) against the oracle's sums over the same points (Eq. (4)'s per-span
    terms), per slice token and per element of d;
  * the state equals the index-ordered sum of all 6,400 span partials, within
    the rounding bound of float32 addition in runs of 64 and then 100 (the
    fold of Eq. (4));
  * sum_m d[h, m] = N and sum_m s_raw[h, m, :] = sum_i x_i for every head
    (for a state of projected sums, sum_m t_raw[h, m, :] = (sum_i x_i) W1_h);
  * reruns, and 10M-point tiles, give bitwise equal states and outputs.
Pass 2 over the whole mesh decodes an injected random state, checked against
the oracle on 64 seeded whole 256-row blocks and 4,096 seeded points, per row,
per block and overall.  The kernel's own state at the benchmark's launch is
compared with the oracle on a 1M-point window in test_gpu_headline.py.
"""
import numpy as np
import pytest

import oracle
from gpu_helpers import assert_bf16_close, assert_state_close, banner, to_host
from ts3_synth import WORKLOADS, make_weights

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
N_SPANS_SAMPLED = 16


@pytest.fixture(scope="module")
def mesh():
    import torch
    from ts3_synth.device_gen import DeviceVolume
    wl = WORKLOADS["volume_100m_bf16"]
    banner(f"{wl.name}: generating {wl.N} points on the device")
    x = torch.empty((wl.N, wl.C), device="cuda", dtype=torch.bfloat16)
    DeviceVolume(wl.seed, wl.C).fill(x)
    torch.cuda.synchronize()
    yield wl, x
    del x
    torch.cuda.empty_cache()


def _layer(wl):
    from paper_2602_04940_amd import PhysicsAttention
    return PhysicsAttention(wl.C, wl.H, wl.M, wl.dh, wl.tau, "bf16", group_span=wl.group_span,
                            max_points=wl.N)


def test_pass1_spans_fold_invariants_tiling_and_determinism_at_100m(mesh):
    import torch
    from paper_2602_04940_amd import LayerWeights, _lib as L
    from oracle.pool import OraclePool
    wl, x = mesh
    N, Q, H, M, C = wl.N, wl.group_span, wl.H, wl.M, wl.C
    nspan = N // Q
    W = make_weights(C, H, M, wl.dh, seed=0)
    lw = LayerWeights(W)
    banner("pass 1 + state at 100M, 1M tiles")
    out = torch.empty_like(x)
    with _layer(wl) as layer:
        layer.forward(lw, x, tile=wl.tile, chunk=wl.chunk, out=out)
        proj = layer.projected()
        key = L.TS3_T_RAW if proj else L.TS3_S_RAW
        R = wl.dh if proj else C  # columns of a sums row before its weight sum
        s_raw, d, Z = layer.get(key).astype(np.float64), layer.get(L.TS3_D).astype(np.float64), layer.get(L.TS3_ZP)
        banner(f"all {nspan} span partials")
        parts = layer.get_spans(0, nspan)
        first = out.clone()
        banner("rerun, then 10M tiles")
        layer.forward(lw, x, tile=wl.tile, chunk=wl.chunk, out=out)
        assert np.array_equal(layer.get(L.TS3_ZP), Z)
        assert torch.equal(out, first)
        layer.forward(lw, x, tile=10 * wl.tile, chunk=wl.chunk, out=out)
        assert np.array_equal(layer.get(key).astype(np.float64), s_raw)
        assert np.array_equal(layer.get(L.TS3_ZP), Z)
        assert torch.equal(out, first)
        del first

    # Sampled span partials against the oracle's sums over the same points.
    spans = np.sort(np.random.default_rng(50).choice(nspan, N_SPANS_SAMPLED, replace=False))
    banner(f"oracle sums over spans {spans.tolist()}")
    xs = [to_host(x[j * Q:(j + 1) * Q]) for j in spans]
    name = "t_raw" if proj else "s_raw"
    with OraclePool(min(N_SPANS_SAMPLED, 16)) as pool:
        refs = (pool.projected_sums(xs, W["W2"], W["b2"], W["W1"], H, M, 1.0 / wl.tau) if proj else
                pool.sums(xs, W["W2"], W["b2"], H, M, 1.0 / wl.tau))
    for j, (sr, dj) in zip(spans, refs):
        p = parts[j]
        assert_state_close({name: p[:, :, :R], "d": p[:, :, R]}, {name: sr, "d": dj}, f"span {j}", BF16_TOL)

    # The fold: float32 sums of 64 consecutive spans, then of the 100 run sums,
    # in index order.  Each element's error is at most (63 + 99) * 2^-24 times
    # the sum of the magnitudes it adds (first order), against the float64 sum.
    p64 = parts.astype(np.float64)
    exact = p64.sum(axis=0)
    mag = np.abs(p64).sum(axis=0)
    del p64
    bound = (63 + 99) * 2.0 ** -24 * mag + 1e-30
    got = np.concatenate([s_raw, d[:, :, None]], axis=2)
    excess = np.abs(got - exact) / bound
    print(f"fold: worst error / bound {excess.max():.3f}", flush=True)
    assert (excess <= 1.0).all()

    # Each point's bf16-rounded weights sum to 1 within 2^-9 (RNE on each
    # term, sum of w = 1); the reciprocal, exp2 and float32 accumulation add
    # well under 1e-5 relative.
    np.testing.assert_allclose(d.sum(axis=1), N, rtol=2.0 ** -9 + 1e-5)
    # sum_m s_raw[h, m, c] - sum_i x_ic = sum_i eps_i x_ic with |eps_i| <= 2^-9.
    # Projected sums: sum_m t_raw[h, m, j] - (sum_i x_i W1_h)_j also carries the
    # bfloat16 rounding of W1 and of each point's projected row (2^-9 each,
    # relative to sum_c |x_ic W1_cj|): at most (2^-8 + 1e-5) (sum_i |x_i|) |W1_h|.
    colsum = np.zeros(C)
    abssum = np.zeros(C)
    for c0 in range(0, N, wl.chunk):
        xc = x[c0:c0 + wl.chunk].double()
        colsum += xc.sum(dim=0).cpu().numpy()
        abssum += xc.abs().sum(dim=0).cpu().numpy()
    for h in range(H):
        if proj:
            W1h = W["W1"][:, h * wl.dh:(h + 1) * wl.dh].astype(np.float64)
            err = np.abs(s_raw[h].sum(axis=0) - colsum @ W1h)
            lim = (2.0 ** -8 + 1e-5) * (abssum @ np.abs(W1h))
        else:
            err = np.abs(s_raw[h].sum(axis=0) - colsum)
            lim = (2.0 ** -9 + 1e-5) * abssum
        assert (err <= lim).all(), (h, (err / lim).max())


def test_pass2_on_injected_state_at_100m_sampled(mesh):
    import torch
    from paper_2602_04940_amd import LayerWeights
    wl, x = mesh
    W = make_weights(wl.C, wl.H, wl.M, wl.dh, seed=0, bias_seed=1)
    lw = LayerWeights(W)
    rng = np.random.default_rng(7)
    Z = (rng.standard_normal((wl.H, wl.M, wl.C)) * 0.3).astype(np.float32)
    b3 = W["b3"]
    banner("pass 2 over 100M points with an injected state")
    out = torch.empty_like(x)
    with _layer(wl) as layer:
        layer.set_state(lw, Z, b3)
        for c0 in range(0, wl.N, wl.chunk):
            layer.deslice(lw, x[c0:c0 + wl.chunk], out[c0:c0 + wl.chunk])
        torch.cuda.synchronize()
    it = 1.0 / wl.tau
    blocks = np.sort(rng.choice(wl.N // 256, 64, replace=False))
    rows = (blocks[:, None] * 256 + np.arange(256)).ravel()
    t = torch.from_numpy(rows).cuda()
    got = to_host(out[t])
    ref = oracle.deslice(to_host(x[t]), W["W2"], W["b2"], Z, b3, wl.H, wl.M, it)
    assert_bf16_close(got, ref, "64 sampled 256-row blocks", BF16_TOL, block=256)
    idx = np.sort(rng.choice(wl.N, 4096, replace=False))
    t = torch.from_numpy(idx).cuda()
    got = to_host(out[t])
    ref = oracle.deslice(to_host(x[t]), W["W2"], W["b2"], Z, b3, wl.H, wl.M, it)
    assert_bf16_close(got, ref, "4,096 sampled points", BF16_TOL, block=256)
