"""The layer backward at the training workload's full size: 2M points drawn by
seed without replacement from a 160M-point volume mesh (section 3.2's training
on subsets of the full mesh), C=128, H=8, M=64, float32, 1M-point tiles and
group span 15,625 (the launch configuration ``bench.py --backward`` times).

The drawn rows are first checked to be the mesh's rows at the drawn indices.
The float64 backward oracle needs minutes for 2M points, so the full size is
checked through properties that hold at any size, and the oracle itself is
compared on the first 40,000 points of the same subset (two spans and a ragged
third, the mesh's own feature distribution):
  * reruns, and untiled (one 2M-point tile) runs, are bitwise equal;
  * scaling g by 2 scales every gradient by exactly 2 (the backward is linear
    in g and a power-of-two scale commutes with rounding);
  * db3 is the column sum of g;
  * the loss is linear in W3, so <dW3, V> equals the loss of a forward with
    W3 := V and b3 := 0;
  * along random directions of x, W2, W1 and Wq the gradient matches a
    fourth-order central difference of the GPU forward's loss.
"""
import numpy as np
import pytest

from gpu_helpers import banner, normwise, to_host
from oracle import backward as BW
from ts3_synth import WORKLOADS, make_weights

pytestmark = pytest.mark.gpu

TOL = 1e-4
NAMES = ("dW2", "db2", "dW1", "db1", "dWq", "dWk", "dWv", "dW3", "db3")


@pytest.fixture(scope="module")
def problem():
    import torch
    from ts3_synth.device_gen import DeviceVolume
    from ts3_synth.workloads import subset_indices
    wl = WORKLOADS["volume_2m_fp32"]
    banner(f"{wl.name}: drawing {wl.N} of {wl.source_N} mesh points and an output gradient on the device")
    x = torch.empty((wl.N, wl.C), device="cuda", dtype=torch.float32)
    DeviceVolume(wl.seed, wl.C, dtype=torch.float32).gather(x, subset_indices(wl), wl.source_N)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(wl.seed + 1000)
    g = torch.randn((wl.N, wl.C), device="cuda", dtype=torch.float32, generator=gen)
    W = make_weights(wl.C, wl.H, wl.M, wl.dh, seed=0, bias_seed=1)
    torch.cuda.synchronize()
    yield wl, x, g, W
    del x, g
    torch.cuda.empty_cache()


def test_the_drawn_rows_are_the_mesh_rows_at_the_drawn_indices():
    """gather() on the device against fill() of the same mesh: a 5M-point
    volume mesh, 40,000 indices drawn as the training subset is, bitwise."""
    import torch
    from ts3_synth.device_gen import DeviceVolume
    wl = WORKLOADS["volume_2m_fp32"]
    source = 5_000_000
    idx = np.sort(np.random.default_rng(wl.subset_seed).choice(source, 40_000, replace=False))
    banner(f"gather of {len(idx)} rows of a {source}-point mesh vs fill")
    gen = DeviceVolume(wl.seed, wl.C, dtype=torch.float32)
    full = torch.empty((source, wl.C), device="cuda", dtype=torch.float32)
    gen.fill(full)
    x = torch.empty((len(idx), wl.C), device="cuda", dtype=torch.float32)
    gen.gather(x, idx, source)
    assert torch.equal(x, full[torch.from_numpy(idx).cuda()])


def _layer(wl, N):
    from paper_2602_04940_amd import PhysicsAttention
    return PhysicsAttention(wl.C, wl.H, wl.M, wl.dh, wl.tau, "fp32", group_span=wl.group_span, max_points=N)


def _backward(layer, wl, W, x, g, tile):
    from paper_2602_04940_amd import LayerWeights
    import torch
    lw = LayerWeights(W)
    layer.forward(lw, x, tile=tile, chunk=wl.chunk)
    dx, grads = layer.backward(lw, x, g, tile=tile)
    torch.cuda.synchronize()
    return dx, grads


def _loss(layer, wl, W, x, g):
    """sum(g * forward(x)) accumulated in float64 on the device."""
    from paper_2602_04940_amd import LayerWeights
    out = layer.forward(LayerWeights(W), x, tile=wl.tile, chunk=wl.chunk)
    return float((out.double() * g.double()).sum())


def test_backward_tiling_rerun_and_g_scaling_are_exact_at_2m(problem):
    import torch
    wl, x, g, W = problem
    with _layer(wl, wl.N) as layer:
        banner("backward at 2M, 1M tiles")
        dx, gr = _backward(layer, wl, W, x, g, wl.tile)
        dx, gr = dx.clone(), {k: v.clone() for k, v in gr.items()}
        banner("rerun")
        dx2, gr2 = _backward(layer, wl, W, x, g, wl.tile)
        assert torch.equal(dx, dx2) and all(torch.equal(gr[k], gr2[k]) for k in NAMES)
        banner("one 2M tile")
        dx2, gr2 = _backward(layer, wl, W, x, g, wl.N)
        assert torch.equal(dx, dx2) and all(torch.equal(gr[k], gr2[k]) for k in NAMES)
        banner("g scaled by 2")
        dx2, gr2 = _backward(layer, wl, W, x, 2 * g, wl.tile)
        assert torch.equal(2 * dx, dx2) and all(torch.equal(2 * gr[k], gr2[k]) for k in NAMES)
        assert torch.isfinite(dx).all()
    # db3 = sum_i g_i: float32 folds of 15,625-point span sums stay far below
    # 1e-4 of the column's absolute sum.
    gd = g.double()
    colsum, abssum = gd.sum(dim=0).cpu().numpy(), gd.abs().sum(dim=0).cpu().numpy()
    err = np.abs(gr["db3"].double().cpu().numpy() - colsum)
    print(f"db3 max error / column abs sum {(err / abssum).max():.2e}", flush=True)
    assert (err <= 1e-4 * abssum).all()


def test_dW3_equals_the_loss_of_the_linear_map_at_2m(problem):
    wl, x, g, W = problem
    rng = np.random.default_rng(21)
    V = rng.standard_normal(np.shape(W["W3"])).astype(np.float32) * 0.1
    with _layer(wl, wl.N) as layer:
        _, gr = _backward(layer, wl, W, x, g, wl.tile)
        lhs = float((gr["dW3"].double().cpu().numpy() * V).sum())
        WV = dict(W, W3=V, b3=np.zeros_like(W["b3"]))
        from paper_2602_04940_amd import LayerWeights
        out = layer.forward(LayerWeights(WV), x, tile=wl.tile, chunk=wl.chunk)
        prod = out.double() * g.double()
        rhs, scale = float(prod.sum()), float(prod.abs().sum())
    print(f"<dW3, V> {lhs:.6e}, loss of W3 := V {rhs:.6e}, |diff| / sum|g out| {abs(lhs - rhs) / scale:.2e}",
          flush=True)
    assert abs(lhs - rhs) <= 1e-5 * scale


def _directional(layer, wl, W, x, g, which, V, eps):
    """Fourth-order central difference of the loss along V (x or a weight)."""
    vals = []
    for k in (2, 1, -1, -2):
        if which == "x":
            vals.append(_loss(layer, wl, W, x + (k * eps) * V, g))
        else:
            Wk = dict(W)
            Wk[which] = (np.asarray(W[which], np.float64) + (k * eps) * V).astype(np.float32)
            vals.append(_loss(layer, wl, Wk, x, g))
    return (-vals[0] + 8 * vals[1] - 8 * vals[2] + vals[3]) / (12 * eps)


@pytest.mark.parametrize("which,eps", [("x", 2e-2), ("W2", 2e-2), ("W1", 5e-2), ("Wq", 5e-2)])
def test_gradient_matches_central_differences_of_the_forward_at_2m(problem, which, eps):
    import torch
    wl, x, g, W = problem
    rng = np.random.default_rng(31)
    with _layer(wl, wl.N) as layer:
        dx, gr = _backward(layer, wl, W, x, g, wl.tile)
        if which == "x":
            gen = torch.Generator(device="cuda")
            gen.manual_seed(41)
            V = torch.randn(x.shape, device="cuda", dtype=torch.float32, generator=gen)
            analytic = float((dx.double() * V.double()).sum())
        else:
            V = rng.standard_normal(np.shape(W[which])) * np.abs(np.asarray(W[which])).mean()
            analytic = float((gr["d" + which].double().cpu().numpy() * V).sum())
        numeric = _directional(layer, wl, W, x, g, which, V, eps)
    rel = abs(analytic - numeric) / abs(numeric)
    print(f"{which}: analytic {analytic:.6e}, differences {numeric:.6e}, rel {rel:.2e}", flush=True)
    assert rel <= 1e-2


def test_backward_matches_oracle_on_the_first_40k_points_of_the_subset(problem):
    wl, x, g, W = problem
    N = 40_000
    xs, gs = x[:N].contiguous(), g[:N].contiguous()
    banner(f"backward on the first {N} points, tile {wl.group_span} vs the float64 oracle")
    with _layer(wl, N) as layer:
        dx, gr = _backward(layer, wl, W, xs, gs, wl.group_span)
        dx, gr = to_host(dx), {k: v.cpu().numpy().astype(np.float64) for k, v in gr.items()}
    W64 = {k: np.asarray(v, np.float64) for k, v in W.items()}
    ref = BW.layer_backward(to_host(xs), W64, to_host(gs), wl.H, wl.M, 1.0 / wl.tau, tile=wl.group_span)
    err = normwise(dx, ref["dx"])
    print(f"dx normwise {err:.2e}", flush=True)
    assert err <= TOL
    for k in NAMES:
        e = normwise(gr[k], ref[k])
        print(f"{k} normwise {e:.2e}", flush=True)
        assert e <= TOL, k
