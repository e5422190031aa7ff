"""Parity at the benchmark's launch configuration, against the float64 oracle.

Workload: the 100M-point volume mesh's recipe (C=128, H=8, M=64, dh=16, tau=0.5,
bf16 storage, the benchmark's zero-bias weights), group span Q = 15,625, pass-1
tiles and pass-2 chunks of 1M points.

A seeded window of 1M points is taken from the mesh: one of its 100 generator
chunks, the rows [k*1M, (k+1)*1M) that bench.py holds.  It runs as a mesh of its
own through ts3_layer_forward with the benchmark's kernels and launch shape.
That is one pass-1 launch over 64 spans of 15,625 points (489 blocks per span)
and one pass-2 launch of 256 persistent workgroups.  Checked against the
oracle (Eq. (1), (3)-(5), Algorithm 1):
  * the state: the slice sums (s_raw, or t_raw for a state of projected sums)
    and Z per slice token, d per element;
  * the output: every row, each 256-row block, and the whole window.
With random-init weights the token attention nearly averages each head's
tokens, so all output rows are close to one vector, and the output check alone
is weak.  The same window is therefore also decoded from an injected random
state, whose output varies strongly from point to point, under the same bars.
"""
import numpy as np
import pytest

from gpu_helpers import assert_bf16_close, assert_state_close, banner, to_host
from ts3_synth import WORKLOADS, make_weights

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
WINDOW_SEED = 40
CHUNK = 1_000_000


@pytest.fixture(scope="module")
def window():
    import torch
    from ts3_synth.device_gen import DeviceVolume
    wl = WORKLOADS["volume_100m_bf16"]
    k = int(np.random.default_rng(WINDOW_SEED).integers(wl.N // CHUNK))
    banner(f"{wl.name}: window = generator chunk {k} (mesh rows {k * CHUNK}..{(k + 1) * CHUNK - 1})")
    gen = DeviceVolume(wl.seed, wl.C)
    x = gen.features(gen.points(k, CHUNK)).contiguous()
    torch.cuda.synchronize()
    return wl, k, x, to_host(x)


@pytest.fixture(scope="module")
def pool():
    from oracle.pool import OraclePool
    with OraclePool() as p:
        yield p


def test_window_state_and_output_at_the_bench_launch(window, pool):
    import torch
    from paper_2602_04940_amd import LayerWeights, PhysicsAttention, _lib as L
    wl, k, x, x64 = window
    W = make_weights(wl.C, wl.H, wl.M, wl.dh, seed=0)
    lw = LayerWeights(W)
    banner(f"GPU layer on window {k}: Q={wl.group_span}, tile={wl.tile}, chunk={wl.chunk}")
    with PhysicsAttention(wl.C, wl.H, wl.M, wl.dh, wl.tau, "bf16", group_span=wl.group_span,
                          max_points=CHUNK) as layer:
        out = layer.forward(lw, x, tile=wl.tile, chunk=wl.chunk)
        torch.cuda.synchronize()
        proj = layer.projected()
        st = {"d": layer.get(L.TS3_D), "Z": layer.get(L.TS3_ZP)}
        st["t_raw" if proj else "s_raw"] = layer.get(L.TS3_T_RAW if proj else L.TS3_S_RAW)
    got = to_host(out)
    banner(f"oracle on window {k} ({pool.workers} host processes)")
    it = 1.0 / wl.tau
    ref_st = pool.state(x64, W, wl.H, wl.M, it)
    if proj:
        parts = pool.projected_tile_sums(x64, W["W2"], W["b2"], W["W1"], wl.H, wl.M, it, 65536)
        ref_st["t_raw"] = sum((t[0] for t in parts), np.zeros((wl.H, wl.M, wl.dh)))
    ref = pool.decode(x64, W["W2"], W["b2"], ref_st["Z"], W["b3"], wl.H, wl.M, it)
    assert_state_close(st, ref_st, "state", BF16_TOL)
    assert_bf16_close(got, ref, "out", BF16_TOL)


def test_window_decoded_from_an_injected_state_at_the_bench_launch(window, pool):
    import torch
    from paper_2602_04940_amd import LayerWeights, PhysicsAttention
    wl, k, x, x64 = window
    W = make_weights(wl.C, wl.H, wl.M, wl.dh, seed=0)
    lw = LayerWeights(W)
    rng = np.random.default_rng(41)
    Z = (rng.standard_normal((wl.H, wl.M, wl.C)) * 0.3).astype(np.float32)
    b3 = (rng.standard_normal(wl.C) * 0.1).astype(np.float32)
    banner(f"pass 2 on window {k} from an injected state, one 1M-point chunk")
    with PhysicsAttention(wl.C, wl.H, wl.M, wl.dh, wl.tau, "bf16", group_span=wl.group_span,
                          max_points=CHUNK) as layer:
        layer.set_state(lw, Z, b3)
        out = layer.deslice(lw, x)
        torch.cuda.synchronize()
    ref = pool.decode(x64, W["W2"], W["b2"], Z, b3, wl.H, wl.M, 1.0 / wl.tau)
    assert_bf16_close(to_host(out), ref, "out (injected state)", BF16_TOL)
