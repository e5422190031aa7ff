"""The block stack at the benchmark's full size: 8 blocks over the 10M-point car
surface, C=256, H=8, M=64, dh=32, F=1024, bf16, 1M-point tiles and chunks,
group span 31,250 (the launch configuration ``bench.py --stack`` times).

The float64 oracle cannot run eight blocks over 1e7 points in test time, so:
  * reruns, and runs with 2M-point tiles, are bitwise equal;
  * decoding 4,096 sampled mesh points from the cached states reproduces the
    forward's outputs at those points bitwise;
  * with random states injected into every block, decoding 4,096 sampled query
    points matches the oracle's decoding from the same states.
"""
import numpy as np
import pytest

from gpu_helpers import assert_bf16_close, banner, rel_l2, to_host
from oracle import block as BK
from ts3_synth import WORKLOADS, make_block_weights

pytestmark = pytest.mark.gpu

BLOCKS = 8
BF16_TOL = 2e-2


@pytest.fixture(scope="module")
def mesh():
    import torch
    from ts3_synth.device_gen import DeviceSurface
    wl = WORKLOADS["car_10m_bf16"]
    banner(f"{wl.name}: generating {wl.N} car-surface points on the device")
    x0 = torch.empty((wl.N, wl.C), device="cuda", dtype=torch.bfloat16)
    DeviceSurface(wl.seed, wl.C).fill(x0)
    blocks = [make_block_weights(wl.C, wl.H, wl.M, wl.dh, 4 * wl.C, seed=100 + l, bias_seed=200 + l)
              for l in range(BLOCKS)]
    torch.cuda.synchronize()
    yield wl, x0, blocks
    del x0
    torch.cuda.empty_cache()


def _stack(wl):
    from paper_2602_04940_amd import TransolverStack
    return TransolverStack(wl.C, wl.H, wl.M, BLOCKS, 4 * wl.C, wl.dh, wl.tau, group_span=wl.group_span,
                           max_points=wl.N)


def test_stack_at_10m_is_tiling_independent_and_decodes_its_mesh(mesh):
    import torch
    from paper_2602_04940_amd import BlockWeights
    wl, x0, blocks = mesh
    dev = [BlockWeights(b) for b in blocks]
    rng = np.random.default_rng(5)
    idx = torch.from_numpy(np.sort(rng.choice(wl.N, 4096, replace=False))).cuda()
    with _stack(wl) as st:
        banner("8 blocks at 10M, 1M tiles")
        x = x0.clone()
        st.forward(dev, x, tile=wl.tile, chunk=wl.chunk)
        torch.cuda.synchronize()
        assert torch.isfinite(x.float()).all()
        banner("rerun, then 2M tiles")
        y = x0.clone()
        st.forward(dev, y, tile=wl.tile, chunk=wl.chunk)
        assert torch.equal(x, y)
        y.copy_(x0)
        st.forward(dev, y, tile=2 * wl.tile, chunk=wl.chunk)
        assert torch.equal(x, y)
        del y
        banner("decode 4,096 mesh points from the cached states")
        q = x0[idx].contiguous()
        st.decode(dev, q, chunk=wl.chunk)
        torch.cuda.synchronize()
        assert torch.equal(q, x[idx])


def test_stack_decode_from_injected_states_at_10m_sampled(mesh):
    import torch
    from paper_2602_04940_amd import BlockWeights
    wl, x0, blocks = mesh
    dev = [BlockWeights(b) for b in blocks]
    rng = np.random.default_rng(7)
    Zs = [(rng.standard_normal((wl.H, wl.M, wl.C)) * 0.3).astype(np.float32) for _ in range(BLOCKS)]
    idx = np.sort(rng.choice(wl.N, 4096, replace=False))
    banner("8 blocks decoding 4,096 sampled points of the 10M mesh from injected states")
    with _stack(wl) as st:
        for l in range(BLOCKS):
            st.layer(l).set_state(dev[l].pa, Zs[l], blocks[l]["b3"])
        q = x0[torch.from_numpy(idx).cuda()].contiguous()
        qs = to_host(q)
        st.decode(dev, q, chunk=wl.chunk)
        torch.cuda.synchronize()
        got = to_host(q)
    b64 = [{k: np.asarray(v, np.float64) for k, v in b.items()} for b in blocks]
    ref = BK.stack_decode(qs, b64, [z.astype(np.float64) for z in Zs], wl.H, wl.M, 1.0 / wl.tau)
    assert_bf16_close(got, ref, "sampled", BF16_TOL)
