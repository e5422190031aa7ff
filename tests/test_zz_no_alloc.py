"""ts3_layer_forward_noalloc (the layer forward without a state object, for
callers that cannot allocate) against ts3_layer_forward on the same inputs.

The no-allocation path runs the same kernels and folds each tile's span
partials into their runs in the same order, so its outputs must equal the
state-based entry point's bit for bit.  Two calls in a row share the library's
scratch array; the second, smaller and with a ragged last span, must not see
anything of the first.
"""
import numpy as np
import pytest

from gpu_helpers import banner, to_device
from ts3_synth import WORKLOADS, make_weights

pytestmark = pytest.mark.gpu


def _state_forward(C, H, M, dtype, Q, x, lw, tile, chunk, accum="fp32"):
    from paper_2602_04940_amd import PhysicsAttention
    with PhysicsAttention(C, H, M, C // H, 0.5, dtype, group_span=Q, max_points=x.shape[0], accum=accum) as layer:
        return layer.forward(lw, x, tile=tile, chunk=chunk).clone()


def test_noalloc_matches_the_state_entry_point_bitwise_on_two_calls():
    import torch
    from paper_2602_04940_amd import LayerWeights
    from paper_2602_04940_amd.layer import layer_forward_noalloc
    from ts3_synth.device_gen import DeviceVolume
    wl = WORKLOADS["volume_100m_bf16"]
    C, H, M, Q = wl.C, wl.H, wl.M, wl.group_span
    n1, n2 = 2_500_000, 300_001
    banner(f"no-alloc forward, call 1: {n1} volume points, Q={Q}, 1M tiles and chunks, bf16")
    x = torch.empty((n1, C), device="cuda", dtype=torch.bfloat16)
    DeviceVolume(wl.seed, C).fill(x)
    lw = LayerWeights(make_weights(C, H, M, C // H, seed=0, bias_seed=1))
    ref1 = _state_forward(C, H, M, "bf16", Q, x, lw, 1_000_000, 1_000_000)
    out1 = torch.empty_like(x)
    layer_forward_noalloc(C, H, M, lw, x, 1_000_000, 1_000_000, out1, temperature=wl.tau, group_span=Q)
    torch.cuda.synchronize()
    assert torch.equal(out1, ref1)
    banner(f"no-alloc forward, call 2: {n2} points (ragged last span), 250k tiles, 100k chunks")
    x2 = x[n1 - n2:].contiguous()
    ref2 = _state_forward(C, H, M, "bf16", Q, x2, lw, 250_000, 100_000)
    out2 = torch.empty_like(x2)
    layer_forward_noalloc(C, H, M, lw, x2, 250_000, 100_000, out2, temperature=wl.tau, group_span=Q)
    torch.cuda.synchronize()
    assert torch.equal(out2, ref2)


def test_noalloc_fp32_with_the_float64_fold_and_an_empty_mesh():
    import torch
    from paper_2602_04940_amd import LayerWeights
    from paper_2602_04940_amd.layer import layer_forward_noalloc
    C, H, M, Q, N = 64, 4, 16, 1024, 5000
    banner(f"no-alloc forward fp32, float64 fold, N={N}, Q={Q}, 2048-point tiles")
    rng = np.random.default_rng(12)
    x = to_device(rng.standard_normal((N, C)), "fp32")
    lw = LayerWeights(make_weights(C, H, M, C // H, seed=4, bias_seed=5))
    ref = _state_forward(C, H, M, "fp32", Q, x, lw, 2048, 1500, accum="fp64")
    out = torch.empty_like(x)
    layer_forward_noalloc(C, H, M, lw, x, 2048, 1500, out, dtype="fp32", group_span=Q, accum="fp64")
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    empty = torch.empty((0, C), device="cuda", dtype=torch.float32)
    layer_forward_noalloc(C, H, M, lw, empty, 2048, 1500, empty, dtype="fp32", group_span=Q)
    torch.cuda.synchronize()
