"""GPU parity of the Transolver block stack (ts3_stack_*) against the float64
block oracle, through the C ABI: bf16 activations, so the bar is relative L2
<= 2e-2 on the stack's output; tiled and untiled runs agree bitwise; decoding
the mesh's own points from the cached states reproduces the forward bitwise;
decoding new query points matches the oracle's decoding from its own states,
and from injected states."""
import numpy as np
import pytest

from gpu_helpers import assert_bf16_close, banner, rel_l2, to_device, to_host
from oracle import block as BK
from ts3_synth import make_block_weights, round_bf16

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


def _blocks(C, H, M, F, L, seed=0):
    return [make_block_weights(C, H, M, C // H, F, seed=seed + 3 * l, bias_seed=seed + 3 * l + 1) for l in range(L)]


def _stack(C, H, M, L, Q, N):
    from paper_2602_04940_amd import TransolverStack
    return TransolverStack(C, H, M, L, group_span=Q, max_points=N)


def _dev_blocks(blocks):
    from paper_2602_04940_amd import BlockWeights
    return [BlockWeights(b) for b in blocks]


def _f64(blocks):
    return [{k: np.asarray(v, np.float64) for k, v in b.items()} for b in blocks]


SHAPES = [(256, 8, 64, 2, 3000, 384), (128, 8, 32, 3, 2000, 256)]


@pytest.mark.parametrize("C,H,M,L,N,Q", SHAPES)
def test_stack_matches_oracle_and_is_tiling_independent(C, H, M, L, N, Q):
    import torch
    F = 4 * C
    banner(f"stack C={C} H={H} M={M} F={F} L={L} N={N} Q={Q}")
    rng = np.random.default_rng(C + L)
    x64 = round_bf16(rng.standard_normal((N, C)))
    blocks = _blocks(C, H, M, F, L)
    dev = _dev_blocks(blocks)
    outs = []
    with _stack(C, H, M, L, Q, N) as st:
        for tile, chunk in ((2 * Q, 500), (N + Q - N % Q, N)):
            x = to_device(x64, "bf16")
            st.forward(dev, x, tile=tile, chunk=chunk)
            torch.cuda.synchronize()
            outs.append(to_host(x))
    assert np.array_equal(outs[0], outs[1])
    ref = BK.stack_forward(x64, _f64(blocks), H, M, 2.0)
    assert_bf16_close(outs[0], ref, "stack", BF16_TOL)


def test_decoding_the_mesh_reproduces_the_forward_and_query_points_match_the_oracle():
    import torch
    C, H, M, L, N, Q = 256, 8, 64, 2, 2500, 384
    F = 4 * C
    banner(f"stack decode C={C} L={L} N={N}")
    rng = np.random.default_rng(9)
    x64 = round_bf16(rng.standard_normal((N, C)))
    q64 = round_bf16(rng.standard_normal((700, C)))
    blocks = _blocks(C, H, M, F, L, seed=20)
    dev = _dev_blocks(blocks)
    with _stack(C, H, M, L, Q, N) as st:
        x = to_device(x64, "bf16")
        st.forward(dev, x, tile=2 * Q, chunk=1000)
        x0 = to_device(x64, "bf16")
        st.decode(dev, x0, chunk=333)
        q = to_device(q64, "bf16")
        st.decode(dev, q, chunk=256)
        torch.cuda.synchronize()
        assert torch.equal(x0, x)
        got = to_host(q)
    b64 = _f64(blocks)
    Zs = BK.stack_states(x64, b64, H, M, 2.0)
    ref = BK.stack_decode(q64, b64, Zs, H, M, 2.0)
    assert_bf16_close(got, ref, "query decode", BF16_TOL)


def test_decoding_from_injected_states():
    import torch
    C, H, M, L, n = 256, 8, 64, 3, 1200
    F = 4 * C
    banner(f"stack decode from injected states C={C} L={L} n={n}")
    rng = np.random.default_rng(17)
    q64 = round_bf16(rng.standard_normal((n, C)))
    blocks = _blocks(C, H, M, F, L, seed=40)
    Zs = [rng.standard_normal((H, M, C)) * 0.3 for _ in range(L)]
    dev = _dev_blocks(blocks)
    with _stack(C, H, M, L, 1024, n) as st:
        for l in range(L):
            st.layer(l).set_state(dev[l].pa, Zs[l].astype(np.float32), blocks[l]["b3"])
        q = to_device(q64, "bf16")
        st.decode(dev, q, chunk=500)
        torch.cuda.synchronize()
        got = to_host(q)
    Zs32 = [z.astype(np.float32).astype(np.float64) for z in Zs]
    ref = BK.stack_decode(q64, _f64(blocks), Zs32, H, M, 2.0)
    assert_bf16_close(got, ref, "injected-state decode", BF16_TOL)


def test_feedforward_half_matches_the_oracle_and_writes_the_next_layernorm():
    import torch
    C, H, M, L, n = 256, 8, 64, 2, 1000
    F = 4 * C
    banner(f"feed-forward half C={C} F={F} n={n} (ragged 128-point workgroups)")
    rng = np.random.default_rng(23)
    x64 = round_bf16(rng.standard_normal((n, C)))
    pa64 = round_bf16(0.5 * rng.standard_normal((n, C)))
    blocks = _blocks(C, H, M, F, L, seed=60)
    dev = _dev_blocks(blocks)
    with _stack(C, H, M, L, 1024, n) as st:
        x = to_device(x64, "bf16")
        xn = torch.empty_like(x)
        st.feedforward(dev, 0, x, to_device(pa64, "bf16"), xn_next=xn)
        torch.cuda.synchronize()
        got, got_xn = to_host(x), to_host(xn)
    b = _f64(blocks)
    y = x64 + pa64
    ref = y + BK.mlp(BK.layer_norm(y, b[0]["ln2_g"], b[0]["ln2_b"]), b[0]["Wa"], b[0]["ba"], b[0]["Wb"], b[0]["bb"])
    assert_bf16_close(got, ref, "feed-forward", BF16_TOL)
    assert_bf16_close(got_xn, BK.layer_norm(ref, b[1]["ln1_g"], b[1]["ln1_b"]), "next LN1", BF16_TOL)
