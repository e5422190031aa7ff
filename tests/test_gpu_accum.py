"""The float64 fold of span partials (ts3_desc.accum = TS3_ACCUM_FP64): the
sum over tiles of Eq. (4) taken in float64 and rounded once, for accumulation
over very large meshes (Appendix A.4).

  * at small sizes it matches the float64 oracle like the float32 fold, and is
    bitwise independent of the tiling;
  * on a 160M-point float32 volume mesh (the size of the paper's largest
    volume meshes) both folds are checked against what holds at any size,
    sum_m d[h, m] = N and sum_m s_raw[h, m, :] = sum_i x_i, and their drift is
    printed side by side.
"""
import numpy as np
import pytest

import oracle
from gpu_helpers import banner, normwise, to_device, to_host
from ts3_synth import make_weights

pytestmark = pytest.mark.gpu


def _layer(C, H, M, Q, N, accum, dtype="fp32"):
    from paper_2602_04940_amd import PhysicsAttention
    return PhysicsAttention(C, H, M, C // H, 0.5, dtype, group_span=Q, max_points=N, accum=accum)


def test_fp64_fold_matches_oracle_and_is_tiling_independent():
    import torch
    from paper_2602_04940_amd import LayerWeights, _lib as L
    C, H, M, N, Q = 128, 8, 64, 70_000, 512
    banner(f"fp64 fold, fp32 storage, N={N}, Q={Q}")
    rng = np.random.default_rng(5)
    x64 = rng.standard_normal((N, C)).astype(np.float32).astype(np.float64)
    W = make_weights(C, H, M, C // H, seed=2, bias_seed=3)
    x = to_device(x64, "fp32")
    lw = LayerWeights(W)
    got = {}
    for accum, tile in (("fp64", 8192), ("fp64", N + 512 - N % 512), ("fp32", 8192)):
        with _layer(C, H, M, Q, N + 512, accum) as layer:
            out = layer.forward(lw, x, tile=tile, chunk=8192)
            torch.cuda.synchronize()
            got[(accum, tile)] = (to_host(out), layer.get(L.TS3_S_RAW), layer.get(L.TS3_D))
    a, b = got[("fp64", 8192)], got[("fp64", N + 512 - N % 512)]
    assert all(np.array_equal(u, v) for u, v in zip(a, b))
    it = 2.0
    st = oracle.build_state(x64, {k: np.asarray(v, np.float64) for k, v in W.items()}, H, M, it, tile=N)
    ref_out = oracle.deslice(x64, W["W2"], W["b2"], st["Z"], W["b3"], H, M, it)
    for accum in ("fp64", "fp32"):
        out, s_raw, d = got[(accum, 8192)]
        e = (normwise(out, ref_out), normwise(s_raw, st["s_raw"]), normwise(d, st["d"]))
        print(f"{accum} fold: out {e[0]:.2e}, s_raw {e[1]:.2e}, d {e[2]:.2e}", flush=True)
        assert max(e) <= 1e-4


def test_fp64_fold_of_projected_sums_bf16():
    """bfloat16 storage at C = 128, head width 16: the span partials hold
    projected rows (dh + 1 floats); the float64 fold of them matches the
    oracle's projected sums and is bitwise independent of the tiling."""
    import torch
    from paper_2602_04940_amd import LayerWeights, _lib as L
    from gpu_helpers import assert_bf16_close, assert_state_close, match_sums
    from ts3_synth import round_bf16
    C, H, M, N, Q = 128, 8, 64, 70_000, 512
    banner(f"fp64 fold of projected sums, bf16 storage, N={N}, Q={Q}")
    rng = np.random.default_rng(6)
    x64 = round_bf16(rng.standard_normal((N, C)))
    W = make_weights(C, H, M, C // H, seed=2, bias_seed=3)
    x = to_device(x64, "bf16")
    lw = LayerWeights(W)
    got = {}
    for accum, tile in (("fp64", 8192), ("fp64", N + 512 - N % 512), ("fp32", 8192)):
        with _layer(C, H, M, Q, N + 512, accum, "bf16") as layer:
            assert layer.projected()
            out = layer.forward(lw, x, tile=tile, chunk=8192)
            torch.cuda.synchronize()
            got[(accum, tile)] = (to_host(out), layer.get(L.TS3_T_RAW), layer.get(L.TS3_D), layer.get(L.TS3_ZP))
    a, b = got[("fp64", 8192)], got[("fp64", N + 512 - N % 512)]
    assert all(np.array_equal(u, v) for u, v in zip(a, b))
    it = 2.0
    st = oracle.build_state(x64, W, H, M, it, tile=N)
    ref_out = oracle.deslice(x64, W["W2"], W["b2"], st["Z"], W["b3"], H, M, it)
    for accum in ("fp64", "fp32"):
        out, t_raw, d, Z = got[(accum, 8192)]
        g = {"t_raw": t_raw, "d": d, "Z": Z}
        match_sums(g, st, x64, W, H, M, it)
        assert_state_close(g, st, f"{accum} fold state", 2e-2)
        assert_bf16_close(out, ref_out, f"{accum} fold out", 2e-2)


def test_fold_drift_on_a_160m_point_mesh():
    import torch
    from paper_2602_04940_amd import LayerWeights, _lib as L
    from ts3_synth.device_gen import DeviceVolume
    N, C, H, M, Q, tile = 160_000_000, 128, 8, 64, 15_625, 10_000_000
    banner(f"generating {N} volume points, fp32")
    x = torch.empty((N, C), device="cuda", dtype=torch.float32)
    DeviceVolume(5, C, dtype=torch.float32).fill(x)
    colsum = torch.zeros(C, dtype=torch.float64, device="cuda")
    abssum = torch.zeros(C, dtype=torch.float64, device="cuda")
    for c0 in range(0, N, tile):
        xc = x[c0:c0 + tile].double()
        colsum += xc.sum(dim=0)
        abssum += xc.abs().sum(dim=0)
    colsum, abssum = colsum.cpu().numpy(), abssum.cpu().numpy()
    lw = LayerWeights(make_weights(C, H, M, C // H, seed=0))
    drift = {}
    for accum in ("fp32", "fp64"):
        banner(f"pass 1 over {N} points, {accum} fold")
        with _layer(C, H, M, Q, N, accum) as layer:
            layer.reset()
            for t0 in range(0, N, tile):
                layer.accumulate(lw, x[t0:t0 + tile], t0)
            layer.finalize(lw)
            torch.cuda.synchronize()
            s_raw = layer.get(L.TS3_S_RAW).astype(np.float64)
            d = layer.get(L.TS3_D).astype(np.float64)
        dd = np.abs(d.sum(axis=1) - N).max() / N
        ds = max((np.abs(s_raw[h].sum(axis=0) - colsum) / abssum).max() for h in range(H))
        drift[accum] = (dd, ds)
        print(f"{accum} fold: max_h |sum_m d - N| / N = {dd:.3e}; "
              f"max_h,c |sum_m s_raw - sum_i x| / sum_i |x| = {ds:.3e}", flush=True)
    del x
    torch.cuda.empty_cache()
    # Bound for either fold: each point's float32 weights sum to one within
    # M * 2^-24 (exp2, one reciprocal and one product per weight, then the
    # sum), and each float32 add of the span, run and final chains loses at
    # most 2^-24 relative: 122 in-span block adds (15,625 points over four
    # waves of 32-point blocks), 64 run adds and 160 final adds (the float64
    # fold drops the last two).
    bound = (M + 122 + 64 + 160) * 2.0 ** -24
    for accum, (dd, ds) in drift.items():
        assert dd <= bound and ds <= bound, (accum, dd, ds, bound)
