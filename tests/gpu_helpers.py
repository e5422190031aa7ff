"""Shared helpers of the GPU tests: device copies of seeded inputs, running the
layer through the C ABI, and the error measures the acceptance bar uses."""
import numpy as np


def normwise(got, ref):
    """max |got - ref| / max |ref|  (the fp32 bar, 1e-4)."""
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.abs(np.asarray(got, dtype=np.float64) - ref).max() / max(np.abs(ref).max(), 1e-300))


def rel_l2(got, ref):
    """||got - ref||_2 / ||ref||_2  (relative L2, the bf16 bar, 2e-2)."""
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(np.asarray(got, dtype=np.float64) - ref) / max(np.linalg.norm(ref), 1e-300))


def to_device(x64, dtype_name, device="cuda"):
    """Stored-precision float64 values -> device tensor of the io dtype (exact)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x64, dtype=np.float32))
    return t.to(device=device, dtype=torch.bfloat16 if dtype_name == "bf16" else torch.float32).contiguous()


def to_host(t):
    return t.float().cpu().numpy().astype(np.float64)


def banner(msg):
    print(f"\n[gpu case] {msg}", flush=True)


def block_rel_l2(got, ref, block=256):
    """Largest relative L2 over consecutive blocks of `block` rows (the last
    block may be short): a single wrong block of a large array fails it."""
    got = np.asarray(got, dtype=np.float64).reshape(len(got), -1)
    ref = np.asarray(ref, dtype=np.float64).reshape(len(ref), -1)
    n = len(ref)
    if n == 0:
        return 0.0
    nb = -(-n // block)
    pad = nb * block - n
    d2 = np.pad(((got - ref) ** 2).sum(axis=1), (0, pad)).reshape(nb, block).sum(axis=1)
    r2 = np.pad((ref ** 2).sum(axis=1), (0, pad)).reshape(nb, block).sum(axis=1)
    return float(np.sqrt(d2 / np.maximum(r2, 1e-300)).max())


def row_rel(got, ref):
    """Largest per-row error ||got_i - ref_i|| / max(||ref_i||, rms row norm):
    relative to the row itself, with rows much smaller than the array's typical
    row measured against that typical size instead."""
    got = np.asarray(got, dtype=np.float64).reshape(len(got), -1)
    ref = np.asarray(ref, dtype=np.float64).reshape(len(ref), -1)
    if len(ref) == 0:
        return 0.0
    rn = np.linalg.norm(ref, axis=1)
    floor = np.sqrt((rn ** 2).mean())
    return float((np.linalg.norm(got - ref, axis=1) / np.maximum(np.maximum(rn, floor), 1e-300)).max())


def assert_bf16_close(got, ref, what, tol=2e-2, block=256):
    """The bf16 bar applied globally and locally: relative L2 over the whole
    array, over every block of `block` consecutive rows, and per row (see
    row_rel).  Rows are points for outputs and slice tokens for states."""
    g, b, r = rel_l2(got, ref), block_rel_l2(got, ref, block), row_rel(got, ref)
    print(f"{what}: rel L2 {g:.3e}, worst {block}-row block {b:.3e}, worst row {r:.3e}", flush=True)
    assert g <= tol, (what, "global", g)
    assert b <= tol, (what, "block", b)
    assert r <= tol, (what, "row", r)
    return g, b, r


def assert_state_close(st, ref, what, tol=2e-2):
    """bf16-path state against the oracle: the slice sums (s_raw [H, M, C] or
    the projected t_raw [H, M, dh]) and Z per slice token, d element by
    element, each within the bf16 bar."""
    H, M = np.asarray(ref["d"]).shape
    for k in ("s_raw", "t_raw", "Z"):
        if k in st:
            assert_bf16_close(np.asarray(st[k]).reshape(H * M, -1), np.asarray(ref[k]).reshape(H * M, -1),
                              f"{what} {k}", tol, block=M)
    dr = np.asarray(ref["d"], dtype=np.float64)
    dg = np.asarray(st["d"], dtype=np.float64)
    ed = float((np.abs(dg - dr) / np.maximum(np.abs(dr), 1e-300)).max()) if dr.size else 0.0
    print(f"{what} d: worst element rel {ed:.3e}", flush=True)
    assert ed <= tol, (what, "d", ed)


def sums_key(st):
    """'t_raw' for a state that sums projected rows (x_i W1_h per head), else 's_raw'."""
    return "t_raw" if "t_raw" in st else "s_raw"


def state_of(layer):
    """The layer's state buffers as float32 host arrays: d, s, s1, Z and the
    slice sums in the form the state keeps them (s_raw or t_raw)."""
    from paper_2602_04940_amd import _lib as L
    st = {"d": layer.get(L.TS3_D), "s": layer.get(L.TS3_S), "s1": layer.get(L.TS3_S1), "Z": layer.get(L.TS3_ZP)}
    if layer.projected():
        st["t_raw"] = layer.get(L.TS3_T_RAW)
    else:
        st["s_raw"] = layer.get(L.TS3_S_RAW)
    return st


def match_sums(st, ref_st, x, W, H, M, inv_tau, tile=None):
    """Give the oracle state the sums the GPU state holds: for a projected
    state, t_raw from oracle.projected_accumulate over consecutive tiles of
    `tile` points (the whole mesh at once when tile is None)."""
    if "t_raw" in st and "t_raw" not in ref_st:
        import oracle
        N = len(x)
        step = tile or max(N, 1)
        dh = W["W1"].shape[1] // H
        t = np.zeros((H, M, dh))
        for i in range(0, N, step):
            t += oracle.projected_accumulate(x[i:i + step], W["W2"], W["b2"], W["W1"], H, M, inv_tau)[0]
        ref_st["t_raw"] = t
    return ref_st
