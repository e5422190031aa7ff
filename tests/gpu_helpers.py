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
