"""Helpers shared by the GPU tests (not collected as tests)."""
import numpy as np


def torch():
    import torch as t
    return t


def seeds_tensor(seeds):
    t = torch()
    return t.from_numpy(np.asarray(seeds, dtype=np.uint64).view(np.int64)).cuda()


def rel_err(got, ref):
    """Normwise relative error max|got - ref| / max|ref| (per last axis)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    num = np.abs(got - ref).max(axis=-1)
    den = np.maximum(np.abs(ref).max(axis=-1), 1e-30)
    return num / den


def bf16_to_f64(t):
    """torch bf16 tensor -> float64 numpy (exact)."""
    return t.float().cpu().numpy().astype(np.float64)


def sample_gpu(rgd, z_np, T, pmin, seeds, ctr=0, stream0=0, draws=1):
    t = torch()
    z = t.from_numpy(np.ascontiguousarray(z_np, dtype=np.float32)).cuda()
    R, V = z.shape
    ws = t.empty(rgd.sampler_workspace_bytes(R, V), dtype=t.uint8, device="cuda")
    out = t.full((R, draws), -1, dtype=t.int32, device="cuda")
    rgd.kernel_sample(z, T, pmin, seeds_tensor(seeds), ctr, stream0, draws, ws, out)
    t.cuda.synchronize()
    return out.cpu().numpy()


def argmax_gpu(rgd, z_np):
    t = torch()
    z = t.from_numpy(np.ascontiguousarray(z_np, dtype=np.float32)).cuda()
    R, V = z.shape
    ws = t.empty(rgd.sampler_workspace_bytes(R, V), dtype=t.uint8, device="cuda")
    out = t.full((R,), -1, dtype=t.int32, device="cuda")
    rgd.kernel_argmax(z, ws, out)
    t.cuda.synchronize()
    return out.cpu().numpy()
