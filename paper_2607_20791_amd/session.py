"""Device-side setup for a decoder workload: uploads weights and allocates the
KV buffers the C ABI works on (PyTorch supplies the device memory).

Weights arrive as numpy arrays (bf16 bit patterns in uint16, or float32) and
become torch tensors on the current GPU; nothing here computes any part of
the decode path.
"""
from __future__ import annotations

import numpy as np

from . import DTYPE_BF16, DTYPE_F32, KV, Model, ModelConfig


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("no GPU visible: the HIP path cannot run")
    return torch


def to_device(a: np.ndarray):
    torch = _torch()
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    if a.dtype == np.float32:
        return torch.from_numpy(a).cuda()
    if a.dtype == np.int32:
        return torch.from_numpy(a).cuda()
    raise TypeError(f"unsupported dtype {a.dtype}")


def model_config(w, max_pos: int) -> ModelConfig:
    return ModelConfig(w.n_layers, w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.ffn, w.vocab,
                       DTYPE_BF16 if w.dtype == "bf16" else DTYPE_F32, w.rms_eps, w.rope_theta,
                       max_pos)


def build_model(weights, max_rows: int, max_pos: int) -> Model:
    """weights: a synth.Weights (numpy) -> Model with device copies."""
    w = weights.w
    tensors = {"embed": to_device(weights.embed), "final_norm": to_device(weights.final_norm),
               "lm_head": to_device(weights.lm_head)}
    layers = [{k: to_device(v) for k, v in L.items()} for L in weights.layers]
    return Model(model_config(w, max_pos), tensors, layers, max_rows)


def alloc_kv(model: Model, w, max_prompts: int, max_prefix: int, n_pages: int,
             page_size: int = 16) -> KV:
    torch = _torch()
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    H, D = w.n_kv_heads, w.head_dim
    pre_k = (w.n_layers, max_prompts, H, max_prefix, D)
    pre_v = (w.n_layers, max_prompts, H, v_stride(max_prefix) // 64, D, 64)
    pool_k = (w.n_layers, max(n_pages, 1), H, page_size, D)
    pool_v = (w.n_layers, max(n_pages, 1), H, D, page_size)
    pk = torch.zeros(pre_k, dtype=dt, device="cuda")
    pv = torch.zeros(pre_v, dtype=dt, device="cuda")
    qk = torch.zeros(pool_k, dtype=dt, device="cuda")
    qv = torch.zeros(pool_v, dtype=dt, device="cuda")
    return KV(model, max_prompts, max_prefix, n_pages, page_size, pk, pv, qk, qv)


def v_stride(max_prefix: int) -> int:
    """Positions per prompt and head in the V cache: max_prefix rounded up to 64."""
    return (max_prefix + 63) // 64 * 64


def k_cache_layout(k: np.ndarray) -> np.ndarray:
    """[B][P][Hkv][D] -> the K cache layout [B][Hkv][P][D]."""
    return np.ascontiguousarray(k.transpose(0, 2, 1, 3))


def v_cache_layout(v: np.ndarray, VP: int) -> np.ndarray:
    """[B][P][Hkv][D] -> the V cache layout [B][Hkv][VP/64][D][64] (zero padded)."""
    B, P, H, D = v.shape
    out = np.zeros((B, H, VP // 64, D, 64), v.dtype)
    vt = v.transpose(0, 2, 3, 1)                 # [B][H][D][P]
    for blk in range((P + 63) // 64):
        n = min(64, P - blk * 64)
        out[:, :, blk, :, :n] = vt[:, :, :, blk * 64:blk * 64 + n]
    return out


def fill_prefix(kv: KV, layer: int, k: np.ndarray, v: np.ndarray):
    """Writes caller-generated prefix K/V [B][P][Hkv][D] into positions [0, P)."""
    B, P = k.shape[:2]
    kv.prefix_k[layer, :B, :, :P].copy_(to_device(k_cache_layout(k)))
    VP = kv.prefix_v.shape[3] * 64  # [L][B][Hkv][VP/64][D][64]
    vv = v_cache_layout(v, VP)
    kv.prefix_v[layer, :B].copy_(to_device(vv))
