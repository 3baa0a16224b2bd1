"""Python binding of librgd (refusal-gated decoding on MI355X / gfx950).

Argument marshalling only: every step of the decode path runs in the HIP
library.  Tensors are PyTorch tensors on the GPU; their data pointers and the
current HIP stream are passed through the C ABI declared in include/rgd.h.
Importing this module loads the library and raises if it has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

__all__ = [
    "RGDError", "lib", "ModelConfig", "Model", "KV", "Table", "prefill_kv", "probe", "probe_fixed", "gate",
    "sample_continuations", "sample_continuations_pless", "check_status", "kernel_attention", "kernel_lm_head", "kernel_argmax",
    "kernel_sample", "kernel_sample_noalloc", "kernel_sample_pless", "sampler_workspace_bytes", "timing_enable", "timing_read", "TIMERS", "EVENT_INCOMPAT", "EVENT_STOP", "EVENT_MAXLEN",
    "DTYPE_F32", "DTYPE_BF16",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librgd.so")
EXPORTS = (
    "rgd_version", "rgd_last_error", "rgd_model_create", "rgd_model_destroy", "rgd_kv_create",
    "rgd_kv_destroy", "rgd_kv_set_prefix_len", "rgd_table_create", "rgd_table_destroy",
    "rgd_prefill_kv", "rgd_prefill_kv_scored", "rgd_probe", "rgd_probe_fixed", "rgd_probe_soft", "rgd_probe_adaptive", "rgd_gate", "rgd_sample_continuations", "rgd_sample_continuations_pless", "rgd_check_status",
    "rgd_kernel_attention", "rgd_kernel_lm_head", "rgd_sampler_workspace_bytes",
    "rgd_kernel_argmax", "rgd_kernel_sample", "rgd_kernel_sample_noalloc", "rgd_kernel_sample_pless", "rgd_kernel_probe_step", "rgd_timing_enable", "rgd_timing_read",
)

DTYPE_F32, DTYPE_BF16 = 0, 1
EVENT_INCOMPAT, EVENT_STOP, EVENT_MAXLEN, EVENT_SKIPPED = 0, 1, 2, 3
STATUS = {0: "OK", 1: "INVALID_ARG", 2: "OOM", 3: "HIP", 4: "UNSUPPORTED", 5: "NONFINITE", 6: "STATE"}

# PyTorch ships its own HIP runtime (same soname as the system one).  Loading it
# first makes librgd bind to that instance; loading librgd first would bring in
# the system runtime and leave the process with two HIP/HSA runtimes, of which
# the second sees no device.
try:
    import torch  # noqa: F401
except ImportError:  # CPU-only use of the binding (export checks) needs no torch
    pass

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with paper_2607_20791_amd/build.py "
                      "(there is no fallback path)")
lib = C.CDLL(LIB_PATH)

VP, I32, U32, F32, U64 = C.c_void_p, C.c_int32, C.c_uint32, C.c_float, C.c_uint64
I32P = C.POINTER(C.c_int32)


class ModelConfig(C.Structure):
    _fields_ = [("n_layers", I32), ("d_model", I32), ("n_heads", I32), ("n_kv_heads", I32),
                ("head_dim", I32), ("ffn_dim", I32), ("vocab", I32), ("dtype", I32),
                ("rms_eps", F32), ("rope_theta", F32), ("max_pos", I32)]


class LayerWeights(C.Structure):
    _fields_ = [(n, VP) for n in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate",
                                  "w_up", "w_down")]


class Weights(C.Structure):
    _fields_ = [("embed", VP), ("final_norm", VP), ("lm_head", VP),
                ("layers", C.POINTER(LayerWeights))]


def _sig(name, res, *args):
    f = getattr(lib, name)
    f.restype = res
    f.argtypes = list(args)
    return f


_sig("rgd_version", C.c_char_p)
_sig("rgd_last_error", C.c_char_p)
_sig("rgd_model_create", I32, C.POINTER(ModelConfig), C.POINTER(Weights), I32, C.POINTER(VP))
_sig("rgd_model_destroy", None, VP)
_sig("rgd_kv_create", I32, VP, I32, I32, I32, I32, VP, VP, VP, VP, C.POINTER(VP))
_sig("rgd_kv_destroy", None, VP)
_sig("rgd_kv_set_prefix_len", I32, VP, I32, I32)
_sig("rgd_table_create", I32, I32P, I32P, I32, I32P, I32, C.POINTER(VP))
_sig("rgd_table_destroy", None, VP)
_sig("rgd_prefill_kv", I32, VP, VP, VP, I32, I32, I32, VP, VP)
_sig("rgd_probe", I32, VP, VP, VP, VP, I32, I32, I32, I32, VP, VP, VP, VP)
_sig("rgd_probe_fixed", I32, VP, VP, VP, VP, I32, I32, I32, I32, VP, VP, VP, VP)
_sig("rgd_probe_soft", I32, VP, VP, VP, VP, I32, I32, I32, I32, I32, C.c_float, VP, VP, VP, VP)
_sig("rgd_probe_adaptive", I32, VP, VP, VP, VP, I32, I32, I32, I32, I32, C.c_float, VP, C.c_float, VP, VP, VP, VP)
_sig("rgd_prefill_kv_scored", I32, VP, VP, VP, I32, I32, I32, VP, I32, VP, C.c_float, VP, VP)
_sig("rgd_kernel_probe_step", I32, VP, VP, I32, VP, I32, I32, I32, I32, C.c_float, VP, VP, VP, VP)
_sig("rgd_gate", I32, VP, VP, I32, I32P, I32P, I32P, VP)
_sig("rgd_sample_continuations", I32, VP, VP, VP, I32P, I32, I32, I32, F32, F32, VP, VP, VP, VP, VP)
_sig("rgd_sample_continuations_pless", I32, VP, VP, VP, I32P, I32, I32, I32, F32, VP, VP, VP, VP, VP)
_sig("rgd_check_status", I32, VP, VP)
_sig("rgd_kernel_attention", I32, VP, VP, I32, I32P, I32P, VP, VP, I32, I32, VP, VP, I32, VP, I32,
     I32, I32, VP, VP)
_sig("rgd_kernel_lm_head", I32, VP, VP, I32, VP, VP)
_sig("rgd_sampler_workspace_bytes", U64, I32, I32)
_sig("rgd_kernel_argmax", I32, VP, I32, I32, VP, VP, VP)
_sig("rgd_kernel_sample", I32, VP, I32, I32, F32, F32, VP, U32, U32, I32, VP, VP, VP)
_sig("rgd_kernel_sample_noalloc", I32, VP, I32, I32, F32, F32, VP, U32, U32, I32, VP, VP)
_sig("rgd_kernel_sample_pless", I32, VP, I32, I32, F32, VP, U32, U32, I32, VP, VP, VP)
_sig("rgd_timing_enable", I32, VP, I32)
_sig("rgd_timing_read", I32, VP, C.POINTER(C.c_double), C.POINTER(C.c_int64))

TIMERS = ("lm_head", "attention", "attn_prefix", "sampler", "step")


class RGDError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"rgd error {STATUS.get(code, code)}: {msg}")
        self.code = code


def _check(rc):
    if rc != 0:
        raise RGDError(rc, lib.rgd_last_error().decode())


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream():
    import torch
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _host_i32(seq):
    import numpy as np
    a = np.ascontiguousarray(np.asarray(seq, dtype=np.int32))
    return a, a.ctypes.data_as(I32P)


class Model:
    """A model handle over caller-owned device weights (kept alive here)."""

    def __init__(self, cfg: ModelConfig, tensors: dict, layers: list, max_rows: int):
        self.cfg = cfg
        self._keep = (tensors, layers)
        lw = (LayerWeights * len(layers))()
        for i, L in enumerate(layers):
            for n in LayerWeights._fields_:
                setattr(lw[i], n[0], L[n[0]].data_ptr())
        self._lw = lw
        w = Weights(tensors["embed"].data_ptr(), tensors["final_norm"].data_ptr(),
                    tensors["lm_head"].data_ptr(), lw)
        h = VP()
        _check(lib.rgd_model_create(C.byref(cfg), C.byref(w), max_rows, C.byref(h)))
        self.h = h

    def close(self):
        if self.h:
            lib.rgd_model_destroy(self.h)
            self.h = VP()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class KV:
    """Prompt-KV and tail-page state over caller-owned device buffers."""

    def __init__(self, model: Model, max_prompts, max_prefix, n_pages, page_size, prefix_k,
                 prefix_v, pool_k, pool_v):
        self.model = model
        self._keep = (prefix_k, prefix_v, pool_k, pool_v)
        self.prefix_k, self.prefix_v, self.pool_k, self.pool_v = prefix_k, prefix_v, pool_k, pool_v
        h = VP()
        _check(lib.rgd_kv_create(model.h, max_prompts, max_prefix, n_pages, page_size,
                                 _ptr(prefix_k), _ptr(prefix_v), _ptr(pool_k), _ptr(pool_v),
                                 C.byref(h)))
        self.h = h

    def set_prefix_len(self, prompt, length):
        _check(lib.rgd_kv_set_prefix_len(self.h, prompt, length))

    def close(self):
        if self.h:
            lib.rgd_kv_destroy(self.h)
            self.h = VP()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Table:
    """Refusal-prefix table (CSR host arrays, copied to the device)."""

    def __init__(self, offsets, tokens, owner=None, min_match=2):
        import numpy as np
        off, offp = _host_i32(offsets)
        tok, tokp = _host_i32(tokens if len(tokens) else np.zeros(1, np.int32))
        n = len(off) - 1
        ownp = None
        if owner is not None:
            own, ownp = _host_i32(owner)
        h = VP()
        _check(lib.rgd_table_create(offp, tokp, n, ownp, min_match, C.byref(h)))
        self.h = h

    def close(self):
        if self.h:
            lib.rgd_table_destroy(self.h)
            self.h = VP()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def prefill_kv(model, kv, tokens, start_pos, last_logits):
    B, n = tokens.shape
    _check(lib.rgd_prefill_kv(model.h, kv.h, _ptr(tokens), B, n, start_pos, _ptr(last_logits),
                              _stream()))


def probe(model, kv, last_logits, table, B, k, c, eos, probe_tokens, probe_len, event):
    """table None: fixed-length probe (no refusal set)."""
    _check(lib.rgd_probe(model.h, kv.h, _ptr(last_logits), table.h if table is not None else None, B, k, c,
                         eos, _ptr(probe_tokens), _ptr(probe_len), _ptr(event), _stream()))


def probe_fixed(model, kv, last_logits, table, B, k, c, eos, probe_tokens, probe_len, event):
    """Probe with no early exit: k greedy tokens (or up to eos), then the table
    judges the finished probe (table None: every probe is a hit)."""
    _check(lib.rgd_probe_fixed(model.h, kv.h, _ptr(last_logits), table.h if table is not None else None, B, k,
                               c, eos, _ptr(probe_tokens), _ptr(probe_len), _ptr(event), _stream()))


def kernel_probe_step(model, logits, table, k, c, eos, topk, rho, probe_tokens, probe_len, event):
    """One probe step for prompts 0..R-1 (R = logits rows) on given logits."""
    _check(lib.rgd_kernel_probe_step(model.h, _ptr(logits), logits.shape[0],
                                     table.h if table is not None else None, k, c, eos, topk, float(rho),
                                     _ptr(probe_tokens), _ptr(probe_len), _ptr(event), _stream()))


def prefill_kv_scored(model, kv, tokens, start_pos, last_logits, cls_layer, cls_w, cls_b, scores):
    """Prefill plus the residual-stream pre-check score of each prompt."""
    B, n = tokens.shape
    _check(lib.rgd_prefill_kv_scored(model.h, kv.h, _ptr(tokens), B, n, start_pos, _ptr(last_logits), cls_layer,
                                     _ptr(cls_w), float(cls_b), _ptr(scores), _stream()))


def probe_adaptive(model, kv, last_logits, table, B, k, c, eos, topk, rho, scores, theta, probe_tokens,
                   probe_len, event):
    """Adaptive gate: prompts scored <= theta are SKIPPED, the others probed."""
    _check(lib.rgd_probe_adaptive(model.h, kv.h, _ptr(last_logits), table.h if table is not None else None, B,
                                  k, c, eos, topk, float(rho), _ptr(scores), float(theta), _ptr(probe_tokens),
                                  _ptr(probe_len), _ptr(event), _stream()))


def probe_soft(model, kv, last_logits, table, B, k, c, eos, topk, rho, probe_tokens, probe_len, event):
    """Probe with the soft compatibility gate: tokens 1..c are soft steps."""
    _check(lib.rgd_probe_soft(model.h, kv.h, _ptr(last_logits), table.h if table is not None else None, B, k,
                              c, eos, topk, float(rho), _ptr(probe_tokens), _ptr(probe_len), _ptr(event),
                              _stream()))


def gate(kv, event, B):
    """Returns (decision list, miss index list)."""
    import numpy as np
    dec = np.zeros(B, np.int32)
    miss = np.zeros(B, np.int32)
    nm = C.c_int32(0)
    _check(lib.rgd_gate(kv.h, _ptr(event), B, dec.ctypes.data_as(I32P), C.byref(nm),
                        miss.ctypes.data_as(I32P), _stream()))
    return dec, miss[:nm.value]


def sample_continuations(model, kv, last_logits, prompt_idx, N, steps, T, min_p, seeds, out,
                         forced=None, logits_tap=None):
    pi, pip = _host_i32(prompt_idx)
    _check(lib.rgd_sample_continuations(model.h, kv.h, _ptr(last_logits), pip, len(pi), N, steps,
                                        T, min_p, _ptr(seeds), _ptr(forced), _ptr(logits_tap),
                                        _ptr(out), _stream()))


def sample_continuations_pless(model, kv, last_logits, prompt_idx, N, steps, T, seeds, out,
                               forced=None, logits_tap=None):
    pi, pip = _host_i32(prompt_idx)
    _check(lib.rgd_sample_continuations_pless(model.h, kv.h, _ptr(last_logits), pip, len(pi), N, steps,
                                              T, _ptr(seeds), _ptr(forced), _ptr(logits_tap),
                                              _ptr(out), _stream()))


def check_status(model):
    _check(lib.rgd_check_status(model.h, _stream()))


def kernel_attention(model, q, row_prompt, plen, prefix_k, prefix_v, max_prompts, max_prefix,
                     pool_k, pool_v, page_size, pages, max_pages, tail_len, out, splits=0):
    rp, rpp = _host_i32(row_prompt)
    pl, plp = _host_i32(plen)
    _check(lib.rgd_kernel_attention(model.h, _ptr(q), len(rp), rpp, plp, _ptr(prefix_k),
                                    _ptr(prefix_v), max_prompts, max_prefix, _ptr(pool_k),
                                    _ptr(pool_v), page_size, _ptr(pages), max_pages, tail_len,
                                    splits, _ptr(out), _stream()))


def kernel_lm_head(model, h, logits):
    _check(lib.rgd_kernel_lm_head(model.h, _ptr(h), h.shape[0], _ptr(logits), _stream()))


def timing_enable(model, period=1):
    """period >= 1 times every period-th launch of each unit; 0 (or False) stops."""
    _check(lib.rgd_timing_enable(model.h, int(period)))


def timing_read(model):
    """{unit: (total ms, launches)} since the last read."""
    ms = (C.c_double * len(TIMERS))()
    n = (C.c_int64 * len(TIMERS))()
    _check(lib.rgd_timing_read(model.h, ms, n))
    return {k: (ms[i], n[i]) for i, k in enumerate(TIMERS)}


def sampler_workspace_bytes(R, V):
    return int(lib.rgd_sampler_workspace_bytes(R, V))


def kernel_argmax(z, workspace, out):
    R, V = z.shape
    _check(lib.rgd_kernel_argmax(_ptr(z), R, V, _ptr(workspace), _ptr(out), _stream()))


def kernel_sample(z, T, min_p, seeds, ctr, stream0, draws, workspace, out):
    R, V = z.shape
    _check(lib.rgd_kernel_sample(_ptr(z), R, V, T, min_p, _ptr(seeds), ctr, stream0, draws,
                                 _ptr(workspace), _ptr(out), _stream()))


NOALLOC_SCRATCH_BYTES = 1 << 20


def kernel_sample_noalloc(z, T, min_p, seeds, ctr, stream0, draws, out):
    """rgd_kernel_sample without a workspace: the library's fixed device scratch
    (RGD_NOALLOC_SCRATCH_BYTES) is used; nothing is allocated."""
    R, V = z.shape
    _check(lib.rgd_kernel_sample_noalloc(_ptr(z), R, V, T, min_p, _ptr(seeds), ctr, stream0, draws, _ptr(out),
                                         _stream()))


def kernel_sample_pless(z, T, seeds, ctr, stream0, draws, workspace, out):
    R, V = z.shape
    _check(lib.rgd_kernel_sample_pless(_ptr(z), R, V, T, _ptr(seeds), ctr, stream0, draws,
                                       _ptr(workspace), _ptr(out), _stream()))
