"""Seeded synthetic inputs for refusal-gated decoding workloads.

This module only draws random numbers and lays them out; it performs none of the
method's arithmetic (no normalisation, attention, softmax, sampling or gating).
Both the GPU path and the CPU oracle take their inputs from here, so neither
depends on the other for data.

Every array is a pure function of (workload id, tensor name): the generator is
seeded with a SeedSequence built from the fixed tag 2607_20791, the workload id
and a CRC32 of the tensor name, and large tensors are filled in fixed-size
chunks from spawned child sequences, so the values never depend on thread
scheduling.

bf16 tensors are returned as numpy ``uint16`` arrays holding bf16 bit patterns
(round-to-nearest-even from a float32 draw); fp32 tensors as ``float32``.
"""
from __future__ import annotations

import zlib
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

TAG = (2607, 20791)
_CHUNK = 1 << 22


# --------------------------------------------------------------------------- #
# Workloads.  Shapes follow the Llama-3-8B layer (d=4096, 32/8 heads, D=128,
# SwiGLU 14336, vocab 128256) for the bf16 cases and a tiny decoder for fp32.
# --------------------------------------------------------------------------- #
@dataclass(frozen=True)
class Workload:
    name: str
    index: int
    dtype: str                 # "f32" | "bf16"
    n_layers: int = 0
    d_model: int = 0
    n_heads: int = 0
    n_kv_heads: int = 0
    head_dim: int = 0
    ffn: int = 0
    vocab: int = 0
    weight_std: float = 0.02
    rms_eps: float = 1e-5
    rope_theta: float = 500000.0
    # prompts: either real token prompts (prompt_len > 0, prefilled from 0) or a
    # synthetic N(0,1) prefix of `synthetic_prefix` positions plus one real
    # "last prompt token" prefilled at that position.
    n_prompts: int = 1
    prompt_len: int = 0
    synthetic_prefix: int = 0
    # gate
    probe_k: int = 16
    n_entries: int = 64
    entry_len: tuple = (3, 6)
    per_prompt_table: bool = False
    # sampling
    n_branches: int = 1
    steps: int = 1
    temperature: float = 1.0
    min_p: float = 0.1
    page_size: int = 16

    @property
    def prefix_positions(self) -> int:
        """Positions in the shared prompt KV once the prompt is prefilled."""
        return self.prompt_len if self.prompt_len else self.synthetic_prefix + 1


TINY_FP32 = Workload("tiny-fp32-2layer", 0, "f32", n_layers=2, d_model=256, n_heads=4,
              n_kv_heads=2, head_dim=64, ffn=1024, vocab=8192, n_prompts=16,
              prompt_len=64, probe_k=8, n_entries=16, per_prompt_table=True,
              n_branches=1, steps=32, temperature=2.0, min_p=0.1)
LAYER_P512 = Workload("8b-layer-p512", 1, "bf16", n_layers=1, d_model=4096, n_heads=32,
              n_kv_heads=8, head_dim=128, ffn=14336, vocab=128256, n_prompts=1,
              synthetic_prefix=512, probe_k=16, n_entries=64, n_branches=16,
              steps=64, temperature=1.5, min_p=0.1)
LAYER_P8192 = Workload("8b-layer-p8192", 2, "bf16", n_layers=1, d_model=4096, n_heads=32,
              n_kv_heads=8, head_dim=128, ffn=14336, vocab=128256, n_prompts=1,
              synthetic_prefix=8192, probe_k=16, n_entries=64, n_branches=64,
              steps=128, temperature=2.0, min_p=0.05)
MODEL_8LAYER = Workload("8b-8layer-32x1024", 4, "bf16", n_layers=8, d_model=4096, n_heads=32,
              n_kv_heads=8, head_dim=128, ffn=14336, vocab=128256, n_prompts=32,
              prompt_len=1024, probe_k=16, n_entries=64, n_branches=8, steps=256,
              temperature=2.0, min_p=0.1)


@dataclass(frozen=True)
class SamplerSweep:
    name: str = "sampler-sweep-256x152064"
    index: int = 3
    vocab: int = 152064
    rows: int = 256
    temperatures: tuple = (0.7, 1.0, 1.5, 2.0, 3.0)
    min_ps: tuple = (0.05, 0.1, 0.2)
    draws: int = 1000
    zipf_s: float = 1.1
    max_gap: float = 12.0


SWEEP = SamplerSweep()

WORKLOADS = {w.name: w for w in (TINY_FP32, LAYER_P512, LAYER_P8192, SWEEP, MODEL_8LAYER)}


def scaled(w: Workload, **kw) -> Workload:
    """A copy of a workload with some fields replaced (used for small test cases)."""
    d = dict(w.__dict__)
    d.update(kw)
    return Workload(**d)


# --------------------------------------------------------------------------- #
# Seeding and raw draws
# --------------------------------------------------------------------------- #
def seed_sequence(index: int, name: str) -> np.random.SeedSequence:
    return np.random.SeedSequence([TAG[0], TAG[1], int(index), zlib.crc32(name.encode())])


def rng(index: int, name: str) -> np.random.Generator:
    return np.random.Generator(np.random.SFC64(seed_sequence(index, name)))


def normal_f32(index: int, name: str, n: int, std: float = 1.0, threads: int = 8) -> np.ndarray:
    """n float32 draws of N(0, std^2), filled chunk-by-chunk from spawned streams."""
    out = np.empty(n, np.float32)
    nch = (n + _CHUNK - 1) // _CHUNK
    kids = seed_sequence(index, name).spawn(nch)

    def fill(i):
        g = np.random.Generator(np.random.SFC64(kids[i]))
        seg = out[i * _CHUNK:(i + 1) * _CHUNK]
        g.standard_normal(out=seg, dtype=np.float32)
        if std != 1.0:
            seg *= np.float32(std)

    if nch == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(fill, range(nch)))
    return out


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + r) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


def tensor(w: Workload, name: str, shape, std: float) -> np.ndarray:
    """A weight-like tensor in the workload's storage type."""
    n = int(np.prod(shape))
    x = normal_f32(w.index, name, n, std).reshape(shape)
    return to_bf16_bits(x) if w.dtype == "bf16" else x


# --------------------------------------------------------------------------- #
# Model weights (Llama-style decoder; W[out][in] row-major, y = W x)
# --------------------------------------------------------------------------- #
@dataclass
class Weights:
    w: Workload
    embed: np.ndarray
    final_norm: np.ndarray
    lm_head: np.ndarray
    layers: list = field(default_factory=list)


LAYER_TENSORS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def layer_shapes(w: Workload) -> dict:
    d, hq, hk, D, f = w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.ffn
    return {"wq": (hq * D, d), "wk": (hk * D, d), "wv": (hk * D, d), "wo": (d, hq * D),
            "w_gate": (f, d), "w_up": (f, d), "w_down": (d, f)}


def layer_weights(w: Workload, layer: int) -> dict:
    out = {}
    for name, shp in layer_shapes(w).items():
        out[name] = tensor(w, f"layer{layer}.{name}", shp, w.weight_std)
    # RMSNorm gains are 1 (Llama initialisation); kept float32.
    out["attn_norm"] = np.ones(w.d_model, np.float32)
    out["ffn_norm"] = np.ones(w.d_model, np.float32)
    return out


def model_weights(w: Workload, layers: bool = True) -> Weights:
    emb = tensor(w, "embed", (w.vocab, w.d_model), w.weight_std)
    head = tensor(w, "lm_head", (w.vocab, w.d_model), w.weight_std)
    ws = Weights(w, emb, np.ones(w.d_model, np.float32), head)
    if layers:
        ws.layers = [layer_weights(w, i) for i in range(w.n_layers)]
    return ws


# --------------------------------------------------------------------------- #
# Prompts, synthetic prefix KV, refusal tables, seeds, forced histories
# --------------------------------------------------------------------------- #
def prompt_tokens(w: Workload) -> np.ndarray:
    """[n_prompts][prompt_len] uniform token ids (or [n_prompts][1] last tokens
    for synthetic-prefix workloads)."""
    n = w.prompt_len if w.prompt_len else 1
    return rng(w.index, "prompts").integers(0, w.vocab, size=(w.n_prompts, n), dtype=np.int32)


def synthetic_prefix_kv(w: Workload, layer: int):
    """K, V ~ N(0,1) for positions [0, synthetic_prefix) of every prompt, shaped
    [n_prompts][P][Hkv][D] (values stand for already-rotated keys)."""
    shp = (w.n_prompts, w.synthetic_prefix, w.n_kv_heads, w.head_dim)
    k = tensor(w, f"prefix{layer}.k", shp, 1.0)
    v = tensor(w, f"prefix{layer}.v", shp, 1.0)
    return k, v


def random_table(w: Workload, name: str = "table", n_entries: int | None = None):
    """A refusal-prefix table in CSR form: offsets[n+1], tokens[offsets[-1]].
    Entry lengths are uniform on [entry_len[0], entry_len[1]], ids uniform."""
    n = w.n_entries if n_entries is None else n_entries
    g = rng(w.index, name)
    lens = g.integers(w.entry_len[0], w.entry_len[1] + 1, size=n)
    offsets = np.zeros(n + 1, np.int32)
    offsets[1:] = np.cumsum(lens)
    toks = g.integers(0, w.vocab, size=int(offsets[-1]), dtype=np.int32)
    return offsets, toks


def branch_seeds(n_prompts: int, n_branches: int, base: int = 0) -> np.ndarray:
    """uint64 Philox keys, one per branch: prompt index * N + branch, offset by base."""
    return (np.arange(n_prompts * n_branches, dtype=np.uint64) + np.uint64(base))


def forced_history(w: Workload, rows: int, steps: int, name: str = "forced") -> np.ndarray:
    """[rows][steps] token ids used to teacher-force a decode loop."""
    return rng(w.index, name).integers(0, w.vocab, size=(rows, steps), dtype=np.int32)


def sweep_logits(s: SamplerSweep = SWEEP, rows: int | None = None, vocab: int | None = None) -> np.ndarray:
    """[rows][V] float32 logits: z_i = eps_i + b_{pi(i)}, eps ~ N(0,1), with rank
    bias b_r = gap * (r^-s - V^-s) / (1 - V^-s), r = 1..V, and pi a uniform random
    permutation per row, so b_1 - b_V = gap exactly."""
    rows = s.rows if rows is None else rows
    V = s.vocab if vocab is None else vocab
    eps = normal_f32(s.index, f"eps{V}", rows * V).reshape(rows, V)
    r = np.arange(1, V + 1, dtype=np.float64)
    vs = float(V) ** (-s.zipf_s)
    bias = s.max_gap * (r ** (-s.zipf_s) - vs) / (1.0 - vs)
    g = rng(s.index, f"perm{V}")
    out = np.empty((rows, V), np.float32)
    for i in range(rows):
        out[i] = eps[i] + bias[g.permutation(V)].astype(np.float32)
    return out
