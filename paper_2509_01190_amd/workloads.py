"""Seeded synthetic inputs for the pruned layer-stack forward.

This module only draws numbers and fixes shapes. It holds none of the
method's arithmetic, so both the HIP path (through the binding) and the
CPU oracle can be fed from it without sharing any computation.

Every tensor has its own stream ``numpy.random.default_rng([seed, layer,
tensor_id])`` (PCG64). Linear weights and biases are N(0, 0.02); norm gains
are 1 and LayerNorm shifts 0 (standard initialisation), unless
``norm_jitter`` asks for gains 1 + N(0, 0.1) and shifts N(0, 0.1) so that a
test exercises those paths. Hidden inputs are N(0, 1) per row. Values are
drawn in float32; for bf16 workloads they are rounded to bf16 (nearest-even,
by torch's CPU conversion) *before* either side sees them, so the GPU and
the oracle consume the same numbers.

The presets follow the paper's two attention forms (bidirectional encoder,
causal decoder; Sec. 3.2) and the backbone features it lists as shared by
current models (pre-norm residual, GELU/SwiGLU, RoPE; Appendix A, Table 1),
at the sizes of the workloads this library is measured on.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence

import numpy as np

ENCODER = 0
DECODER = 1

# tensor ids of the per-layer RNG streams
_TID = {
    "norm1_w": 0, "norm1_b": 1, "w_qkv": 2, "b_qkv": 3, "w_o": 4, "b_o": 5,
    "norm2_w": 6, "norm2_b": 7, "w_up": 8, "b_up": 9, "w_down": 10, "b_down": 11,
}
_HIDDEN_LAYER = 10_000   # stream "layer" index used for the hidden inputs
_LENGTH_LAYER = 10_001   # ... for ragged lengths
_RATE_LAYER = 10_002     # ... for per-sequence keep rates
_SCORE_LAYER = 10_003    # ... for injected importance scores


@dataclasses.dataclass(frozen=True)
class Preset:
    name: str
    kind: int                 # ENCODER or DECODER
    n_layers: int
    d_model: int
    n_heads: int
    d_ff: int
    batch: int
    seq_len: int              # fixed length; ragged presets override via lengths()
    dtype: str                # "f32" or "bf16"
    causal: bool
    prune_after: tuple        # 1-based layer indices whose output is compacted
    keep_rates: tuple         # sweep (ignored when per_seq_rates)
    tau: int = 5              # floor on preserved rows (paper: fixed at 5)
    ragged: bool = False
    min_len: int = 0
    per_seq_rates: bool = False
    rate_lo: float = 0.0
    rate_hi: float = 1.0
    norm_eps: float = 1e-5
    rope_theta: float = 10000.0
    n_kv_heads: int = 0       # key/value heads (grouped-query attention); 0: n_heads
    force_keep_last: bool = False
    mark_only: bool = False   # pruning points mark rows instead of removing them

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    @property
    def kv_heads(self) -> int:
        return self.n_heads if self.n_kv_heads == 0 else self.n_kv_heads


PRESETS: Dict[str, Preset] = {
    # 2-layer encoder small enough for the oracle to finish in well under a second
    "tiny": Preset("tiny", ENCODER, 2, 128, 4, 512, 4, 64, "f32", False, (1,), (0.5,)),
    # BERT-base-shaped encoder, pruned after layers 3/6/9
    "bert": Preset("bert", ENCODER, 12, 768, 12, 3072, 32, 512, "bf16", False, (3, 6, 9),
                   (1.0, 0.7, 0.5, 0.3, 0.1)),
    # 1B-shaped decoder prefill, pruned every 4 layers
    "dec1b": Preset("dec1b", DECODER, 16, 2048, 32, 8192, 8, 2048, "bf16", True, (4, 8, 12),
                    (1.0, 0.5, 0.25, 0.1)),
    # 7B-shaped decoder prefill, a 4-layer slice at real width, pruned after layer 1
    "dec7b": Preset("dec7b", DECODER, 4, 4096, 32, 11008, 4, 4096, "bf16", True, (1,),
                    (0.5, 0.2, 0.09)),
    # the paper's own schedule: Eq. 2 after every layer (tau = 5) on a
    # GPT-2-small-shaped causal stack (pre-LN, GELU, biases, no rotary; the
    # learned position embeddings are part of the synthetic input rows)
    "gpt2": Preset("gpt2", ENCODER, 12, 768, 12, 3072, 32, 512, "bf16", True,
                   tuple(range(1, 13)), (1.0, 0.9, 0.8, 0.7, 0.5, 0.3, 0.1, 0.02)),
    # ... the same stack at the other sequence lengths, 16384 rows per batch
    "gpt2_n128": Preset("gpt2_n128", ENCODER, 12, 768, 12, 3072, 128, 128, "bf16", True,
                        tuple(range(1, 13)), (1.0, 0.9, 0.8, 0.7, 0.5, 0.3, 0.1, 0.02)),
    "gpt2_n1024": Preset("gpt2_n1024", ENCODER, 12, 768, 12, 3072, 16, 1024, "bf16", True,
                         tuple(range(1, 13)), (1.0, 0.9, 0.8, 0.7, 0.5, 0.3, 0.1, 0.02)),
    # LLaMA-3-8B-shaped prefill slice: grouped-query attention (32 query heads
    # over 8 key/value heads), FFN 14336; the last input row always survives
    # (the first generated token is predicted from it)
    "llama3_8b": Preset("llama3_8b", DECODER, 4, 4096, 32, 14336, 4, 4096, "bf16", True, (1,),
                        (1.0, 0.5, 0.2, 0.09), rope_theta=500000.0, n_kv_heads=8,
                        force_keep_last=True),
    # one 7B-shaped layer over a ragged batch with per-sequence keep rates
    "ragged": Preset("ragged", DECODER, 1, 4096, 32, 11008, 64, 4096, "bf16", True, (1,), (),
                     ragged=True, min_len=128, per_seq_rates=True, rate_lo=0.05, rate_hi=1.0),
}


def shrink(p: Preset, **kw) -> Preset:
    """A copy of a preset with some fields replaced (smaller test shapes)."""
    return dataclasses.replace(p, **kw)


def _rng(seed: int, layer: int, tid: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(layer), int(tid)])


def lengths(p: Preset, seed: int = 0) -> List[int]:
    """Sequence lengths: fixed, or uniform integers in [min_len, seq_len]."""
    if not p.ragged:
        return [p.seq_len] * p.batch
    g = _rng(seed, _LENGTH_LAYER, 0)
    return [int(v) for v in g.integers(p.min_len, p.seq_len + 1, size=p.batch)]


def cu_seqlens(lens: Sequence[int]) -> np.ndarray:
    """Row offsets of each sequence in the packed [T, d] layout (int32, B+1)."""
    cu = np.zeros(len(lens) + 1, dtype=np.int64)
    cu[1:] = np.cumsum(np.asarray(lens, dtype=np.int64))
    return cu.astype(np.int32)


def keep_rates(p: Preset, seed: int = 0, alpha: Optional[float] = None) -> np.ndarray:
    """Per-sequence keep rates (float64): all equal to ``alpha``, or, for
    presets with per-sequence rates, uniform in [rate_lo, rate_hi]."""
    if p.per_seq_rates and alpha is None:
        g = _rng(seed, _RATE_LAYER, 0)
        return g.uniform(p.rate_lo, p.rate_hi, size=p.batch).astype(np.float64)
    a = 1.0 if alpha is None else float(alpha)
    return np.full(p.batch, a, dtype=np.float64)


def hidden(p: Preset, seed: int = 0, lens: Optional[Sequence[int]] = None) -> np.ndarray:
    """Packed hidden inputs [sum(lens), d_model], float32, N(0, 1)."""
    if lens is None:
        lens = lengths(p, seed)
    t = int(sum(lens))
    g = _rng(seed, _HIDDEN_LAYER, 0)
    return g.standard_normal((t, p.d_model), dtype=np.float32)


def positions(lens: Sequence[int]) -> np.ndarray:
    """Original position of every packed row (0..n_b-1 per sequence), int32."""
    return np.concatenate([np.arange(n, dtype=np.int32) for n in lens]) if len(lens) else \
        np.zeros(0, dtype=np.int32)


def layer_weights(p: Preset, layer: int, seed: int = 0, norm_jitter: bool = False,
                  zero_wq: bool = False) -> Dict[str, Optional[np.ndarray]]:
    """Weights of one layer (PyTorch Linear layout [out, in], float32).

    w_qkv rows are [q; k; v]: d_model query rows, then kv_heads*head_dim key
    rows and as many value rows, head h at rows h*head_dim ..
    (h+1)*head_dim of its block. For the decoder, w_up has 2*d_ff rows that
    interleave gate and up projections: row 2f is gate f, row 2f+1 is up f.
    ``zero_wq`` zeroes the query rows (and their bias): every query is then
    the zero vector, which makes attention exactly uniform.
    """
    d, f = p.d_model, p.d_ff
    qkv = d + 2 * p.kv_heads * p.head_dim

    def normal(name, shape, std=0.02):
        return (_rng(seed, layer, _TID[name]).standard_normal(shape, dtype=np.float32)
                * np.float32(std)).astype(np.float32)

    def gain(name, shape):
        if norm_jitter:
            return (1.0 + normal(name, shape, 0.1)).astype(np.float32)
        return np.ones(shape, dtype=np.float32)

    def shift(name, shape):
        if norm_jitter:
            return normal(name, shape, 0.1)
        return np.zeros(shape, dtype=np.float32)

    w: Dict[str, Optional[np.ndarray]] = {}
    if p.kind == ENCODER:
        w["norm1_w"] = gain("norm1_w", (d,))
        w["norm1_b"] = shift("norm1_b", (d,))
        w["w_qkv"] = normal("w_qkv", (qkv, d))
        w["b_qkv"] = normal("b_qkv", (qkv,))
        w["w_o"] = normal("w_o", (d, d))
        w["b_o"] = normal("b_o", (d,))
        w["norm2_w"] = gain("norm2_w", (d,))
        w["norm2_b"] = shift("norm2_b", (d,))
        w["w_up"] = normal("w_up", (f, d))
        w["b_up"] = normal("b_up", (f,))
        w["w_down"] = normal("w_down", (d, f))
        w["b_down"] = normal("b_down", (d,))
    else:
        w["norm1_w"] = gain("norm1_w", (d,))
        w["norm1_b"] = None
        w["w_qkv"] = normal("w_qkv", (qkv, d))
        w["b_qkv"] = None
        w["w_o"] = normal("w_o", (d, d))
        w["b_o"] = None
        w["norm2_w"] = gain("norm2_w", (d,))
        w["norm2_b"] = None
        w["w_up"] = normal("w_up", (2 * f, d))
        w["b_up"] = None
        w["w_down"] = normal("w_down", (d, f))
        w["b_down"] = None
    if zero_wq:
        w["w_qkv"][:d] = 0.0
        if w["b_qkv"] is not None:
            w["b_qkv"][:d] = 0.0
    return w


def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def stack_weights(p: Preset, seed: int = 0, norm_jitter: bool = False,
                  zero_wq: bool = False) -> List[Dict[str, Optional[np.ndarray]]]:
    """Every layer's weights. Layers are drawn on a few threads at once (the
    generator releases the interpreter lock); each tensor has its own stream,
    so the numbers do not depend on the order or the thread count."""
    if p.n_layers <= 1:
        return [layer_weights(p, l, seed, norm_jitter, zero_wq) for l in range(p.n_layers)]
    with ThreadPoolExecutor(max_workers=min(_workers(), p.n_layers)) as ex:
        return list(ex.map(lambda l: layer_weights(p, l, seed, norm_jitter, zero_wq),
                           range(p.n_layers)))


def injected_scores(lens: Sequence[int], seed: int = 0) -> np.ndarray:
    """Importance scores [sum(lens)] float32 built to stress tie handling.

    Sequence b gets, by b % 4: (0) scores quantised to multiples of 1/16 in
    [0, 4), so many equal values straddle any cut; (1) one constant value
    (a plateau: every score ties); (2) continuous uniform values; (3) a
    plateau with a few distinct larger values and both +0.0 and -0.0.
    """
    out = []
    for b, n in enumerate(lens):
        g = _rng(seed, _SCORE_LAYER, b)
        kind = b % 4
        if kind == 0:
            s = g.integers(0, 64, size=n).astype(np.float32) / np.float32(16.0)
        elif kind == 1:
            s = np.full(n, np.float32(g.uniform(0.5, 2.0)), dtype=np.float32)
        elif kind == 2:
            s = g.uniform(0.0, 8.0, size=n).astype(np.float32)
        else:
            s = np.full(n, np.float32(1.0), dtype=np.float32)
            if n:
                hi = g.choice(n, size=min(n, 7), replace=False)
                s[hi] = g.uniform(2.0, 3.0, size=hi.size).astype(np.float32)
                z = g.choice(n, size=min(n, 4), replace=False)
                s[z[: len(z) // 2]] = np.float32(0.0)
                s[z[len(z) // 2:]] = np.float32(-0.0)
        out.append(s)
    return np.concatenate(out) if out else np.zeros(0, dtype=np.float32)


def to_storage(a: np.ndarray, dtype: str):
    """A CPU torch tensor holding ``a`` in the storage dtype ("f32"/"bf16").
    bf16 uses torch's round-to-nearest-even conversion from float32."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if dtype == "bf16":
        return t.to(torch.bfloat16)
    if dtype == "f32":
        return t
    raise ValueError(f"unknown dtype {dtype!r}")


def as_f64(t) -> np.ndarray:
    """Exact float64 copy of a CPU/GPU torch tensor (for the oracle)."""
    import torch
    return t.detach().to("cpu").to(torch.float64).numpy()
