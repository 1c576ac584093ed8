"""Python binding of libzsa: argument marshalling only.

Every function here checks shapes, takes raw pointers out of torch tensors
(device memory) and numpy arrays (host metadata) and calls the C entry point
of the same name; all arithmetic runs in the library's HIP kernels. If the
library has not been built this module raises instead of doing anything
else.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libzsa.so")

OK, EINVAL, ESHAPE, EALIGN, EUNSUPPORTED, EWORKSPACE, EHIP = 0, -1, -2, -3, -4, -5, -6
F32, BF16 = 0, 1
ENCODER, DECODER = 0, 1
NORM_LAYER, NORM_RMS = 0, 1
EPI_NONE, EPI_GELU, EPI_SWIGLU, EPI_RESIDUAL, EPI_ROPE = 0, 1, 2, 3, 4
K_GEMM, K_ATTENTION, K_SCORE, K_SELECT, K_GATHER, K_NORM, K_MISC = range(7)
KCLASS_NAMES = ["gemm", "attention", "score", "select", "gather", "norm", "misc"]

_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_f32 = ctypes.c_float
_f64 = ctypes.c_double
_sz = ctypes.c_size_t
_pi32 = ctypes.POINTER(ctypes.c_int32)
_pf64 = ctypes.POINTER(ctypes.c_double)


class ZsaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libzsa error {code}: {msg}")
        self.code = code


class LayerCfg(ctypes.Structure):
    _fields_ = [("kind", _i32), ("d_model", _i32), ("n_heads", _i32), ("head_dim", _i32),
                ("d_ff", _i32), ("causal", _i32), ("dtype", _i32), ("tau", _i32),
                ("norm_eps", _f32), ("rope_theta", _f32), ("n_kv_heads", _i32),
                ("force_keep_last", _i32), ("mark_only", _i32)]


WEIGHT_NAMES = ["norm1_w", "norm1_b", "w_qkv", "b_qkv", "w_o", "b_o",
                "norm2_w", "norm2_b", "w_up", "b_up", "w_down", "b_down"]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, _vp) for n in WEIGHT_NAMES]


class LayerGrads(ctypes.Structure):
    _fields_ = [(n, _vp) for n in WEIGHT_NAMES]


_SIGS = {
    "zsa_last_error": (ctypes.c_char_p, []),
    "zsa_version": (ctypes.c_char_p, []),
    "zsa_keep_count": (ctypes.c_int, [_i32, _f64, _i32, _pi32]),
    "zsa_keep_schedule": (ctypes.c_int, [_i32, _pi32, _pf64, _i32, _i32, _pi32]),
    "zsa_norm": (ctypes.c_int, [_vp, _i32, _i32, _vp, _vp, _vp, _i32, _i32, _f32, _vp]),
    "zsa_linear": (ctypes.c_int, [_vp, _i32, _vp, _i32, _i32, _vp, _i32, _vp, _i32, _vp, _vp,
                                  _i32, _i32, _f32, _vp, _vp, _sz]),
    "zsa_linear_workspace_size": (_sz, [_i32, _i32, _i32, _i32]),
    "zsa_attention_with_scores": (ctypes.c_int, [_vp, _i32, _vp, _vp, _vp, _i64, _i32, _i32,
                                                 _i32, _i32, _f32, _i32, _pi32, _vp, _vp, _i64,
                                                 _vp, _vp, _vp, _sz]),
    "zsa_attention_workspace_size": (_sz, [_i32, _i32, _i32]),
    "zsa_attention_with_scores_static": (ctypes.c_int, [_vp, _i32, _vp, _vp, _vp, _i64, _i32, _i32,
                                                        _i32, _i32, ctypes.c_float, _i32, _pi32,
                                                        _vp, _vp, _i64, _vp, _vp]),
    "zsa_static_scratch_bytes": (_sz, []),
    "zsa_score_positions": (ctypes.c_int, [_vp, _i32, _vp, _vp, _i64, _vp, _i32, _i32, _i32,
                                           _i32, _f32, _i32, _pi32, _vp, _vp, _vp, _sz]),
    "zsa_score_workspace_size": (_sz, [_i32, _i32]),
    "zsa_select_topk": (ctypes.c_int, [_vp, _vp, _i32, _pi32, _vp, _pi32, _i32, _vp, _vp, _sz]),
    "zsa_select_workspace_size": (_sz, [_i32]),
    "zsa_compact_gather": (ctypes.c_int, [_vp, _i32, _vp, _i32, _vp, _i32, _vp, _i32, _vp, _vp]),
    "zsa_layer_forward": (ctypes.c_int, [_vp, ctypes.POINTER(LayerCfg),
                                         ctypes.POINTER(LayerWeights), _vp, _vp, _i32, _pi32, _vp,
                                         _pf64, _vp, _vp, _pi32, _vp, _vp, _vp, _vp, _sz]),
    "zsa_layer_workspace_size": (_sz, [ctypes.POINTER(LayerCfg), _i32, _i32]),
    "zsa_stack_forward": (ctypes.c_int, [_vp, ctypes.POINTER(LayerCfg),
                                         ctypes.POINTER(LayerWeights), _i32, _pi32, _i32, _pf64,
                                         _vp, _vp, _i32, _pi32, _vp, _vp, _vp, _pi32, _vp, _pi32,
                                         _vp, _vp, _vp, _vp, _i32, _vp, _sz]),
    "zsa_decode_step": (ctypes.c_int, [_vp, ctypes.POINTER(LayerCfg), ctypes.POINTER(LayerWeights),
                                       _i32, _i32, _vp, _pi32, _vp, _i32, _pi32, _vp, _vp, _sz]),
    "zsa_decode_workspace_size": (_sz, [ctypes.POINTER(LayerCfg), _i32, _i32, _i32]),
    "zsa_stack_backward": (ctypes.c_int, [_vp, ctypes.POINTER(LayerCfg),
                                          ctypes.POINTER(LayerWeights), ctypes.POINTER(LayerGrads),
                                          _i32, _pi32, _i32, _pf64, _vp, _vp, _i32, _pi32, _vp,
                                          _vp, _vp, _vp, _sz]),
    "zsa_stack_backward_workspace_size": (_sz, [ctypes.POINTER(LayerCfg), _i32, _i32, _i32, _i32]),
    "zsa_stack_workspace_size": (_sz, [ctypes.POINTER(LayerCfg), _i32, _i32, _i32]),
    "zsa_timing_arm": (ctypes.c_int, [_i32, _i32]),
    "zsa_timing_read": (ctypes.c_int, [_i32, _pi32, ctypes.POINTER(ctypes.c_double)]),
}

EXPORTED = sorted(_SIGS)
_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               f"(python -m paper_2509_01190_amd._build)")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(l, name)
            fn.restype = res
            fn.argtypes = args
        _lib = l
    return _lib


def _check(rc: int) -> None:
    if rc != OK:
        raise ZsaError(rc, lib().zsa_last_error().decode())


def _p(t: Optional[torch.Tensor]):
    return None if t is None else _vp(t.data_ptr())


def _stream(dev: Optional[torch.device] = None):
    return _vp(torch.cuda.current_stream(dev).cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _host_i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _host_f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _hp32(a: np.ndarray):
    return a.ctypes.data_as(_pi32)


def _hpf64(a: np.ndarray):
    return a.ctypes.data_as(_pf64)


def _require_cuda(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("expected a device tensor")


class Seqs:
    """Packed sequence offsets, held on the host and on the device."""

    def __init__(self, lengths: Sequence[int], device="cuda"):
        cu = np.zeros(len(lengths) + 1, dtype=np.int64)
        cu[1:] = np.cumsum(np.asarray(lengths, dtype=np.int64))
        self.host = cu.astype(np.int32)
        self.dev = torch.from_numpy(self.host.copy()).to(device)
        self.batch = len(lengths)
        self.total = int(self.host[-1])

    @classmethod
    def from_cu(cls, cu, device="cuda"):
        cu = np.asarray(cu, dtype=np.int64)
        return cls(np.diff(cu), device)

    @property
    def lengths(self) -> List[int]:
        return [int(v) for v in np.diff(self.host)]


# ------------------------------------------------------------------ host helpers
def version() -> str:
    return lib().zsa_version().decode()


def keep_count(n: int, keep_rate: float, tau: int = 5) -> int:
    out = ctypes.c_int32()
    _check(lib().zsa_keep_count(int(n), float(keep_rate), int(tau), ctypes.byref(out)))
    return out.value


def keep_schedule(lengths, keep_rates, tau: int, n_points: int) -> np.ndarray:
    ln = _host_i32(lengths)
    kr = _host_f64(keep_rates)
    out = np.zeros((n_points, len(ln)), dtype=np.int32)
    _check(lib().zsa_keep_schedule(len(ln), _hp32(ln), _hpf64(kr), int(tau), int(n_points),
                                   _hp32(out)))
    return out


# ------------------------------------------------------------------ device ops
def norm(x: torch.Tensor, gain: torch.Tensor, shift: Optional[torch.Tensor], kind: int,
         eps: float = 1e-5, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    _require_cuda(x, gain, shift)
    rows, d = x.shape
    y = torch.empty_like(x) if out is None else out
    _check(lib().zsa_norm(_stream(x.device), _dtype_code(x), kind, _p(x), _p(gain), _p(shift),
                          rows, d, eps, _p(y)))
    return y


def linear_workspace_size(dtype: int, m: int, n: int, k: int) -> int:
    return int(lib().zsa_linear_workspace_size(dtype, m, n, k))


def linear(x: torch.Tensor, w: torch.Tensor, bias: Optional[torch.Tensor] = None,
           epilogue: int = EPI_NONE, residual: Optional[torch.Tensor] = None,
           pos: Optional[torch.Tensor] = None, head_dim: int = 0, rope_cols: int = 0,
           rope_theta: float = 10000.0, out: Optional[torch.Tensor] = None,
           split: bool = True, ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """y = epilogue(x w^T + bias). With ``split`` (and no ``ws``) a split-K
    workspace is allocated when the shape asks for one; ``split=False``
    never splits K."""
    _require_cuda(x, w, bias, residual, pos)
    m, k = x.shape
    n, k2 = w.shape
    if k2 != k:
        raise ValueError("inner dimensions differ")
    ncols = n // 2 if epilogue == EPI_SWIGLU else n
    y = torch.empty((m, ncols), dtype=x.dtype, device=x.device) if out is None else out
    if ws is None and split:
        need = linear_workspace_size(_dtype_code(x), m, n, k)
        if epilogue == EPI_ROPE and _dtype_code(x) == BF16 and m > 0:
            # room for the per-row rotary table past the split-K partials
            need = (need + 255) // 256 * 256 + m * head_dim * 4
        if need:
            ws = torch.empty(need, dtype=torch.uint8, device=x.device)
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().zsa_linear(_stream(x.device), _dtype_code(x), _p(x), m, k, _p(w), n, _p(bias),
                            epilogue, _p(residual), _p(pos), head_dim, rope_cols, rope_theta,
                            _p(y), _p(ws), ws_bytes))
    return y


def attention_with_scores(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, n_heads: int,
                          seqs: Seqs, causal: bool, want_lse: bool = True,
                          want_scores: bool = True, scale: Optional[float] = None,
                          n_kv_heads: int = 0):
    """q: [T, n_heads*hd], k, v: [T, n_kv_heads*hd] views sharing one row
    stride (e.g. slices of one fused [T, (n_heads + 2 n_kv_heads) hd]
    tensor); n_kv_heads 0 means n_heads. Returns (out, lse or None, scores
    or None)."""
    _require_cuda(q, k, v)
    T, width = q.shape
    hd = width // n_heads
    # no rows: nothing is read, and torch may give empty views any strides
    rs = q.stride(0) if T > 0 else width
    if T > 0 and (k.stride(0) != rs or v.stride(0) != rs or q.stride(1) != 1):
        raise ValueError("q, k, v must share one row stride")
    if scale is None:
        scale = 1.0 / float(np.sqrt(hd))
    out = torch.empty((T, width), dtype=q.dtype, device=q.device)
    lse = torch.empty((n_heads, T), dtype=torch.float32, device=q.device) if want_lse else None
    scores = torch.empty(T, dtype=torch.float32, device=q.device) if want_scores else None
    wsz = lib().zsa_attention_workspace_size(n_heads, T, int(want_scores))
    ws = torch.empty(max(int(wsz), 1), dtype=torch.uint8, device=q.device)
    _check(lib().zsa_attention_with_scores(
        _stream(q.device), _dtype_code(q), _p(q), _p(k), _p(v), rs, n_heads, n_kv_heads, hd,
        int(causal), scale, seqs.batch, _hp32(seqs.host), _p(seqs.dev), _p(out), width, _p(lse),
        _p(scores), _p(ws), wsz))
    return out, lse, scores


def score_positions(q: torch.Tensor, k: torch.Tensor, lse: torch.Tensor, n_heads: int,
                    seqs: Seqs, causal: bool, scale: Optional[float] = None,
                    n_kv_heads: int = 0) -> torch.Tensor:
    _require_cuda(q, k, lse)
    T, width = q.shape
    hd = width // n_heads
    rs = q.stride(0) if T > 0 else width
    if T > 0 and k.stride(0) != rs:
        raise ValueError("q and k must share one row stride")
    if scale is None:
        scale = 1.0 / float(np.sqrt(hd))
    scores = torch.empty(T, dtype=torch.float32, device=q.device)
    wsz = lib().zsa_score_workspace_size(n_heads, T)
    ws = torch.empty(max(int(wsz), 1), dtype=torch.uint8, device=q.device)
    _check(lib().zsa_score_positions(
        _stream(q.device), _dtype_code(q), _p(q), _p(k), rs, _p(lse), n_heads, n_kv_heads, hd,
        int(causal), scale, seqs.batch, _hp32(seqs.host), _p(seqs.dev), _p(scores), _p(ws), wsz))
    return scores


def select_topk(scores: torch.Tensor, seqs: Seqs, k, keep_last: bool = False) -> torch.Tensor:
    _require_cuda(scores)
    kh = _host_i32(k)
    kept = torch.empty(max(int(kh.sum()), 1), dtype=torch.int32, device=scores.device)
    wsz = lib().zsa_select_workspace_size(seqs.batch)
    ws = torch.empty(max(int(wsz), 1), dtype=torch.uint8, device=scores.device)
    _check(lib().zsa_select_topk(_stream(scores.device), _p(scores), seqs.batch,
                                 _hp32(seqs.host), _p(seqs.dev), _hp32(kh), int(keep_last),
                                 _p(kept), _p(ws), wsz))
    return kept[: int(kh.sum())]


def compact_gather(hidden: torch.Tensor, pos: Optional[torch.Tensor],
                   kept_rows: torch.Tensor):
    _require_cuda(hidden, pos, kept_rows)
    t_in, d = hidden.shape
    t_out = kept_rows.shape[0]
    out = torch.empty((t_out, d), dtype=hidden.dtype, device=hidden.device)
    pos_out = None if pos is None else torch.empty(t_out, dtype=torch.int32, device=hidden.device)
    _check(lib().zsa_compact_gather(_stream(hidden.device), _dtype_code(hidden), _p(hidden), d,
                                    _p(pos), t_in, _p(kept_rows), t_out, _p(out), _p(pos_out)))
    return out, pos_out


# ------------------------------------------------------------------ blocks
def make_cfg(kind: int, d_model: int, n_heads: int, d_ff: int, causal: bool, dtype: int,
             tau: int = 5, norm_eps: float = 1e-5, rope_theta: float = 10000.0,
             n_kv_heads: int = 0, force_keep_last: bool = False,
             mark_only: bool = False) -> LayerCfg:
    return LayerCfg(kind, d_model, n_heads, d_model // n_heads, d_ff, int(causal), dtype, tau,
                    norm_eps, rope_theta, n_kv_heads, int(force_keep_last), int(mark_only))


def weight_shapes(cfg: LayerCfg) -> Dict[str, tuple]:
    """Shape of every weight of one block under ``cfg`` (PyTorch Linear
    layout; the fused projection is [q | k | v] with grouped-query k/v)."""
    d, hd, F = cfg.d_model, cfg.head_dim, cfg.d_ff
    kv = cfg.n_kv_heads or cfg.n_heads
    qkv = d + 2 * kv * hd
    up = 2 * F if cfg.kind == DECODER else F
    return {"norm1_w": (d,), "norm1_b": (d,), "w_qkv": (qkv, d), "b_qkv": (qkv,),
            "w_o": (d, d), "b_o": (d,), "norm2_w": (d,), "norm2_b": (d,),
            "w_up": (up, d), "b_up": (up,), "w_down": (d, F), "b_down": (d,)}


def _check_weight_shapes(cfg: LayerCfg, w: Dict[str, Optional[torch.Tensor]], layer: int) -> None:
    # the library takes raw pointers: a wrongly sized weight would be read out
    # of bounds, so shapes are checked here, before any launch
    required = {"norm1_w", "w_qkv", "w_o", "norm2_w", "w_up", "w_down"}
    for name, shape in weight_shapes(cfg).items():
        t = w.get(name)
        if t is None:
            if name in required:
                raise ValueError(f"layer {layer}: {name} is missing")
            continue
        if tuple(t.shape) != shape or not t.is_contiguous():
            raise ValueError(f"layer {layer}: {name} has shape {tuple(t.shape)}, "
                             f"expected contiguous {shape}")


def _weights_struct(w: Dict[str, Optional[torch.Tensor]]) -> LayerWeights:
    return LayerWeights(*[None if w.get(n) is None else w[n].data_ptr() for n in WEIGHT_NAMES])


class Stack:
    """Device weights of a layer stack plus its configuration.

    ``weights`` is a list of dicts (names as in LayerWeights) of contiguous
    device tensors in the storage dtype."""

    def __init__(self, cfg: LayerCfg, weights: List[Dict[str, Optional[torch.Tensor]]]):
        for l, w in enumerate(weights):
            _check_weight_shapes(cfg, w, l)
        self.cfg = cfg
        self.weights = weights
        self._wstructs = (LayerWeights * len(weights))(*[_weights_struct(w) for w in weights])
        self._ws: Optional[torch.Tensor] = None

    @property
    def n_layers(self) -> int:
        return len(self.weights)

    def workspace(self, total_rows: int, batch: int, n_prune: int, device) -> torch.Tensor:
        need = int(lib().zsa_stack_workspace_size(ctypes.byref(self.cfg), total_rows, batch,
                                                  n_prune))
        if self._ws is None or self._ws.numel() < need or self._ws.device != torch.device(device):
            self._ws = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
        return self._ws

    def layer_forward(self, layer: int, hidden: torch.Tensor, pos: torch.Tensor, seqs: Seqs,
                      keep_rate=None, want_scores: bool = False, want_kept: bool = False):
        """One block (0-based ``layer``); returns a dict with x, pos, seqs
        and optionally scores / kept_rows."""
        _require_cuda(hidden, pos)
        dev = hidden.device
        T = seqs.total
        t_kept = T
        if keep_rate is not None:
            kr = _host_f64(keep_rate)
            counts = keep_schedule(seqs.lengths, kr, self.cfg.tau, 1)[0]
            t_kept = int(counts.sum())
            kr_p = _hpf64(kr)
        else:
            kr_p = None
        t_out = T if self.cfg.mark_only else t_kept     # mark-only keeps every row
        x_out = torch.empty((max(t_out, 1), self.cfg.d_model), dtype=hidden.dtype, device=dev)
        pos_out = torch.empty(max(t_out, 1), dtype=torch.int32, device=dev)
        cu_out = np.zeros(seqs.batch + 1, dtype=np.int32)
        cu_out_dev = torch.empty(seqs.batch + 1, dtype=torch.int32, device=dev)
        scores = torch.empty(max(T, 1), dtype=torch.float32, device=dev) if want_scores else None
        kept = torch.empty(max(t_kept, 1), dtype=torch.int32, device=dev) if want_kept else None
        wsz = int(lib().zsa_layer_workspace_size(ctypes.byref(self.cfg), T, seqs.batch))
        ws = torch.empty(max(wsz, 1), dtype=torch.uint8, device=dev)
        w = _weights_struct(self.weights[layer])
        _check(lib().zsa_layer_forward(
            _stream(dev), ctypes.byref(self.cfg), ctypes.byref(w), _p(hidden), _p(pos),
            seqs.batch, _hp32(seqs.host), _p(seqs.dev), kr_p, _p(x_out), _p(pos_out),
            _hp32(cu_out), _p(cu_out_dev), _p(scores), _p(kept), _p(ws), wsz))
        out_seqs = Seqs.from_cu(cu_out, dev)
        res = {"x": x_out[:t_out], "pos": pos_out[:t_out], "seqs": out_seqs,
               "cu_dev": cu_out_dev}
        if want_scores:
            res["scores"] = scores[:T]
        if want_kept:
            res["kept_rows"] = kept[:t_kept]
        return res

    def plan(self, seqs: Seqs, prune_after: Sequence[int], keep_rate) -> Dict:
        """Host-side shapes of a stack call (the Eq. 2 schedule)."""
        kr = _host_f64(keep_rate)
        counts = keep_schedule(seqs.lengths, kr, self.cfg.tau, len(prune_after))
        marked = [int(c.sum()) for c in counts]
        if self.cfg.mark_only:        # rows are marked, not removed
            return {"counts": counts, "final_rows": seqs.total, "marked": marked,
                    "rows_in": [seqs.total] * (len(marked) + 1)}
        final = marked[-1] if len(prune_after) else seqs.total
        rows_in = [seqs.total] + marked
        return {"counts": counts, "final_rows": final, "rows_in": rows_in, "marked": marked}

    def layer_out_rows(self, seqs: Seqs, prune_after: Sequence[int], keep_rate) -> List[int]:
        """Rows leaving each block of a stack call (the row counts of the
        per-block debug output)."""
        plan = self.plan(seqs, prune_after, keep_rate)
        pset = list(prune_after)
        out, point = [], 0
        cur = seqs.total
        for l in range(1, self.n_layers + 1):
            if point < len(pset) and pset[point] == l:
                point += 1
                if not self.cfg.mark_only:
                    cur = plan["rows_in"][point]
            out.append(cur)
        return out

    def kv_cache(self, batch: int, capacity: int, device) -> torch.Tensor:
        """An empty key/value cache [layers, batch, capacity, 2 * kvd]."""
        kvd = (self.cfg.n_kv_heads or self.cfg.n_heads) * self.cfg.head_dim
        dtype = torch.bfloat16 if self.cfg.dtype == BF16 else torch.float32
        return torch.empty((self.n_layers, batch, capacity, 2 * kvd), dtype=dtype, device=device)

    def kv_lengths(self, seqs: Seqs, prune_after: Sequence[int], keep_rate) -> np.ndarray:
        """Rows each sequence has in each layer's cache after a prefill:
        [layers, batch] int32 (the count after the last pruning point before
        the layer)."""
        counts = self.plan(seqs, prune_after, keep_rate)["counts"]
        cur = np.asarray(seqs.lengths, dtype=np.int32)
        out = np.zeros((self.n_layers, seqs.batch), dtype=np.int32)
        pset = list(prune_after)
        point = 0
        for l in range(1, self.n_layers + 1):
            out[l - 1] = cur
            if point < len(pset) and pset[point] == l:
                cur = np.asarray(counts[point], dtype=np.int32)
                point += 1
        return out

    def backward(self, hidden: torch.Tensor, pos: torch.Tensor, seqs: Seqs,
                 prune_after: Sequence[int], keep_rate, dy: torch.Tensor):
        """Gradients of sum(forward(...)["x"] * dy): returns (dx, grads) with
        grads[l][name] fp32 tensors shaped like the weights (None where the
        weight is absent). The kept rows are constants."""
        _require_cuda(hidden, pos, dy)
        dev = hidden.device
        pa = _host_i32(prune_after)
        kr = _host_f64(keep_rate)
        shapes = weight_shapes(self.cfg)
        grads = []
        for w in self.weights:
            grads.append({n: (None if w.get(n) is None else
                              torch.empty(shapes[n], dtype=torch.float32, device=dev))
                          for n in WEIGHT_NAMES})
        gstructs = (LayerGrads * len(grads))(
            *[LayerGrads(*[None if g[n] is None else g[n].data_ptr() for n in WEIGHT_NAMES])
              for g in grads])
        dx = torch.empty_like(hidden)
        wsz = int(lib().zsa_stack_backward_workspace_size(ctypes.byref(self.cfg), seqs.total,
                                                          seqs.batch, self.n_layers, len(pa)))
        ws = torch.empty(max(wsz, 1), dtype=torch.uint8, device=dev)
        _check(lib().zsa_stack_backward(
            _stream(dev), ctypes.byref(self.cfg), self._wstructs, gstructs, self.n_layers,
            _hp32(pa), len(pa), _hpf64(kr), _p(hidden), _p(pos), seqs.batch, _hp32(seqs.host),
            _p(seqs.dev), _p(dy), _p(dx), _p(ws), wsz))
        return dx, grads

    def decode_step(self, x_new: torch.Tensor, pos_new, kv_cache: torch.Tensor,
                    kv_len: np.ndarray, out: Optional[torch.Tensor] = None) -> torch.Tensor:
        """One generated row per sequence (x_new [batch, d]) at original
        positions pos_new; appends its k / v to kv_cache at rows kv_len
        ([layers, batch] host, incremented in place) and returns the
        outputs [batch, d]."""
        _require_cuda(x_new, kv_cache)
        batch = x_new.shape[0]
        if kv_cache.shape[:2] != (self.n_layers, batch) or not kv_cache.is_contiguous():
            raise ValueError("kv_cache must be a contiguous [layers, batch, capacity, 2*kvd] tensor")
        cap = kv_cache.shape[2]
        lens = np.ascontiguousarray(kv_len, dtype=np.int32)
        if lens.shape != (self.n_layers, batch):
            raise ValueError("kv_len must be [layers, batch]")
        y = torch.empty_like(x_new) if out is None else out
        wsz = int(lib().zsa_decode_workspace_size(ctypes.byref(self.cfg), self.n_layers, batch,
                                                  cap))
        ws = torch.empty(max(wsz, 1), dtype=torch.uint8, device=x_new.device)
        _check(lib().zsa_decode_step(_stream(x_new.device), ctypes.byref(self.cfg), self._wstructs,
                                     self.n_layers, batch, _p(x_new), _hp32(_host_i32(pos_new)),
                                     _p(kv_cache), cap, _hp32(lens), _p(y), _p(ws), wsz))
        kv_len += 1
        return y

    def forward(self, hidden: torch.Tensor, pos: torch.Tensor, seqs: Seqs,
                prune_after: Sequence[int], keep_rate, debug: bool = False,
                out: Optional[Dict] = None, kv_cache: Optional[torch.Tensor] = None) -> Dict:
        """The whole stack. With ``out`` (a dict from a previous call with the
        same shapes) the outputs are written into its tensors again, so the
        call allocates nothing and may be captured in a HIP graph. With
        ``kv_cache`` (from ``kv_cache()``) every layer's keys and values are
        stored for decoding."""
        _require_cuda(hidden, pos)
        dev = hidden.device
        pa = _host_i32(prune_after)
        kr = _host_f64(keep_rate)
        if out is None:
            plan = self.plan(seqs, pa, kr)
            t_fin = plan["final_rows"]
            out = {
                "x": torch.empty((max(t_fin, 1), self.cfg.d_model), dtype=hidden.dtype, device=dev),
                "pos": torch.empty(max(t_fin, 1), dtype=torch.int32, device=dev),
                "cu_host": np.zeros(seqs.batch + 1, dtype=np.int32),
                "cu_dev": torch.empty(seqs.batch + 1, dtype=torch.int32, device=dev),
                "counts": np.zeros((len(pa), seqs.batch), dtype=np.int32),
                "t_final": t_fin,
                "ws": self.workspace(seqs.total, seqs.batch, len(pa), dev),
                "pa": pa, "kr": kr,
            }
            if debug:
                sc_rows = sum(plan["rows_in"][:len(pa)])
                pos_rows = sum(plan["marked"])
                out["scores_dbg"] = torch.empty(max(sc_rows, 1), dtype=torch.float32, device=dev)
                out["pos_dbg"] = torch.empty(max(pos_rows, 1), dtype=torch.int32, device=dev)
                out["rows_in"] = plan["rows_in"]
                # every block's output rows, concatenated in block order
                out["layer_rows"] = self.layer_out_rows(seqs, pa, kr)
                out["hidden_dbg"] = torch.empty((max(sum(out["layer_rows"]), 1), self.cfg.d_model),
                                                dtype=hidden.dtype, device=dev)
        ws = out["ws"]
        _check(lib().zsa_stack_forward(
            _stream(dev), ctypes.byref(self.cfg), self._wstructs, self.n_layers,
            _hp32(out["pa"]), len(out["pa"]), _hpf64(out["kr"]), _p(hidden), _p(pos),
            seqs.batch, _hp32(seqs.host), _p(seqs.dev), _p(out["x"]), _p(out["pos"]),
            _hp32(out["cu_host"]), _p(out["cu_dev"]),
            _hp32(out["counts"]) if len(out["pa"]) else None,
            _p(out.get("scores_dbg")), _p(out.get("pos_dbg")), _p(out.get("hidden_dbg")),
            _p(kv_cache),
            0 if kv_cache is None else kv_cache.shape[2], _p(ws), ws.numel()))
        return out


# ------------------------------------------------------------------ timing hook
def timing_arm(kclass: int, capacity: int) -> None:
    _check(lib().zsa_timing_arm(kclass, capacity))


def timing_read(kclass: int):
    n = ctypes.c_int32()
    ms = ctypes.c_double()
    _check(lib().zsa_timing_read(kclass, ctypes.byref(n), ctypes.byref(ms)))
    return n.value, ms.value
