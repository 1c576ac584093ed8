"""CPU oracle of the pruned transformer layer stack -- TEST INFRASTRUCTURE.

Plain, slow, float64 NumPy. Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this module; the product path (the
HIP library and its binding) never does, and shares no code with it.

What it computes (Kachuee & Sharifkhani, "Efficient Large Language Models
with Zero-Shot Adjustable Acceleration"):

* attention as in Eq. 1: softmax(Q K^T / sqrt(d_k) + M) V, with M = 0
  (bidirectional) or -inf on future positions (causal), Sec. 3.2;
* the contribution of hidden activation j to the layer output: the weight
  its V row receives from the softmax matrix (the "soft-score"), Sec. 3.2
  and 3.3. Reading used here: s_j = sum over heads h and query rows i of
  P_h[i, j] -- a plain column sum, no normalisation by the number of
  attending queries, no V-row norm;
* the number of rows kept at a pruning layer, Eq. 2:
  N_l = max(alpha * N_{l-1}, tau), with tau = 5 (Sec. 4.2); reading:
  floor(alpha*N + 1e-9) in float64, and never more than N;
* removal of the lowest-contribution rows, which then take no part in the
  later layers (Sec. 3.3). Reading: layer l runs fully on its N_{l-1} input
  rows, its output rows are ranked by (score desc, index asc), the first
  N_l are kept, they stay in their original order and keep their original
  positions (for RoPE and the causal mask).

The backbone (pre-norm residual block, LayerNorm or RMSNorm, GELU or
SwiGLU, RoPE) follows the common blueprint of Appendix A / Table 1; the
constants the paper leaves open (eps = 1e-5, RoPE theta = 1e4 with
rotate-half pairing (i, i + hd/2), SwiGLU gate/up rows interleaved) are
readings shared with the library's documented interface.

Grouped-query attention (the LLaMA 3 / Gemma 2 backbones of Table 1):
query head h reads key/value head h // (H / H_kv); H_kv = H is ordinary
multi-head attention and H_kv = 1 multi-query attention. The score still
sums the soft-score matrices of all H query heads.

``force_keep_last`` (a reading for generation, where the first new token is
predicted from the last input row): that row is always kept and the other
k - 1 rows are chosen by score as above.

``mark_only`` (the visualisation mode of Appendix B: rows "pruned but not
removed"): every row continues through every layer, so the hidden states
are those of the unpruned stack; each pruning point ranks all current rows
by score and marks the Eq. 2 count, compounded on the previous point's
marked count, as kept. A row marked pruned at one point can be marked kept
again later (reactivated).

``mode="exact"`` keeps everything in float64. ``mode="bf16"`` rounds to
bfloat16 (nearest-even) exactly where the GPU path stores bfloat16: norm
outputs, Q/K/V (after RoPE), attention output, MLP intermediate and the
residual stream after each add; and where it feeds bfloat16 to the matrix
cores without storing it: the attention probabilities (relative to the row
maximum, before the division by the row sum) in the P V product of a
prefill layer. A generated row's attention keeps them in float32.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np
from scipy.special import erf as _erf

ENCODER = 0
DECODER = 1


# ---------------------------------------------------------------------------
# Eq. 2: how many rows survive a pruning layer
# ---------------------------------------------------------------------------
def keep_count(n: int, alpha: float, tau: int = 5) -> int:
    """Eq. 2, N_l = max(alpha * N_{l-1}, tau_l), for one sequence.

    alpha*N is made an integer by flooring the float64 product after adding
    1e-9, so that decimal rates such as 0.57 * 100 give 57 rather than the
    56 that the raw IEEE product 56.99999... would floor to. The result
    never exceeds N (a sequence shorter than tau keeps every row).
    """
    if isinstance(alpha, float) and math.isnan(alpha):
        raise ValueError("keep rate is NaN")
    alpha = float(alpha)
    if not (0.0 <= alpha <= 1.0):
        raise ValueError(f"keep rate {alpha} outside [0, 1]")
    if tau < 1:
        raise ValueError("tau must be >= 1")
    if n < 0:
        raise ValueError("negative length")
    product = alpha * float(n)              # one IEEE double multiply
    kept = int(math.floor(product + 1e-9))  # one IEEE double add, then floor
    return min(int(n), max(kept, int(tau)))


def keep_schedule(lengths: Sequence[int], keep_rates: Sequence[float], tau: int,
                  n_prune: int) -> List[List[int]]:
    """Eq. 2 compounded over ``n_prune`` pruning points: entry p is the list
    of per-sequence counts after pruning point p (each relative to the count
    after point p-1)."""
    cur = [int(n) for n in lengths]
    out = []
    for _ in range(n_prune):
        cur = [keep_count(n, a, tau) for n, a in zip(cur, keep_rates)]
        out.append(list(cur))
    return out


# ---------------------------------------------------------------------------
# storage rounding used by the "bf16" emulation mode
# ---------------------------------------------------------------------------
def bf16_round(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (8 significant bits),
    ties to even, returned as float64. Valid for the normal bf16 range
    (|x| >= 2**-126), which is all this stack produces; +-inf and NaN pass
    through unchanged."""
    x = np.asarray(x, dtype=np.float64)
    mant, expo = np.frexp(x)                       # x = mant * 2**expo, 0.5 <= |mant| < 1
    return np.ldexp(np.rint(np.ldexp(mant, 8)), expo - 8)


def _identity(x):
    return x


def _rounder(mode: str):
    if mode == "exact":
        return _identity
    if mode == "bf16":
        return bf16_round
    raise ValueError(f"unknown mode {mode!r}")


# ---------------------------------------------------------------------------
# backbone pieces (Appendix A: pre-norm residual, LayerNorm, GELU/SwiGLU, RoPE)
# ---------------------------------------------------------------------------
def layer_norm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    """(x - mean) / sqrt(biased variance + eps) * g + b, over the last axis."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g, over the last axis."""
    ms = (x * x).mean(axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def gelu(z: np.ndarray) -> np.ndarray:
    """Exact GELU: z * Phi(z) = 0.5 z (1 + erf(z / sqrt 2))."""
    return 0.5 * z * (1.0 + _erf(z / math.sqrt(2.0)))


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def rope(x: np.ndarray, pos: np.ndarray, n_heads: int, theta: float) -> np.ndarray:
    """Rotary embedding on [n, n_heads*hd]: in every head, channel i and
    channel i + hd/2 (i < hd/2) form a pair rotated by the angle
    pos * theta**(-2i/hd)."""
    n, d = x.shape
    hd = d // n_heads
    half = hd // 2
    i = np.arange(half, dtype=np.float64)
    inv_freq = theta ** (-2.0 * i / hd)                       # [half]
    ang = pos.astype(np.float64)[:, None] * inv_freq[None, :]  # [n, half]
    c, s = np.cos(ang), np.sin(ang)
    out = np.empty_like(x)
    for h in range(n_heads):
        a = x[:, h * hd: h * hd + half]
        b = x[:, h * hd + half: (h + 1) * hd]
        out[:, h * hd: h * hd + half] = a * c - b * s
        out[:, h * hd + half: (h + 1) * hd] = b * c + a * s
    return out


# ---------------------------------------------------------------------------
# Eq. 1 attention and the soft-score contribution of each position
# ---------------------------------------------------------------------------
def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, pos: np.ndarray, n_heads: int,
              causal: bool, want_scores: bool = True, n_kv_heads: Optional[int] = None,
              p_round=None):
    """Eq. 1 for one sequence, per head, plus the column sums of the
    soft-score matrix (Sec. 3.2-3.3).

    q: [n, n_heads*hd]; k, v: [n, n_kv_heads*hd] (n_kv_heads divides
    n_heads; None means n_heads), query head h reading key/value head
    h // (n_heads // n_kv_heads). pos: [n] original positions; under the
    causal mask, row i may attend to row j iff pos[j] <= pos[i].
    Returns (o [n, d], lse [n_heads, n], s [n] or None) where lse is the
    natural-log log-sum-exp of each scaled, masked score row and
    s[j] = sum_h sum_i P_h[i, j].

    ``p_round`` (storage emulation only) rounds the unnormalised
    probabilities exp(S - row max) where they enter the P V product, which
    is then divided by the unrounded row sum; the scores and the
    log-sum-exp use the unrounded probabilities.
    """
    n, d = q.shape
    hd = d // n_heads
    hkv = n_heads if n_kv_heads is None else int(n_kv_heads)
    if hkv <= 0 or n_heads % hkv != 0 or k.shape[1] != hkv * hd or v.shape[1] != hkv * hd:
        raise ValueError("key/value heads do not divide the query heads")
    group = n_heads // hkv
    scale = 1.0 / math.sqrt(hd)
    o = np.zeros((n, d))
    lse = np.zeros((n_heads, n))
    s = np.zeros(n) if want_scores else None
    if n == 0:
        return o, lse, s
    future = pos[None, :] > pos[:, None]      # [i, j]: j is after i
    for h in range(n_heads):
        cols = slice(h * hd, (h + 1) * hd)
        kv = slice((h // group) * hd, (h // group + 1) * hd)
        S = (q[:, cols] @ k[:, kv].T) * scale
        if causal:
            S = np.where(future, -np.inf, S)   # M of Eq. 1
        row_max = S.max(axis=1, keepdims=True)
        E = np.exp(S - row_max)
        Z = E.sum(axis=1, keepdims=True)
        P = E / Z                               # the soft-score matrix of head h
        if p_round is None:
            o[:, cols] = P @ v[:, kv]
        else:
            o[:, cols] = (p_round(E) @ v[:, kv]) / Z
        lse[h] = row_max[:, 0] + np.log(Z[:, 0])
        if want_scores:
            s += P.sum(axis=0)                  # weight each V row receives
    return o, lse, s


def select_topk(s: np.ndarray, k: int, keep_last: bool = False) -> np.ndarray:
    """Indices of the k highest scores, ties going to the lower index
    (total order: score descending, then index ascending), returned in
    ascending index order. -0.0 and +0.0 compare equal. NaN is rejected.
    With ``keep_last`` the last index is always kept (if k >= 1) and the
    other k - 1 are the highest of the remaining scores."""
    s = np.asarray(s, dtype=np.float64)
    if np.isnan(s).any():
        raise ValueError("NaN score")
    n = s.shape[0]
    if not (0 <= k <= n):
        raise ValueError("k out of range")
    if keep_last and 1 <= k < n:
        rest = select_topk(s[:n - 1], k - 1)
        return np.concatenate([rest, [n - 1]]).astype(np.int64)
    idx = np.arange(n)
    order = np.lexsort((idx, -s))              # primary -s, secondary index
    return np.sort(order[:k])


# ---------------------------------------------------------------------------
# one layer and the stack
# ---------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class LayerCfg:
    kind: int            # ENCODER: pre-LN, biases, GELU; DECODER: RMSNorm, RoPE, SwiGLU
    d_model: int
    n_heads: int
    d_ff: int
    causal: bool
    norm_eps: float = 1e-5
    rope_theta: float = 10000.0
    tau: int = 5
    n_kv_heads: int = 0          # key/value heads (0: n_heads)
    force_keep_last: bool = False

    @property
    def kv_heads(self) -> int:
        return self.n_heads if self.n_kv_heads == 0 else self.n_kv_heads


def _linear(x, w, b):
    y = x @ w.T
    if b is not None:
        y = y + b
    return y


def sequence_layer(x: np.ndarray, pos: np.ndarray, w: Dict[str, Optional[np.ndarray]],
                   cfg: LayerCfg, mode: str = "exact", want_scores: bool = False) -> Dict:
    """One pre-norm block on one sequence (no pruning). Returns the output
    rows and the intermediates a test may compare."""
    r = _rounder(mode)
    d = cfg.d_model
    if cfg.kind == ENCODER:
        h = r(layer_norm(x, w["norm1_w"], w["norm1_b"], cfg.norm_eps))
    else:
        h = r(rms_norm(x, w["norm1_w"], cfg.norm_eps))
    qkv = _linear(h, w["w_qkv"], w["b_qkv"])
    kvd = cfg.kv_heads * (d // cfg.n_heads)
    q, k, v = qkv[:, :d], qkv[:, d:d + kvd], qkv[:, d + kvd:d + 2 * kvd]
    if cfg.kind == DECODER:
        q = rope(q, pos, cfg.n_heads, cfg.rope_theta)
        k = rope(k, pos, cfg.kv_heads, cfg.rope_theta)
    q, k, v = r(q), r(k), r(v)
    # under bf16 storage the probabilities also enter the P V product as
    # bf16 (the matrix-core operand); exact mode leaves them alone
    o, lse, s = attention(q, k, v, pos, cfg.n_heads, cfg.causal, want_scores, cfg.kv_heads,
                          p_round=None if mode == "exact" else r)
    o = r(o)
    x1 = r(x + _linear(o, w["w_o"], w["b_o"]))
    if cfg.kind == ENCODER:
        h2 = r(layer_norm(x1, w["norm2_w"], w["norm2_b"], cfg.norm_eps))
        f = r(gelu(_linear(h2, w["w_up"], w["b_up"])))
    else:
        h2 = r(rms_norm(x1, w["norm2_w"], cfg.norm_eps))
        z = _linear(h2, w["w_up"], w["b_up"])
        f = r(silu(z[:, 0::2]) * z[:, 1::2])   # rows 2f / 2f+1 = gate / up
    x2 = r(x1 + _linear(f, w["w_down"], w["b_down"]))
    return {"x": x2, "scores": s, "lse": lse, "q": q, "k": k, "v": v, "o": o,
            "h": h, "x_mid": x1, "f": f}


def layer_forward(x: np.ndarray, pos: np.ndarray, cu: Sequence[int], w: Dict,
                  cfg: LayerCfg, keep_rate: Optional[Sequence[float]] = None,
                  mode: str = "exact", kept_override: Optional[Sequence[np.ndarray]] = None,
                  keep_intermediates: bool = False, want_kv: bool = False,
                  want_scores: bool = False) -> Dict:
    """One layer over a packed batch ([T, d] rows, sequence b at rows
    cu[b]..cu[b+1]). With ``keep_rate`` (one rate per sequence) the layer is
    a pruning layer: its output rows are cut down to the Eq. 2 count by
    score (Sec. 3.3). ``kept_override[b]`` (local row indices) replaces the
    oracle's own choice, so a comparison can continue on another
    implementation's kept set."""
    cu = [int(c) for c in cu]
    B = len(cu) - 1
    prune = keep_rate is not None
    xs, ps, ss, kept_all, ks, lses, inter, kvs = [], [], [], [], [], [], [], []
    cu_out = [0]
    for b in range(B):
        lo, hi = cu[b], cu[b + 1]
        res = sequence_layer(x[lo:hi], pos[lo:hi], w, cfg, mode, want_scores=prune or want_scores)
        lses.append(res["lse"])
        if keep_intermediates or (want_scores and not prune):
            inter.append(res)
        if want_kv:
            kvs.append((res["k"], res["v"]))
        if prune:
            n = hi - lo
            kb = keep_count(n, float(keep_rate[b]), cfg.tau)
            if kept_override is not None:
                kept = np.asarray(kept_override[b], dtype=np.int64)
            else:
                kept = select_topk(res["scores"], kb, cfg.force_keep_last)
            ss.append(res["scores"])
            ks.append(kb)
            kept_all.append(kept + lo)
            xs.append(res["x"][kept])
            ps.append(pos[lo:hi][kept])
            cu_out.append(cu_out[-1] + len(kept))
        else:
            xs.append(res["x"])
            ps.append(pos[lo:hi])
            cu_out.append(cu_out[-1] + hi - lo)
    d = x.shape[1]
    out = {
        "x": np.concatenate(xs) if xs else np.zeros((0, d)),
        "pos": np.concatenate(ps) if ps else np.zeros(0, dtype=pos.dtype),
        "cu": np.asarray(cu_out, dtype=np.int64),
        "lse": np.concatenate(lses, axis=1) if lses else np.zeros((cfg.n_heads, 0)),
    }
    if want_scores and not prune:
        out["scores"] = np.concatenate([r["scores"] for r in inter]) if inter else np.zeros(0)
    if prune:
        out["scores"] = np.concatenate(ss) if ss else np.zeros(0)
        out["kept_rows"] = np.concatenate(kept_all) if kept_all else np.zeros(0, dtype=np.int64)
        out["k"] = ks
    if keep_intermediates:
        out["per_seq"] = inter
    if want_kv:
        out["kv"] = kvs
    return out


def stack_forward(x: np.ndarray, pos: np.ndarray, cu: Sequence[int], weights: Sequence[Dict],
                  cfg: LayerCfg, prune_after: Sequence[int], keep_rate: Sequence[float],
                  mode: str = "exact",
                  kept_override: Optional[Dict[int, Sequence[np.ndarray]]] = None,
                  record: bool = False, want_kv: bool = False, mark_only: bool = False) -> Dict:
    """The layer stack: layers 1..L in order; after each layer listed in
    ``prune_after`` (1-based) the output is pruned at the per-sequence keep
    rates. Returns the final rows, their original positions and row offsets,
    and per pruning point the scores, counts and kept positions.
    ``kept_override`` maps a 1-based layer index to per-sequence kept local
    indices. With ``record`` every layer's output is kept too. With
    ``want_kv`` the result holds, per layer and sequence, the keys and values
    (after RoPE) of the rows that entered that layer: the cache a decode step
    attends to. With ``mark_only`` nothing is removed: each pruning point
    marks its kept rows (``points``) and every row continues."""
    prune_set = set(int(p) for p in prune_after)
    cur_x, cur_pos, cur_cu = x, pos, np.asarray(cu, dtype=np.int64)
    points, layers, kv = [], [], []
    if mark_only:
        active = [int(cur_cu[b + 1] - cur_cu[b]) for b in range(len(cur_cu) - 1)]
        for l, w in enumerate(weights, start=1):
            pr = l in prune_set
            res = layer_forward(cur_x, cur_pos, cur_cu, w, cfg, None, mode, want_kv=want_kv,
                                want_scores=pr)
            if want_kv:
                kv.append(res["kv"])
            if pr:
                ks, kept_all, cu_k = [], [], [0]
                for b in range(len(active)):
                    lo, hi = int(cur_cu[b]), int(cur_cu[b + 1])
                    kb = keep_count(active[b], float(keep_rate[b]), cfg.tau)
                    ov = kept_override.get(l) if kept_override else None
                    kept = (np.asarray(ov[b], dtype=np.int64) if ov is not None else
                            select_topk(res["scores"][lo:hi], kb, cfg.force_keep_last))
                    active[b] = kb
                    ks.append(kb)
                    kept_all.append(kept + lo)
                    cu_k.append(cu_k[-1] + len(kept))
                kr = np.concatenate(kept_all) if kept_all else np.zeros(0, dtype=np.int64)
                points.append({"layer": l, "scores": res["scores"], "k": ks, "kept_rows": kr,
                               "pos": cur_pos[kr], "cu": np.asarray(cu_k, dtype=np.int64)})
            cur_x = res["x"]
            if record:
                layers.append({"x": cur_x, "pos": cur_pos, "cu": cur_cu})
        return {"x": cur_x, "pos": cur_pos, "cu": cur_cu, "points": points, "layers": layers,
                "kv": kv}
    for l, w in enumerate(weights, start=1):
        pr = l in prune_set
        ov = kept_override.get(l) if (kept_override and pr) else None
        res = layer_forward(cur_x, cur_pos, cur_cu, w, cfg, keep_rate if pr else None, mode, ov,
                            want_kv=want_kv)
        if want_kv:
            kv.append(res["kv"])
        if pr:
            points.append({"layer": l, "scores": res["scores"], "k": res["k"],
                           "kept_rows": res["kept_rows"], "pos": res["pos"], "cu": res["cu"]})
        cur_x, cur_pos, cur_cu = res["x"], res["pos"], res["cu"]
        if record:
            layers.append({"x": cur_x, "pos": cur_pos, "cu": cur_cu})
    return {"x": cur_x, "pos": cur_pos, "cu": cur_cu, "points": points, "layers": layers,
            "kv": kv}


# ---------------------------------------------------------------------------
# generation after a pruned prefill
# ---------------------------------------------------------------------------
def decode_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int,
                     n_kv_heads: Optional[int] = None) -> np.ndarray:
    """Eq. 1 for one new query row over m cached rows (all of them earlier
    positions, so the causal mask removes nothing): q [n_heads*hd], k, v
    [m, n_kv_heads*hd]; query head h reads key/value head
    h // (n_heads // n_kv_heads). Returns o [n_heads*hd]."""
    d = q.shape[0]
    hd = d // n_heads
    hkv = n_heads if n_kv_heads is None else int(n_kv_heads)
    group = n_heads // hkv
    o = np.zeros(d)
    for h in range(n_heads):
        g = h // group
        S = k[:, g * hd:(g + 1) * hd] @ q[h * hd:(h + 1) * hd] / math.sqrt(hd)
        P = np.exp(S - S.max())
        P /= P.sum()
        o[h * hd:(h + 1) * hd] = P @ v[:, g * hd:(g + 1) * hd]
    return o


def decode_step(x_new: np.ndarray, pos_new: np.ndarray, cache: List[List[tuple]],
                weights: Sequence[Dict], cfg: LayerCfg, mode: str = "exact") -> Dict:
    """One generated token per sequence through the stack (causal models).

    Reading: generated rows are never pruned; at layer l the new row of
    sequence b attends to the keys and values of the rows that entered
    layer l in the (pruned) prefill, plus every earlier generated row, plus
    itself. ``cache[l][b]`` = (k, v) of those earlier rows ([m, kvd] each,
    after RoPE); it is not modified. x_new [B, d], pos_new [B] (original
    position of the new row). Returns the new rows' outputs "x" [B, d] and,
    per layer and sequence, the (k, v) rows to append ("kv")."""
    if not cfg.causal:
        raise ValueError("decoding needs the causal mask")
    r = _rounder(mode)
    d = cfg.d_model
    kvd = cfg.kv_heads * (d // cfg.n_heads)
    x = np.asarray(x_new, dtype=np.float64)
    appended = []
    for l, w in enumerate(weights):
        x1s, new_kv = [], []
        for b in range(x.shape[0]):
            xb = x[b:b + 1]
            pb = np.asarray([pos_new[b]])
            if cfg.kind == ENCODER:
                h = r(layer_norm(xb, w["norm1_w"], w["norm1_b"], cfg.norm_eps))
            else:
                h = r(rms_norm(xb, w["norm1_w"], cfg.norm_eps))
            qkv = _linear(h, w["w_qkv"], w["b_qkv"])
            q, k, v = qkv[:, :d], qkv[:, d:d + kvd], qkv[:, d + kvd:d + 2 * kvd]
            if cfg.kind == DECODER:
                q = rope(q, pb, cfg.n_heads, cfg.rope_theta)
                k = rope(k, pb, cfg.kv_heads, cfg.rope_theta)
            q, k, v = r(q), r(k), r(v)
            ck, cv = cache[l][b]
            o = r(decode_attention(q[0], np.concatenate([ck, k]), np.concatenate([cv, v]),
                                   cfg.n_heads, cfg.kv_heads))
            x1s.append(r(xb[0] + _linear(o[None, :], w["w_o"], w["b_o"])[0]))
            new_kv.append((k, v))
        x1 = np.stack(x1s)
        if cfg.kind == ENCODER:
            h2 = r(layer_norm(x1, w["norm2_w"], w["norm2_b"], cfg.norm_eps))
            f = r(gelu(_linear(h2, w["w_up"], w["b_up"])))
        else:
            h2 = r(rms_norm(x1, w["norm2_w"], cfg.norm_eps))
            z = _linear(h2, w["w_up"], w["b_up"])
            f = r(silu(z[:, 0::2]) * z[:, 1::2])
        x = r(x1 + _linear(f, w["w_down"], w["b_down"]))
        appended.append(new_kv)
    return {"x": x, "kv": appended}
