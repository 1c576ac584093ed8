"""Planted mistakes in the oracle (on the CPU) must fail at least one pin.

Each case swaps one oracle function for a plausible wrong variant and runs
the pin that should catch it; the pin has to raise. This shows the pins are
not restating the oracle.
"""
import math

import numpy as np
import pytest

from oracle import zsa_oracle as O
from tests import test_oracle_pins as P


def _attention_no_scale(q, k, v, pos, n_heads, causal, want_scores=True, n_kv_heads=None,
                        p_round=None):
    return _orig_attention(q * math.sqrt(q.shape[1] // n_heads), k, v, pos, n_heads, causal,
                           want_scores, n_kv_heads, p_round)


def _attention_mask_excludes_diagonal(q, k, v, pos, n_heads, causal, want_scores=True,
                                      n_kv_heads=None, p_round=None):
    return _attention_shifted(q, k, v, pos, n_heads, want_scores)


def _attention_shifted(q, k, v, pos, n_heads, want_scores):
    n, d = q.shape
    hd = d // n_heads
    o = np.zeros((n, d))
    lse = np.zeros((n_heads, n))
    s = np.zeros(n)
    for h in range(n_heads):
        c = slice(h * hd, (h + 1) * hd)
        S = q[:, c] @ k[:, c].T / math.sqrt(hd)
        S = np.where(pos[None, :] >= pos[:, None] + 1, -np.inf, S)
        S[np.arange(1, n), np.arange(1, n)] = -np.inf          # drop the diagonal
        m = S.max(axis=1, keepdims=True)
        E = np.exp(S - m)
        Pm = E / E.sum(axis=1, keepdims=True)
        o[:, c] = Pm @ v[:, c]
        lse[h] = m[:, 0] + np.log(E.sum(axis=1))
        s += Pm.sum(axis=0)
    return o, lse, s


def _attention_row_sums(q, k, v, pos, n_heads, causal, want_scores=True, n_kv_heads=None,
                        p_round=None):
    o, lse, s = _orig_attention(q, k, v, pos, n_heads, causal, want_scores, n_kv_heads, p_round)
    if s is not None:
        s = np.full_like(s, float(n_heads))   # what summing each row (axis 1) gives
    return o, lse, s


def _attention_kv_modulo(q, k, v, pos, n_heads, causal, want_scores=True, n_kv_heads=None,
                         p_round=None):
    # query head h reads key/value head h % H_kv instead of h // (H / H_kv)
    hkv = n_heads if n_kv_heads is None else n_kv_heads
    hd = q.shape[1] // n_heads
    idx = np.concatenate([np.arange((h % hkv) * hd, (h % hkv + 1) * hd) for h in range(n_heads)])
    return _orig_attention(q, k[:, idx], v[:, idx], pos, n_heads, causal, want_scores,
                           p_round=p_round)


def _select_ignores_keep_last(s, k, keep_last=False):
    return _orig_select(s, k)


def _select_ties_high(s, k, keep_last=False):
    s = np.asarray(s, dtype=np.float64)
    idx = np.arange(s.shape[0])
    order = np.lexsort((-idx, -s))
    return np.sort(order[:k])


def _keep_count_round(n, alpha, tau=5):
    return min(int(n), max(int(round(alpha * n)), tau))


def _rope_adjacent(x, pos, n_heads, theta):
    n, d = x.shape
    hd = d // n_heads
    out = np.empty_like(x)
    for h in range(n_heads):
        for i in range(hd // 2):
            ang = pos.astype(np.float64) * theta ** (-2.0 * i / hd)
            a = x[:, h * hd + 2 * i]
            b = x[:, h * hd + 2 * i + 1]
            out[:, h * hd + 2 * i] = a * np.cos(ang) - b * np.sin(ang)
            out[:, h * hd + 2 * i + 1] = b * np.cos(ang) + a * np.sin(ang)
    return out


def _layer_norm_unbiased(x, g, b, eps):
    mu = x.mean(axis=-1, keepdims=True)
    var = x.var(axis=-1, ddof=1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def _gelu_tanh(z):
    return 0.5 * z * (1 + np.tanh(math.sqrt(2 / math.pi) * (z + 0.044715 * z ** 3)))


def _bf16_truncate(x):
    x = np.asarray(x, dtype=np.float64)
    mant, expo = np.frexp(x)
    return np.ldexp(np.trunc(np.ldexp(mant, 8)), expo - 8)


_orig_attention = O.attention
_orig_select = O.select_topk
_orig_decode_attention = O.decode_attention


def _decode_attention_skips_self(q, k, v, n_heads, n_kv_heads=None):
    # the new row does not attend to its own key/value
    return _orig_decode_attention(q, k[:-1], v[:-1], n_heads, n_kv_heads)

MUTANTS = [
    ("attention", _attention_no_scale, lambda: P.test_attention_brute_force(False)),
    ("attention", _attention_mask_excludes_diagonal, lambda: P.test_attention_brute_force(True)),
    ("attention", _attention_row_sums,
     lambda: P.test_scores_closed_form_uniform_attention(P.W.DECODER)),
    ("attention", _attention_kv_modulo, lambda: P.test_gqa_vs_torch_sdpa(True, 2)),
    ("select_topk", _select_ties_high, P.test_select_topk_brute_force),
    ("select_topk", _select_ignores_keep_last, P.test_select_topk_keep_last),
    ("decode_attention", _decode_attention_skips_self,
     lambda: P.test_decode_equals_forward_on_the_extended_sequence(P.W.DECODER, 2)),
    ("keep_count", _keep_count_round, P.test_keep_schedule_golden),
    ("rope", _rope_adjacent, P.test_rope_hand_example),
    ("layer_norm", _layer_norm_unbiased, P.test_layer_norm_vs_torch),
    ("gelu", _gelu_tanh, P.test_gelu_and_silu),
    ("bf16_round", _bf16_truncate, P.test_bf16_round_matches_torch_conversion),
]


@pytest.mark.parametrize("name,mutant,pin", MUTANTS, ids=[m[1].__name__ for m in MUTANTS])
def test_planted_mistake_is_caught(monkeypatch, name, mutant, pin):
    monkeypatch.setattr(O, name, mutant)
    with pytest.raises(AssertionError):
        pin()
