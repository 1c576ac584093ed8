"""Generation after a pruned prefill: the key/value cache the stack writes
and the decode step over it, against the oracle continued on the GPU's kept
sets (generated rows are never pruned)."""
import numpy as np
import pytest
import torch

from oracle import zsa_oracle as O
from paper_2509_01190_amd import workloads as W
from paper_2509_01190_amd import zsa
from tests.helpers import (SEQ_TOL, assert_rel_l2, assert_rows_vs_exact, dev, f64, row_errors,
                           to_dev, weights_f64)

from tests.test_gpu_stack import build, gpu_kept_overrides

TOL = SEQ_TOL["bf16"]


def check_rows(got, ref_x, ref_e, what):
    """Rows that each belong to another sequence (the generated row of every
    sequence, or one appended cache row): the per-sequence tolerance applies
    to every row, against the exact oracle; the emulation oracle only names
    what bf16 storage alone does, in the message."""
    for i in range(got.shape[0]):
        assert_rel_l2(got[i:i + 1], ref_x[i:i + 1], TOL,
                      f"{what} row {i} (bf16 storage alone: "
                      f"{row_errors(ref_e[i:i + 1], ref_x[i:i + 1])[0]:.3e})")

pytestmark = pytest.mark.gpu


CASES = [
    # kind, kv heads, pruning points, force_keep_last, head_dim
    (W.DECODER, 2, (1, 2), True, 64),
    (W.DECODER, 1, (2,), False, 128),
    (W.ENCODER, 0, (1,), True, 64),
    (W.DECODER, 4, (), False, 64),
]


@pytest.mark.parametrize("kind,hkv,prune,keep_last,hd", CASES)
def test_prefill_cache_and_decode(kind, hkv, prune, keep_last, hd):
    H = 4
    p = W.shrink(W.PRESETS["dec1b"], kind=kind, causal=True, n_layers=3, d_model=H * hd,
                 n_heads=H, d_ff=256, batch=3, prune_after=prune, n_kv_heads=hkv,
                 force_keep_last=keep_last)
    lens = [200, 33, 129]
    lens, stack, xd, posd, dws, ocfg = build(p, 6, lens, sharp=3.0)
    seqs = zsa.Seqs(lens, dev())
    rates = [0.5, 0.3, 0.7]
    cap = max(lens) + 3
    cache = stack.kv_cache(len(lens), cap, dev())
    out = stack.forward(xd, posd, seqs, p.prune_after, rates, debug=True, kv_cache=cache)
    torch.cuda.synchronize()
    kv_len = stack.kv_lengths(seqs, p.prune_after, rates)
    overrides = gpu_kept_overrides(p, lens, seqs, out) if prune else [{} for _ in lens]
    x_all = f64(xd)
    ws64 = [weights_f64(w) for w in dws]
    kvd = p.kv_heads * hd
    caches = {"exact": [], "bf16": []}
    for b, n in enumerate(lens):
        lo = int(seqs.host[b])
        for mode in caches:
            ref = O.stack_forward(x_all[lo:lo + n], np.arange(n), [0, n], ws64, ocfg, p.prune_after,
                                  [rates[b]], mode=mode, kept_override=overrides[b], want_kv=True)
            caches[mode].append([ref["kv"][l][0] for l in range(p.n_layers)])
    # the cache rows the prefill stored
    gc = f64(cache)
    for l in range(p.n_layers):
        for b in range(len(lens)):
            k_ref, v_ref = caches["bf16"][b][l]
            k_x, v_x = caches["exact"][b][l]
            m = int(kv_len[l, b])
            assert m == k_ref.shape[0]
            got = gc[l, b, :m]
            assert_rel_l2(got[:, :kvd], k_x, TOL, f"layer {l} seq {b} k")
            assert_rel_l2(got[:, kvd:], v_x, TOL, f"layer {l} seq {b} v")
            assert_rows_vs_exact(got[:, :kvd], k_x, k_ref, TOL, f"layer {l} seq {b} k")
            assert_rows_vs_exact(got[:, kvd:], v_x, v_ref, TOL, f"layer {l} seq {b} v")
    # two generated rows per sequence
    g = np.random.default_rng(17)
    ocache = {mode: [[caches[mode][b][l] for b in range(len(lens))] for l in range(p.n_layers)]
              for mode in caches}
    for step in range(2):
        x_new = to_dev(g.standard_normal((len(lens), p.d_model)).astype(np.float32), "bf16")
        pos_new = [n + step for n in lens]
        before = kv_len.copy()
        y = stack.decode_step(x_new, pos_new, cache, kv_len)
        y2 = stack.decode_step(x_new, pos_new, cache, before.copy())   # same rows again
        torch.cuda.synchronize()
        assert torch.equal(y, y2)
        assert np.array_equal(kv_len, before + 1)
        x64 = f64(x_new)
        res = {mode: O.decode_step(x64, np.array(pos_new), ocache[mode], ws64, ocfg, mode=mode)
               for mode in ocache}
        # one row per sequence: per-sequence relative L2 is per row
        check_rows(f64(y), res["exact"]["x"], res["bf16"]["x"], f"decode step {step}")
        gc = f64(cache)
        for l in range(p.n_layers):
            for b in range(len(lens)):
                nk, nv = res["bf16"]["kv"][l][b]
                xk, xv = res["exact"]["kv"][l][b]
                row = gc[l, b, before[l, b]]
                check_rows(row[None, :kvd], xk, nk, f"appended k, layer {l} seq {b}")
                check_rows(row[None, kvd:], xv, nv, f"appended v, layer {l} seq {b}")
        for mode in ocache:
            ocache[mode] = [[(np.concatenate([ocache[mode][l][b][0], res[mode]["kv"][l][b][0]]),
                              np.concatenate([ocache[mode][l][b][1], res[mode]["kv"][l][b][1]]))
                             for b in range(len(lens))] for l in range(p.n_layers)]


LONG_CASES = [
    # kind, query heads, key/value heads, head_dim, rows in layer 0's cache per sequence
    (W.DECODER, 8, 1, 128, [8500, 0, 300]),   # 8 query heads per cache head, 2 blocks per split
    (W.DECODER, 8, 2, 64, [1030, 1, 257]),
    (W.DECODER, 4, 4, 64, [700, 256, 255]),
    (W.ENCODER, 4, 0, 128, [3000, 9, 511]),
    (W.DECODER, 32, 8, 128, [600, 5, 0]),     # LLaMA-3-8B widths: d = 4096, 4 query heads per cache head
    (W.ENCODER, 16, 0, 128, [400, 1, 70]),    # d = 2048, LayerNorm
]


@pytest.mark.parametrize("kind,H,hkv,hd,kv0", LONG_CASES)
def test_decode_long_cache(kind, H, hkv, hd, kv0):
    """Decode steps over long caches given directly (random k / v rows, a
    second layer holding about half as many, as after pruning): several
    splits per (sequence, head group) merged in-kernel, several row blocks
    per split, splits past a short sequence's rows, and a cache holding
    only the new row. Two steps against the oracle continued on the GPU's
    cache, each step reproducible."""
    B = len(kv0)
    p = W.shrink(W.PRESETS["dec1b"], kind=kind, causal=True, n_layers=2, d_model=H * hd,
                 n_heads=H, d_ff=512, batch=B, prune_after=(), n_kv_heads=hkv)
    _, stack, _, _, dws, ocfg = build(p, 3, [8] * B, sharp=3.0)
    kvd = p.kv_heads * hd
    g = np.random.default_rng(sum(kv0) + hd)
    kv_len = np.array([kv0, [n // 2 for n in kv0]], dtype=np.int32)
    cap = int(kv_len.max()) + 3
    host = np.zeros((2, B, cap, 2 * kvd), np.float32)
    for l in range(2):
        for b, n in enumerate(kv_len[l]):
            host[l, b, :n, :kvd] = 2.0 * g.standard_normal((n, kvd))
            host[l, b, :n, kvd:] = g.standard_normal((n, kvd))
    cache = to_dev(host, "bf16").contiguous()
    ws64 = [weights_f64(w) for w in dws]
    for step in range(2):
        gc = f64(cache)
        ocache = [[(gc[l, b, :kv_len[l, b], :kvd], gc[l, b, :kv_len[l, b], kvd:])
                   for b in range(B)] for l in range(2)]
        x_new = to_dev(g.standard_normal((B, p.d_model)).astype(np.float32), "bf16")
        pos_new = [int(n) + step for n in kv0]
        before = kv_len.copy()
        y = stack.decode_step(x_new, pos_new, cache, kv_len)
        y2 = stack.decode_step(x_new, pos_new, cache, before.copy())
        torch.cuda.synchronize()
        assert torch.equal(y, y2)
        x64 = f64(x_new)
        res = {mode: O.decode_step(x64, np.array(pos_new), ocache, ws64, ocfg, mode=mode)
               for mode in ("exact", "bf16")}
        check_rows(f64(y), res["exact"]["x"], res["bf16"]["x"], f"decode step {step}")
        gc = f64(cache)
        for l in range(2):
            for b in range(B):
                nk, nv = res["bf16"]["kv"][l][b]
                xk, xv = res["exact"]["kv"][l][b]
                row = gc[l, b, before[l, b]]
                check_rows(row[None, :kvd], xk, nk, f"appended k, layer {l} seq {b}")
                check_rows(row[None, kvd:], xv, nv, f"appended v, layer {l} seq {b}")
                # rows before the new one are untouched
                old = np.concatenate([ocache[l][b][0], ocache[l][b][1]], axis=1)
                assert np.array_equal(gc[l, b, :before[l, b]], old)
