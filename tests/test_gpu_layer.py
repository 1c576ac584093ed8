"""One pre-norm block through zsa_layer_forward against the oracle, with and
without pruning, encoder and decoder, fp32 and bf16, ragged batches."""
import numpy as np
import pytest
import torch

from oracle import zsa_oracle as O
from paper_2509_01190_amd import workloads as W
from paper_2509_01190_amd import zsa
from tests.helpers import (SEQ_TOL, assert_close, assert_rel_l2, check_kept_sets, dev,
                           dev_weights, f64, modes, score_eps, to_dev, weights_f64)

pytestmark = pytest.mark.gpu

# (name, kind, dtype, d, H, F)
CASES = [
    ("enc_bf16_hd64", W.ENCODER, "bf16", 256, 4, 512),
    ("dec_bf16_hd128", W.DECODER, "bf16", 256, 2, 384),
    ("dec_bf16_hd64", W.DECODER, "bf16", 512, 8, 256),
    ("enc_f32_hd32", W.ENCODER, "f32", 128, 4, 512),
    ("dec_f32_hd32", W.DECODER, "f32", 128, 4, 256),
]


def _setup(kind, dtype, d, H, F, lens, seed, sharp=None):
    # query/key weights are scaled up so attention is far from uniform: score
    # logits reach a std of ~10 in fp32 and ~1-2 in bf16 (random-init N(0,
    # 0.02) weights give 0.3-1.6 at the benchmark shapes); at std ~20 single
    # bf16 rounding flips of recomputed Q/K alone move scores by ~1e-2
    if sharp is None:
        sharp = 10.0 if dtype == "f32" else 3.0
    causal = kind == W.DECODER
    p = W.shrink(W.PRESETS["tiny"], kind=kind, causal=causal, n_layers=1, d_model=d, n_heads=H,
                 d_ff=F, dtype=dtype, batch=len(lens))
    w = W.layer_weights(p, 0, seed, norm_jitter=True)
    w["w_qkv"] = (w["w_qkv"] * np.float32(sharp)).astype(np.float32)
    x = W.hidden(p, seed, lens)
    wd = dev_weights(w, dtype)
    cfg = zsa.make_cfg(kind, d, H, F, causal, zsa.BF16 if dtype == "bf16" else zsa.F32)
    stack = zsa.Stack(cfg, [wd])
    xd = to_dev(x, dtype)
    ocfg = O.LayerCfg(kind, d, H, F, causal)
    return p, stack, xd, wd, ocfg


@pytest.mark.parametrize("name,kind,dtype,d,H,F", CASES, ids=[c[0] for c in CASES])
@pytest.mark.parametrize("prune", [False, True])
def test_layer_forward(name, kind, dtype, d, H, F, prune):
    lens = [5, 64, 150, 257, 1]
    rates = [0.5, 0.3, 0.9, 1.0, 0.2]
    p, stack, xd, wd, ocfg = _setup(kind, dtype, d, H, F, lens, seed=31)
    seqs = zsa.Seqs(lens, dev())
    # non-trivial original positions: a pruned earlier layer left gaps
    pos = np.concatenate([np.sort(np.random.default_rng(b).choice(3 * n + 1, n, replace=False))
                          for b, n in enumerate(lens)]).astype(np.int32)
    posd = torch.from_numpy(pos).to(dev())
    res = stack.layer_forward(0, xd, posd, seqs, keep_rate=rates if prune else None,
                              want_scores=prune, want_kept=prune)
    torch.cuda.synchronize()
    x64 = f64(xd)
    w64 = weights_f64(wd)
    cu = seqs.host
    m_l2, m_el = modes(dtype)
    tol_x = SEQ_TOL[dtype]

    def check_x(got, ref_l2, ref_el, cu_rows):
        for b in range(len(lens)):
            lo, hi = cu_rows[b], cu_rows[b + 1]
            assert_rel_l2(got[lo:hi], ref_l2[lo:hi], tol_x, f"{name} seq {b}")
        assert_close(got, ref_el, tol_x, name)

    if not prune:
        ref = O.layer_forward(x64, pos.astype(np.int64), cu, w64, ocfg, mode=m_l2)
        ref_e = O.layer_forward(x64, pos.astype(np.int64), cu, w64, ocfg, mode=m_el)
        check_x(f64(res["x"]), ref["x"], ref_e["x"], cu)
        assert np.array_equal(res["pos"].cpu().numpy(), pos)
        assert np.array_equal(res["seqs"].host, cu)
        return
    own = O.layer_forward(x64, pos.astype(np.int64), cu, w64, ocfg, keep_rate=rates, mode=m_el)
    own_x = O.layer_forward(x64, pos.astype(np.int64), cu, w64, ocfg, keep_rate=rates, mode=m_l2)
    kept_gpu = res["kept_rows"].cpu().numpy()
    s_gpu = res["scores"].cpu().numpy()
    assert np.array_equal(res["seqs"].host, own["cu"])
    override, swaps = [], 0
    for b, n in enumerate(lens):
        lo = cu[b]
        kb = own["k"][b]
        kg = kept_gpu[res["seqs"].host[b]:res["seqs"].host[b + 1]] - lo
        kr = own["kept_rows"][own["cu"][b]:own["cu"][b + 1]] - lo
        s_e, s_x = own["scores"][lo:lo + n], own_x["scores"][lo:lo + n]
        swaps += check_kept_sets(s_gpu[lo:lo + n], s_e, kb, kg, kr, score_eps(s_e, s_x, dtype),
                                 f"{name} seq {b}", exact_scores=s_x)
        override.append(kg)
    if dtype == "f32":
        assert swaps == 0
    ref = O.layer_forward(x64, pos.astype(np.int64), cu, w64, ocfg, keep_rate=rates,
                          mode=m_l2, kept_override=override)
    ref_e = O.layer_forward(x64, pos.astype(np.int64), cu, w64, ocfg, keep_rate=rates,
                            mode=m_el, kept_override=override)
    assert np.array_equal(res["pos"].cpu().numpy(), ref["pos"])
    check_x(f64(res["x"]), ref["x"], ref_e["x"], res["seqs"].host)


def test_layer_keep_rate_one_equals_unpruned_bitwise():
    lens = [40, 129, 7]
    p, stack, xd, wd, ocfg = _setup(W.DECODER, "bf16", 256, 4, 256, lens, seed=5)
    seqs = zsa.Seqs(lens, dev())
    posd = torch.from_numpy(W.positions(lens)).to(dev())
    a = stack.layer_forward(0, xd, posd, seqs, keep_rate=[1.0, 1.0, 1.0], want_kept=True)
    b = stack.layer_forward(0, xd, posd, seqs, keep_rate=None)
    torch.cuda.synchronize()
    assert torch.equal(a["x"], b["x"])
    assert torch.equal(a["pos"], b["pos"])
    assert np.array_equal(a["kept_rows"].cpu().numpy(), np.arange(sum(lens)))
