"""The whole pruned stack through zsa_stack_forward against the oracle:
the small fp32 encoder exactly (kept positions identical), small bf16
encoder/decoder stacks under the margin protocol, determinism and the
keep_rate = 1 identity."""
import numpy as np
import pytest
import torch

from oracle import zsa_oracle as O
from paper_2509_01190_amd import workloads as W
from paper_2509_01190_amd import zsa
from tests.helpers import (SEQ_TOL, assert_rel_l2, assert_rows_vs_exact, check_kept_sets, dev,
                           dev_weights, f64, modes, rel_l2, score_eps, score_eps_from,
                           score_err, to_dev, weights_f64)

pytestmark = pytest.mark.gpu


def build(p, seed, lens=None, norm_jitter=True, sharp=1.0, qk_sharp=1.0):
    """Device weights, inputs and configurations of a test stack. ``sharp``
    scales the whole fused q|k|v projection; ``qk_sharp`` only its query and
    key rows (attention logits grow by its square, values stay)."""
    lens = W.lengths(p, seed) if lens is None else lens
    ws = W.stack_weights(p, seed, norm_jitter=norm_jitter)
    qk_rows = p.d_model + p.kv_heads * (p.d_model // p.n_heads)
    for w in ws:
        w["w_qkv"] = (w["w_qkv"] * np.float32(sharp)).astype(np.float32)
        w["w_qkv"][:qk_rows] *= np.float32(qk_sharp)
        if w["b_qkv"] is not None:
            w["b_qkv"][:qk_rows] *= np.float32(qk_sharp)
    dws = [dev_weights(w, p.dtype) for w in ws]
    cfg = zsa.make_cfg(p.kind, p.d_model, p.n_heads, p.d_ff, p.causal,
                       zsa.BF16 if p.dtype == "bf16" else zsa.F32, p.tau, p.norm_eps, p.rope_theta,
                       p.n_kv_heads, p.force_keep_last, p.mark_only)
    stack = zsa.Stack(cfg, dws)
    x = W.hidden(p, seed, lens)
    xd = to_dev(x, p.dtype)
    posd = torch.from_numpy(W.positions(lens)).to(dev())
    ocfg = O.LayerCfg(p.kind, p.d_model, p.n_heads, p.d_ff, p.causal, p.norm_eps, p.rope_theta,
                      p.tau, p.n_kv_heads, p.force_keep_last)
    return lens, stack, xd, posd, dws, ocfg


def gpu_kept_overrides(p, lens, seqs, out):
    """Per sequence, the GPU's kept sets at every pruning point as local row
    indices among the rows entering that point (for kept_override)."""
    n_pts = len(p.prune_after)
    rows_in = out["rows_in"]
    pos_dbg = out["pos_dbg"].cpu().numpy()
    cus = [seqs.host.astype(np.int64)]
    for pt in range(n_pts):
        c = np.zeros(len(lens) + 1, dtype=np.int64)
        c[1:] = np.cumsum(out["counts"][pt])
        cus.append(c)
    p_off = np.concatenate([[0], np.cumsum(rows_in[1:n_pts + 1])])
    overrides = []
    for b, n in enumerate(lens):
        posb = np.arange(n)
        override = {}
        for pt, layer in enumerate(p.prune_after):
            prev_pos = posb if pt == 0 else pos_dbg[p_off[pt - 1] + cus[pt][b]:p_off[pt - 1] + cus[pt][b + 1]]
            kept_pos = pos_dbg[p_off[pt] + cus[pt + 1][b]:p_off[pt] + cus[pt + 1][b + 1]]
            override[layer] = [np.searchsorted(prev_pos, kept_pos)]
        overrides.append(override)
    return overrides


def _split_dbg(p, lens, seqs, out):
    """Offsets of the debug outputs: per pruning point the row offsets of the
    rows entering (scores) and leaving it (positions); per block the offsets
    of its output rows inside hidden_dbg."""
    n_pts = len(p.prune_after)
    rows_in = out["rows_in"]
    cus = [seqs.host.astype(np.int64)]
    for pt in range(n_pts):
        c = np.zeros(len(lens) + 1, dtype=np.int64)
        c[1:] = np.cumsum(out["counts"][pt])
        cus.append(c)
    s_off = np.concatenate([[0], np.cumsum(rows_in[:n_pts])])
    p_off = np.concatenate([[0], np.cumsum(rows_in[1:n_pts + 1])])
    l_off = np.concatenate([[0], np.cumsum(out["layer_rows"])])
    # cu of the rows leaving block l (1-based): after the last point at or before l
    layer_cu, point = [], 0
    for l in range(1, len(out["layer_rows"]) + 1):
        if point < n_pts and p.prune_after[point] == l:
            point += 1
        layer_cu.append(cus[0] if p.mark_only else cus[point])
    return cus, s_off, p_off, l_off, layer_cu


def compare_stack(p, lens, stack, xd, posd, dws, ocfg, rates, seqs_check=None, tol=None,
                  exact_only=False, label=""):
    """Run the stack on the GPU (with debug outputs) and check it against the
    oracle, sequence by sequence (sequences are independent), continuing the
    oracle on the GPU's kept sets:

    * every block's output rows: relative L2 error per sequence against the
      exact oracle within the sequence tolerance, and every row within
      ROW_FACTOR of what bf16 storage alone does to it;
    * every pruning point: scores within SCORE_FACTOR of the emulation
      oracle's own error, the GPU's kept set exactly the top-k of its own
      scores, and any disagreement with the oracle's choice inside the
      score tolerance around the k-th score;
    * final positions exactly the oracle's.

    Returns statistics (kept-set swaps, score errors against their bounds,
    the worst row ratio, the worst per-sequence error) and prints them."""
    seqs = zsa.Seqs(lens, dev())
    out = stack.forward(xd, posd, seqs, p.prune_after, rates, debug=True)
    torch.cuda.synchronize()
    dt = "bf16" if p.dtype == "bf16" else "f32"
    tol = tol if tol is not None else SEQ_TOL[dt]
    n_pts = len(p.prune_after)
    s_dbg = out["scores_dbg"].cpu().numpy()
    pos_dbg = out["pos_dbg"].cpu().numpy()
    h_dbg = f64(out["hidden_dbg"])
    cus, s_off, p_off, l_off, layer_cu = _split_dbg(p, lens, seqs, out)
    assert np.array_equal(out["cu_host"], cus[-1])
    sched = O.keep_schedule(lens, list(rates), p.tau, n_pts)
    assert np.array_equal(out["counts"], np.array(sched).reshape(n_pts, len(lens)))
    x_all = f64(xd)
    ws64 = [weights_f64(w) for w in dws]
    x_fin = f64(out["x"][: out["t_final"]])
    pos_fin = out["pos"][: out["t_final"]].cpu().numpy()
    # the last block's debug rows are the output itself
    assert np.array_equal(h_dbg[l_off[-2]:l_off[-1]], x_fin)
    stats = {"swaps": 0, "kept": 0, "score_err_over_eps": 0.0, "row_ratio": 0.0,
             "seq_err": 0.0, "emul_seq_err": 0.0, "points": []}
    check = range(len(lens)) if seqs_check is None else seqs_check
    m_l2, m_el = ("exact", "exact") if exact_only else modes(p.dtype)
    for b in check:
        n = lens[b]
        lo = int(seqs.host[b])
        xb = x_all[lo:lo + n]
        posb = np.arange(n)
        override = {}
        for pt, layer in enumerate(p.prune_after):
            # GPU kept original positions -> local indices among the rows entering this point
            prev_pos = posb if pt == 0 else pos_dbg[p_off[pt - 1] + cus[pt][b]:p_off[pt - 1] + cus[pt][b + 1]]
            kept_pos = pos_dbg[p_off[pt] + cus[pt + 1][b]:p_off[pt] + cus[pt + 1][b + 1]]
            override[layer] = [np.searchsorted(prev_pos, kept_pos)]
        # oracle continuing on the GPU's kept sets: exact, and rounding at the
        # GPU's storage points
        ref = O.stack_forward(xb, posb, [0, n], ws64, ocfg, p.prune_after, [rates[b]],
                              mode=m_l2, kept_override=override, record=True)
        ref_e = ref if m_el == m_l2 else O.stack_forward(
            xb, posb, [0, n], ws64, ocfg, p.prune_after, [rates[b]], mode=m_el,
            kept_override=override, record=True)
        # the sequence's score budget: twice the largest error bf16 storage
        # causes at any of its pruning points (a point with few rows alone is
        # a noisy estimate of the error at that depth)
        emul_worst = max([score_err(ref_e["points"][pt]["scores"], ref["points"][pt]["scores"])
                          for pt in range(n_pts)] or [0.0])
        eps = score_eps_from(emul_worst, dt)
        for pt, layer in enumerate(p.prune_after):
            s_gpu = s_dbg[s_off[pt] + cus[pt][b]:s_off[pt] + cus[pt][b + 1]]
            s_x = ref["points"][pt]["scores"]
            s_e = ref_e["points"][pt]["scores"]
            k = ref["points"][pt]["k"][0]
            kg = override[layer][0]
            # the oracle's own choice given identical inputs to this point
            kr = O.select_topk(s_e, k, ocfg.force_keep_last)
            sw = check_kept_sets(s_gpu, s_e, k, kg, kr, eps, f"{label} seq {b} point {pt}",
                                 ocfg.force_keep_last, exact_scores=s_x)
            err = score_err(s_gpu, s_x)
            stats["swaps"] += sw
            stats["kept"] += k
            stats["score_err_over_eps"] = max(stats["score_err_over_eps"], err / eps)
            stats["points"].append({"seq": b, "point": pt, "k": int(k), "swaps": sw,
                                    "score_err": err, "emul_score_err": score_err(s_e, s_x),
                                    "eps": eps})
        for l in range(1, p.n_layers + 1):
            cu_l = layer_cu[l - 1]
            got = h_dbg[l_off[l - 1] + cu_l[b]:l_off[l - 1] + cu_l[b + 1]]
            rx = ref["layers"][l - 1]["x"]
            re_ = ref_e["layers"][l - 1]["x"]
            what = f"{label} seq {b} layer {l}"
            stats["emul_seq_err"] = max(stats["emul_seq_err"], rel_l2(re_, rx))
            assert_rel_l2(got, rx, tol, what + f" (bf16 storage alone: {rel_l2(re_, rx):.3e})")
            stats["seq_err"] = max(stats["seq_err"], rel_l2(got, rx))
            stats["row_ratio"] = max(stats["row_ratio"],
                                     assert_rows_vs_exact(got, rx, re_, tol, what))
        fo, fe = out["cu_host"][b], out["cu_host"][b + 1]
        assert np.array_equal(pos_fin[fo:fe], ref["pos"])
    print(f"[parity] {label or p.name}: seqs {list(check)}, worst seq rel-L2 {stats['seq_err']:.3e} "
          f"(tol {tol:.0e}; bf16 storage alone {stats['emul_seq_err']:.3e}), "
          f"worst row error / bound {stats['row_ratio']:.3f}, "
          f"worst score error / eps {stats['score_err_over_eps']:.3f}, "
          f"kept-set swaps {stats['swaps']} of {stats['kept']} kept", flush=True)
    for q in stats["points"]:
        print(f"[parity]   seq {q['seq']} point {q['point']}: k {q['k']}, swaps {q['swaps']}, "
              f"score err {q['score_err']:.3e} (emulation {q['emul_score_err']:.3e}, "
              f"eps {q['eps']:.3e})", flush=True)
    return stats


def test_tiny_encoder_exact():
    p = W.PRESETS["tiny"]
    lens, stack, xd, posd, dws, ocfg = build(p, 0)
    rates = W.keep_rates(p, 0, 0.5)
    assert compare_stack(p, lens, stack, xd, posd, dws, ocfg, rates)["swaps"] == 0


@pytest.mark.parametrize("kind", [W.ENCODER, W.DECODER])
def test_small_bf16_stack(kind):
    causal = kind == W.DECODER
    p = W.shrink(W.PRESETS["bert"], kind=kind, causal=causal, n_layers=4, d_model=256, n_heads=4,
                 d_ff=512, batch=5, prune_after=(1, 3))
    lens = [300, 64, 129, 17, 512]
    lens, stack, xd, posd, dws, ocfg = build(p, 1, lens, sharp=3.0)
    rates = [0.5, 0.7, 0.3, 0.9, 0.1]
    compare_stack(p, lens, stack, xd, posd, dws, ocfg, rates)


def test_stack_with_empty_sequences():
    """Empty sequences inside a batch pass every pruning point with zero rows
    (their kept counts are 0) and leave the other sequences' rows, scores,
    kept sets and positions as the oracle has them."""
    p = W.shrink(W.PRESETS["dec1b"], n_layers=3, d_model=256, n_heads=4, d_ff=256, batch=5,
                 prune_after=(1, 2))
    lens, stack, xd, posd, dws, ocfg = build(p, 2, [0, 37, 0, 120, 5])
    compare_stack(p, lens, stack, xd, posd, dws, ocfg, [0.5, 0.5, 0.3, 0.7, 0.9],
                  seqs_check=[1, 3, 4], label="empty sequences")
    # a batch of empty sequences only: nothing to compute, zero rows out
    seqs0 = zsa.Seqs([0, 0, 0], dev())
    out = stack.forward(xd[:0], posd[:0], seqs0, p.prune_after, [0.5, 0.5, 0.5])
    torch.cuda.synchronize()
    assert out["t_final"] == 0 and not np.any(out["cu_host"])


def test_stack_deterministic_and_keep_one():
    p = W.shrink(W.PRESETS["dec1b"], n_layers=3, d_model=256, n_heads=4, d_ff=256, batch=3,
                 prune_after=(1, 2))
    lens = [200, 33, 450]
    lens, stack, xd, posd, dws, ocfg = build(p, 2, lens, sharp=8.0)
    seqs = zsa.Seqs(lens, dev())
    a = stack.forward(xd, posd, seqs, p.prune_after, [0.4, 0.6, 0.25], debug=True)
    a_x = a["x"].clone()
    a_s = a["scores_dbg"].clone()
    b = stack.forward(xd, posd, seqs, p.prune_after, [0.4, 0.6, 0.25], debug=True)
    torch.cuda.synchronize()
    assert torch.equal(a_x, b["x"])
    assert torch.equal(a_s, b["scores_dbg"])
    one = stack.forward(xd, posd, seqs, p.prune_after, [1.0] * 3)
    none = stack.forward(xd, posd, seqs, (), [1.0] * 3)
    torch.cuda.synchronize()
    assert torch.equal(one["x"][: one["t_final"]], none["x"][: none["t_final"]])
    assert torch.equal(one["pos"][: one["t_final"]], none["pos"][: none["t_final"]])


def test_graph_replay_matches_eager():
    p = W.shrink(W.PRESETS["bert"], n_layers=3, d_model=256, n_heads=4, d_ff=512, batch=4,
                 prune_after=(1, 2))
    lens = [128, 300, 77, 512]
    lens, stack, xd, posd, dws, ocfg = build(p, 3, lens, sharp=8.0)
    seqs = zsa.Seqs(lens, dev())
    rates = [0.5, 0.3, 0.8, 0.6]
    eager = stack.forward(xd, posd, seqs, p.prune_after, rates)
    ref_x = eager["x"].clone()
    ref_pos = eager["pos"].clone()
    out = stack.forward(xd, posd, seqs, p.prune_after, rates)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            stack.forward(xd, posd, seqs, p.prune_after, rates, out=out)
    torch.cuda.current_stream().wait_stream(s)
    for i in range(3):
        out["x"].zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out["x"], ref_x), f"replay {i}"
        assert torch.equal(out["pos"], ref_pos), f"replay {i}"


def test_small_every_layer_schedule():
    # the paper's default: Eq. 2 after every layer, tau = 5, causal GPT-2-like
    # blocks, down to the tau floor
    p = W.shrink(W.PRESETS["gpt2"], n_layers=5, d_model=256, n_heads=4, d_ff=512, batch=4,
                 prune_after=(1, 2, 3, 4, 5))
    lens = [300, 64, 129, 17]
    lens, stack, xd, posd, dws, ocfg = build(p, 4, lens, sharp=3.0)
    for rates in ([0.5, 0.7, 0.3, 0.9], [0.02, 0.1, 0.05, 1.0]):
        compare_stack(p, lens, stack, xd, posd, dws, ocfg, rates)


@pytest.mark.parametrize("kind", ["gpt2", "dec1b"])
def test_floor_points_run_unpruned(kind):
    # Pruning after every layer at low keep rates leaves every sequence at
    # its floor tau after a few layers; from there Eq. 2 keeps all rows, and
    # without score debugging the stack runs those blocks unpruned (no
    # scores, selection or gather). The result must be bitwise that of the
    # run that scores, selects and gathers at every point (debug outputs on).
    p = W.shrink(W.PRESETS[kind], n_layers=5, d_model=256, n_heads=4, d_ff=512, batch=4,
                 prune_after=(1, 2, 3, 4, 5))
    lens = [300, 64, 129, 17]
    lens, stack, xd, posd, dws, ocfg = build(p, 6, lens, sharp=3.0)
    seqs = zsa.Seqs(lens, dev())
    rates = [0.02, 0.1, 0.05, 0.3]
    plan = stack.plan(seqs, list(p.prune_after), rates)
    counts = [lens] + [list(c) for c in plan["counts"]]
    assert any(counts[i] == counts[i + 1] for i in range(len(p.prune_after))), counts
    fast = stack.forward(xd, posd, seqs, p.prune_after, rates)
    full = stack.forward(xd, posd, seqs, p.prune_after, rates, debug=True)
    torch.cuda.synchronize()
    assert fast["t_final"] == full["t_final"]
    t = fast["t_final"]
    assert torch.equal(fast["x"][:t], full["x"][:t])
    assert torch.equal(fast["pos"][:t], full["pos"][:t])
    assert np.array_equal(fast["cu_host"], full["cu_host"])
    assert np.array_equal(fast["counts"], full["counts"])


@pytest.mark.parametrize("hkv", [2, 1])
def test_small_gqa_stack_keep_last(hkv):
    # grouped-query (and multi-query) decoder, every-layer schedule, the last
    # row of each sequence forced to survive every pruning point
    p = W.shrink(W.PRESETS["dec1b"], n_layers=3, d_model=256, n_heads=4, d_ff=256, batch=4,
                 prune_after=(1, 2, 3), n_kv_heads=hkv, force_keep_last=True)
    lens = [300, 64, 129, 17]
    lens, stack, xd, posd, dws, ocfg = build(p, 5, lens, sharp=3.0)
    rates = [0.5, 0.3, 0.7, 0.1]
    compare_stack(p, lens, stack, xd, posd, dws, ocfg, rates)
    out = stack.forward(xd, posd, zsa.Seqs(lens, dev()), p.prune_after, rates)
    torch.cuda.synchronize()
    pos = out["pos"][: out["t_final"]].cpu().numpy()
    cu = out["cu_host"]
    assert [int(pos[cu[b + 1] - 1]) for b in range(len(lens))] == [n - 1 for n in lens]


@pytest.mark.parametrize("kind", [W.ENCODER, W.DECODER])
def test_mark_only_stack(kind):
    # rows are marked, not removed: the outputs are the unpruned stack's, and
    # every point marks the Eq. 2 count (compounded on the marked counts) by
    # the scores of all rows at that layer
    causal = kind == W.DECODER
    p = W.shrink(W.PRESETS["bert"], kind=kind, causal=causal, n_layers=3, d_model=256, n_heads=4,
                 d_ff=512, batch=3, prune_after=(1, 2, 3), mark_only=True)
    lens = [300, 64, 129]
    lens, stack, xd, posd, dws, ocfg = build(p, 8, lens, sharp=3.0)
    seqs = zsa.Seqs(lens, dev())
    rates = [0.5, 0.3, 0.7]
    out = stack.forward(xd, posd, seqs, p.prune_after, rates, debug=True)
    torch.cuda.synchronize()
    T = sum(lens)
    assert out["t_final"] == T and np.array_equal(out["cu_host"], seqs.host)
    assert torch.equal(out["pos"][:T], posd)
    sched = O.keep_schedule(lens, rates, p.tau, 3)
    assert np.array_equal(out["counts"], np.array(sched).reshape(3, len(lens)))
    x_all = f64(xd)
    ws64 = [weights_f64(w) for w in dws]
    s_dbg = out["scores_dbg"].cpu().numpy()
    pos_dbg = out["pos_dbg"].cpu().numpy()
    h_dbg = f64(out["hidden_dbg"])
    assert out["layer_rows"] == [T] * p.n_layers
    m_off = np.concatenate([[0], np.cumsum([int(np.sum(c)) for c in sched])])
    for b, n in enumerate(lens):
        lo = int(seqs.host[b])
        ref = O.stack_forward(x_all[lo:lo + n], np.arange(n), [0, n], ws64, ocfg, p.prune_after,
                              [rates[b]], mode="exact", mark_only=True, record=True)
        ref_e = O.stack_forward(x_all[lo:lo + n], np.arange(n), [0, n], ws64, ocfg, p.prune_after,
                                [rates[b]], mode="bf16", mark_only=True, record=True)
        for l in range(p.n_layers):
            got = h_dbg[l * T + lo:l * T + lo + n]
            what = f"seq {b} layer {l + 1}"
            assert_rel_l2(got, ref["layers"][l]["x"], SEQ_TOL["bf16"], what)
            assert_rows_vs_exact(got, ref["layers"][l]["x"], ref_e["layers"][l]["x"],
                                 SEQ_TOL["bf16"], what)
        for pt in range(3):
            k = sched[pt][b]
            c0 = m_off[pt] + int(np.sum(sched[pt][:b]))
            kept_gpu = pos_dbg[c0:c0 + k]                 # positions = local indices here
            s_gpu = s_dbg[pt * T + lo:pt * T + lo + n]
            s_x = ref["points"][pt]["scores"]
            s_e = ref_e["points"][pt]["scores"]
            check_kept_sets(s_gpu, s_e, k, kept_gpu, ref_e["points"][pt]["kept_rows"],
                            score_eps(s_e, s_x, "bf16"), f"seq {b} point {pt}",
                            exact_scores=s_x)
