"""Pins of the gradient oracle: its torch forward is the NumPy oracle's
(same kept sets), and its gradients are the NumPy oracle's finite
differences (central, float64)."""
import numpy as np
import pytest

from oracle import zsa_grad as G
from oracle import zsa_oracle as O
from paper_2509_01190_amd import workloads as W


def _setup(kind, hkv, n, seed, d=32, H=4, F=64, L=2, sharp=4.0):
    causal = True if kind == W.DECODER else False
    p = W.shrink(W.PRESETS["tiny"], kind=kind, causal=causal, n_layers=L, batch=1, d_model=d,
                 n_heads=H, d_ff=F, n_kv_heads=hkv)
    ws = [{k: (None if v is None else v.astype(np.float64)) for k, v in wd.items()}
          for wd in W.stack_weights(p, seed, norm_jitter=True)]
    for wd in ws:
        wd["w_qkv"] *= sharp
    cfg = O.LayerCfg(kind, d, H, F, causal, n_kv_heads=hkv)
    x = W.hidden(p, seed, [n]).astype(np.float64)
    return ws, cfg, x


def _kept(x, ws, cfg, prune, rate):
    n = x.shape[0]
    ref = O.stack_forward(x, np.arange(n), [0, n], ws, cfg, prune, [rate])
    return {pt["layer"]: pt["kept_rows"] for pt in ref["points"]}, ref


@pytest.mark.parametrize("kind,hkv", [(W.ENCODER, 0), (W.DECODER, 2), (W.DECODER, 0)])
def test_torch_forward_is_the_oracle(kind, hkv):
    ws, cfg, x = _setup(kind, hkv, 23, 3, L=3)
    kept, ref = _kept(x, ws, cfg, (1, 2), 0.5)
    dy = np.zeros_like(ref["x"])
    out, _, _ = G.stack_backward(x, np.arange(23), ws, cfg, (1, 2), kept, dy)
    assert np.allclose(out, ref["x"], rtol=1e-12, atol=1e-12)


def _loss(x, ws, cfg, prune, kept, dy):
    n = x.shape[0]
    over = {l: [k] for l, k in kept.items()}
    out = O.stack_forward(x, np.arange(n), [0, n], ws, cfg, prune, [0.5], kept_override=over)
    return float(np.sum(out["x"] * dy))


@pytest.mark.parametrize("kind,hkv", [(W.ENCODER, 0), (W.DECODER, 2)])
def test_gradients_match_finite_differences(kind, hkv):
    ws, cfg, x = _setup(kind, hkv, 9, 5, d=16, H=4, F=32)
    prune = (1,)
    kept, ref = _kept(x, ws, cfg, prune, 0.5)
    g = np.random.default_rng(7)
    dy = g.standard_normal(ref["x"].shape)
    _, dx, grads = G.stack_backward(x, np.arange(9), ws, cfg, prune, kept, dy)
    eps = 1e-6
    # a row the pruning point drops still gets gradient through that layer's
    # keys and values if some kept row attends to it; under the causal mask a
    # dropped row after every kept row gets none
    dropped = sorted(set(range(9)) - set(kept[1].tolist()))
    last_kept = int(kept[1].max())
    seen = [j for j in dropped if not cfg.causal or j < last_kept]
    unseen = [j for j in dropped if cfg.causal and j > last_kept]
    assert seen or unseen
    if seen:
        assert np.abs(dx[seen]).max() > 0
    if unseen:
        assert np.abs(dx[unseen]).max() == 0
    u = g.standard_normal(x.shape)
    fd = (_loss(x + eps * u, ws, cfg, prune, kept, dy) - _loss(x - eps * u, ws, cfg, prune, kept, dy)) / (2 * eps)
    assert abs(fd - np.sum(dx * u)) <= 1e-6 * max(1.0, abs(fd))
    # every weight of every layer along a random direction
    for l in range(len(ws)):
        for name, gw in grads[l].items():
            if gw is None:
                continue
            u = g.standard_normal(gw.shape)
            wp = [dict(w) for w in ws]
            wm = [dict(w) for w in ws]
            wp[l][name] = ws[l][name] + eps * u
            wm[l][name] = ws[l][name] - eps * u
            fd = (_loss(x, wp, cfg, prune, kept, dy) - _loss(x, wm, cfg, prune, kept, dy)) / (2 * eps)
            assert abs(fd - np.sum(gw * u)) <= 1e-6 * max(1.0, abs(fd)), (l, name, fd, np.sum(gw * u))
