"""Kernel-level parity of the HIP path against the CPU oracle, through the
C-ABI (select, gather, norms, projections with every epilogue, attention,
contribution scores)."""
import math

import numpy as np
import pytest
import torch

from oracle import zsa_oracle as O
from paper_2509_01190_amd import workloads as W
from paper_2509_01190_amd import zsa
from tests.helpers import assert_close, dev, f64, to_dev

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------------ top-k
@pytest.mark.parametrize("case", ["ragged_ties", "long_rows", "edges", "one_magnitude", "all_equal"])
def test_select_topk_bit_exact(case):
    if case == "ragged_ties":
        lens = W.lengths(W.PRESETS["ragged"], 0)
    elif case == "long_rows":
        lens = [20000, 16384, 16385, 3, 4097]
    else:
        lens = [0, 1, 5, 6, 64, 1000, 2, 2048, 2049, 3000]
    g = np.random.default_rng(3)
    scores = W.injected_scores(lens, seed=1)
    if case == "one_magnitude":
        # every key shares its top two bytes (the radix passes there put all
        # rows in one bin), with ties among the rest
        scores = (10.0 + np.round(g.uniform(0.0, 0.03, len(scores)), 3)).astype(np.float32)
    elif case == "all_equal":
        scores = np.full(len(scores), 3.25, np.float32)
    ks = []
    for b, n in enumerate(lens):
        if b % 5 == 3:
            ks.append(0)
        elif b % 5 == 4:
            ks.append(n)
        else:
            ks.append(O.keep_count(n, float(g.uniform(0.0, 1.0)), 5))
    seqs = zsa.Seqs(lens, dev())
    kept = zsa.select_topk(torch.from_numpy(scores).to(dev()), seqs, ks)
    torch.cuda.synchronize()
    got = kept.cpu().numpy()
    ref = []
    for b, n in enumerate(lens):
        lo = int(seqs.host[b])
        ref.append(O.select_topk(scores[lo:lo + n].astype(np.float64), ks[b]) + lo)
    ref = np.concatenate(ref) if ref else np.zeros(0)
    assert np.array_equal(got, ref)


def test_select_topk_keep_last_bit_exact():
    lens = [1, 2, 5, 6, 64, 1000, 20000, 777]
    g = np.random.default_rng(13)
    scores = W.injected_scores(lens, seed=2)
    ks = [O.keep_count(n, float(g.uniform(0.0, 1.0)), 5) for n in lens]
    ks[3] = 1
    seqs = zsa.Seqs(lens, dev())
    kept = zsa.select_topk(torch.from_numpy(scores).to(dev()), seqs, ks, keep_last=True)
    torch.cuda.synchronize()
    ref = []
    for b, n in enumerate(lens):
        lo = int(seqs.host[b])
        ref.append(O.select_topk(scores[lo:lo + n].astype(np.float64), ks[b], keep_last=True) + lo)
    assert np.array_equal(kept.cpu().numpy(), np.concatenate(ref))


def test_select_topk_deterministic():
    lens = [4096, 777, 3000]
    scores = np.random.default_rng(4).standard_normal(sum(lens)).astype(np.float32)
    seqs = zsa.Seqs(lens, dev())
    s = torch.from_numpy(scores).to(dev())
    a = zsa.select_topk(s, seqs, [100, 300, 2999]).cpu()
    b = zsa.select_topk(s, seqs, [100, 300, 2999]).cpu()
    assert torch.equal(a, b)


# ------------------------------------------------------------------ gather
@pytest.mark.parametrize("dtype,d", [("bf16", 768), ("bf16", 4096), ("f32", 128)])
def test_compact_gather_bit_exact(dtype, d):
    g = np.random.default_rng(5)
    t_in = 1000
    x = g.standard_normal((t_in, d)).astype(np.float32)
    pos = g.integers(0, 5000, t_in).astype(np.int32)
    kept = np.sort(g.choice(t_in, 333, replace=False)).astype(np.int32)
    kept = np.concatenate([kept, np.array([-1, t_in], dtype=np.int32)])   # out-of-range rows
    xd = to_dev(x, dtype)
    out, pos_out = zsa.compact_gather(xd, torch.from_numpy(pos).to(dev()),
                                      torch.from_numpy(kept).to(dev()))
    torch.cuda.synchronize()
    ref = xd.cpu()
    assert torch.equal(out[:333].cpu(), ref[kept[:333]])
    assert torch.equal(out[333:].cpu(), torch.zeros_like(out[333:].cpu()))
    assert np.array_equal(pos_out.cpu().numpy(), np.concatenate([pos[kept[:333]], [-1, -1]]))


# ------------------------------------------------------------------ norms
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kind", [zsa.NORM_LAYER, zsa.NORM_RMS])
@pytest.mark.parametrize("d", [128, 768, 4096])
def test_norm(dtype, kind, d):
    g = np.random.default_rng(6)
    rows = 37
    x = (g.standard_normal((rows, d)) * 2 + 0.5).astype(np.float32)
    w = (1 + 0.1 * g.standard_normal(d)).astype(np.float32)
    b = (0.1 * g.standard_normal(d)).astype(np.float32)
    xd, wd, bd = to_dev(x, dtype), to_dev(w, dtype), to_dev(b, dtype)
    y = zsa.norm(xd, wd, bd, kind, 1e-5)
    torch.cuda.synchronize()
    x64, w64, b64 = f64(xd), f64(wd), f64(bd)
    ref = O.layer_norm(x64, w64, b64, 1e-5) if kind == zsa.NORM_LAYER else O.rms_norm(x64, w64, 1e-5)
    assert_close(f64(y), ref, 1e-2 if dtype == "bf16" else 1e-5, f"norm {kind}")


# ------------------------------------------------------------------ projections
EPIS = [zsa.EPI_NONE, zsa.EPI_GELU, zsa.EPI_SWIGLU, zsa.EPI_RESIDUAL, zsa.EPI_ROPE]


@pytest.mark.parametrize("dtype,k", [("bf16", 256), ("bf16", 136), ("f32", 200)])
@pytest.mark.parametrize("epi", EPIS)
def test_linear_epilogues(dtype, k, epi):
    g = np.random.default_rng(7 + epi)
    m, n, hd = 300, 384, 64
    x = g.standard_normal((m, k)).astype(np.float32)
    w = (g.standard_normal((n, k)) / math.sqrt(k)).astype(np.float32)
    bias = (0.1 * g.standard_normal(n)).astype(np.float32)
    xd, wd, bd = to_dev(x, dtype), to_dev(w, dtype), to_dev(bias, dtype)
    res = to_dev(g.standard_normal((m, n)).astype(np.float32), dtype) if epi == zsa.EPI_RESIDUAL else None
    pos = g.integers(0, 4096, m).astype(np.int32)
    posd = torch.from_numpy(pos).to(dev())
    rope_cols = 256
    y = zsa.linear(xd, wd, bd, epi, residual=res, pos=posd if epi == zsa.EPI_ROPE else None,
                   head_dim=hd, rope_cols=rope_cols, rope_theta=10000.0)
    torch.cuda.synchronize()
    z = f64(xd) @ f64(wd).T + f64(bd)
    if epi == zsa.EPI_NONE:
        ref = z
    elif epi == zsa.EPI_GELU:
        ref = O.gelu(z)
    elif epi == zsa.EPI_SWIGLU:
        ref = O.silu(z[:, 0::2]) * z[:, 1::2]
    elif epi == zsa.EPI_RESIDUAL:
        ref = f64(res) + z
    else:
        ref = z.copy()
        ref[:, :rope_cols] = O.rope(z[:, :rope_cols], pos.astype(np.int64), rope_cols // hd, 1e4)
    assert_close(f64(y), ref, 1e-2 if dtype == "bf16" else 2e-5, f"epilogue {epi}")


@pytest.mark.parametrize("epi", EPIS)
@pytest.mark.parametrize("split", [False, True])
def test_linear_zero_rows(epi, split):
    """A product of no rows (a batch whose sequences were all emptied, a
    layer past the last kept row) returns an empty output and launches
    nothing; the operands are views of real allocations."""
    k, n, hd = 256, 384, 64
    g = np.random.default_rng(3 + epi)
    xd = to_dev(g.standard_normal((1, k)).astype(np.float32), "bf16")[:0]
    wd = to_dev((g.standard_normal((n, k)) / math.sqrt(k)).astype(np.float32), "bf16")
    res = to_dev(g.standard_normal((1, n)).astype(np.float32), "bf16")[:0] if epi == zsa.EPI_RESIDUAL else None
    posd = torch.zeros(1, dtype=torch.int32, device=dev())[:0]
    y = zsa.linear(xd, wd, None, epi, residual=res, pos=posd if epi == zsa.EPI_ROPE else None,
                   head_dim=hd, rope_cols=256, rope_theta=1e4, split=split)
    torch.cuda.synchronize()
    assert tuple(y.shape) == (0, n // 2 if epi == zsa.EPI_SWIGLU else n)


@pytest.mark.parametrize("m,n,k", [(1100, 384, 3072), (1500, 768, 8192), (2100, 768, 3072)])
@pytest.mark.parametrize("epi", [zsa.EPI_NONE, zsa.EPI_GELU, zsa.EPI_SWIGLU, zsa.EPI_RESIDUAL,
                                 zsa.EPI_ROPE])
def test_linear_split_k(m, n, k, epi):
    """Small grids split K into slices summed in a fixed order: the result
    matches the oracle like the unsplit product and is reproducible."""
    assert zsa.linear_workspace_size(zsa.BF16, m, n, k) > 0
    g = np.random.default_rng(11 + epi + m)
    hd = 64
    x = g.standard_normal((m, k)).astype(np.float32)
    w = (g.standard_normal((n, k)) / math.sqrt(k)).astype(np.float32)
    bias = (0.1 * g.standard_normal(n)).astype(np.float32)
    xd, wd, bd = to_dev(x, "bf16"), to_dev(w, "bf16"), to_dev(bias, "bf16")
    res = to_dev(g.standard_normal((m, n)).astype(np.float32), "bf16") if epi == zsa.EPI_RESIDUAL else None
    pos = g.integers(0, 4096, m).astype(np.int32)
    posd = torch.from_numpy(pos).to(dev())
    rope_cols = 256
    kw = dict(residual=res, pos=posd if epi == zsa.EPI_ROPE else None, head_dim=hd,
              rope_cols=rope_cols, rope_theta=10000.0)
    y1 = zsa.linear(xd, wd, bd, epi, split=True, **kw)
    y2 = zsa.linear(xd, wd, bd, epi, split=True, **kw)
    y0 = zsa.linear(xd, wd, bd, epi, split=False, **kw)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    z = f64(xd) @ f64(wd).T + f64(bd)
    if epi == zsa.EPI_NONE:
        ref = z
    elif epi == zsa.EPI_GELU:
        ref = O.gelu(z)
    elif epi == zsa.EPI_SWIGLU:
        ref = O.silu(z[:, 0::2]) * z[:, 1::2]
    elif epi == zsa.EPI_RESIDUAL:
        ref = f64(res) + z
    else:
        ref = z.copy()
        ref[:, :rope_cols] = O.rope(z[:, :rope_cols], pos.astype(np.int64), rope_cols // hd, 1e4)
    assert_close(f64(y1), ref, 1e-2, f"split epilogue {epi}")
    assert_close(f64(y0), ref, 1e-2, f"unsplit epilogue {epi}")


@pytest.mark.parametrize("m,n,k", [(4, 6144, 4096),     # one row block, two register rounds
                                   (8, 2048, 8192),     # one row block, long K
                                   (17, 2304, 768),     # two row blocks, one partly filled
                                   (64, 256, 4096),     # two register rounds
                                   (160, 768, 3072),    # one column block per workgroup
                                   (160, 2304, 768),    # two column blocks per workgroup
                                   (256, 3072, 768),
                                   (40, 2048, 8192),    # long K, two register rounds
                                   (100, 48, 64),       # three column blocks, one wave's range
                                   (33, 8, 32),         # N under one column block, K one step
                                   (200, 1000, 96),     # ragged N, K not a whole 64-wide group
                                   (300, 2304, 1024),   # ragged rows, two column blocks
                                   (500, 1000, 2048),   # odd column blocks: the last pair half past N
                                   (512, 768, 3072),    # two column blocks, double-buffered
                                   (1000, 768, 768)])   # ragged, near the last row count
@pytest.mark.parametrize("epi", [zsa.EPI_NONE, zsa.EPI_GELU, zsa.EPI_SWIGLU, zsa.EPI_RESIDUAL])
@pytest.mark.parametrize("split", [True, False])
def test_linear_short_products(m, n, k, epi, split):
    """Products of 4 to 1000 rows (the few-row kernel: one or two 16-row and
    16-column blocks per workgroup, K over its waves in one round or in
    double-buffered rounds), every epilogue but the rotary one, against the
    oracle, and reproducible."""
    if epi == zsa.EPI_SWIGLU:  # the API takes gate/up products of whole 16-column groups
        n = (n + 15) // 16 * 16
    g = np.random.default_rng(m + n + k + epi)
    x = g.standard_normal((m, k)).astype(np.float32)
    w = (g.standard_normal((n, k)) / math.sqrt(k)).astype(np.float32)
    bias = (0.1 * g.standard_normal(n)).astype(np.float32)
    xd, wd, bd = to_dev(x, "bf16"), to_dev(w, "bf16"), to_dev(bias, "bf16")
    res = to_dev(g.standard_normal((m, n)).astype(np.float32), "bf16") if epi == zsa.EPI_RESIDUAL else None
    y1 = zsa.linear(xd, wd, bd, epi, residual=res, split=split)
    y2 = zsa.linear(xd, wd, bd, epi, residual=res, split=split)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    z = f64(xd) @ f64(wd).T + f64(bd)
    if epi == zsa.EPI_GELU:
        z = O.gelu(z)
    elif epi == zsa.EPI_RESIDUAL:
        z = z + f64(res)
    elif epi == zsa.EPI_SWIGLU:
        z = O.silu(z[:, 0::2]) * z[:, 1::2]
    assert_close(f64(y1), z, 1e-2, f"short product {m}x{n}x{k} epilogue {epi}")


@pytest.mark.parametrize("m,n,k,split", [(16129, 3072, 768, False),   # persistent 256x256: whole rounds
                                         (16129, 3072, 128, False),   # two K slices per tile
                                         (16129, 2304, 192, False),   # three, 256x192
                                         (16129, 2304, 768, False),   # persistent 256x192: whole rounds
                                         (12289, 768, 3072, False),   # persistent 256x192: 0.77 round
                                         (4001, 2304, 768, False),    # persistent 256x192: 0.75 round
                                         (4097, 4096, 4096, False),   # persistent 256x256: K > 3072
                                         (12289, 3072, 768, False),   # persistent 128x128
                                         (1000, 768, 768, False),
                                         (4000, 768, 3072, False),
                                         (16385, 2304, 768, False),
                                         (1500, 2048, 8192, False),   # persistent 128x128, long K
                                         (1000, 2048, 8192, True)])   # split K over 4 slices
@pytest.mark.parametrize("epi", [zsa.EPI_NONE, zsa.EPI_GELU, zsa.EPI_RESIDUAL, zsa.EPI_SWIGLU])
@pytest.mark.parametrize("with_bias", [True, False])
def test_linear_kernel_regimes(m, n, k, split, epi, with_bias):
    """Every GEMM the projection shapes dispatch to (by grid size and
    epilogue), with ragged row counts, against the oracle on sampled rows
    (the first and last 64 and 128 drawn at random), and reproducible."""
    g = np.random.default_rng(m + n + k + epi + int(with_bias))
    x = g.standard_normal((m, k)).astype(np.float32)
    w = (g.standard_normal((n, k)) / math.sqrt(k)).astype(np.float32)
    xd, wd = to_dev(x, "bf16"), to_dev(w, "bf16")
    bd = to_dev((0.1 * g.standard_normal(n)).astype(np.float32), "bf16") if with_bias else None
    res = to_dev(g.standard_normal((m, n)).astype(np.float32), "bf16") if epi == zsa.EPI_RESIDUAL else None
    y1 = zsa.linear(xd, wd, bd, epi, residual=res, split=split)
    y2 = zsa.linear(xd, wd, bd, epi, residual=res, split=split)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    rows = np.unique(np.concatenate([np.arange(64), np.arange(m - 64, m),
                                     g.integers(0, m, 128)]))
    rt = torch.from_numpy(rows).to(dev())
    z = f64(xd[rt]) @ f64(wd).T
    if bd is not None:
        z = z + f64(bd)
    if epi == zsa.EPI_GELU:
        z = O.gelu(z)
    elif epi == zsa.EPI_RESIDUAL:
        z = z + f64(res[rt])
    elif epi == zsa.EPI_SWIGLU:
        z = O.silu(z[:, 0::2]) * z[:, 1::2]
    assert_close(f64(y1[rt]), z, 1e-2, f"regime {m}x{n}x{k} epilogue {epi}")


@pytest.mark.parametrize("m,n,k,hd,rope_cols", [(16129, 3072, 768, 64, 2048),   # 256x256 on 8 waves
                                               (8191, 6144, 2048, 64, 4096),    # 1B-shaped QKV
                                               (4097, 4096, 4096, 128, 2048),   # K > 3072
                                               (4097, 6144, 4096, 128, 5120),   # grouped-query
                                               (3000, 3072, 768, 64, 2048),     # 128x128
                                               (40, 6144, 2048, 64, 4096),      # few-row, two column blocks
                                               (163, 3072, 768, 64, 2048),      # few-row, ragged rows
                                               (20, 6144, 4096, 128, 5120)])    # few-row, grouped-query
@pytest.mark.parametrize("with_bias", [True, False])
@pytest.mark.parametrize("table", [False, True])
def test_linear_rope_regimes(m, n, k, hd, rope_cols, with_bias, table):
    """The rotary epilogue in the kernels the decoders' QKV projections
    dispatch to (ragged rows, grouped-query widths), with the angles formed
    per element or read from a per-row table built in the workspace (which
    lets the persistent four-wave kernel take the product: heads past
    rope_cols pass unrotated), against the oracle on sampled rows, and
    reproducible."""
    g = np.random.default_rng(m + n + hd + int(with_bias))
    x = g.standard_normal((m, k)).astype(np.float32)
    w = (g.standard_normal((n, k)) / math.sqrt(k)).astype(np.float32)
    xd, wd = to_dev(x, "bf16"), to_dev(w, "bf16")
    bd = to_dev((0.1 * g.standard_normal(n)).astype(np.float32), "bf16") if with_bias else None
    pos = g.integers(0, 8192, m).astype(np.int32)
    posd = torch.from_numpy(pos).to(dev())
    kw = dict(pos=posd, head_dim=hd, rope_cols=rope_cols, rope_theta=500000.0, split=table)
    y1 = zsa.linear(xd, wd, bd, zsa.EPI_ROPE, **kw)
    y2 = zsa.linear(xd, wd, bd, zsa.EPI_ROPE, **kw)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    rows = np.unique(np.concatenate([np.arange(64), np.arange(m - 64, m), g.integers(0, m, 128)]))
    rows = rows[(rows >= 0) & (rows < m)]
    rt = torch.from_numpy(rows).to(dev())
    z = f64(xd[rt]) @ f64(wd).T
    if bd is not None:
        z = z + f64(bd)
    ref = z.copy()
    ref[:, :rope_cols] = O.rope(z[:, :rope_cols], pos[rows].astype(np.int64), rope_cols // hd, 5e5)
    assert_close(f64(y1[rt]), ref, 1e-2, f"rope regime {m}x{n}x{k} hd {hd}")


@pytest.mark.parametrize("m,n,k,hd", [(1, 384, 256, 64), (4, 6144, 4096, 128),
                                      (4, 4096, 14336, 128), (16, 3072, 768, 64),
                                      (3, 400, 512, 16), (7, 2304, 768, 64), (5, 512, 800, 64),
                                      (17, 2304, 768, 64), (64, 3072, 768, 64),
                                      (160, 768, 768, 64), (237, 768, 1024, 128)])
@pytest.mark.parametrize("epi", EPIS)
def test_linear_few_rows(m, n, k, hd, epi):
    """Short products (generation rows, the short layers of the
    every-layer schedule): W streamed into the matrix cores, one workgroup
    per 16 output columns and 16 rows of x (ragged last blocks: 17, 237
    rows), whose waves split K (k = 800: the last waves get a short range
    or none) and add their sums in a fixed order. Every epilogue against
    the oracle (the rotary one with each workgroup's columns paired across
    half heads), results bit-identical over calls."""
    g = np.random.default_rng(100 * m + n + k + epi)
    x = g.standard_normal((m, k)).astype(np.float32)
    w = (g.standard_normal((n, k)) / math.sqrt(k)).astype(np.float32)
    bias = (0.1 * g.standard_normal(n)).astype(np.float32)
    xd, wd, bd = to_dev(x, "bf16"), to_dev(w, "bf16"), to_dev(bias, "bf16")
    res = to_dev(g.standard_normal((m, n)).astype(np.float32), "bf16") if epi == zsa.EPI_RESIDUAL else None
    pos = g.integers(0, 4096, m).astype(np.int32)
    posd = torch.from_numpy(pos).to(dev())
    rope_cols = min(n, 8 * hd) // hd * hd
    kw = dict(residual=res, pos=posd if epi == zsa.EPI_ROPE else None, head_dim=hd,
              rope_cols=rope_cols, rope_theta=10000.0)
    y1 = zsa.linear(xd, wd, bd, epi, **kw)
    y2 = zsa.linear(xd, wd, bd, epi, **kw)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    z = f64(xd) @ f64(wd).T + f64(bd)
    if epi == zsa.EPI_NONE:
        ref = z
    elif epi == zsa.EPI_GELU:
        ref = O.gelu(z)
    elif epi == zsa.EPI_SWIGLU:
        ref = O.silu(z[:, 0::2]) * z[:, 1::2]
    elif epi == zsa.EPI_RESIDUAL:
        ref = f64(res) + z
    else:
        ref = z.copy()
        ref[:, :rope_cols] = O.rope(z[:, :rope_cols], pos.astype(np.int64), rope_cols // hd, 1e4)
    assert_close(f64(y1), ref, 1e-2, f"few-row {m}x{n}x{k} epilogue {epi}")


def test_linear_in_place_residual():
    g = np.random.default_rng(8)
    m, k, n = 129, 128, 256
    xd = to_dev(g.standard_normal((m, k)).astype(np.float32), "bf16")
    wd = to_dev((g.standard_normal((n, k)) / 11).astype(np.float32), "bf16")
    yd = to_dev(g.standard_normal((m, n)).astype(np.float32), "bf16")
    ref = f64(yd) + f64(xd) @ f64(wd).T
    zsa.linear(xd, wd, None, zsa.EPI_RESIDUAL, residual=yd, out=yd)
    torch.cuda.synchronize()
    assert_close(f64(yd), ref, 1e-2, "in-place residual")


# ------------------------------------------------------------------ attention + scores
def _qkv(lens, H, hd, dtype, seed, sharp=1.5):
    g = np.random.default_rng(seed)
    T = sum(lens)
    d = H * hd
    qkv = g.standard_normal((T, 3 * d)).astype(np.float32)
    qkv[:, :d] *= sharp
    t = to_dev(qkv, dtype)
    return t, t[:, :d], t[:, d:2 * d], t[:, 2 * d:]


ATT_CASES = [("bf16", 64), ("bf16", 128), ("f32", 32), ("f32", 64), ("bf16", 32)]


@pytest.mark.parametrize("dtype,hd", ATT_CASES)
@pytest.mark.parametrize("causal", [False, True])
def test_attention_with_scores(dtype, hd, causal):
    lens = [1, 17, 130, 300, 64]
    H = 4
    qkv, q, k, v = _qkv(lens, H, hd, dtype, seed=hd + causal)
    seqs = zsa.Seqs(lens, dev())
    out, lse, scores = zsa.attention_with_scores(q, k, v, H, seqs, causal)
    torch.cuda.synchronize()
    q64, k64, v64 = f64(q), f64(k), f64(v)
    o_ref, lse_ref, s_ref = [], [], []
    for b, n in enumerate(lens):
        lo = int(seqs.host[b])
        o, l, s = O.attention(q64[lo:lo + n], k64[lo:lo + n], v64[lo:lo + n], np.arange(n), H,
                              causal)
        o_ref.append(o)
        lse_ref.append(l)
        s_ref.append(s)
    o_ref = np.concatenate(o_ref)
    lse_ref = np.concatenate(lse_ref, axis=1)
    s_ref = np.concatenate(s_ref)
    assert_close(f64(out), o_ref, 1e-2 if dtype == "bf16" else 1e-5, "attention output")
    assert np.max(np.abs(lse.cpu().numpy() - lse_ref)) <= 2e-5 * max(1.0, np.abs(lse_ref).max())
    assert np.max(np.abs(scores.cpu().numpy() - s_ref) / s_ref) <= 1e-4
    assert abs(scores.cpu().double().sum() - H * sum(lens)) <= 1e-4 * H * sum(lens)


def test_all_sequences_empty():
    """A batch whose sequences are all empty (T = 0) and a norm of no rows:
    the calls return at once with empty results, through NULL row operands
    (torch gives zero-size tensors a null address)."""
    H, hd = 4, 64
    qkv, q, k, v = _qkv([0, 0, 0], H, hd, "bf16", seed=1)
    seqs = zsa.Seqs([0, 0, 0], dev())
    out, lse, scores = zsa.attention_with_scores(q, k, v, H, seqs, True)
    s2 = zsa.score_positions(q, k, lse, H, seqs, True)
    g = to_dev(np.ones(256, dtype=np.float32), "bf16")
    y = zsa.norm(to_dev(np.zeros((1, 256), dtype=np.float32), "bf16")[:0], g, g, zsa.NORM_LAYER)
    torch.cuda.synchronize()
    assert tuple(out.shape) == (0, H * hd) and tuple(lse.shape) == (H, 0)
    assert scores.numel() == 0 and s2.numel() == 0 and tuple(y.shape) == (0, 256)


@pytest.mark.parametrize("hd", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_attention_empty_sequences(hd, causal):
    """Zero-length sequences among others (every row of a sequence dropped
    upstream): their workgroups exit at once and the other sequences'
    outputs, log-sum-exp and scores match the oracle."""
    lens = [0, 5, 0, 300, 0, 33]
    H = 4
    qkv, q, k, v = _qkv(lens, H, hd, "bf16", seed=hd + 3 * causal)
    seqs = zsa.Seqs(lens, dev())
    out, lse, scores = zsa.attention_with_scores(q, k, v, H, seqs, causal)
    torch.cuda.synchronize()
    q64, k64, v64 = f64(q), f64(k), f64(v)
    o_ref, lse_ref, s_ref = [], [], []
    for b, n in enumerate(lens):
        if n == 0:
            continue
        lo = int(seqs.host[b])
        o, l, s = O.attention(q64[lo:lo + n], k64[lo:lo + n], v64[lo:lo + n], np.arange(n), H,
                              causal)
        o_ref.append(o)
        lse_ref.append(l)
        s_ref.append(s)
    o_ref = np.concatenate(o_ref)
    lse_ref = np.concatenate(lse_ref, axis=1)
    s_ref = np.concatenate(s_ref)
    assert_close(f64(out), o_ref, 1e-2, "attention output")
    assert np.max(np.abs(lse.cpu().numpy() - lse_ref)) <= 2e-5 * max(1.0, np.abs(lse_ref).max())
    assert np.max(np.abs(scores.cpu().numpy() - s_ref) / s_ref) <= 1e-4


@pytest.mark.parametrize("lens", [[100, 37], [300, 700]])   # 128- and 256-query blocks
@pytest.mark.parametrize("hd", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_attention_growing_scores(lens, hd, causal):
    """Key rows whose norm grows fivefold along the sequence: queries' running
    maxima grow by more than 2^8 in exp2 units after their first key tile
    (12 to 3107 such moves per case, counted on the host from these inputs),
    so the kernel moves its reference max and rescales its sums and
    accumulators mid-sequence, not only at the first tile."""
    H = 2
    g = np.random.default_rng(90 + hd + causal + len(lens))
    T, d = sum(lens), H * hd
    qkv = g.standard_normal((T, 3 * d)).astype(np.float32)
    qkv[:, :d] *= 1.5
    lo = 0
    for n in lens:
        qkv[lo:lo + n, d:2 * d] *= (1.0 + 4.0 * np.arange(n) / max(n - 1, 1))[:, None]
        lo += n
    t = to_dev(qkv, "bf16")
    q, k, v = t[:, :d], t[:, d:2 * d], t[:, 2 * d:]
    seqs = zsa.Seqs(lens, dev())
    out, lse, scores = zsa.attention_with_scores(q, k, v, H, seqs, causal)
    torch.cuda.synchronize()
    q64, k64, v64 = f64(q), f64(k), f64(v)
    o_ref, lse_ref, s_ref = [], [], []
    for b, n in enumerate(lens):
        lo = int(seqs.host[b])
        o, l, sc = O.attention(q64[lo:lo + n], k64[lo:lo + n], v64[lo:lo + n], np.arange(n), H,
                               causal)
        o_ref.append(o)
        lse_ref.append(l)
        s_ref.append(sc)
    assert_close(f64(out), np.concatenate(o_ref), 1e-2, "attention output")
    lse_ref = np.concatenate(lse_ref, axis=1)
    assert np.max(np.abs(lse.cpu().numpy() - lse_ref)) <= 2e-5 * max(1.0, np.abs(lse_ref).max())
    s_ref = np.concatenate(s_ref)
    assert np.max(np.abs(scores.cpu().numpy() - s_ref) / s_ref) <= 1e-4


@pytest.mark.parametrize("hd", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_attention_long_sequences(hd, causal):
    """Sequences past 512 rows take 256-query blocks of eight waves (ragged
    last block; a short sequence in the same launch)."""
    lens = [700, 90, 513]
    H = 2
    qkv, q, k, v = _qkv(lens, H, hd, "bf16", seed=70 + hd + causal)
    seqs = zsa.Seqs(lens, dev())
    out, lse, scores = zsa.attention_with_scores(q, k, v, H, seqs, causal)
    torch.cuda.synchronize()
    q64, k64, v64 = f64(q), f64(k), f64(v)
    o_ref, lse_ref, s_ref = [], [], []
    for b, n in enumerate(lens):
        lo = int(seqs.host[b])
        o, l, sc = O.attention(q64[lo:lo + n], k64[lo:lo + n], v64[lo:lo + n], np.arange(n), H,
                               causal)
        o_ref.append(o)
        lse_ref.append(l)
        s_ref.append(sc)
    assert_close(f64(out), np.concatenate(o_ref), 1e-2, "attention output")
    lse_ref = np.concatenate(lse_ref, axis=1)
    assert np.max(np.abs(lse.cpu().numpy() - lse_ref)) <= 2e-5 * max(1.0, np.abs(lse_ref).max())
    s_ref = np.concatenate(s_ref)
    assert np.max(np.abs(scores.cpu().numpy() - s_ref) / s_ref) <= 1e-4


@pytest.mark.parametrize("dtype,hd,hkv", [("bf16", 64, 2), ("bf16", 128, 1), ("f32", 32, 2),
                                          ("bf16", 64, 4)])
@pytest.mark.parametrize("causal", [False, True])
def test_attention_with_scores_gqa(dtype, hd, hkv, causal):
    """Grouped-query (hkv < H) and multi-query (hkv = 1) attention from one
    fused [q | k | v] buffer."""
    lens = [1, 17, 130, 300, 64]
    H = 4
    d, kvd = H * hd, hkv * hd
    g = np.random.default_rng(30 + hd + hkv + causal)
    fused = g.standard_normal((sum(lens), d + 2 * kvd)).astype(np.float32)
    fused[:, :d] *= 1.5
    t = to_dev(fused, dtype)
    q, k, v = t[:, :d], t[:, d:d + kvd], t[:, d + kvd:]
    seqs = zsa.Seqs(lens, dev())
    out, lse, scores = zsa.attention_with_scores(q, k, v, H, seqs, causal, n_kv_heads=hkv)
    torch.cuda.synchronize()
    q64, k64, v64 = f64(q), f64(k), f64(v)
    o_ref, lse_ref, s_ref = [], [], []
    for b, n in enumerate(lens):
        lo = int(seqs.host[b])
        o, l, s = O.attention(q64[lo:lo + n], k64[lo:lo + n], v64[lo:lo + n], np.arange(n), H,
                              causal, True, hkv)
        o_ref.append(o)
        lse_ref.append(l)
        s_ref.append(s)
    o_ref = np.concatenate(o_ref)
    lse_ref = np.concatenate(lse_ref, axis=1)
    s_ref = np.concatenate(s_ref)
    assert_close(f64(out), o_ref, 1e-2 if dtype == "bf16" else 1e-5, "attention output")
    assert np.max(np.abs(lse.cpu().numpy() - lse_ref)) <= 2e-5 * max(1.0, np.abs(lse_ref).max())
    assert np.max(np.abs(scores.cpu().numpy() - s_ref) / s_ref) <= 1e-4


@pytest.mark.parametrize("dtype,hd", [("bf16", 64), ("bf16", 128), ("f32", 32)])
@pytest.mark.parametrize("causal", [False, True])
def test_score_positions_from_oracle_lse(dtype, hd, causal):
    lens = [300, 9, 64, 129]
    H = 3
    qkv, q, k, v = _qkv(lens, H, hd, dtype, seed=11 + hd, sharp=2.0)
    seqs = zsa.Seqs(lens, dev())
    q64, k64, v64 = f64(q), f64(k), f64(v)
    lse_ref, s_ref = [], []
    for b, n in enumerate(lens):
        lo = int(seqs.host[b])
        _, l, s = O.attention(q64[lo:lo + n], k64[lo:lo + n], v64[lo:lo + n], np.arange(n), H, causal)
        lse_ref.append(l)
        s_ref.append(s)
    lse_ref = np.concatenate(lse_ref, axis=1)
    s_ref = np.concatenate(s_ref)
    lse_d = torch.from_numpy(lse_ref.astype(np.float32)).to(dev())
    s = zsa.score_positions(q, k, lse_d, H, seqs, causal)
    torch.cuda.synchronize()
    assert np.max(np.abs(s.cpu().numpy() - s_ref) / s_ref) <= 1e-4
    s2 = zsa.score_positions(q, k, lse_d, H, seqs, causal)
    assert torch.equal(s, s2)   # fixed reduction order: bitwise reproducible


def test_uniform_attention_scores_closed_form():
    # all-zero queries: every row spreads its mass uniformly over the rows it sees
    lens = [50, 7, 200]
    H, hd = 4, 64
    qkv, q, k, v = _qkv(lens, H, hd, "bf16", seed=2)
    q.zero_()
    seqs = zsa.Seqs(lens, dev())
    for causal in (False, True):
        _, _, s = zsa.attention_with_scores(q, k, v, H, seqs, causal)
        torch.cuda.synchronize()
        s = s.cpu().double().numpy()
        for b, n in enumerate(lens):
            lo = int(seqs.host[b])
            if causal:
                harm = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, n + 1))])
                expect = H * (harm[n] - harm[np.arange(n)])
            else:
                expect = np.full(n, float(H))
            assert np.allclose(s[lo:lo + n], expect, rtol=1e-5)
