"""The C-ABI library on the CPU: it loads, exports every symbol the header
declares, its host-only Eq. 2 schedule agrees with the oracle's, and its
argument validation rejects bad calls before touching the GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import zsa_oracle as O
from paper_2509_01190_amd import zsa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "zsa.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(zsa_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = zsa.lib()
    names = _declared()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(zsa.EXPORTED)


def test_version_and_error_text():
    assert "gfx950" in zsa.version()
    with pytest.raises(zsa.ZsaError) as e:
        zsa.keep_count(10, 1.5, 5)
    assert e.value.code == zsa.EINVAL
    assert "keep rate" in zsa.lib().zsa_last_error().decode()


def test_keep_count_matches_oracle():
    rng = np.random.default_rng(0)
    rates = list(np.linspace(0, 1, 201)) + list(rng.uniform(0, 1, 300)) + \
        [0.57, 0.29, 0.09, 0.7, 0.3, 0.1, 0.99, 0.98, 0.97, 0.96]
    for n in [0, 1, 3, 5, 7, 40, 64, 100, 128, 512, 2048, 4096, 9999]:
        for a in rates:
            for tau in (1, 5):
                assert zsa.keep_count(n, float(a), tau) == O.keep_count(n, float(a), tau), (n, a, tau)


def test_keep_schedule_matches_oracle():
    rng = np.random.default_rng(1)
    lens = rng.integers(0, 5000, 64)
    rates = rng.uniform(0.0, 1.0, 64)
    got = zsa.keep_schedule(lens, rates, 5, 4)
    ref = O.keep_schedule(list(lens), list(rates), 5, 4)
    assert np.array_equal(got, np.array(ref))


@pytest.mark.parametrize("bad", [float("nan"), -1e-12, 1.0000001, float("inf")])
def test_keep_schedule_rejects_bad_rates(bad):
    with pytest.raises(zsa.ZsaError) as e:
        zsa.keep_schedule([10, 10], [0.5, bad], 5, 1)
    assert e.value.code == zsa.EINVAL


def test_validation_happens_before_any_launch():
    lib = zsa.lib()
    # unknown dtype
    assert lib.zsa_norm(None, 7, 0, None, None, None, 4, 64, 1e-5, None) == zsa.EINVAL
    # misaligned pointer
    assert lib.zsa_norm(None, zsa.F32, 0, ctypes.c_void_p(0x1004), ctypes.c_void_p(0x2000), None, 4,
                        64, 1e-5, ctypes.c_void_p(0x3000)) == zsa.EALIGN
    # row length not a multiple of 16 bytes
    assert lib.zsa_norm(None, zsa.BF16, 0, ctypes.c_void_p(0x1000), ctypes.c_void_p(0x2000), None,
                        4, 12, 1e-5, ctypes.c_void_p(0x3000)) == zsa.EALIGN
    # unsupported head_dim
    cu = np.array([0, 8], dtype=np.int32)
    rc = lib.zsa_attention_with_scores(None, zsa.BF16, ctypes.c_void_p(0x1000),
                                       ctypes.c_void_p(0x1000), ctypes.c_void_p(0x1000), 96, 2, 0,
                                       48, 0, 0.1, 1, cu.ctypes.data_as(zsa._pi32),
                                       ctypes.c_void_p(0x4000), ctypes.c_void_p(0x5000), 96, None,
                                       None, None, 0)
    assert rc == zsa.EUNSUPPORTED
    # key/value heads that do not divide the query heads
    rc = lib.zsa_attention_with_scores(None, zsa.BF16, ctypes.c_void_p(0x1000),
                                       ctypes.c_void_p(0x1000), ctypes.c_void_p(0x1000), 384, 6, 4,
                                       64, 0, 0.1, 1, cu.ctypes.data_as(zsa._pi32),
                                       ctypes.c_void_p(0x4000), ctypes.c_void_p(0x5000), 384, None,
                                       None, None, 0)
    assert rc == zsa.ESHAPE
    # cu not monotone
    cu = np.array([0, 8, 4], dtype=np.int32)
    rc = lib.zsa_select_topk(None, ctypes.c_void_p(0x1000), 2, cu.ctypes.data_as(zsa._pi32),
                             ctypes.c_void_p(0x2000), cu.ctypes.data_as(zsa._pi32), 0,
                             ctypes.c_void_p(0x3000), ctypes.c_void_p(0x4000), 1024)
    assert rc == zsa.ESHAPE
    # k > n
    cu = np.array([0, 8], dtype=np.int32)
    k = np.array([9], dtype=np.int32)
    rc = lib.zsa_select_topk(None, ctypes.c_void_p(0x1000), 1, cu.ctypes.data_as(zsa._pi32),
                             ctypes.c_void_p(0x2000), k.ctypes.data_as(zsa._pi32), 0,
                             ctypes.c_void_p(0x3000), ctypes.c_void_p(0x4000), 1024)
    assert rc == zsa.ESHAPE
    # workspace too small
    k = np.array([4], dtype=np.int32)
    rc = lib.zsa_select_topk(None, ctypes.c_void_p(0x1000), 1, cu.ctypes.data_as(zsa._pi32),
                             ctypes.c_void_p(0x2000), k.ctypes.data_as(zsa._pi32), 1,
                             ctypes.c_void_p(0x3000), ctypes.c_void_p(0x4000), 4)
    assert rc == zsa.EWORKSPACE


def test_layer_config_validation():
    lib = zsa.lib()
    cfg = zsa.make_cfg(zsa.ENCODER, 768, 12, 3072, False, zsa.BF16)
    cfg.tau = 0
    cu = np.array([0, 16], dtype=np.int32)
    w = zsa.LayerWeights(*([0x1000] * 12))
    rc = lib.zsa_layer_forward(None, ctypes.byref(cfg), ctypes.byref(w), ctypes.c_void_p(0x1000),
                               ctypes.c_void_p(0x2000), 1, cu.ctypes.data_as(zsa._pi32),
                               ctypes.c_void_p(0x3000), None, ctypes.c_void_p(0x4000),
                               ctypes.c_void_p(0x5000), cu.ctypes.data_as(zsa._pi32),
                               ctypes.c_void_p(0x6000), None, None, ctypes.c_void_p(0x7000), 1)
    assert rc == zsa.EINVAL
    cfg = zsa.make_cfg(zsa.DECODER, 768, 12, 3072, True, zsa.BF16, n_kv_heads=5)  # 5 does not divide 12
    rc = lib.zsa_layer_forward(None, ctypes.byref(cfg), ctypes.byref(w), ctypes.c_void_p(0x1000),
                               ctypes.c_void_p(0x2000), 1, cu.ctypes.data_as(zsa._pi32),
                               ctypes.c_void_p(0x3000), None, ctypes.c_void_p(0x4000),
                               ctypes.c_void_p(0x5000), cu.ctypes.data_as(zsa._pi32),
                               ctypes.c_void_p(0x6000), None, None, ctypes.c_void_p(0x7000), 1)
    assert rc == zsa.ESHAPE
    # grouped-query attention shrinks the fused projection (and its workspace)
    mha = zsa.make_cfg(zsa.DECODER, 4096, 32, 14336, True, zsa.BF16)
    gqa = zsa.make_cfg(zsa.DECODER, 4096, 32, 14336, True, zsa.BF16, n_kv_heads=8)
    assert lib.zsa_layer_workspace_size(ctypes.byref(gqa), 4096, 1) < \
        lib.zsa_layer_workspace_size(ctypes.byref(mha), 4096, 1)
    cfg = zsa.make_cfg(zsa.ENCODER, 768, 10, 3072, False, zsa.BF16)   # 768 / 10 is not integral
    assert lib.zsa_layer_workspace_size(ctypes.byref(cfg), 16, 1) > 0
    rc = lib.zsa_layer_forward(None, ctypes.byref(cfg), ctypes.byref(w), ctypes.c_void_p(0x1000),
                               ctypes.c_void_p(0x2000), 1, cu.ctypes.data_as(zsa._pi32),
                               ctypes.c_void_p(0x3000), None, ctypes.c_void_p(0x4000),
                               ctypes.c_void_p(0x5000), cu.ctypes.data_as(zsa._pi32),
                               ctypes.c_void_p(0x6000), None, None, ctypes.c_void_p(0x7000), 1)
    assert rc == zsa.ESHAPE


def test_workspace_sizes_grow_with_rows():
    cfg = zsa.make_cfg(zsa.DECODER, 4096, 32, 11008, True, zsa.BF16)
    lib = zsa.lib()
    a = lib.zsa_stack_workspace_size(ctypes.byref(cfg), 1024, 4, 1)
    b = lib.zsa_stack_workspace_size(ctypes.byref(cfg), 16384, 4, 1)
    assert 0 < a < b
    assert b < 4 << 30   # a 7B-shaped 16k-row slice needs well under 4 GiB of scratch


def test_linear_split_k_workspace():
    ws = zsa.linear_workspace_size
    # a 160-row down projection (12 output tiles) is split; 12 slices of K
    assert ws(zsa.BF16, 160, 768, 3072) == 12 * 160 * 768 * 4
    # grids that fill the GPU, fp32, and K too short to split are not
    assert ws(zsa.BF16, 16384, 2304, 768) == 0
    assert ws(zsa.F32, 160, 768, 3072) == 0
    assert ws(zsa.BF16, 160, 768, 256) == 0
    assert ws(zsa.BF16, 160, 768, 768) == 0
    # 96 tiles of a 2048-row down projection: 5 slices (one round of 480 workgroups)
    assert ws(zsa.BF16, 2048, 768, 3072) == 5 * 2048 * 768 * 4
    assert ws(zsa.BF16, 0, 768, 3072) == 0
    # a workspace below the need is refused before any launch
    lib = zsa.lib()
    rc = lib.zsa_linear(None, zsa.BF16, ctypes.c_void_p(0x1000), 160, 3072, ctypes.c_void_p(0x2000),
                        768, None, zsa.EPI_NONE, None, None, 0, 0, 1e4, ctypes.c_void_p(0x3000),
                        ctypes.c_void_p(0x4000), 1024)
    assert rc == zsa.EWORKSPACE
    # the layer workspace covers the split of every projection at any row count
    cfg = zsa.make_cfg(zsa.ENCODER, 768, 12, 3072, False, zsa.BF16)
    small = lib.zsa_layer_workspace_size(ctypes.byref(cfg), 160, 32)
    assert small >= ws(zsa.BF16, 160, 768, 3072)


def test_stack_rejects_misshaped_weights():
    import torch
    from paper_2509_01190_amd import workloads as W
    p = W.shrink(W.PRESETS["dec1b"], n_layers=1, d_model=256, n_heads=4, d_ff=256, n_kv_heads=2)
    cfg = zsa.make_cfg(p.kind, p.d_model, p.n_heads, p.d_ff, True, zsa.BF16, n_kv_heads=2)
    good = {k: (None if v is None else torch.from_numpy(v)) for k, v in W.layer_weights(p, 0).items()}
    assert tuple(good["w_qkv"].shape) == (256 + 2 * 2 * 64, 256)
    zsa.Stack(cfg, [good])
    bad = dict(good)
    bad["w_qkv"] = torch.zeros(3 * 256, 256)        # the MHA shape under a GQA config
    with pytest.raises(ValueError):
        zsa.Stack(cfg, [bad])
    bad = dict(good)
    bad["w_down"] = None
    with pytest.raises(ValueError):
        zsa.Stack(cfg, [bad])


def test_rows_beyond_32bit_offsets_are_refused():
    # the attention kernels reach a sequence's K/V rows through 32-bit byte
    # offsets: a sequence whose rows span 4 GiB (here 180000 rows of a
    # 7B-shaped fused q|k|v projection, 12288 bf16 wide) is refused up front
    lib = zsa.lib()
    row = 3 * 4096
    cu = np.array([0, 180000], dtype=np.int32)
    rc = lib.zsa_attention_with_scores(None, zsa.BF16, ctypes.c_void_p(0x1000),
                                       ctypes.c_void_p(0x1000), ctypes.c_void_p(0x1000), row, 32,
                                       0, 128, 1, 0.1, 1, cu.ctypes.data_as(zsa._pi32),
                                       ctypes.c_void_p(0x4000), ctypes.c_void_p(0x5000), 4096,
                                       ctypes.c_void_p(0x6000), None, None, 0)
    assert rc == zsa.EUNSUPPORTED
    assert "4 GiB" in lib.zsa_last_error().decode()
    # one row fewer than the limit passes this check (and fails later on the
    # missing workspace, still before any launch)
    n_ok = (1 << 32) // (row * 2) - 256 - 1
    cu = np.array([0, n_ok], dtype=np.int32)
    rc = lib.zsa_attention_with_scores(None, zsa.BF16, ctypes.c_void_p(0x1000),
                                       ctypes.c_void_p(0x1000), ctypes.c_void_p(0x1000), row, 32,
                                       0, 128, 1, 0.1, 1, cu.ctypes.data_as(zsa._pi32),
                                       ctypes.c_void_p(0x4000), ctypes.c_void_p(0x5000), 4096,
                                       None, ctypes.c_void_p(0x7000), None, 0)
    assert rc == zsa.EWORKSPACE
    # the same limit through the layer entry point (its q|k|v rows)
    cfg = zsa.make_cfg(zsa.DECODER, 4096, 32, 11008, True, zsa.BF16)
    w = zsa.LayerWeights(*([0x1000] * 12))
    cu = np.array([0, 180000], dtype=np.int32)
    rc = lib.zsa_layer_forward(None, ctypes.byref(cfg), ctypes.byref(w), ctypes.c_void_p(0x1000),
                               ctypes.c_void_p(0x2000), 1, cu.ctypes.data_as(zsa._pi32),
                               ctypes.c_void_p(0x3000), None, ctypes.c_void_p(0x4000),
                               ctypes.c_void_p(0x5000), cu.ctypes.data_as(zsa._pi32),
                               ctypes.c_void_p(0x6000), None, None, ctypes.c_void_p(0x7000), 1)
    assert rc == zsa.EUNSUPPORTED
    # and for a decode step's cache slot (2 * 4096 bf16 per row: 262144 rows)
    x = ctypes.c_void_p(0x10000)
    pos = np.zeros(1, dtype=np.int32)
    kvl = np.zeros(1, dtype=np.int32)
    rc = lib.zsa_decode_step(None, ctypes.byref(cfg), ctypes.byref(w), 1, 1, x,
                             pos.ctypes.data_as(zsa._pi32), ctypes.c_void_p(0x20000), 262144,
                             kvl.ctypes.data_as(zsa._pi32), x, ctypes.c_void_p(0x30000), 1)
    assert rc == zsa.EUNSUPPORTED
