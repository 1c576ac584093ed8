"""The attention-with-scores entry point that allocates nothing (its scratch
is a static device buffer) against the workspace entry point, through the
C-ABI: identical outputs on two calls in a row, the second smaller, and a
clear refusal of a call whose scratch would not fit."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2509_01190_amd import zsa
from tests.helpers import dev

pytestmark = pytest.mark.gpu


def _inputs(lens, H, Hkv, hd, seed):
    g = torch.Generator().manual_seed(seed)
    T = sum(lens)
    width = (H + 2 * Hkv) * hd
    qkv = (torch.randn(T, width, generator=g) * 0.7).to(torch.bfloat16).to(dev())
    return qkv, zsa.Seqs(lens, dev())


def _run(static, qkv, seqs, H, Hkv, hd, causal, want_lse, want_scores):
    lib = zsa.lib()
    T = qkv.shape[0]
    d, kvd = H * hd, Hkv * hd
    q, k, v = qkv[:, :d], qkv[:, d:d + kvd], qkv[:, d + kvd:]
    rs = qkv.stride(0)
    out = torch.full((T, d), 7.0, dtype=torch.bfloat16, device=dev())
    lse = torch.full((H, T), 7.0, dtype=torch.float32, device=dev()) if want_lse else None
    scores = torch.full((T,), 7.0, dtype=torch.float32, device=dev()) if want_scores else None
    scale = 1.0 / float(np.sqrt(hd))
    common = (zsa._stream(qkv.device), zsa.BF16, zsa._p(q), zsa._p(k), zsa._p(v), rs, H, Hkv, hd,
              int(causal), scale, seqs.batch, zsa._hp32(seqs.host), zsa._p(seqs.dev), zsa._p(out),
              d, zsa._p(lse), zsa._p(scores))
    if static:
        rc = lib.zsa_attention_with_scores_static(*common)
    else:
        wsz = int(lib.zsa_attention_workspace_size(H, T, int(want_scores)))
        ws = torch.empty(max(wsz, 1), dtype=torch.uint8, device=dev())
        rc = lib.zsa_attention_with_scores(*common, zsa._p(ws), wsz)
    assert rc == zsa.OK, lib.zsa_last_error().decode()
    torch.cuda.synchronize()
    return out, lse, scores


CALLS = [
    # lengths, query heads, key/value heads, head_dim, causal, want lse, want scores
    ([700, 1030, 33, 512], 8, 2, 128, True, False, True),   # lse and partials in the scratch
    ([100, 5], 4, 4, 64, False, True, True),                 # smaller: partials only
]


def test_static_scratch_matches_workspace_entry_point():
    assert zsa.lib().zsa_static_scratch_bytes() == 32 << 20
    for i, (lens, H, Hkv, hd, causal, want_lse, want_scores) in enumerate(CALLS):
        qkv, seqs = _inputs(lens, H, Hkv, hd, seed=11 + i)
        ref = _run(False, qkv, seqs, H, Hkv, hd, causal, want_lse, want_scores)
        got = _run(True, qkv, seqs, H, Hkv, hd, causal, want_lse, want_scores)
        for name, a, b in zip(("out", "lse", "scores"), got, ref):
            if b is None:
                assert a is None
                continue
            assert torch.equal(a, b), f"call {i}: {name} differs"
        # the scores are those of a normalised soft-score matrix: total mass
        # is the number of heads times the rows of each sequence
        s = got[2].cpu().numpy().astype(np.float64)
        lo = 0
        for n in lens:
            assert abs(s[lo:lo + n].sum() - H * n) <= 1e-4 * H * n
            lo += n


def test_static_scratch_refuses_what_does_not_fit():
    lib = zsa.lib()
    # 32 heads x 200000 rows: log-sum-exp rows and partials need about 51 MB
    cu = np.array([0, 200000], dtype=np.int32)
    fake = ctypes.c_void_p(0x1000)
    rc = lib.zsa_attention_with_scores_static(None, zsa.BF16, fake, fake, fake, 3 * 4096, 32, 0,
                                              128, 1, 0.1, 1, cu.ctypes.data_as(zsa._pi32),
                                              fake, fake, 4096, None, fake)
    assert rc == zsa.EUNSUPPORTED
    assert "static scratch" in lib.zsa_last_error().decode()
