"""Shared helpers of the parity tests (no tests here)."""
import numpy as np
import torch

from oracle import zsa_oracle as O
from paper_2509_01190_amd import workloads as W


def dev():
    return torch.device("cuda:0")


def to_dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    return W.to_storage(a, dtype).to(dev())


def f64(t: torch.Tensor) -> np.ndarray:
    return W.as_f64(t)


def rel_l2(got: np.ndarray, ref: np.ndarray) -> float:
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def assert_close(got: np.ndarray, ref: np.ndarray, rtol: float, what: str = "") -> None:
    """Relative L2 error <= rtol, and elementwise |d| <= rtol*|ref| + rtol*rms(ref)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if ref.size == 0:
        return
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    e = rel_l2(got, ref)
    assert e <= rtol, f"{what}: relative L2 error {e:.3e} > {rtol:.1e}"
    rms = float(np.sqrt(np.mean(ref * ref)))
    bound = rtol * np.abs(ref) + rtol * rms
    worst = np.max(np.abs(got - ref) - bound)
    assert worst <= 0, f"{what}: elementwise error above bound by {worst:.3e}"


def assert_rel_l2(got: np.ndarray, ref: np.ndarray, tol: float, what: str = "") -> None:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    e = rel_l2(got, ref)
    assert e <= tol, f"{what}: relative L2 error {e:.3e} > {tol:.1e}"


def assert_rows_close(got: np.ndarray, ref: np.ndarray, tol: float, what: str = "") -> None:
    """Every row's relative L2 error <= tol (a row that went to the wrong
    place, or was rotated with the wrong position, is off by O(1))."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if ref.size == 0:
        return
    num = np.linalg.norm(got - ref, axis=1)
    den = np.maximum(np.linalg.norm(ref, axis=1), 1e-30)
    worst = int(np.argmax(num / den))
    assert num[worst] / den[worst] <= tol, \
        f"{what}: row {worst} relative error {num[worst] / den[worst]:.3e} > {tol:.1e}"


def modes(dtype: str):
    """(mode for hidden-state L2 tolerance, mode for scores / kept sets and
    the elementwise check): bf16 storage is judged in L2 against the exact
    oracle and elementwise against the oracle that rounds at the same
    storage points."""
    return ("exact", "bf16") if dtype == "bf16" else ("exact", "exact")


def weights_f64(w):
    return {k: (None if v is None else W.as_f64(v)) for k, v in w.items()}


def dev_weights(w_np, dtype):
    return {k: (None if v is None else to_dev(v, dtype)) for k, v in w_np.items()}


def check_kept_sets(gpu_scores, ref_scores, k, kept_gpu, kept_ref, eps, what="",
                    keep_last=False):
    """Kept-set agreement for one sequence.

    Exact: the GPU kept set is the oracle's top-k of the GPU's own scores.
    Margin: the GPU scores are within eps of the oracle's, and every row the
    two kept sets disagree on has an oracle score within eps of the oracle's
    k-th score (the decision there is inside the numerical tolerance).
    Returns the number of such swaps."""
    gpu_scores = np.asarray(gpu_scores, dtype=np.float64)
    ref_scores = np.asarray(ref_scores, dtype=np.float64)
    kept_gpu = np.asarray(kept_gpu, dtype=np.int64)
    kept_ref = np.asarray(kept_ref, dtype=np.int64)
    own = O.select_topk(gpu_scores, k, keep_last)
    assert np.array_equal(kept_gpu, own), f"{what}: GPU kept set is not the top-k of its own scores"
    scale = np.maximum(np.abs(ref_scores), 1e-30)
    rel = np.max(np.abs(gpu_scores - ref_scores) / scale) if ref_scores.size else 0.0
    assert rel <= eps, f"{what}: score error {rel:.3e} > {eps:.1e}"
    diff = np.setxor1d(kept_gpu, kept_ref)
    if diff.size == 0 or k == 0:
        return 0
    # with keep_last the last row is fixed and k - 1 are chosen among the rest
    cand, kk = (ref_scores[:-1], k - 1) if keep_last else (ref_scores, k)
    assert kk > 0, f"{what}: kept sets differ where only the last row is kept"
    s_star = np.sort(cand)[::-1][kk - 1]
    amb = np.abs(ref_scores[diff] - s_star) <= 2 * eps * abs(s_star)
    assert amb.all(), f"{what}: kept sets differ at unambiguous rows {diff[~amb]}"
    return int(diff.size // 2)
