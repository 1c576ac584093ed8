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


# Tolerances (the reasoning and the measurements behind them are recorded with
# the design notes on precision):
#  * hidden states: relative L2 error per sequence against the exact float64
#    oracle, at every layer output: 2e-2 (bf16 storage) or 1e-4 (fp32);
#  * every row: its relative L2 error against the exact oracle is at most
#    ROW_FACTOR times the error bf16 storage alone causes on that row (the
#    oracle that rounds where the GPU stores bf16, against the exact one), and
#    never needs to be below the sequence tolerance;
#  * scores: the largest error against the exact oracle, relative to
#    max(|score|, mean score), is at most SCORE_FACTOR times the emulation
#    oracle's own, and never needs to be below SCORE_FLOOR (what identical
#    bf16 inputs give: fp32 sums and exp2).
SEQ_TOL = {"bf16": 2e-2, "f32": 1e-4}
ROW_FACTOR = 2.0
SCORE_FACTOR = 2.0
SCORE_FLOOR = {"bf16": 1e-4, "f32": 1e-5}


def row_errors(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    num = np.linalg.norm(np.asarray(got, np.float64) - np.asarray(ref, np.float64), axis=1)
    den = np.maximum(np.linalg.norm(np.asarray(ref, np.float64), axis=1), 1e-30)
    return num / den


def assert_rows_vs_exact(got: np.ndarray, ref_x: np.ndarray, ref_e: np.ndarray, tol: float,
                         what: str = "", factor: float = ROW_FACTOR) -> float:
    """Every row's relative L2 error against the exact oracle ``ref_x`` is at
    most max(tol, factor * the emulation oracle ``ref_e``'s error on that
    row). Returns the largest ratio of a row's error to its bound."""
    got = np.asarray(got, dtype=np.float64)
    assert got.shape == ref_x.shape == ref_e.shape, (what, got.shape, ref_x.shape, ref_e.shape)
    if ref_x.size == 0:
        return 0.0
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    e_gpu = row_errors(got, ref_x)
    e_emu = row_errors(ref_e, ref_x)
    bound = np.maximum(tol, factor * e_emu)
    worst = int(np.argmax(e_gpu / bound))
    assert e_gpu[worst] <= bound[worst], (
        f"{what}: row {worst} relative error {e_gpu[worst]:.3e} > bound {bound[worst]:.3e} "
        f"(bf16 storage alone: {e_emu[worst]:.3e})")
    return float(e_gpu[worst] / bound[worst])


def max_rel(a: np.ndarray, ref: np.ndarray) -> float:
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    return float(np.max(np.abs(a - ref) / np.maximum(np.abs(ref), 1e-30)))


def score_err(a: np.ndarray, ref: np.ndarray) -> float:
    """Largest score error relative to max(|score|, mean score): relative
    for the scores that can decide a kept set, and measured against the
    mean (the number of heads: each query row's probabilities sum to one)
    for the small scores of rows far below any threshold, whose own
    relative error says nothing about the selection."""
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    scale = np.maximum(np.abs(ref), max(float(np.mean(np.abs(ref))), 1e-30))
    return float(np.max(np.abs(a - ref) / scale))


def score_eps_from(emul_err: float, dtype: str) -> float:
    """Score tolerance from the emulation oracle's largest relative score
    error: SCORE_FACTOR times it, at least the floor."""
    return max(SCORE_FLOOR[dtype], SCORE_FACTOR * emul_err)


def score_eps(s_emu: np.ndarray, s_exact: np.ndarray, dtype: str) -> float:
    """The score tolerance of one sequence at one pruning point: SCORE_FACTOR
    times the emulation oracle's largest relative error, at least the floor."""
    return score_eps_from(score_err(s_emu, s_exact), dtype)


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
                    keep_last=False, exact_scores=None):
    """Kept-set agreement for one sequence.

    Exact: the GPU kept set is the oracle's top-k of the GPU's own scores.
    Margin: the GPU scores are within eps of the oracle's (of
    ``exact_scores`` when given), and every row the two kept sets disagree on
    has an oracle score within 2 eps of the oracle's k-th score (the decision
    there is inside the numerical tolerance). Returns the number of such
    swaps."""
    gpu_scores = np.asarray(gpu_scores, dtype=np.float64)
    ref_scores = np.asarray(ref_scores, dtype=np.float64)
    kept_gpu = np.asarray(kept_gpu, dtype=np.int64)
    kept_ref = np.asarray(kept_ref, dtype=np.int64)
    own = O.select_topk(gpu_scores, k, keep_last)
    assert np.array_equal(kept_gpu, own), f"{what}: GPU kept set is not the top-k of its own scores"
    against = ref_scores if exact_scores is None else np.asarray(exact_scores, np.float64)
    rel = score_err(gpu_scores, against)
    assert rel <= eps, f"{what}: score error {rel:.3e} > {eps:.3e}"
    diff = np.setxor1d(kept_gpu, kept_ref)
    if diff.size == 0 or k == 0:
        return 0
    # with keep_last the last row is fixed and k - 1 are chosen among the rest
    cand, kk = (ref_scores[:-1], k - 1) if keep_last else (ref_scores, k)
    assert kk > 0, f"{what}: kept sets differ where only the last row is kept"
    s_star = np.sort(cand)[::-1][kk - 1]
    band = 2 * eps * max(abs(s_star), float(np.mean(np.abs(ref_scores))))
    amb = np.abs(ref_scores[diff] - s_star) <= band
    assert amb.all(), f"{what}: kept sets differ at unambiguous rows {diff[~amb]}"
    return int(diff.size // 2)
