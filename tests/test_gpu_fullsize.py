"""Parity at the full workload sizes, in the launch configuration the
benchmark times, at every keep rate the benchmark sweeps: the GPU runs the
whole batch, the oracle recomputes sampled sequences one by one (sequences
are independent under the method), continuing on the GPU's kept sets.
Standard random-init weights. Every layer's output is held to the
per-sequence relative-L2 tolerance against the exact float64 oracle and
every row to twice what bf16 storage alone does to it; scores to twice the
emulation oracle's own error; kept sets exactly to the top-k of the GPU's
scores, and to the oracle's choice up to swaps inside the score tolerance,
whose number is reported and bounded."""
import pytest

from paper_2509_01190_amd import workloads as W
from tests.test_gpu_stack import build, compare_stack

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

# Swaps with the oracle's kept set happen only between rows whose scores lie
# within the score tolerance of the k-th score. On random-init weights the
# scores crowd around it (a quarter to two fifths of a bert sequence's rows
# lie within 1 % of it), yet at most one kept row in a few hundred was seen
# to swap; more than one in a hundred would mean scores off by more than
# their error budget near the threshold.
MAX_SWAP_SHARE = 0.01


def run(name, seed, rate, seqs, qk_sharp=1.0):
    p = W.PRESETS[name]
    lens, stack, xd, posd, dws, ocfg = build(p, seed, norm_jitter=False, qk_sharp=qk_sharp)
    rates = W.keep_rates(p, seed, rate)
    st = compare_stack(p, lens, stack, xd, posd, dws, ocfg, rates, seqs_check=seqs,
                       label=f"{name} seed {seed} keep rate {rate}"
                             + (f" query/key scale {qk_sharp}" if qk_sharp != 1.0 else ""))
    assert st["swaps"] <= MAX_SWAP_SHARE * max(st["kept"], 1) + 1, st["swaps"]
    return st


@pytest.mark.parametrize("rate", [1.0, 0.7, 0.5, 0.3, 0.1])
def test_bert_full(rate):
    run("bert", 0, rate, [0, 21])


@pytest.mark.parametrize("seed,seqs", [(1, [7]), (2, [30])])
def test_bert_full_other_seeds(seed, seqs):
    run("bert", seed, 0.5, seqs)


def test_bert_full_sharpened():
    # query and key weights scaled by 2 (attention logits by 4, from a std of
    # about 0.3 to 1.3): scores spread out, so fewer rows sit near the
    # threshold and the kept set is decided by wider margins
    run("bert", 0, 0.5, [4], qk_sharp=2.0)


@pytest.mark.parametrize("rate", [1.0, 0.5, 0.25, 0.1])
def test_dec1b_full(rate):
    run("dec1b", 0, rate, [5])


@pytest.mark.parametrize("seed,seqs", [(1, [2]), (2, [6])])
def test_dec1b_full_other_seeds(seed, seqs):
    run("dec1b", seed, 0.5, seqs)


@pytest.mark.parametrize("rate", [1.0, 0.5, 0.2, 0.09])
def test_dec7b_full(rate):
    run("dec7b", 0, rate, [2])


def test_ragged_full():
    p = W.PRESETS["ragged"]
    lens = W.lengths(p, 0)
    order = sorted(range(len(lens)), key=lambda b: lens[b])
    run("ragged", 0, None, [order[0], order[-1]])


@pytest.mark.parametrize("rate", [0.7, 0.3])
def test_gpt2_every_layer_full(rate):
    run("gpt2", 0, rate, [3])


@pytest.mark.parametrize("name,rate,seq", [("gpt2_n128", 0.3, 100), ("gpt2_n1024", 0.5, 9)])
def test_gpt2_every_layer_other_lengths(name, rate, seq):
    run(name, 0, rate, [seq])


def test_llama3_gqa_keep_last_full():
    run("llama3_8b", 0, 0.2, [1])
