"""Pins of the fp64 selection oracle (Sec. 5.3) against hand-worked examples, exact-rational
brute force, the budget table and a distributional fact of the synthetic inputs."""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2602_06161_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "select_examples.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


@pytest.mark.parametrize("ex", _golden()["examples"], ids=lambda e: e["name"])
def test_hand_worked_examples(ex):
    f32 = lambda x: np.array([x], np.float32)
    si, ns, score = oracle.select(f32(ex["logp"]), f32(ex["d_in"]), f32(ex["d_out"]),
                                  np.array([ex["flags"]], np.uint8), ex["max_seeds"], ex["pos_offset"])
    assert si[0].tolist() == ex["seed_idx"], ex["why"]
    assert int(ns[0]) == ex["n_seed"], ex["why"]
    assert score[0].tolist() == [float(v) for v in ex["score"]], ex["why"]


def test_budget_table():
    t = _golden()["budget_table"]
    for c, k in zip(t["c"], t["k"]):
        # c positions scoring 2 and one scoring 0: mean 2c/(c+1) < 2, so exactly c lie above it
        logp = np.array([[-2.0] * c + [0.0]], np.float32)
        z = np.zeros_like(logp)
        fl = np.ones(logp.shape, np.uint8)
        si, ns, _ = oracle.select(logp, z, z, fl, 64)
        assert int(ns[0]) == k, (c, k)
        assert si[0, :k].tolist() == list(range(k))


def _brute(logp, d_in, d_out, flags, max_seeds):
    """Exact-rational reference on dyadic inputs: the score, mean and count are exact."""
    U = [j for j in range(len(logp)) if flags[j] & 1]
    s = {j: Fraction(-float(logp[j])) * (1 + Fraction(float(d_in[j]))) / (1 + Fraction(float(d_out[j])))
         for j in U}
    if not U:
        return []
    mean = sum(s.values()) / len(U)
    c = sum(1 for j in U if s[j] > mean)
    k = math.isqrt(c)
    k = k if k * k == c else k + 1
    E = [j for j in U if not flags[j] & 2]
    k = min(k, len(E), max_seeds)
    best = sorted(E, key=lambda j: (-s[j], j))[:k]
    return sorted(best)


def test_brute_force_small_rows_with_ties():
    rng = np.random.default_rng(1)
    for trial in range(3000):
        n = int(rng.integers(1, 13))
        # dyadic values: every sum and quotient below is exact in fp64
        logp = -rng.integers(0, 6, n).astype(np.float32)
        d_in = rng.choice([0.0, 0.5, 1.0, 3.0], n).astype(np.float32)
        d_out = rng.choice([0.0, 1.0, 3.0], n).astype(np.float32)
        flags = rng.choice([0, 1, 1, 1, 3], n).astype(np.uint8)
        ms = int(rng.integers(0, 5))
        si, ns, _ = oracle.select(logp[None], d_in[None], d_out[None], flags[None], ms)
        ref = _brute(logp, d_in, d_out, flags, ms)
        assert si[0, : ns[0]].tolist() == ref, (trial, logp, d_in, d_out, flags, ms)
        assert (si[0, ns[0]:] == -1).all()


def test_excluded_never_selected_and_budget_unchanged():
    s = synth.select_inputs(4, 256, seed=3, n_excl_prev=20, n_excl_budget=10)
    fl = s["flags"].numpy()
    si, ns, _ = oracle.select(s["logp"], s["d_in"], s["d_out"], fl, 64)
    si2, ns2, _ = oracle.select(s["logp"], s["d_in"], s["d_out"], fl & 1, 64)
    for b in range(4):
        chosen = si[b, : ns[b]]
        assert not (fl[b, chosen] & 2).any()
        assert (fl[b, chosen] & 1).all()
        assert ns[b] == ns2[b]  # budget comes from all of U_t, not from the eligible set
        assert list(chosen) == sorted(chosen)


def test_budget_fraction_matches_exponential_tail():
    # conf ~ Beta(5,1) => u = -log conf ~ Exp(rate 5); with d_in = d_out = 0 the fraction of
    # scores above the mean tends to P(u > E[u]) = e^{-1}.
    B, Lr = 1, 200000
    s = synth.select_inputs(B, Lr, seed=5, unmasked=Lr, n_excl_prev=0, n_excl_budget=0)
    z = np.zeros((B, Lr), np.float32)
    _, _, score = oracle.select(s["logp"], z, z, s["flags"], 1000)
    frac = (score[0] > score[0].mean()).mean()
    assert abs(frac - math.exp(-1)) < 0.005


def test_subnormal_and_zero_inputs_are_exact():
    tiny = np.float32(1e-40)  # fp32 subnormal
    logp = np.array([[-0.0, -tiny, -1.0, -2.0]], np.float32)
    d_in = np.array([[tiny, 0.0, tiny, 0.0]], np.float32)
    d_out = np.array([[0.0, tiny, 0.0, 0.0]], np.float32)
    fl = np.ones((1, 4), np.uint8)
    si, ns, score = oracle.select(logp, d_in, d_out, fl, 4)
    assert score[0, 0] == 0.0
    assert score[0, 1] == float(tiny) / (1.0 + float(tiny))  # widened exactly, not flushed
    assert score[0, 1] > 0.0
    assert score[0, 2] == 1.0 * (1.0 + float(tiny))
    assert si[0, : ns[0]].tolist() == [2, 3]  # mean 0.75: scores 1 and 2 lie above, budget 2


def test_non_finite_inputs_raise():
    logp = np.array([[-1.0, np.nan]], np.float32)
    z = np.zeros((1, 2), np.float32)
    with pytest.raises(oracle.OracleError):
        oracle.select(logp, z, z, np.ones((1, 2), np.uint8), 2)
    # a masked position is not read
    si, ns, _ = oracle.select(logp, z, z, np.array([[1, 0]], np.uint8), 2)
    assert ns[0] == 0
    with pytest.raises(oracle.OracleError):
        oracle.select(np.array([[-1.0]], np.float32), np.array([[-0.5]], np.float32),
                      np.zeros((1, 1), np.float32), np.ones((1, 1), np.uint8), 1)


def test_empty_region_and_empty_batch():
    e = np.zeros((1, 0), np.float32)
    si, ns, score = oracle.select(e, e, e, np.zeros((1, 0), np.uint8), 3)
    assert ns.tolist() == [0] and si.tolist() == [[-1, -1, -1]] and score.shape == (1, 0)
    e = np.zeros((0, 5), np.float32)
    si, ns, score = oracle.select(e, e, e, np.zeros((0, 5), np.uint8), 3)
    assert si.shape == (0, 3) and ns.shape == (0,)
