"""GPU cover_select_seeds (through the C ABI) against the fp64 oracle: seed lists, counts and
fp64 scores must be bitwise equal."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from helpers import announce
from paper_2602_06161_amd import cover, synth

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "select_examples.json")


def _both(logp, d_in, d_out, flags, max_seeds, pos_offset=0, want_score=True):
    t = lambda x, dt: torch.as_tensor(np.ascontiguousarray(x)).to(dt).cuda()
    si, ns, sc = cover.cover_select_seeds(t(logp, torch.float32), t(d_in, torch.float32),
                                          t(d_out, torch.float32), t(flags, torch.uint8),
                                          max_seeds, pos_offset, want_score=want_score)
    torch.cuda.synchronize()
    r_si, r_ns, r_sc = oracle.select(logp, d_in, d_out, flags, max_seeds, pos_offset)
    assert np.array_equal(ns.cpu().numpy(), r_ns), "n_seed differs"
    assert np.array_equal(si.cpu().numpy(), r_si), "seed_idx differs"
    if want_score:
        g = sc.cpu().numpy()
        assert np.array_equal(g.view(np.uint64), r_sc.view(np.uint64)), "scores differ bitwise"
    return r_si, r_ns


def test_hand_worked_examples_on_gpu():
    ex = json.load(open(GOLDEN))["examples"]
    for e in ex:
        announce(f"select golden {e['name']}")
        f = lambda k: np.array([e[k]], np.float32)
        si, ns = _both(f("logp"), f("d_in"), f("d_out"), np.array([e["flags"]], np.uint8),
                       e["max_seeds"], e["pos_offset"])
        assert si[0].tolist() == e["seed_idx"]


@pytest.mark.parametrize("Lr,B", [(1, 64), (7, 64), (64, 256), (256, 64), (1000, 16), (2048, 8),
                                  (16384, 4)])
def test_random_rows(Lr, B):
    announce(f"select random Lr{Lr} B{B}")
    rng = np.random.default_rng(Lr)
    s = synth.select_inputs(B, Lr, seed=Lr, unmasked=int(rng.integers(0, Lr + 1)),
                            n_excl_prev=int(rng.integers(0, 1 + Lr // 8)), n_excl_budget=3)
    for ms in (0, 3, 64):
        _both(s["logp"].numpy(), s["d_in"].numpy(), s["d_out"].numpy(), s["flags"].numpy(), ms, 17)


def test_ten_thousand_rows():
    announce("select 10^4 rows Lr64")
    rng = np.random.default_rng(42)
    B, Lr = 10000, 64
    logp = np.log(rng.beta(5, 1, (B, Lr))).astype(np.float32)
    d_in = rng.exponential(0.1, (B, Lr)).astype(np.float32)
    d_out = rng.exponential(0.02, (B, Lr)).astype(np.float32)
    flags = rng.choice([0, 1, 1, 3], (B, Lr)).astype(np.uint8)
    _both(logp, d_in, d_out, flags, 16, 0)


def test_adversarial_rows():
    announce("select adversarial ties/subnormals/zeros")
    rng = np.random.default_rng(7)
    B, Lr = 512, 96
    logp = -rng.integers(0, 4, (B, Lr)).astype(np.float32)          # many ties
    logp[::7] = -0.0
    logp[1::11] = 0.0
    d_in = rng.choice(np.array([0.0, 1e-40, 0.5, 3.0], np.float32), (B, Lr))   # incl. subnormal
    d_out = rng.choice(np.array([0.0, 1e-45, 1.0, 3.0], np.float32), (B, Lr))
    flags = rng.choice([0, 1, 1, 1, 3], (B, Lr)).astype(np.uint8)
    flags[0] = 0          # nothing unmasked
    flags[1] = 3          # everything excluded
    flags[2] = 1
    logp[2] = -1.0        # all equal: budget 0
    _both(logp, d_in, d_out, flags, 32, 5)
    _both(logp, d_in, d_out, flags, 1, 0)


def test_llada_step_selection():
    announce("select LLaDA step inputs Lr256")
    a = synth.step_inputs("llada", seed=0)
    si, ns = _both(a["logp"].numpy(), a["d_in"].numpy(), a["d_out"].numpy(), a["flags"].numpy(),
                   16, a["pos_offset"])
    assert 1 <= ns[0] <= 16
    assert (si[0, : ns[0]] >= 768).all()


def test_no_score_buffer_same_selection():
    announce("select without score output")
    s = synth.select_inputs(4, 300, seed=3)
    _both(s["logp"].numpy(), s["d_in"].numpy(), s["d_out"].numpy(), s["flags"].numpy(), 20, 0,
          want_score=False)


def test_empty_region_on_gpu():
    announce("select empty region Lr0")
    B, ms = 3, 5
    e = torch.empty((B, 0), device="cuda")
    si, ns, _ = cover.cover_select_seeds(e, e.clone(), e.clone(),
                                         torch.empty((B, 0), device="cuda", dtype=torch.uint8),
                                         ms, 0, want_score=False)
    torch.cuda.synchronize()
    assert ns.cpu().tolist() == [0] * B
    assert (si.cpu() == -1).all()


@pytest.mark.parametrize("Lr", [64, 256, 1000])
def test_signed_zero_ties(Lr):
    """logp of +0.0 gives the score -0.0 and logp of -0.0 gives +0.0: the two compare equal, so
    the position decides between them; the emitted score keeps its sign bit."""
    announce(f"select signed-zero ties Lr{Lr}")
    rng = np.random.default_rng(11 + Lr)
    B = 16
    logp = rng.choice(np.array([0.0, -0.0, -0.5, -2.0], np.float32), (B, Lr))
    d_in = rng.choice(np.array([0.0, 0.25], np.float32), (B, Lr))
    d_out = np.zeros((B, Lr), np.float32)
    flags = rng.choice([1, 1, 1, 3], (B, Lr)).astype(np.uint8)
    for ms in (4, 32):
        _both(logp, d_in, d_out, flags, ms, 0)


@pytest.mark.parametrize("Lr", [64, 256, 1000])
def test_near_ties_below_the_high_word(Lr):
    """Scores 2 + k 2^-23 (logp = -1, d_out = 0, d_in = 1 + k 2^-23 in fp32) agree in the upper
    32 bits of their fp64 encoding and differ only below, while equal k give exact ties: the
    ranking must use all 64 bits and then the position."""
    announce(f"select near ties Lr{Lr}")
    rng = np.random.default_rng(5 + Lr)
    B = 16
    k = rng.integers(0, 8, (B, Lr))
    d_in = (1.0 + k * 2.0 ** -23).astype(np.float32)
    assert np.array_equal(d_in.astype(np.float64), 1.0 + k * 2.0 ** -23)
    logp = np.full((B, Lr), -1.0, np.float32)
    d_out = np.zeros((B, Lr), np.float32)
    logp[:, ::5] = -0.5   # a lower group, so that the budget is not zero
    flags = rng.choice([1, 1, 1, 3], (B, Lr)).astype(np.uint8)
    for ms in (8, 64):
        _both(logp, d_in, d_out, flags, ms, 0)
