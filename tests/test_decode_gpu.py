"""cover_decode_update through the C ABI against the oracle's decode_update, bit-exact on
every output (tokens, ReMask counters, flags, drafted, counts): the LLaDA decoding region,
ties that push the draft cap's radix select down to the position bits, every cap regime,
ragged and maximum region lengths, seed lists with out-of-region, masked and repeated
entries, and several steps chained on the same state."""
import numpy as np
import pytest
import torch

import oracle
from helpers import announce
from paper_2602_06161_amd import cover, synth

pytestmark = pytest.mark.gpu


def _both(a, tau, cap, budget, seeds=True, last=None, min_draft=0):
    announce(f"decode update B{a['tokens'].shape[0]} Lr{a['tokens'].shape[1]} tau{tau} cap{cap}")
    si = a["seed_idx"] if seeds else np.zeros((a["tokens"].shape[0], 0), np.int32)
    ns = a["n_seed"] if seeds else np.zeros(a["tokens"].shape[0], np.int32)
    exp = oracle.decode_update(a["tokens"].numpy(), a["argmax"].numpy(), a["conf"].numpy(),
                               np.asarray(si), np.asarray(ns), a["remask_count"].numpy(),
                               a["mask_id"], tau, cap, budget, a["pos_offset"],
                               min_draft=min_draft,
                               **({} if last is None else {"last_unmask": last}))
    tok, cnt = a["tokens"].cuda(), a["remask_count"].cuda()
    lt = None if last is None else torch.from_numpy(np.ascontiguousarray(last)).cuda()
    r = cover.cover_decode_update(
        tok, a["argmax"].cuda(), a["conf"].cuda(), a["seed_idx"].cuda() if seeds else None,
        a["n_seed"].cuda() if seeds else None, cnt, a["mask_id"], tau, cap, budget,
        a["pos_offset"], last_unmask=lt, min_draft=min_draft)
    torch.cuda.synchronize()
    got = (tok.cpu().numpy(), cnt.cpu().numpy(), r[0].cpu().numpy(), r[1].cpu().numpy(),
           r[2].cpu().numpy())
    if last is not None:
        got = got + (lt.cpu().numpy(), r[3].cpu().numpy())
    names = ("tokens", "remask_count", "flags", "drafted", "counts", "last_unmask", "flipflops")
    for name, g, e in zip(names, got, exp):
        assert np.array_equal(g, e), f"{name}: {np.argwhere(g != e)[:8].tolist()}"
    return got


def test_llada_region():
    a = synth.update_inputs(1, 256, seed=0)
    _both(a, 0.9, 15, 2)


@pytest.mark.parametrize("cap", [0, 1, 7, 100, 255, 10000])
def test_caps_with_ties(cap):
    # four confidence values: long runs of equal keys, decided by position
    a = synth.update_inputs(2, 700, seed=cap, conf_levels=4, masked_frac=0.8)
    _both(a, 0.05, cap, 1)


@pytest.mark.parametrize("B,Lr,levels", [(3, 1000, 0), (1, 1, 0), (2, 63, 3), (2, 65, 0),
                                          (1, 4097, 2), (1, cover.COVER_MAX_LR, 3),
                                          (4, 2048, 0)])
def test_region_lengths(B, Lr, levels):
    a = synth.update_inputs(B, Lr, seed=Lr, conf_levels=levels, n_seeds=64, max_seeds=64)
    _both(a, 0.5, max(1, Lr // 7), 2)


def test_empty_region_writes_zero_counts():
    a = synth.update_inputs(2, 0, seed=0, n_seeds=0)
    _, _, _, _, counts = _both(a, 0.9, 4, 2)
    assert not counts.any()


def test_without_seeds():
    a = synth.update_inputs(2, 300, seed=5)
    _both(a, 0.7, 20, 2, seeds=False)


def test_seed_lists_outside_the_contract_of_selection():
    # entries outside the region, at masked positions, repeated, and n_seed beyond the row
    a = synth.update_inputs(2, 200, seed=9, n_seeds=6, max_seeds=10)
    si = a["seed_idx"].clone()
    masked = np.nonzero(a["tokens"][0].numpy() == a["mask_id"])[0]
    si[0, 6:10] = torch.tensor([5, 768 + 200, 768 + int(masked[0]), int(si[0, 0])], dtype=torch.int32)
    a["seed_idx"], a["n_seed"] = si, torch.tensor([10, 99], dtype=torch.int32)
    _both(a, 0.6, 9, 2)
    a["n_seed"] = torch.tensor([-3, 4], dtype=torch.int32)
    _both(a, 0.6, 9, 2)


def test_negative_confidences_and_threshold():
    a = synth.update_inputs(1, 500, seed=11)
    a["conf"] = a["conf"] - 0.5
    a["conf"][0, :5] = torch.tensor([0.0, -0.0, -0.25, -0.25, 0.25])
    _both(a, -0.3, 60, 2)


def test_chained_steps_keep_state():
    # twelve steps on one state: each step's tokens, counters, flags and last unmasked tokens
    # feed the next; a vocabulary of 4 makes restored tokens (flip-flops) common
    a = synth.update_inputs(2, 256, seed=21, vocab=5)
    last = np.full((2, 256), -1, np.int32)
    total_ff = 0
    for t in range(12):
        nxt = synth.update_inputs(2, 256, seed=100 + t, vocab=5)
        a["argmax"], a["conf"] = nxt["argmax"], nxt["conf"]
        tok, cnt, flags, drafted, _, last, ff = _both(a, 0.5, 40, 3, last=last)
        total_ff += int(ff.sum())
        a["tokens"], a["remask_count"] = torch.from_numpy(tok), torch.from_numpy(cnt)
        # next seeds: unmasked, not excluded positions (any such set is a valid selection)
        for b in range(2):
            ok = np.nonzero((flags[b] & 3) == 1)[0][:16]
            a["seed_idx"][b] = -1
            a["seed_idx"][b, :ok.size] = torch.from_numpy(768 + ok.astype(np.int32))
            a["n_seed"][b] = ok.size
    assert total_ff > 0


@pytest.mark.parametrize("tau,min_draft,levels", [(0.999, 1, 0), (0.999, 15, 3), (0.5, 4, 0),
                                                  (2.0, 15, 0)])
def test_min_draft(tau, min_draft, levels):
    # forced drafting when too few pass tau (ties among few levels), unchanged otherwise
    a = synth.update_inputs(2, 700, seed=min_draft, conf_levels=levels)
    _both(a, tau, 15, 5, min_draft=min_draft)
