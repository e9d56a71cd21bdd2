"""GPU parity of cover_attn_rect (a block of query rows against all keys, the prefix-cache
form of Sec. 6.6) through the C ABI: each output row must equal the oracle's COVER attention
row at the same absolute position of the full-length problem (Sec. 5.1, App. B.1), within
the bf16 tolerance of the square kernel.  Cases: the LLaDA generated block, small blocks,
every key-split count regime (including splits with no keys), GQA, ragged lengths with
seeds on the first and last positions, seeds outside the block, every position a seed, the
whole sequence as the block, a single position, no seeds."""
import numpy as np
import pytest
import torch

import oracle
from helpers import announce, check_attn, to_dev
from paper_2602_06161_amd import cover, synth

pytestmark = pytest.mark.gpu


def _custom(seed, B, Hq, Hkv, L, n_seeds, positions=None):
    cfg = synth.AttnConfig("custom", B, Hq, Hkv, L, 128, "bf16", 0, L, n_seeds, "independent")
    a = synth.attn_inputs(cfg, seed=seed)
    if positions is not None:
        pos = np.array(sorted(positions), np.int32)
        a["seed_idx"] = torch.from_numpy(np.tile(pos, (B, 1)))
        a["n_seed"] = torch.full((B,), len(pos), dtype=torch.int32)
    return a


def _check(a, q_off, Lq, n_split=None, seeds=True, where=""):
    announce(f"rect {where} q_off={q_off} Lq={Lq} n_split={n_split}")
    q, kl, vl, kc, vc, si, ns = to_dev(a)
    if not seeds:
        si = ns = None
    qb = q[:, :, q_off:q_off + Lq].contiguous()
    out, lse = cover.cover_attn_rect(qb, kl, vl, kc, vc, q_off, si, ns, n_split=n_split)
    torch.cuda.synchronize()
    B, Hq, L, d = a["q"].shape
    rows = np.array([(b * Hq + h) * L + i for b in range(B) for h in range(Hq)
                     for i in range(q_off, q_off + Lq)], np.int64)
    osi = a["seed_idx"] if seeds else torch.zeros((B, 0), dtype=torch.int32)
    ons = a["n_seed"] if seeds else torch.zeros(B, dtype=torch.int32)
    ref_o, ref_l = oracle.attn(a["q"], a["k_live"], a["v_live"], a["k_cache"], a["v_cache"], osi,
                               ons, scale=a["scale"], mode="fast", rows=rows)
    check_attn(out, lse, ref_o.reshape(B, Hq, Lq, d), ref_l.reshape(B, Hq, Lq), torch.bfloat16,
               where)
    return out, lse


def test_llada_generated_block():
    a = synth.attn_inputs("llada", seed=0)
    _check(a, 768, 256, where="llada")


@pytest.mark.parametrize("q_off,Lq", [(800, 32), (896, 64), (768, 32), (992, 32)])
def test_small_blocks(q_off, Lq):
    a = synth.attn_inputs("llada", seed=1)
    _check(a, q_off, Lq, where="llada small block")


@pytest.mark.parametrize("n_split", [1, 3, 7, 32, 40])
def test_split_counts(n_split):
    # 40 splits of a 32-stage sequence leave splits without keys
    a = synth.attn_inputs("llada", seed=2)
    _check(a, 768, 256, n_split=n_split, where="splits")


def test_gqa_dream_block():
    a = synth.attn_inputs("dream", seed=0)
    _check(a, 512, 256, where="dream")


def test_ragged_with_edge_seeds():
    a = _custom(3, 2, 4, 2, 1000, 0, positions=[5, 900, 910, 933, 976, 999])
    _check(a, 900, 77, n_split=3, where="ragged")
    _check(a, 923, 77, n_split=5, where="ragged block at the end")


def test_every_position_a_seed():
    a = _custom(4, 1, 2, 2, 256, 0, positions=list(range(256)))
    _check(a, 100, 100, where="all seeds")


def test_whole_sequence_matches_square_kernel():
    a = synth.attn_inputs("llada", seed=5)
    out, lse = _check(a, 0, 1024, where="whole sequence")
    q, kl, vl, kc, vc, si, ns = to_dev(a)
    sq, slse = cover.cover_attn_fwd(q, kl, vl, kc, vc, si, ns)
    torch.cuda.synchronize()
    assert (out.float() - sq.float()).abs().max().item() < 4e-2
    assert (lse - slse).abs().max().item() < 4e-2


def test_single_position_and_no_seeds():
    a = _custom(6, 1, 2, 2, 1, 0, positions=[0])
    _check(a, 0, 1, where="L=1 seed")
    a = synth.attn_inputs("llada", seed=7)
    _check(a, 768, 256, seeds=False, where="no seeds")


@pytest.mark.parametrize("case", ["llada256", "llada32", "llada64_896", "dream", "ragged",
                                  "ragged_end", "all_seeds", "short", "L1", "no_seeds",
                                  "long_seed_list", "batch_gqa"])
def test_single_launch_form(case):
    """n_split = 1: the single-launch kernel (key split across the waves of a workgroup,
    merged in LDS), on every case shape above plus short sequences (waves without stages)
    and seed lists longer than the part fetched into LDS."""
    if case == "llada256":
        _check(synth.attn_inputs("llada", seed=10), 768, 256, n_split=1, where=case)
    elif case == "llada32":
        _check(synth.attn_inputs("llada", seed=11), 992, 32, n_split=1, where=case)
    elif case == "llada64_896":
        _check(synth.attn_inputs("llada", seed=12), 896, 64, n_split=1, where=case)
    elif case == "dream":
        _check(synth.attn_inputs("dream", seed=13), 512, 256, n_split=1, where=case)
    elif case == "ragged":
        _check(_custom(14, 2, 4, 2, 1000, 0, positions=[5, 900, 910, 933, 976, 999]), 900, 77,
               n_split=1, where=case)
    elif case == "ragged_end":
        _check(_custom(15, 2, 4, 2, 1000, 0, positions=[0, 31, 32, 923, 999]), 923, 77,
               n_split=1, where=case)
    elif case == "all_seeds":
        _check(_custom(16, 1, 2, 2, 256, 0, positions=list(range(256))), 100, 100, n_split=1,
               where=case)
    elif case == "short":  # 4 stages for 8 waves; 3 stages, the last ragged
        _check(_custom(17, 1, 2, 1, 100, 0, positions=[3, 50, 99]), 40, 60, n_split=1, where=case)
        _check(_custom(18, 1, 2, 2, 70, 0, positions=[69]), 0, 70, n_split=1, where=case)
    elif case == "L1":
        _check(_custom(19, 1, 2, 2, 1, 0, positions=[0]), 0, 1, n_split=1, where=case)
    elif case == "no_seeds":
        _check(synth.attn_inputs("llada", seed=20), 768, 256, n_split=1, seeds=False, where=case)
    elif case == "long_seed_list":  # 700 seeds: 512 through LDS, the rest by plain loads
        rng = np.random.default_rng(21)
        pos = rng.choice(1024, size=700, replace=False)
        _check(_custom(21, 1, 2, 2, 1024, 0, positions=pos.tolist()), 600, 200, n_split=1,
               where=case)
    elif case == "batch_gqa":
        _check(_custom(22, 3, 8, 2, 640, 0, positions=[1, 100, 333, 500, 639]), 480, 160,
               n_split=1, where=case)


def test_single_launch_long_sequence():
    """The single launch at L = 4200 (132 stages of 32 keys, 16-17 per wave, the last ragged)
    with seeds in the first, middle and last stages and a block of 256 rows whose 256
    workgroups keep the single launch the default form."""
    pos = [0, 31, 1500, 2047, 2048, 2049, 3999, 4000, 4100, 4191, 4199]
    a = _custom(23, 1, 32, 32, 4200, 0, positions=pos)
    assert cover.rect_splits(1, 32, 256, 4200) == 1
    _check(a, 3944, 256, where="L4200 block at the end")
    _check(a, 1900, 64, n_split=1, where="L4200 middle block")


@pytest.mark.parametrize("n_split", [1, 3])
def test_distinct_seed_lists_per_batch_row(n_split):
    """Each batch row has its own seed list and count: none, a few in and out of the block,
    and a long list with entries past its count (padded with -1, ignored)."""
    L, ms = 700, 40
    cfg = synth.AttnConfig("custom", 3, 4, 2, L, 128, "bf16", 0, L, ms, "independent")
    a = synth.attn_inputs(cfg, seed=24)
    rng = np.random.default_rng(24)
    si = np.full((3, ms), -1, np.int32)
    counts = [0, 5, 33]
    si[1, :5] = [0, 333, 500, 517, 699]
    si[2, :33] = np.sort(rng.choice(L, size=33, replace=False))
    si[2, 33:] = rng.choice(L, size=ms - 33)  # past the count: must be ignored
    a["seed_idx"] = torch.from_numpy(si)
    a["n_seed"] = torch.tensor(counts, dtype=torch.int32)
    osi = torch.from_numpy(np.where(np.arange(ms)[None, :] < np.array(counts)[:, None], si, -1).astype(np.int32))
    q, kl, vl, kc, vc, sid, nsd = to_dev(a)
    q_off, Lq = 480, 150
    announce(f"rect distinct seeds per row n_split={n_split}")
    qb = q[:, :, q_off:q_off + Lq].contiguous()
    out, lse = cover.cover_attn_rect(qb, kl, vl, kc, vc, q_off, sid, nsd, n_split=n_split)
    torch.cuda.synchronize()
    B, Hq, _, d = a["q"].shape
    rows = np.array([(b * Hq + h) * L + i for b in range(B) for h in range(Hq)
                     for i in range(q_off, q_off + Lq)], np.int64)
    ref_o, ref_l = oracle.attn(a["q"], a["k_live"], a["v_live"], a["k_cache"], a["v_cache"], osi,
                               a["n_seed"], scale=a["scale"], mode="fast", rows=rows)
    check_attn(out, lse, ref_o.reshape(B, Hq, Lq, d), ref_l.reshape(B, Hq, Lq), torch.bfloat16,
               "distinct seeds")
