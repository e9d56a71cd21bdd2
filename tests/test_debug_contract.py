"""COVER_DEBUG=1 contract checks through the C ABI: every violation of the device-data
contracts sets its status bit (read back with cover_debug_status), valid inputs set none,
and without COVER_DEBUG nothing is checked.  The checked kernels still run on the bad
inputs: they must complete (the contracts promise no out-of-bounds access)."""
import numpy as np
import pytest
import torch

from helpers import announce
from paper_2602_06161_amd import cover, synth

pytestmark = pytest.mark.gpu


@pytest.fixture
def debug(monkeypatch):
    monkeypatch.setenv("COVER_DEBUG", "1")
    cover.debug_status(clear=True)
    yield
    cover.debug_status(clear=True)


def _attn(seeds, n_seed, max_seeds, L=256, dtype="bf16", d=128):
    a = synth.attn_inputs("tiny", seed=3, L=L, d=d, dtype=dtype, Hq=2, Hkv=2, prompt=0,
                          unmasked_gen=L, n_seeds=0, max_seeds=max(max_seeds, 1))
    dev = lambda x: x.cuda()
    si = torch.full((1, max_seeds), -1, dtype=torch.int32)
    si[0, :len(seeds)] = torch.tensor(seeds, dtype=torch.int32)
    ns = torch.tensor([n_seed], dtype=torch.int32)
    out, lse = cover.cover_attn_fwd(dev(a["q"]), dev(a["k_live"]), dev(a["v_live"]),
                                    dev(a["k_cache"]), dev(a["v_cache"]), dev(si), dev(ns))
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("bf16", 64), ("f32", 64)])
def test_valid_seed_lists_set_no_bit(debug, dtype, d):
    announce(f"debug valid seeds {dtype} d{d}")
    _attn([5, 17, 200, 3], 4, 8, dtype=dtype, d=d)   # any order is allowed
    _attn([], 0, 8, dtype=dtype, d=d)
    assert cover.debug_status() == 0


@pytest.mark.parametrize("seeds,n_seed,bit", [
    ([5, 300], 2, cover.COVER_DEBUG_SEED_RANGE),       # position >= L
    ([-3, 7], 2, cover.COVER_DEBUG_SEED_RANGE),        # negative position
    ([9, 4, 9], 3, cover.COVER_DEBUG_SEED_DUPLICATE),  # listed twice
    (list(range(8)), 9, cover.COVER_DEBUG_SEED_COUNT),  # n_seed > max_seeds (row full)
    ([1, 2], -1, cover.COVER_DEBUG_SEED_COUNT),        # negative n_seed
])
def test_each_seed_violation_sets_its_bit(debug, seeds, n_seed, bit):
    announce(f"debug seeds {seeds} n{n_seed}")
    _attn(seeds, n_seed, 8)
    assert cover.debug_status(clear=True) == bit


def test_bits_accumulate_until_cleared(debug):
    announce("debug accumulate")
    _attn([5, 300], 2, 8)
    _attn([9, 9], 2, 8)
    assert cover.debug_status() == cover.COVER_DEBUG_SEED_RANGE | cover.COVER_DEBUG_SEED_DUPLICATE
    assert cover.debug_status(clear=True) != 0
    assert cover.debug_status() == 0


def test_no_checks_without_the_variable(monkeypatch):
    announce("debug off")
    monkeypatch.delenv("COVER_DEBUG", raising=False)
    cover.debug_status(clear=True)
    _attn([5, 300, 300], 3, 8)
    assert cover.debug_status() == 0


def _select(logp, d_in, d_out, flags):
    t = lambda x, dt: torch.as_tensor(np.ascontiguousarray(x)).to(dt).cuda()
    cover.cover_select_seeds(t(logp, torch.float32), t(d_in, torch.float32),
                             t(d_out, torch.float32), t(flags, torch.uint8), 8)
    torch.cuda.synchronize()


def test_selection_inputs(debug):
    announce("debug selection inputs")
    s = synth.select_inputs(2, 64, seed=1, unmasked=40)
    logp, d_in, d_out, flags = (s[k].numpy().copy() for k in ("logp", "d_in", "d_out", "flags"))
    _select(logp, d_in, d_out, flags)
    assert cover.debug_status() == 0
    um = np.argwhere(flags & 1)
    out_u = np.argwhere((flags & 1) == 0)
    # non-finite values and negative masses outside U_t are allowed
    l2, a2 = logp.copy(), d_in.copy()
    l2[tuple(out_u[0])] = np.nan
    a2[tuple(out_u[1])] = -1.0
    _select(l2, a2, d_out, flags)
    assert cover.debug_status() == 0
    l2 = logp.copy()
    l2[tuple(um[3])] = np.inf
    _select(l2, d_in, d_out, flags)
    assert cover.debug_status(clear=True) == cover.COVER_DEBUG_SELECT_NONFINITE
    o2 = d_out.copy()
    o2[tuple(um[5])] = -0.5
    _select(logp, d_in, o2, flags)
    assert cover.debug_status(clear=True) == cover.COVER_DEBUG_SELECT_NEGATIVE


def test_attention_masses_check_their_seed_lists(debug):
    announce("debug attn stats seeds")
    a = synth.stats_inputs("llada", seed=2)
    dev = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in a.items()}
    _, lse = cover.cover_attn_fwd(dev["q"], dev["k_live"], dev["v_live"], dev["k_cache"],
                                  dev["v_cache"], dev["seed_idx"], dev["n_seed"])
    assert cover.debug_status() == 0
    si = dev["seed_idx"].clone()
    si[0, 1] = si[0, 0]   # a duplicate
    cover.cover_attn_stats(dev["q"], dev["k_live"], dev["k_cache"], si, dev["n_seed"], lse,
                           dev["masked"], dev["drafted"], a["r0"])
    torch.cuda.synchronize()
    assert cover.debug_status(clear=True) == cover.COVER_DEBUG_SEED_DUPLICATE


def test_block_attention_checks_its_seed_list(debug):
    announce("debug rect seeds")
    a = synth.attn_inputs("llada", seed=4)
    q, kl, vl, kc, vc = (a[k].cuda() for k in ("q", "k_live", "v_live", "k_cache", "v_cache"))
    si = a["seed_idx"].clone()
    si[0, 1] = si[0, 0]  # a duplicate
    qb = q[:, :, 768:].contiguous()
    cover.cover_attn_rect(qb, kl, vl, kc, vc, 768, si.cuda(), a["n_seed"].cuda())
    torch.cuda.synchronize()
    assert cover.debug_status(clear=True) == cover.COVER_DEBUG_SEED_DUPLICATE
