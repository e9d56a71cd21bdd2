"""cover_attn_stats_noalloc (the attention masses with the library's own per-GPU workspace)
through the C ABI: its outputs equal those of cover_attn_stats with a caller workspace, bit for
bit (the same kernels and the same fixed summation order), on two calls in a row, the second
with a smaller problem than the first, and a problem whose workspace exceeds the array is
refused before anything is enqueued."""
import numpy as np
import pytest
import torch

from helpers import announce
from paper_2602_06161_amd import cover, synth

pytestmark = pytest.mark.gpu


def _inputs(a):
    t = {k: a[k].cuda() for k in ("q", "k_live", "v_live", "k_cache", "v_cache", "seed_idx", "n_seed")}
    _, lse = cover.cover_attn_fwd(t["q"], t["k_live"], t["v_live"], t["k_cache"], t["v_cache"],
                                  t["seed_idx"], t["n_seed"])
    return t, lse


def _compare(t, lse, masked, drafted, r0):
    m, d = torch.as_tensor(masked).cuda(), torch.as_tensor(drafted).cuda()
    B, Lr = m.shape
    ref_in, ref_out = cover.cover_attn_stats(t["q"], t["k_live"], t["k_cache"], t["seed_idx"],
                                             t["n_seed"], lse, m, d, r0)
    d_in = torch.full((B, Lr), float("nan"), device="cuda")
    d_out = torch.full((B, Lr), float("nan"), device="cuda")
    cover.cover_attn_stats_noalloc(t["q"], t["k_live"], t["k_cache"], t["seed_idx"], t["n_seed"],
                                   lse, m, d, r0, d_in, d_out)
    torch.cuda.synchronize()
    assert torch.equal(d_in, ref_in) and torch.equal(d_out, ref_out)
    return d_in, d_out


def test_noalloc_matches_workspace_entry_point_twice():
    announce("attn stats noalloc: LLaDA block, then a smaller problem")
    a = synth.stats_inputs("llada", seed=3)
    t, lse = _inputs(a)
    _compare(t, lse, a["masked"].numpy(), a["drafted"].numpy(), a["r0"])
    # second call: fewer heads, a shorter region, other seeds (the array keeps the first call's
    # partial sums; none may leak into this one)
    b = synth.attn_inputs("tiny", seed=11, max_seeds=6, B=2, Hq=4, Hkv=2, L=200, d=128,
                          dtype="bf16", prompt=0, unmasked_gen=200, n_seeds=6)
    t2, lse2 = _inputs(b)
    rng = np.random.default_rng(5)
    masked = rng.integers(0, 2, (2, 70)).astype(np.uint8)
    drafted = (rng.integers(0, 4, (2, 70)) == 0).astype(np.uint8)
    _compare(t2, lse2, masked, drafted, 90)


def test_noalloc_refuses_problems_beyond_its_array():
    announce("attn stats noalloc: oversize refused")
    B, Hq, L, d = 1, 257, 2048, 128
    assert cover.attn_stats_workspace(B, Hq, L) > cover.COVER_STATS_SCRATCH_FLOATS
    q = torch.zeros((B, Hq, L, d), device="cuda", dtype=torch.bfloat16)
    k = torch.zeros((B, Hq, L, d), device="cuda", dtype=torch.bfloat16)
    lse = torch.zeros((B, Hq, L), device="cuda")
    m = torch.zeros((B, L), device="cuda", dtype=torch.uint8)
    d_in = torch.zeros((B, L), device="cuda")
    d_out = torch.zeros((B, L), device="cuda")
    with pytest.raises(cover.CoverError) as e:
        cover.cover_attn_stats_noalloc(q, k, k, None, None, lse, m, m, 0, d_in, d_out)
    assert e.value.status == cover.COVER_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert torch.count_nonzero(d_in) == 0 and torch.count_nonzero(d_out) == 0
