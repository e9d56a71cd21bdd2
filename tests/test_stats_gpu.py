"""GPU producers of the selection signals (cover_token_stats, cover_attn_stats, through the
C ABI) against the fp64 oracle.

Tolerances, from the arithmetic:
  token stats: the log-sum-exp is an fp32 sum of V exp2 terms (each within 2 ulp), taken as
    per-thread runs of at most ~V/8192 chunks and a 1024-way tree, so the relative error of
    the sum stays below (V/8192*8 + 10) * 2^-23 ~ 2e-5 for V = 126464; logp = x_y - lz then
    errs by that much absolutely, conf = 1/sum relatively.  argmax is decided on the stored
    values, which both sides compare exactly: bit-exact.
  attention masses: the weights are exp(s - lse) with the lse of cover_attn_fwd, whose row
    sum adds the bf16-rounded probabilities the PV product uses (each within 2^-9); the lse
    is therefore within 2^-9 of the exact one and every weight within that relative error,
    which sums of positive weights keep: rtol 2^-9 ~ 2e-3 (plus 1e-6 absolute for masses of
    rows with nothing in them)."""
import numpy as np
import pytest
import torch

import oracle
from helpers import announce
from paper_2602_06161_amd import cover, synth

pytestmark = pytest.mark.gpu

TOK_ATOL = 3e-5
TOK_RTOL = 3e-5
MASS_RTOL = 2e-3
MASS_ATOL = 1e-6


def _dev(t):
    """The logits on the GPU with their padded row stride."""
    V = t["logits"].shape[1]
    return t["buffer"].cuda()[:, :V]


def _token_check(t):
    logits, tokens = t["logits"], t["tokens"]
    lg, cf, am = cover.cover_token_stats(_dev(t), tokens.cuda())
    torch.cuda.synchronize()
    r_lp, r_cf, r_am = oracle.token_stats(oracle._f64(logits), tokens.numpy())
    assert np.array_equal(am.cpu().numpy(), r_am), "argmax differs"
    np.testing.assert_allclose(lg.cpu().numpy(), r_lp, rtol=0, atol=TOK_ATOL)
    np.testing.assert_allclose(cf.cpu().numpy(), r_cf, rtol=TOK_RTOL, atol=0)


@pytest.mark.parametrize("R,V,dtype", [(8, 126464, "bf16"), (5, 1003, "f32"), (3, 1001, "bf16"),
                                       (2, 1, "f32"), (7, 8, "bf16"), (4, 50000, "f32")])
def test_token_stats_vs_oracle(R, V, dtype):
    announce(f"token stats R{R} V{V} {dtype}")
    t = synth.token_inputs(R, V, seed=V, dtype=dtype)
    _token_check(t)


def test_token_stats_llada_block():
    """The LM-head output of the 256 generated positions of a LLaDA-8B step (vocab 126464)."""
    announce("token stats R256 V126464 bf16")
    t = synth.token_inputs(256, 126464, seed=1)
    _token_check(t)


def test_token_stats_ties_and_bad_tokens():
    announce("token stats ties / bad tokens")
    t = synth.token_inputs(6, 4096, seed=3, dtype="f32")
    x = t["buffer"]  # V = 4096 needs no padding: the buffer is the logits
    x[1, 100] = x[1, 3000] = x[1].max() + 1.0     # tie: the smaller index wins
    x[2, :] = 0.5                                   # all equal: index 0, conf = 1/V
    tok = t["tokens"].clone()
    tok[3], tok[4] = -1, 4096                       # outside [0, V): NaN, no read
    lg, cf, am = cover.cover_token_stats(x.cuda(), tok.cuda())
    torch.cuda.synchronize()
    am, lg, cf = am.cpu().numpy(), lg.cpu().numpy(), cf.cpu().numpy()
    assert am[1] == 100 and am[2] == 0
    assert abs(cf[2] - 1.0 / 4096) < 1e-9
    assert np.isnan(lg[3]) and np.isnan(lg[4])
    ok = [0, 1, 2, 5]
    r_lp, r_cf, r_am = oracle.token_stats(oracle._f64(x[ok]), tok[ok].numpy())
    np.testing.assert_allclose(lg[ok], r_lp, atol=TOK_ATOL, rtol=0)
    assert np.array_equal(am[ok], r_am)


def _stats_case(a, r0, masked, drafted):
    t = {k: a[k].cuda() for k in ("q", "k_live", "v_live", "k_cache", "v_cache", "seed_idx", "n_seed")}
    _, lse = cover.cover_attn_fwd(t["q"], t["k_live"], t["v_live"], t["k_cache"], t["v_cache"],
                                  t["seed_idx"], t["n_seed"])
    m, d = torch.as_tensor(masked).cuda(), torch.as_tensor(drafted).cuda()
    d_in, d_out = cover.cover_attn_stats(t["q"], t["k_live"], t["k_cache"], t["seed_idx"],
                                         t["n_seed"], lse, m, d, r0)
    d_in2, d_out2 = cover.cover_attn_stats(t["q"], t["k_live"], t["k_cache"], t["seed_idx"],
                                           t["n_seed"], lse, m, d, r0)
    torch.cuda.synchronize()
    assert torch.equal(d_in, d_in2) and torch.equal(d_out, d_out2), "not deterministic"
    r_in, r_out = oracle.attn_stats(a["q"], a["k_live"], a["k_cache"], a["seed_idx"].numpy(),
                                    a["n_seed"].numpy(), r0, np.asarray(masked), np.asarray(drafted))
    np.testing.assert_allclose(d_in.cpu().numpy(), r_in, rtol=MASS_RTOL, atol=MASS_ATOL)
    np.testing.assert_allclose(d_out.cpu().numpy(), r_out, rtol=MASS_RTOL, atol=MASS_ATOL)


@pytest.mark.parametrize("d,r0,Lr", [(64, 120, 80), (128, 0, 200), (128, 150, 50), (64, 199, 1),
                                     (128, 37, 96)])
def test_attn_stats_vs_oracle(d, r0, Lr):
    """Ragged regions and query blocks, GQA, seeds inside the region (their diagonal takes the
    live key) and outside it."""
    announce(f"attn stats d{d} r0 {r0} Lr {Lr}")
    a = synth.attn_inputs("tiny", seed=d + r0, max_seeds=12, B=2, Hq=4, Hkv=2, L=200, d=d,
                          dtype="bf16", prompt=0, unmasked_gen=200, n_seeds=12)
    rng = np.random.default_rng(r0 + Lr)
    # put some seeds inside the region so its diagonal is exercised
    si = a["seed_idx"].numpy().copy()
    for b in range(2):
        inside = np.sort(rng.choice(np.arange(r0, r0 + Lr), size=min(4, Lr), replace=False))
        rest = np.setdiff1d(si[b][si[b] >= 0], inside)[:8]
        row = np.sort(np.concatenate([inside, rest])).astype(np.int32)
        si[b, :] = -1
        si[b, :row.size] = row
        a["n_seed"][b] = row.size
    a["seed_idx"] = torch.from_numpy(si)
    masked = (rng.integers(0, 2, (2, Lr))).astype(np.uint8)
    drafted = (rng.integers(0, 4, (2, Lr)) == 0).astype(np.uint8)
    _stats_case(a, r0, masked, drafted)


@pytest.mark.parametrize("B,Hq,Hkv,L,r0,Lr", [
    (2, 4, 2, 1100, 0, 1100),    # 35 key tiles in 18 groups of 2, the last group one tile
    (1, 32, 32, 2048, 0, 2048),  # 64 key tiles in 8 groups of 8
    (1, 28, 4, 1500, 300, 1111),  # 35 tiles in 9 groups of 4, the last group three tiles (GQA)
])
def test_attn_stats_key_groups(B, Hq, Hkv, L, r0, Lr):
    """Key groups of several 32-key tiles (the next tile of a group is prefetched while the
    current one is used) and a shorter last group, with seeds inside and outside the region."""
    announce(f"attn stats key groups B{B} Hq{Hq} Hkv{Hkv} L{L} r0 {r0} Lr {Lr}")
    a = synth.attn_inputs("tiny", seed=L + Hq, max_seeds=40, B=B, Hq=Hq, Hkv=Hkv, L=L, d=128,
                          dtype="bf16", prompt=0, unmasked_gen=L, n_seeds=40)
    rng = np.random.default_rng(Lr)
    masked = (rng.integers(0, 2, (B, Lr))).astype(np.uint8)
    drafted = (rng.integers(0, 8, (B, Lr)) == 0).astype(np.uint8)
    _stats_case(a, r0, masked, drafted)


def test_attn_stats_long_seed_lists():
    """Seed lists longer than the 512 positions fetched with the seed count (the rest are read
    in a loop), with entries outside [0, L) inside the count and junk past it (ignored), and a
    batch row without seeds; the oracle gets the cleaned lists."""
    B, Hq, Hkv, L, r0, Lr, ms = 2, 4, 2, 1100, 100, 900, 800
    announce(f"attn stats long seed lists B{B} Hq{Hq} L{L} max_seeds {ms}")
    a = synth.attn_inputs("tiny", seed=77, max_seeds=ms, B=B, Hq=Hq, Hkv=Hkv, L=L, d=128,
                          dtype="bf16", prompt=0, unmasked_gen=L, n_seeds=0)
    rng = np.random.default_rng(77)
    si = rng.integers(-50, L + 50, size=(B, ms)).astype(np.int32)  # junk everywhere
    good = np.sort(rng.choice(L, size=700, replace=False)).astype(np.int32)
    si[0, :700] = good
    si[0, 700:703] = [-5, L, L + 9]  # inside the count, outside [0, L)
    counts = np.array([703, 0], np.int32)
    clean = np.full((B, ms), -1, np.int32)
    clean[0, :700] = good
    a["seed_idx"], a["n_seed"] = torch.from_numpy(si), torch.from_numpy(counts)
    masked = (rng.integers(0, 2, (B, Lr))).astype(np.uint8)
    drafted = (rng.integers(0, 4, (B, Lr)) == 0).astype(np.uint8)
    t = {k: a[k].cuda() for k in ("q", "k_live", "v_live", "k_cache", "v_cache", "seed_idx", "n_seed")}
    _, lse = cover.cover_attn_fwd(t["q"], t["k_live"], t["v_live"], t["k_cache"], t["v_cache"],
                                  t["seed_idx"], t["n_seed"])
    m, d = torch.as_tensor(masked).cuda(), torch.as_tensor(drafted).cuda()
    d_in, d_out = cover.cover_attn_stats(t["q"], t["k_live"], t["k_cache"], t["seed_idx"],
                                         t["n_seed"], lse, m, d, r0)
    torch.cuda.synchronize()
    r_in, r_out = oracle.attn_stats(a["q"], a["k_live"], a["k_cache"], clean,
                                    np.array([700, 0], np.int32), r0, masked, drafted)
    np.testing.assert_allclose(d_in.cpu().numpy(), r_in, rtol=MASS_RTOL, atol=MASS_ATOL)
    np.testing.assert_allclose(d_out.cpu().numpy(), r_out, rtol=MASS_RTOL, atol=MASS_ATOL)


def test_attn_stats_workspace_checked():
    """A caller workspace smaller than the launch needs, or of the wrong dtype, is refused
    before anything is enqueued."""
    announce("attn stats workspace checks")
    a = synth.stats_inputs("llada", seed=0)
    t = {k: a[k].cuda() for k in ("q", "k_live", "v_live", "k_cache", "v_cache", "seed_idx", "n_seed")}
    _, lse = cover.cover_attn_fwd(t["q"], t["k_live"], t["v_live"], t["k_cache"], t["v_cache"],
                                  t["seed_idx"], t["n_seed"])
    m, d = a["masked"].cuda(), a["drafted"].cuda()
    B, Hq, _, _ = a["q"].shape
    need = cover.attn_stats_workspace(B, Hq, m.shape[1])
    args = (t["q"], t["k_live"], t["k_cache"], t["seed_idx"], t["n_seed"], lse, m, d, a["r0"])
    with pytest.raises(ValueError):
        cover.cover_attn_stats(*args, workspace=torch.empty(need - 1, device="cuda"))
    with pytest.raises(ValueError):
        cover.cover_attn_stats(*args, workspace=torch.empty(need, device="cuda", dtype=torch.float64))
    d_in, d_out = cover.cover_attn_stats(*args, workspace=torch.empty(need, device="cuda"))
    r_in, r_out = cover.cover_attn_stats(*args)
    torch.cuda.synchronize()
    assert torch.equal(d_in, r_in) and torch.equal(d_out, r_out)


@pytest.mark.parametrize("name", ["llada", "dream"])
def test_attn_stats_workload(name):
    """The generated block of the LLaDA-8B and Dream-7B layer shapes: 256 region positions,
    128 still masked, 15 drafted."""
    announce(f"attn stats {name}")
    a = synth.stats_inputs(name, seed=0)
    _stats_case(a, a["r0"], a["masked"].numpy(), a["drafted"].numpy())
