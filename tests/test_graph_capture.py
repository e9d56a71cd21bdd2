"""The layer step's entry points (cover_attn_fwd, cover_select_seeds) captured in a HIP graph:
they allocate nothing and make no host call besides the launch, so a replay must give the
same bits as the eager calls.  Replays alternate with eager steps and device
synchronisations, and every replay is checked."""
import pytest
import torch

from helpers import announce
from paper_2602_06161_amd import cover, synth

pytestmark = pytest.mark.gpu


def _same(a, b):
    if a.dtype == torch.float64:
        a, b = a.view(torch.int64), b.view(torch.int64)
    elif a.dtype in (torch.float32, torch.bfloat16):
        a, b = a.view(torch.int32 if a.dtype == torch.float32 else torch.int16), \
            b.view(torch.int32 if b.dtype == torch.float32 else torch.int16)
    return torch.equal(a, b)


@pytest.mark.parametrize("workload", ["llada", "dream"])
def test_step_replays_match_eager(workload):
    announce(f"graph capture of the layer step, {workload}")
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream(device=dev)
    a = synth.step_inputs(workload, seed=3)
    c = a["cfg"]
    t = {k: a[k].to(dev) for k in ("q", "k_live", "v_live", "k_cache", "v_cache", "seed_idx",
                                   "n_seed", "logp", "d_in", "d_out", "flags")}
    out = torch.empty_like(t["q"])
    lse = torch.empty((c.B, c.Hq, c.L), device=dev, dtype=torch.float32)
    nsi = torch.empty((c.B, c.n_seeds), device=dev, dtype=torch.int32)
    nns = torch.empty((c.B,), device=dev, dtype=torch.int32)
    score = torch.empty((c.B, a["Lr"]), device=dev, dtype=torch.float64)
    attn = cover.PreparedAttn(t["q"], t["k_live"], t["v_live"], t["k_cache"], t["v_cache"],
                              t["seed_idx"], t["n_seed"], out=out, lse=lse, stream=stream)
    select = cover.PreparedSelect(t["logp"], t["d_in"], t["d_out"], t["flags"], c.n_seeds,
                                  a["pos_offset"], seed_idx=nsi, n_seed=nns, score=score,
                                  stream=stream)
    outs = (out, lse, nsi, nns, score)
    with torch.cuda.stream(stream):
        attn()
        select()
    torch.cuda.synchronize()
    ref = [x.clone() for x in outs]

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for _ in range(2):
            attn()
            select()
    torch.cuda.synchronize()
    for rep in range(3):
        with torch.cuda.stream(stream):
            for x in outs:
                x.fill_(0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, r, x in zip(("out", "lse", "seed_idx", "n_seed", "score"), ref, outs):
            assert _same(r, x), f"replay {rep}: {name} differs from the eager result"
        with torch.cuda.stream(stream):
            attn()
            select()
        torch.cuda.synchronize()
        for name, r, x in zip(("out", "lse", "seed_idx", "n_seed", "score"), ref, outs):
            assert _same(r, x), f"eager step after replay {rep}: {name} differs"
