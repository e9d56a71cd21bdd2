"""Seeded synthetic inputs for the COVER hot path.

This module holds none of the method's arithmetic: only random draws (numpy PCG64,
``default_rng(seed)``), rounding to the storage dtype (round-to-nearest-even through
torch's CPU conversion) and index bookkeeping.  The tests, the benchmark and the smoke
check all draw their inputs here, so both sides of every comparison see identical values.

Workloads (no trained weights or datasets are available, so these stand in for the
paper's LLaDA-8B / Dream-7B decoding steps; the shapes follow those models):
  tiny     B1 H2 L64 d64 fp32, 4 seeds anywhere in the sequence
  llada    B1 H32 L1024 d128 bf16 (MHA); prompt 768 + generated block 256, 128 of the
           generated positions unmasked, 16 seeds among them; cache rows independent
  dream    B1 Hq28/Hkv4 L768 d128 bf16 (GQA); prompt 512 + generated 256, 128 unmasked,
           32 seeds; cache = live + 0.1 N(0,1) at unmasked positions, = live elsewhere
  batched  B8 H32 L2048 d128 bf16; generated region [1536, 2048) with 256 unmasked per
           row, 64 seeds per row drawn independently per row
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch


@dataclass(frozen=True)
class AttnConfig:
    name: str
    B: int
    Hq: int
    Hkv: int
    L: int
    d: int
    dtype: str          # "f32" or "bf16"
    prompt: int         # positions [0, prompt) are the prompt (always unmasked)
    unmasked_gen: int   # unmasked positions inside the generated region [prompt, L)
    n_seeds: int        # seeds per batch row, drawn from the unmasked generated positions
    cache: str          # "independent" | "perturb"


CONFIGS = {
    "tiny": AttnConfig("tiny", 1, 2, 2, 64, 64, "f32", 0, 64, 4, "independent"),
    "llada": AttnConfig("llada", 1, 32, 32, 1024, 128, "bf16", 768, 128, 16, "independent"),
    "dream": AttnConfig("dream", 1, 28, 4, 768, 128, "bf16", 512, 128, 32, "perturb"),
    "batched": AttnConfig("batched", 8, 32, 32, 2048, 128, "bf16", 1536, 256, 64, "independent"),
}

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


def _normal(rng: np.random.Generator, shape, dtype: str) -> torch.Tensor:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    return torch.from_numpy(x).to(TORCH_DTYPE[dtype])


def attn_inputs(cfg: AttnConfig | str, seed: int = 0, max_seeds: int | None = None,
                **overrides) -> dict:
    """Host (CPU) tensors for one attention call.

    Returns q [B,Hq,L,d]; k_live, v_live, k_cache, v_cache [B,Hkv,L,d] in the storage dtype;
    seed_idx int32 [B,max_seeds] (ascending, -1 padded); n_seed int32 [B]; unmasked bool
    [B,L]; plus the config.  ``overrides`` replaces config fields (shape sweeps).
    """
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    if overrides:
        cfg = AttnConfig(**{**cfg.__dict__, **overrides})
    rng = np.random.default_rng(seed)
    B, Hq, Hkv, L, d = cfg.B, cfg.Hq, cfg.Hkv, cfg.L, cfg.d
    if max_seeds is None:
        max_seeds = cfg.n_seeds
    q = _normal(rng, (B, Hq, L, d), cfg.dtype)
    k_live = _normal(rng, (B, Hkv, L, d), cfg.dtype)
    v_live = _normal(rng, (B, Hkv, L, d), cfg.dtype)
    unmasked = np.zeros((B, L), dtype=bool)
    unmasked[:, : cfg.prompt] = True
    gen = L - cfg.prompt
    seed_idx = np.full((B, max_seeds), -1, dtype=np.int32)
    n_seed = np.zeros((B,), dtype=np.int32)
    for b in range(B):
        um = cfg.prompt + np.sort(rng.choice(gen, size=min(cfg.unmasked_gen, gen), replace=False))
        unmasked[b, um] = True
        ns = min(cfg.n_seeds, um.size, max_seeds)
        s = np.sort(rng.choice(um, size=ns, replace=False)).astype(np.int32)
        seed_idx[b, :ns] = s
        n_seed[b] = ns
    if cfg.cache == "independent":
        k_cache = _normal(rng, (B, Hkv, L, d), cfg.dtype)
        v_cache = _normal(rng, (B, Hkv, L, d), cfg.dtype)
    elif cfg.cache == "perturb":
        um = torch.from_numpy(unmasked)[:, None, :, None]
        k_cache = torch.where(um, (k_live.float() + 0.1 * _normal(rng, k_live.shape, "f32"))
                              .to(k_live.dtype), k_live)
        v_cache = torch.where(um, (v_live.float() + 0.1 * _normal(rng, v_live.shape, "f32"))
                              .to(v_live.dtype), v_live)
    else:
        raise ValueError(cfg.cache)
    return dict(cfg=cfg, q=q, k_live=k_live, v_live=v_live, k_cache=k_cache, v_cache=v_cache,
                seed_idx=torch.from_numpy(seed_idx), n_seed=torch.from_numpy(n_seed),
                unmasked=torch.from_numpy(unmasked), scale=1.0 / float(np.sqrt(d)))


def select_inputs(B: int, Lr: int, seed: int = 0, unmasked: int | None = None,
                  n_excl_prev: int = 16, n_excl_budget: int = 4, n_masked_q: int | None = None,
                  n_draft: int = 15, L_total: int | None = None,
                  unmasked_mask: np.ndarray | None = None,
                  prev_seeds: np.ndarray | None = None) -> dict:
    """Host tensors for one selection call over a region of Lr positions per batch row.

    Stand-ins for the signals of the paper's decoding step:
      confidence of the assigned token ~ Beta(5, 1); logp = fp32(log conf)
      d_in(j)  = (1/L_total) sum over the still-masked queries of exp(z - 1/2), z ~ N(0,1)
      d_out(j) = (1/L_total) sum over n_draft drafted columns of exp(z - 1/2)
    (the mass an N(0,1)-logit softmax row over L_total positions puts on one column, summed
    over the contributing rows/columns).  flags bit0 = unmasked, bit1 = excluded: the
    previous step's seeds plus positions that reached their ReMask budget.
    """
    rng = np.random.default_rng(seed + 7919)
    if unmasked is None:
        unmasked = Lr // 2
    if L_total is None:
        L_total = 4 * Lr
    flags = np.zeros((B, Lr), dtype=np.uint8)
    for b in range(B):
        if unmasked_mask is not None:
            um = np.nonzero(unmasked_mask[b])[0]
        else:
            um = np.sort(rng.choice(Lr, size=min(unmasked, Lr), replace=False))
        flags[b, um] = 1
        if prev_seeds is not None:
            ex = prev_seeds[b][prev_seeds[b] >= 0]
        else:
            ex = rng.choice(um, size=min(n_excl_prev, um.size), replace=False) if um.size else um
        rest = np.setdiff1d(um, ex)
        nb = min(n_excl_budget, rest.size)
        ex2 = rng.choice(rest, size=nb, replace=False) if nb else rest[:0]
        flags[b, ex] |= 2
        flags[b, ex2] |= 2
    conf = rng.beta(5.0, 1.0, size=(B, Lr))
    logp = np.log(conf).astype(np.float32)
    nm = n_masked_q if n_masked_q is not None else int((flags & 1 == 0).sum(axis=1).max())
    nm = max(nm, 1)
    z_in = rng.standard_normal(size=(B, Lr, nm))
    z_out = rng.standard_normal(size=(B, Lr, max(n_draft, 1)))
    d_in = (np.exp(z_in - 0.5).sum(axis=2) / L_total).astype(np.float32)
    d_out = (np.exp(z_out - 0.5).sum(axis=2) / L_total).astype(np.float32)
    if n_draft == 0:
        d_out[:] = 0.0
    return dict(logp=torch.from_numpy(logp), d_in=torch.from_numpy(d_in),
                d_out=torch.from_numpy(d_out), flags=torch.from_numpy(flags))


def step_inputs(cfg: AttnConfig | str = "llada", seed: int = 0) -> dict:
    """One hot-path pass at an attention config: attention inputs plus the selection inputs
    of the generated region [prompt, L) (its unmasked set and the current seeds as the
    previous-step exclusion), region offset = prompt."""
    a = attn_inputs(cfg, seed)
    c = a["cfg"]
    Lr = c.L - c.prompt
    um = a["unmasked"].numpy()[:, c.prompt:]
    prev = a["seed_idx"].numpy().copy()
    prev = np.where(prev >= 0, prev - c.prompt, -1)
    s = select_inputs(c.B, Lr, seed, unmasked_mask=um, prev_seeds=prev,
                      n_masked_q=int(Lr - um.sum(axis=1).min()), L_total=c.L)
    a.update(s)
    a["pos_offset"] = c.prompt
    a["Lr"] = Lr
    return a


def token_inputs(R: int, V: int, seed: int = 0, dtype: str = "bf16", peak: float = 14.0) -> dict:
    """Logits of R positions over a vocabulary of V (stand-in for the LM head's output on the
    generated block): N(0, 2^2) with one token per row raised by U(0, peak), so the maximum
    probability spans near-uniform to near-certain rows.  logits is a [R, V] view of
    `buffer`, whose rows are padded to 16 bytes (move the buffer, then slice, to keep the
    padded row stride on the device).  tokens: the raised token for even rows, a
    uniformly random token for odd rows."""
    rng = np.random.default_rng(seed + 104729)
    x = rng.standard_normal(size=(R, V)).astype(np.float32) * 2.0
    top = rng.integers(0, V, size=R)
    x[np.arange(R), top] += rng.uniform(0.0, peak, size=R).astype(np.float32)
    per = 8 if dtype == "bf16" else 4
    stride = (V + per - 1) // per * per
    buf = torch.zeros((R, stride), dtype=TORCH_DTYPE[dtype])
    buf[:, :V] = torch.from_numpy(x).to(TORCH_DTYPE[dtype])
    tokens = np.where(np.arange(R) % 2 == 0, top, rng.integers(0, V, size=R)).astype(np.int32)
    return dict(logits=buf[:, :V], buffer=buf, tokens=torch.from_numpy(tokens))


def stats_inputs(cfg: AttnConfig | str = "llada", seed: int = 0, n_draft: int = 15) -> dict:
    """Attention inputs plus the masks of the generated region [prompt, L): masked = the
    positions still masked, drafted = up to n_draft of them chosen uniformly."""
    a = attn_inputs(cfg, seed)
    c = a["cfg"]
    rng = np.random.default_rng(seed + 15485863)
    Lr = c.L - c.prompt
    masked = (~a["unmasked"].numpy()[:, c.prompt:]).astype(np.uint8)
    drafted = np.zeros_like(masked)
    for b in range(c.B):
        mpos = np.nonzero(masked[b])[0]
        if mpos.size:
            drafted[b, rng.choice(mpos, size=min(n_draft, mpos.size), replace=False)] = 1
    a.update(masked=torch.from_numpy(masked), drafted=torch.from_numpy(drafted), r0=c.prompt,
             Lr=Lr)
    return a


def update_inputs(B: int, Lr: int, seed: int = 0, vocab: int = 126464, masked_frac: float = 0.5,
                  n_seeds: int = 16, max_seeds: int = 16, conf_levels: int = 0,
                  keep_frac: float = 0.4, pos_offset: int = 768) -> dict:
    """Host tensors for one decoding-state update over a region of Lr positions per row:
    tokens with about masked_frac at mask_id (= vocab - 1), the step's argmax tokens (equal to
    the current token at about keep_frac of the unmasked positions), confidences (uniform on
    [0, 1) in fp32, or drawn from conf_levels distinct values when conf_levels > 0, which
    makes ties), seeds = min(n_seeds, #unmasked) distinct unmasked positions per row (absolute
    positions, region start pos_offset, listed in random order, then -1), ReMask counters in
    [0, 3]."""
    rng = np.random.default_rng(seed)
    mask_id = vocab - 1
    tokens = rng.integers(0, vocab - 1, (B, Lr))
    tokens[rng.random((B, Lr)) < masked_frac] = mask_id
    argmax = rng.integers(0, vocab - 1, (B, Lr))
    same = (rng.random((B, Lr)) < keep_frac) & (tokens != mask_id)
    argmax[same] = tokens[same]
    if conf_levels > 0:
        conf = rng.choice(rng.random(conf_levels), (B, Lr))
    else:
        conf = rng.random((B, Lr))
    seed_idx = np.full((B, max(max_seeds, 0)), -1, np.int64)
    n_seed = np.zeros(B, np.int64)
    for b in range(B):
        um = np.nonzero(tokens[b] != mask_id)[0]
        k = min(n_seeds, um.size, max_seeds)
        seed_idx[b, :k] = pos_offset + rng.choice(um, k, replace=False)
        n_seed[b] = k
    t = lambda x, dt: torch.from_numpy(np.ascontiguousarray(x)).to(dt)
    return {"tokens": t(tokens, torch.int32), "argmax": t(argmax, torch.int32),
            "conf": t(conf.astype(np.float32), torch.float32),
            "seed_idx": t(seed_idx, torch.int32), "n_seed": t(n_seed, torch.int32),
            "remask_count": t(rng.integers(0, 4, (B, Lr)), torch.int32),
            "mask_id": mask_id, "pos_offset": pos_offset}
