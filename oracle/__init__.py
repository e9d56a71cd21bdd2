"""COVER fp64 CPU oracle -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The HIP library and its Python binding never
call it; the two share no code.

The arithmetic lives in ``cover_oracle.c`` (plain C, fp64, built with
``-ffp-contract=off`` so no multiply-add is fused).  This module only marshals numpy
arrays in and out through ctypes.  Paper: arXiv 2602.06161.

Functions (each cites the passage it follows):
  attn              Sec. 5.1 + App. B.1, materialised leave-one-out view per row
  attn_closed_form  App. B.2-B.4, the paper's post-hoc diagonal correction
  select            Sec. 5.3, score / adaptive budget / exclusion / top-k
  token_stats       Sec. 5.3 u(j) and Sec. 3 confidence, from logits
  attn_stats        Sec. 5.3 d_in / d_out from the head-averaged attention
  decode_update     Sec. 5.2 drafting with a cap and the Keep/Replace/ReMask revision rule;
                    Sec. 3 state update; Sec. 5.3 exclusion inputs of the next selection
                    (plain numpy here, in the order the paper states the rules)
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cover_oracle.c")
_LIB = os.path.join(_HERE, "libcover_oracle.so")
_CFLAGS = ["-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared"]

_ERRORS = {1: "invalid sizes", 2: "seed contract violated (out of range or duplicate)",
           3: "non-finite or negative selection input", 4: "allocation failure"}


class OracleError(RuntimeError):
    pass


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (host only)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", *_CFLAGS, "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        P = ctypes.c_void_p
        I = ctypes.c_int
        I64 = ctypes.c_int64
        D = ctypes.c_double
        lib.cover_oracle_attn.argtypes = [P, P, P, P, P, P, P, I, I, I, I, I, I, D, I, P, I64, P, P]
        lib.cover_oracle_attn_closed.argtypes = [P, P, P, P, P, P, P, I, I, I, I, I, I, D, P, P]
        lib.cover_oracle_select.argtypes = [P, P, P, P, I, I, I, I, P, P, P]
        lib.cover_oracle_token_stats.argtypes = [P, P, I64, I64, P, P, P]
        lib.cover_oracle_attn_stats.argtypes = [P, P, P, P, P, I, I, I, I, I, I, D, I, I, P, P, P, P]
        lib.cover_oracle_threads.argtypes = []
        lib.cover_oracle_threads.restype = ctypes.c_int
        lib.cover_oracle_set_threads.argtypes = [ctypes.c_int]
        lib.cover_oracle_set_threads.restype = None
        for f in (lib.cover_oracle_attn, lib.cover_oracle_attn_closed, lib.cover_oracle_select,
                  lib.cover_oracle_token_stats, lib.cover_oracle_attn_stats):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_load().cover_oracle_threads())


def set_threads(n: int) -> None:
    """Sets the OpenMP threads of the oracle's parallel loops (results do not depend on it)."""
    _load().cover_oracle_set_threads(int(n))


def _f64(x) -> np.ndarray:
    """Exact widening of any stored float (bf16, fp16, fp32, fp64) to a contiguous fp64 array."""
    if hasattr(x, "detach"):  # a torch tensor: widen on the host
        x = x.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _i32(x) -> np.ndarray:
    if hasattr(x, "detach"):
        x = x.detach().to("cpu").numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int):
    if rc != 0:
        raise OracleError(_ERRORS.get(rc, f"oracle error {rc}"))


def _attn_args(q, k_live, v_live, k_cache, v_cache, seed_idx, n_seed, scale):
    q, kl, vl, kc, vc = (_f64(t) for t in (q, k_live, v_live, k_cache, v_cache))
    if q.ndim != 4 or kl.ndim != 4:
        raise ValueError("q is [B,Hq,L,d] and k/v are [B,Hkv,L,d]")
    B, Hq, L, d = q.shape
    Hkv = kl.shape[1]
    for t in (kl, vl, kc, vc):
        if t.shape != (B, Hkv, L, d):
            raise ValueError(f"k/v shape {t.shape} != {(B, Hkv, L, d)}")
    si = _i32(seed_idx).reshape(B, -1) if seed_idx is not None else np.zeros((B, 0), np.int32)
    ns = _i32(n_seed).reshape(B) if n_seed is not None else np.zeros((B,), np.int32)
    si = np.ascontiguousarray(si)
    if scale is None or scale == 0.0:
        scale = 1.0 / np.sqrt(d)
    return q, kl, vl, kc, vc, si, ns, (B, Hq, Hkv, L, d, si.shape[1]), float(scale)


def attn(q, k_live, v_live, k_cache, v_cache, seed_idx, n_seed, scale=None, mode="literal",
         rows=None):
    """Leave-one-out COVER attention (Sec. 5.1, App. B.1), fp64.

    Returns (out, lse).  With rows=None: out [B,Hq,L,d], lse [B,Hq,L].  With rows (flat
    indices (b*Hq+h)*L+i): out [n,d], lse [n].  mode: "literal" (a materialised L x d view
    per row) or "fast" (shared override view for non-seed rows; bitwise identical).
    """
    q, kl, vl, kc, vc, si, ns, dims, scale = _attn_args(q, k_live, v_live, k_cache, v_cache,
                                                        seed_idx, n_seed, scale)
    B, Hq, Hkv, L, d, ms = dims
    if rows is None:
        out = np.zeros((B, Hq, L, d))
        lse = np.zeros((B, Hq, L))
        rp, nr = None, 0
    else:
        rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64).reshape(-1))
        out = np.zeros((rows.size, d))
        lse = np.zeros((rows.size,))
        rp, nr = _ptr(rows), rows.size
    rc = _load().cover_oracle_attn(_ptr(q), _ptr(kl), _ptr(vl), _ptr(kc), _ptr(vc), _ptr(si),
                                   _ptr(ns), B, Hq, Hkv, L, d, ms, scale,
                                   1 if mode == "literal" else 0, rp, nr, _ptr(out), _ptr(lse))
    _check(rc)
    return out, lse


def attn_closed_form(q, k_live, v_live, k_cache, v_cache, seed_idx, n_seed, scale=None):
    """Override attention + the paper's closed-form diagonal correction (App. B.2-B.4)."""
    q, kl, vl, kc, vc, si, ns, dims, scale = _attn_args(q, k_live, v_live, k_cache, v_cache,
                                                        seed_idx, n_seed, scale)
    B, Hq, Hkv, L, d, ms = dims
    out = np.zeros((B, Hq, L, d))
    lse = np.zeros((B, Hq, L))
    rc = _load().cover_oracle_attn_closed(_ptr(q), _ptr(kl), _ptr(vl), _ptr(kc), _ptr(vc),
                                          _ptr(si), _ptr(ns), B, Hq, Hkv, L, d, ms, scale,
                                          _ptr(out), _ptr(lse))
    _check(rc)
    return out, lse


def select(logp, d_in, d_out, flags, max_seeds, pos_offset=0):
    """Stability-aware seed selection with adaptive budget (Sec. 5.3).

    Inputs are fp32 [B,Lr] (logp, d_in, d_out) and uint8 flags [B,Lr] (bit0: unmasked,
    bit1: excluded).  Returns (seed_idx int32 [B,max_seeds] ascending, -1 padded;
    n_seed int32 [B]; score fp64 [B,Lr]).
    """
    def f32(x):
        if hasattr(x, "detach"):
            x = x.detach().to("cpu").numpy()
        return np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    lp, di, do = f32(logp), f32(d_in), f32(d_out)
    if lp.ndim == 1:
        lp, di, do = lp[None], di[None], do[None]
    fl = flags.detach().to("cpu").numpy() if hasattr(flags, "detach") else flags
    fl = np.ascontiguousarray(np.asarray(fl, dtype=np.uint8)).reshape(lp.shape)
    B, Lr = lp.shape
    seed_idx = np.full((B, max_seeds), -1, np.int32)
    n_seed = np.zeros((B,), np.int32)
    score = np.zeros((B, Lr))
    rc = _load().cover_oracle_select(_ptr(lp), _ptr(di), _ptr(do), _ptr(fl), B, Lr,
                                     int(max_seeds), int(pos_offset), _ptr(seed_idx),
                                     _ptr(n_seed), _ptr(score))
    _check(rc)
    return seed_idx, n_seed, score


def token_stats(logits, y):
    """Per row: log p(y), max probability, argmax (Sec. 5.3 u(j); Sec. 3 confidence)."""
    x = _f64(logits)
    R, V = x.shape
    yy = _i32(y).reshape(R)
    logp = np.zeros(R)
    conf = np.zeros(R)
    amax = np.zeros(R, np.int32)
    rc = _load().cover_oracle_token_stats(_ptr(x), _ptr(yy), R, V, _ptr(logp), _ptr(conf),
                                          _ptr(amax))
    _check(rc)
    return logp, conf, amax


def attn_stats(q, k_live, k_cache, seed_idx, n_seed, r0, masked, drafted, scale=None):
    """d_in / d_out over the region [r0, r0+Lr) from head-averaged corrected weights (Sec. 5.3)."""
    qq, kl, kc = _f64(q), _f64(k_live), _f64(k_cache)
    B, Hq, L, d = qq.shape
    Hkv = kl.shape[1]
    si = np.ascontiguousarray(_i32(seed_idx).reshape(B, -1))
    ns = _i32(n_seed).reshape(B)
    m = np.ascontiguousarray(np.asarray(masked, dtype=np.uint8)).reshape(B, -1)
    dr = np.ascontiguousarray(np.asarray(drafted, dtype=np.uint8)).reshape(B, -1)
    Lr = m.shape[1]
    if scale is None or scale == 0.0:
        scale = 1.0 / np.sqrt(d)
    d_in = np.zeros((B, Lr))
    d_out = np.zeros((B, Lr))
    rc = _load().cover_oracle_attn_stats(_ptr(qq), _ptr(kl), _ptr(kc), _ptr(si), _ptr(ns), B, Hq,
                                         Hkv, L, d, si.shape[1], float(scale), int(r0), Lr,
                                         _ptr(m), _ptr(dr), _ptr(d_in), _ptr(d_out))
    _check(rc)
    return d_in, d_out


def decode_update(tokens, argmax, conf, seed_idx, n_seed, remask_count, mask_id, tau, cap,
                  remask_budget, pos_offset=0, last_unmask=None, min_draft=0):
    """One decoding step's state update over a region of Lr positions (absolute position =
    pos_offset + region index), for each batch row:

    drafting (Sec. 5.2, Drafting): D = the masked positions (token == mask_id) whose
      confidence exceeds tau (strictly), keeping the `cap` largest confidences when more
      qualify (ties: smaller position first); each drafted position takes its argmax token.
    revision (Sec. 5.2, Revision outcomes), for each previous seed i (seed_idx[b, :n_seed[b]],
      absolute positions; entries outside the region or at masked positions are ignored):
      Keep if argmax_i == token_i; Replace (token_i = argmax_i) if they differ and
      conf_i > tau; otherwise ReMask (token_i = mask_id).  R = the ReMasked seeds.
    state update (Sec. 3, State update): U_t = (U_{t-1} + D) - R.
    counters: remask_count_i += 1 for i in R (Sec. 5.3 per-position ReMask budget).
    next selection's flags (Sec. 5.3, exclusion): bit 0 = unmasked after the update; bit 1 =
      i was a seed this step, or remask_count_i >= remask_budget.

    min_draft (not in the paper; 0 keeps its rule): when fewer than min_draft masked positions
      pass tau, the min_draft most confident masked positions (same order) are drafted
      instead, so that a decoding loop always progresses.
    flip-flops (Sec. 4, Definition): with last_unmask given (the token of each position's most
      recent [MASK] -> token transition, -1 if none yet), a drafted position whose new token
      equals its last_unmask entry is a flip-flop event; every drafted position then records
      its new token there.  Replace is not an unmasking and leaves last_unmask alone.

    Confidences compare with tau in fp32.  Returns (tokens, remask_count, flags, drafted,
    counts) with counts[b] = (|D|, kept, replaced, remasked, masked after the update); with
    last_unmask given, also (last_unmask, flipflops[b]).
    """
    tok = np.array(tokens, dtype=np.int64, copy=True)
    am = np.asarray(argmax, dtype=np.int64)
    c = np.asarray(conf, dtype=np.float32)
    cnt = np.array(remask_count, dtype=np.int64, copy=True)
    si = np.asarray(seed_idx, dtype=np.int64).reshape(tok.shape[0], -1)
    ns = np.asarray(n_seed, dtype=np.int64).reshape(-1)
    t32 = np.float32(tau)
    B, Lr = tok.shape
    flags = np.zeros((B, Lr), np.uint8)
    drafted = np.zeros((B, Lr), np.uint8)
    counts = np.zeros((B, 5), np.int64)
    last = None if last_unmask is None else np.array(last_unmask, dtype=np.int64, copy=True)
    ff = np.zeros(B, np.int64)
    for b in range(B):
        # the previous step's seeds, as region indices (each counted once)
        seeds = set()
        for t in range(max(0, min(int(ns[b]), si.shape[1]))):
            i = int(si[b, t]) - pos_offset
            if 0 <= i < Lr and tok[b, i] != mask_id:
                seeds.add(i)
        # drafting over M_{t-1}
        cand = [i for i in range(Lr) if tok[b, i] == mask_id and c[b, i] > t32]
        cand.sort(key=lambda i: (-float(c[b, i]), i))
        D = cand[:max(0, int(cap))]
        if len(cand) < min_draft:
            masked = [i for i in range(Lr) if tok[b, i] == mask_id and not np.isnan(c[b, i])]
            masked.sort(key=lambda i: (-float(c[b, i]), i))
            D = masked[:min_draft]
        # revision of the seeds
        kept = replaced = 0
        R = []
        for i in sorted(seeds):
            if am[b, i] == tok[b, i]:
                kept += 1
            elif c[b, i] > t32:
                replaced += 1
                tok[b, i] = am[b, i]
            else:
                R.append(i)
        # state update
        for i in D:
            tok[b, i] = am[b, i]
            drafted[b, i] = 1
            if last is not None:
                if last[b, i] == am[b, i]:
                    ff[b] += 1
                last[b, i] = am[b, i]
        for i in R:
            tok[b, i] = mask_id
            cnt[b, i] += 1
        for i in range(Lr):
            excl = i in seeds or cnt[b, i] >= remask_budget
            flags[b, i] = (1 if tok[b, i] != mask_id else 0) | (2 if excl else 0)
        counts[b] = (len(D), kept, replaced, len(R), int(np.sum(tok[b] == mask_id)))
    out = (tok.astype(np.int32), cnt.astype(np.int32), flags, drafted, counts.astype(np.int32))
    if last is not None:
        out = out + (last.astype(np.int32), ff.astype(np.int32))
    return out


# ---- temperature sampling of the draft tokens (stochastic decoding, App. "Robustness under
# stochastic decoding") ----------------------------------------------------------------------

_PHILOX_M = (0xD2511F53, 0xCD9E8D57)  # Philox4x32 multipliers (Salmon et al., SC 2011)
_PHILOX_W = (0x9E3779B9, 0xBB67AE85)  # Weyl key increments
_U32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """The Philox4x32-10 counter-based generator as published (Salmon, Moraes, Dror, Shaw,
    "Parallel random numbers: as easy as 1, 2, 3", SC 2011): ten rounds of two 32x32 -> 64-bit
    multiplications whose halves are mixed with the other two counter words and the key, the
    key advanced by the Weyl constants between rounds.  Arguments: arrays (or scalars) of
    32-bit values; returns the four 32-bit output words as uint64 arrays."""
    c = [np.asarray(x, dtype=np.uint64) & _U32 for x in (c0, c1, c2, c3)]
    k0 = np.asarray(k0, dtype=np.uint64) & _U32
    k1 = np.asarray(k1, dtype=np.uint64) & _U32
    for r in range(10):
        if r:
            k0 = (k0 + np.uint64(_PHILOX_W[0])) & _U32
            k1 = (k1 + np.uint64(_PHILOX_W[1])) & _U32
        p0 = np.uint64(_PHILOX_M[0]) * c[0]
        p1 = np.uint64(_PHILOX_M[1]) * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & _U32
        hi1, lo1 = p1 >> np.uint64(32), p1 & _U32
        c = [hi1 ^ c[1] ^ k0, lo1, hi0 ^ c[3] ^ k1, lo0]
    return c


def sample_uniforms(R, V, seed, step):
    """u[r, v] in (0, 1): word v % 4 of Philox4x32-10 with counter (v // 4, r, step, 0) and
    key (seed mod 2^32, seed >> 32), mapped as ((w >> 9) + 1/2) 2^-23 (exact in fp32)."""
    v = np.arange(V, dtype=np.uint64)
    r = np.arange(R, dtype=np.uint64)[:, None]
    words = philox4x32_10(v[None, :] // np.uint64(4), r, np.uint64(step), np.uint64(0),
                          np.uint64(seed & 0xFFFFFFFF), np.uint64((seed >> 32) & 0xFFFFFFFF))
    w = np.choose((v % np.uint64(4)).astype(np.int64)[None, :].repeat(R, 0),
                  [np.broadcast_to(x, (R, V)) for x in words])
    return ((w >> np.uint64(9)).astype(np.float64) + 0.5) * 2.0 ** -23


def token_sample(logits, temperature, seed, step):
    """Temperature sampling per row of logits [R, V] (the stochastic drafting the paper tests
    at T in {0.1, 0.2, 0.3}) by the Gumbel-max construction: token = argmax_v (x_v / T + g_v)
    with g_v = -ln(-ln u_v) standard Gumbel noise from sample_uniforms (smallest v on ties),
    which draws v with probability softmax(x / T)_v; its probability p = softmax(x / T) at the
    token is the confidence the drafting rule compares with tau.  fp64.  Returns (token int32
    [R], p [R], y [R, V] the perturbed scores)."""
    x = np.asarray(logits, dtype=np.float64)
    R, V = x.shape
    u = sample_uniforms(R, V, seed, step)
    y = x / temperature - np.log(-np.log(u))
    tok = np.argmax(y, axis=1)
    z = x / temperature
    zm = z.max(axis=1, keepdims=True)
    lse = zm[:, 0] + np.log(np.exp(z - zm).sum(axis=1))
    p = np.exp(z[np.arange(R), tok] - lse)
    return tok.astype(np.int32), p, y
