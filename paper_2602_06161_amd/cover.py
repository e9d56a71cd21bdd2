"""ctypes binding of the COVER C ABI (``include/cover.h``).

Argument marshalling only: torch supplies device memory and the stream; every step of the
computation runs in the HIP kernels of ``libcover.so``.  There is no fallback -- if the
library has not been built, or a call is rejected, an exception is raised.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

from .build import LIB

COVER_OK, COVER_ERR_INVALID, COVER_ERR_UNSUPPORTED, COVER_ERR_HIP = 0, -1, -2, -3
COVER_F32, COVER_BF16 = 0, 1
COVER_MAX_L = 65536
COVER_MAX_LR = 16384
COVER_RECT_RECORD = 68

EXPORTED = ("cover_attn_fwd", "cover_attn_rect", "cover_attn_stats", "cover_attn_stats_noalloc",
            "cover_attn_stats_workspace",
            "cover_debug_status", "cover_decode_update",
            "cover_select_seeds", "cover_status_str", "cover_token_sample", "cover_token_stats",
            "cover_version")
# status bits of the contract checks that COVER_DEBUG=1 enables (cover_debug_status)
COVER_DEBUG_SEED_COUNT, COVER_DEBUG_SEED_RANGE, COVER_DEBUG_SEED_DUPLICATE = 1, 2, 4
COVER_DEBUG_SELECT_NONFINITE, COVER_DEBUG_SELECT_NEGATIVE = 8, 16


class CoverError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_str(status)} ({status})")
        self.status = status


class AttnDesc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("Hq", ctypes.c_int32), ("Hkv", ctypes.c_int32),
                ("L", ctypes.c_int32), ("d", ctypes.c_int32), ("max_seeds", ctypes.c_int32),
                ("dtype", ctypes.c_int), ("scale", ctypes.c_float),
                ("q_sb", ctypes.c_int64), ("q_sh", ctypes.c_int64), ("q_sl", ctypes.c_int64),
                ("kv_sb", ctypes.c_int64), ("kv_sh", ctypes.c_int64), ("kv_sl", ctypes.c_int64)]


class SelectDesc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("Lr", ctypes.c_int32), ("max_seeds", ctypes.c_int32),
                ("pos_offset", ctypes.c_int32)]


class TokenDesc(ctypes.Structure):
    _fields_ = [("R", ctypes.c_int32), ("V", ctypes.c_int32), ("dtype", ctypes.c_int),
                ("row_stride", ctypes.c_int64)]


class UpdateDesc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("Lr", ctypes.c_int32), ("max_seeds", ctypes.c_int32),
                ("pos_offset", ctypes.c_int32), ("mask_id", ctypes.c_int32),
                ("draft_cap", ctypes.c_int32), ("remask_budget", ctypes.c_int32),
                ("tau", ctypes.c_float), ("min_draft", ctypes.c_int32)]


class RectDesc(ctypes.Structure):
    _fields_ = [("attn", AttnDesc), ("q_off", ctypes.c_int32), ("Lq", ctypes.c_int32),
                ("n_split", ctypes.c_int32)]


class StatsDesc(ctypes.Structure):
    _fields_ = [("attn", AttnDesc), ("r0", ctypes.c_int32), ("Lr", ctypes.c_int32)]


def attn_stats_workspace(B: int, Hq: int, Lr: int) -> int:
    """Floats of workspace a cover_attn_stats call of this size uses (the library's
    cover_attn_stats_workspace)."""
    n = lib().cover_attn_stats_workspace(int(B), int(Hq), int(Lr))
    if n < 0:
        raise ValueError("negative size")
    return int(n)


_lib = None
_lib_path = LIB


def use_library(path: str) -> None:
    """Load the library from `path` instead of libcover.so (the in-tree timing build of the
    same sources, for measurements).  Must come before the first call."""
    global _lib_path
    if _lib is not None and path != _lib_path:
        raise RuntimeError("the COVER library is already loaded")
    _lib_path = path


def lib():
    """Load libcover.so (built in-tree); raise if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(_lib_path):
            raise RuntimeError(f"COVER HIP library not built ({_lib_path}); run "
                               "`python -m paper_2602_06161_amd.build` or __graft_entry__.build()")
        L = ctypes.CDLL(_lib_path)
        P = ctypes.c_void_p
        L.cover_attn_fwd.argtypes = [P, P, P, P, P, P, P, P, P, ctypes.POINTER(AttnDesc), P]
        L.cover_attn_fwd.restype = ctypes.c_int
        L.cover_select_seeds.argtypes = [P, P, P, P, P, P, P, ctypes.POINTER(SelectDesc), P]
        L.cover_select_seeds.restype = ctypes.c_int
        L.cover_token_stats.argtypes = [P, P, P, P, P, ctypes.POINTER(TokenDesc), P]
        L.cover_attn_rect.argtypes = [P, P, P, P, P, P, P, P, P, P, ctypes.POINTER(RectDesc), P]
        L.cover_attn_rect.restype = ctypes.c_int
        L.cover_decode_update.argtypes = [P, P, P, P, P, P, P, P, P, P, P,
                                          ctypes.POINTER(UpdateDesc), P]
        L.cover_decode_update.restype = ctypes.c_int
        L.cover_token_stats.restype = ctypes.c_int
        L.cover_token_sample.argtypes = [P, ctypes.c_float, ctypes.c_uint64, ctypes.c_uint32, P, P,
                                         ctypes.POINTER(TokenDesc), P]
        L.cover_token_sample.restype = ctypes.c_int
        L.cover_attn_stats.argtypes = [P, P, P, P, P, P, P, P, P, P, P, ctypes.POINTER(StatsDesc), P]
        L.cover_attn_stats.restype = ctypes.c_int
        L.cover_attn_stats_noalloc.argtypes = [P, P, P, P, P, P, P, P, P, P,
                                               ctypes.POINTER(StatsDesc), P]
        L.cover_attn_stats_noalloc.restype = ctypes.c_int
        L.cover_attn_stats_workspace.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]
        L.cover_attn_stats_workspace.restype = ctypes.c_int64
        L.cover_status_str.argtypes = [ctypes.c_int]
        L.cover_status_str.restype = ctypes.c_char_p
        L.cover_version.argtypes = []
        L.cover_version.restype = ctypes.c_int32
        L.cover_debug_status.argtypes = [ctypes.POINTER(ctypes.c_int32), ctypes.c_int32, P]
        L.cover_debug_status.restype = ctypes.c_int
        _lib = L
    return _lib


def status_str(s: int) -> str:
    return lib().cover_status_str(s).decode()


def version() -> int:
    return lib().cover_version()


def debug_status(clear: bool = False, stream=None) -> int:
    """The contract-violation bits recorded under COVER_DEBUG=1 on the current GPU (waits
    for `stream`); optionally reset them."""
    v = ctypes.c_int32(0)
    st = lib().cover_debug_status(ctypes.byref(v), 1 if clear else 0, _stream(stream))
    if st != COVER_OK:
        raise CoverError(st, "cover_debug_status")
    return v.value


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def attn_desc(q: torch.Tensor, k: torch.Tensor, max_seeds: int, scale: float = 0.0) -> AttnDesc:
    B, Hq, L, d = q.shape
    Hkv = k.shape[1]
    dt = {torch.float32: COVER_F32, torch.bfloat16: COVER_BF16}.get(q.dtype)
    if dt is None:
        raise TypeError(f"unsupported dtype {q.dtype}")
    return AttnDesc(B, Hq, Hkv, L, d, max_seeds, dt, float(scale),
                    q.stride(0), q.stride(1), q.stride(2), k.stride(0), k.stride(1), k.stride(2))


def cover_attn_fwd(q, k_live, v_live, k_cache, v_cache, seed_idx=None, n_seed=None, out=None,
                   lse=None, scale: float = 0.0, stream=None, want_lse: bool = True):
    """COVER attention of one layer.  Tensors on the GPU: q [B,Hq,L,d]; k/v [B,Hkv,L,d]
    (head dim contiguous, all four K/V tensors with identical strides); seed_idx int32
    [B,max_seeds]; n_seed int32 [B].  Returns (out, lse)."""
    for t in (k_live, v_live, k_cache, v_cache):
        if t.shape != k_live.shape or t.stride() != k_live.stride() or t.dtype != q.dtype:
            raise ValueError("k_live, v_live, k_cache, v_cache need equal shape, strides and dtype")
    if q.stride(-1) != 1 or k_live.stride(-1) != 1:
        raise ValueError("head dimension must be contiguous")
    max_seeds = 0 if seed_idx is None else seed_idx.shape[-1]
    if seed_idx is not None and (seed_idx.dtype != torch.int32 or n_seed is None
                                 or n_seed.dtype != torch.int32 or not seed_idx.is_contiguous()):
        raise ValueError("seed_idx and n_seed must be contiguous int32 tensors")
    B, Hq, L, d = q.shape
    if out is None:
        out = torch.empty_like(q)
    if out.shape != q.shape or out.stride() != q.stride() or out.dtype != q.dtype:
        raise ValueError("out must match q's shape, strides and dtype")
    if lse is None and want_lse:
        lse = torch.empty((B, Hq, L), device=q.device, dtype=torch.float32)
    desc = attn_desc(q, k_live, max_seeds, scale)
    st = lib().cover_attn_fwd(_ptr(q), _ptr(k_live), _ptr(v_live), _ptr(k_cache), _ptr(v_cache),
                              _ptr(seed_idx), _ptr(n_seed), _ptr(out), _ptr(lse),
                              ctypes.byref(desc), _stream(stream))
    if st != COVER_OK:
        raise CoverError(st, "cover_attn_fwd")
    return out, lse


def rect_workspace(B: int, Hq: int, Lq: int, n_split: int) -> int:
    """Floats of workspace cover_attn_rect needs (COVER_ATTN_RECT_WORKSPACE): none for the
    single launch (n_split == 1)."""
    return B * Hq * n_split * Lq * COVER_RECT_RECORD if n_split > 1 else 0


def rect_splits(B: int, Hq: int, Lq: int, L: int) -> int:
    """Key splits.  1 (the single launch: one workgroup per 32 query rows, its waves split the
    keys) unless the sequence is long and the block leaves most CUs idle: that kernel reads
    all of a head's K and V through one CU per 32 rows, about 100 GB/s per CU, so past 2048
    keys with fewer than 256 workgroups the keys are split across workgroups instead (about
    256 workgroups of at least 128 keys each, merged by a second launch)."""
    if L <= 2048 or B * Hq * ((Lq + 31) // 32) >= 256:
        return 1
    wgs = B * Hq * ((Lq + 127) // 128)
    n = min(-(-256 // wgs), -(-L // 128))
    return max(1, min(n, 256))


def cover_attn_rect(q, k_live, v_live, k_cache, v_cache, q_off: int, seed_idx=None, n_seed=None,
                    out=None, lse=None, scale: float = 0.0, n_split=None, workspace=None,
                    want_lse: bool = True, stream=None):
    """COVER attention of the query block [q_off, q_off + Lq) against all L keys.  q
    [B,Hq,Lq,d] bf16; k/v [B,Hkv,L,d] (equal strides); seeds as for cover_attn_fwd (absolute
    positions).  Returns (out [B,Hq,Lq,d], lse [B,Hq,Lq])."""
    for t in (k_live, v_live, k_cache, v_cache):
        if t.shape != k_live.shape or t.stride() != k_live.stride() or t.dtype != q.dtype:
            raise ValueError("k_live, v_live, k_cache, v_cache need equal shape, strides and dtype")
    if q.stride(-1) != 1 or k_live.stride(-1) != 1:
        raise ValueError("head dimension must be contiguous")
    max_seeds = 0 if seed_idx is None else seed_idx.shape[-1]
    if seed_idx is not None and (seed_idx.dtype != torch.int32 or n_seed is None
                                 or n_seed.dtype != torch.int32 or not seed_idx.is_contiguous()):
        raise ValueError("seed_idx and n_seed must be contiguous int32 tensors")
    B, Hq, Lq, d = q.shape
    L = k_live.shape[2]
    if out is None:
        out = torch.empty_like(q)
    if out.shape != q.shape or out.stride() != q.stride() or out.dtype != q.dtype:
        raise ValueError("out must match q's shape, strides and dtype")
    if lse is None and want_lse:
        lse = torch.empty((B, Hq, Lq), device=q.device, dtype=torch.float32)
    if n_split is None:
        n_split = rect_splits(B, Hq, Lq, L)
    need = rect_workspace(B, Hq, Lq, n_split)
    if need == 0:
        workspace = None  # not used by the single launch
    elif workspace is None:
        workspace = torch.empty(need, device=q.device, dtype=torch.float32)
    if workspace is not None and (workspace.dtype != torch.float32 or workspace.numel() < need
                                  or not workspace.is_contiguous()):
        raise ValueError(f"workspace must be contiguous fp32 with at least {need} elements")
    ad = attn_desc(q, k_live, max_seeds, scale)
    ad.L = L
    desc = RectDesc(ad, q_off, Lq, n_split)
    st = lib().cover_attn_rect(_ptr(q), _ptr(k_live), _ptr(v_live), _ptr(k_cache), _ptr(v_cache),
                               _ptr(seed_idx), _ptr(n_seed), _ptr(out), _ptr(lse), _ptr(workspace),
                               ctypes.byref(desc), _stream(stream))
    if st != COVER_OK:
        raise CoverError(st, "cover_attn_rect")
    return out, lse


def cover_select_seeds(logp, d_in, d_out, flags, max_seeds: int, pos_offset: int = 0,
                       seed_idx=None, n_seed=None, score=None, want_score: bool = True,
                       stream=None):
    """Stability-aware seed selection.  logp/d_in/d_out fp32 [B,Lr], flags uint8 [B,Lr] on the
    GPU (contiguous).  Returns (seed_idx int32 [B,max_seeds], n_seed int32 [B], score fp64
    [B,Lr] or None)."""
    B, Lr = logp.shape
    for t, dt in ((logp, torch.float32), (d_in, torch.float32), (d_out, torch.float32),
                  (flags, torch.uint8)):
        if t.shape != (B, Lr) or t.dtype != dt or not t.is_contiguous():
            raise ValueError("selection inputs must be contiguous [B,Lr] (fp32 x3, uint8 flags)")
    dev = logp.device
    if seed_idx is None:
        seed_idx = torch.empty((B, max_seeds), device=dev, dtype=torch.int32)
    if n_seed is None:
        n_seed = torch.empty((B,), device=dev, dtype=torch.int32)
    if score is None and want_score:
        score = torch.empty((B, Lr), device=dev, dtype=torch.float64)
    desc = SelectDesc(B, Lr, max_seeds, pos_offset)
    st = lib().cover_select_seeds(_ptr(logp), _ptr(d_in), _ptr(d_out), _ptr(flags),
                                  _ptr(seed_idx), _ptr(n_seed), _ptr(score), ctypes.byref(desc),
                                  _stream(stream))
    if st != COVER_OK:
        raise CoverError(st, "cover_select_seeds")
    return seed_idx, n_seed, score


def cover_decode_update(tokens, argmax, conf, seed_idx, n_seed, remask_count, mask_id: int,
                        tau: float, draft_cap: int, remask_budget: int, pos_offset: int = 0,
                        flags=None, drafted=None, counts=None, want_outputs: bool = True,
                        last_unmask=None, flipflops=None, min_draft: int = 0, stream=None):
    """One step's decoding-state update, in place on tokens and remask_count (int32 [B,Lr]);
    argmax int32 / conf fp32 [B,Lr]; seed_idx int32 [B,max_seeds], n_seed int32 [B] (may be
    None: no seeds).  Returns (flags uint8, drafted uint8, counts int32 [B,5]), allocated
    unless given (None when want_outputs is False).  With last_unmask (int32 [B,Lr], in
    place) the step's flip-flop events go to flipflops (int32 [B], allocated unless given),
    returned as a fourth element."""
    B, Lr = tokens.shape
    for t, dt in ((tokens, torch.int32), (argmax, torch.int32), (conf, torch.float32),
                  (remask_count, torch.int32)):
        if t.shape != (B, Lr) or t.dtype != dt or not t.is_contiguous():
            raise ValueError("update inputs must be contiguous [B,Lr] (int32 x3, fp32 conf)")
    max_seeds = 0
    if seed_idx is not None:
        if seed_idx.dim() != 2 or seed_idx.shape[0] != B or seed_idx.dtype != torch.int32 or \
                not seed_idx.is_contiguous() or n_seed is None or n_seed.shape != (B,) or \
                n_seed.dtype != torch.int32:
            raise ValueError("seed_idx must be contiguous int32 [B,max_seeds], n_seed int32 [B]")
        max_seeds = seed_idx.shape[1]
    dev = tokens.device
    if want_outputs:
        flags = torch.empty((B, Lr), device=dev, dtype=torch.uint8) if flags is None else flags
        drafted = torch.empty((B, Lr), device=dev, dtype=torch.uint8) if drafted is None else drafted
        counts = torch.empty((B, 5), device=dev, dtype=torch.int32) if counts is None else counts
    for t, shape, dt in ((flags, (B, Lr), torch.uint8), (drafted, (B, Lr), torch.uint8),
                         (counts, (B, 5), torch.int32), (last_unmask, (B, Lr), torch.int32),
                         (flipflops, (B,), torch.int32)):
        if t is not None and (t.shape != shape or t.dtype != dt or not t.is_contiguous()):
            raise ValueError("flags/drafted must be contiguous uint8 [B,Lr], counts int32 [B,5], "
                             "last_unmask int32 [B,Lr], flipflops int32 [B]")
    if last_unmask is not None and flipflops is None:
        flipflops = torch.empty((B,), device=dev, dtype=torch.int32)
    desc = UpdateDesc(B, Lr, max_seeds, pos_offset, mask_id, draft_cap, remask_budget, tau,
                      min_draft)
    st = lib().cover_decode_update(_ptr(tokens), _ptr(argmax), _ptr(conf),
                                   _ptr(seed_idx) if max_seeds else None,
                                   _ptr(n_seed) if max_seeds else None, _ptr(remask_count),
                                   _ptr(flags), _ptr(drafted), _ptr(counts), _ptr(last_unmask),
                                   _ptr(flipflops), ctypes.byref(desc), _stream(stream))
    if st != COVER_OK:
        raise CoverError(st, "cover_decode_update")
    if last_unmask is not None:
        return flags, drafted, counts, flipflops
    return flags, drafted, counts


def cover_token_sample(logits, temperature: float, seed: int, step: int, want_prob: bool = True,
                       stream=None):
    """Temperature sampling per row of logits [R, V] (bf16 or fp32, last dimension
    contiguous, row stride a multiple of 16 bytes).  Returns (token int32 [R], prob fp32 [R]
    or None)."""
    R, V = logits.shape
    dt = {torch.float32: COVER_F32, torch.bfloat16: COVER_BF16}.get(logits.dtype)
    if dt is None or logits.stride(-1) != 1:
        raise ValueError("logits must be bf16 or fp32 with a contiguous last dimension")
    token = torch.empty(R, device=logits.device, dtype=torch.int32)
    prob = torch.empty(R, device=logits.device, dtype=torch.float32) if want_prob else None
    desc = TokenDesc(R, V, dt, logits.stride(0))
    st = lib().cover_token_sample(_ptr(logits), float(temperature), int(seed) & (2**64 - 1),
                                  int(step) & 0xFFFFFFFF, _ptr(token), _ptr(prob),
                                  ctypes.byref(desc), _stream(stream))
    if st != COVER_OK:
        raise CoverError(st, "cover_token_sample")
    return token, prob


def cover_token_stats(logits, tokens=None, want_logp: bool = True, want_conf: bool = True,
                      want_argmax: bool = True, stream=None):
    """Per-row log p(token), max probability and argmax of logits [R, V] (bf16 or fp32, last
    dimension contiguous, row stride a multiple of 16 bytes).  Returns (logp, conf, argmax),
    each None when not requested."""
    R, V = logits.shape
    dt = {torch.float32: COVER_F32, torch.bfloat16: COVER_BF16}.get(logits.dtype)
    if dt is None or logits.stride(-1) != 1:
        raise ValueError("logits must be bf16 or fp32 with a contiguous last dimension")
    if want_logp and (tokens is None or tokens.dtype != torch.int32 or tokens.shape != (R,)
                      or not tokens.is_contiguous()):
        raise ValueError("tokens must be a contiguous int32 [R] tensor")
    dev = logits.device
    logp = torch.empty(R, device=dev, dtype=torch.float32) if want_logp else None
    conf = torch.empty(R, device=dev, dtype=torch.float32) if want_conf else None
    amax = torch.empty(R, device=dev, dtype=torch.int32) if want_argmax else None
    desc = TokenDesc(R, V, dt, logits.stride(0))
    st = lib().cover_token_stats(_ptr(logits), _ptr(tokens if want_logp else None), _ptr(logp),
                                 _ptr(conf), _ptr(amax), ctypes.byref(desc), _stream(stream))
    if st != COVER_OK:
        raise CoverError(st, "cover_token_stats")
    return logp, conf, amax


def cover_attn_stats(q, k_live, k_cache, seed_idx, n_seed, lse, masked, drafted, r0: int,
                     scale: float = 0.0, workspace=None, stream=None):
    """d_in, d_out [B, Lr] over the region [r0, r0+Lr) (Lr = masked.shape[1]) from the corrected
    attention weights of cover_attn_fwd (lse from that call).  bf16 q/k; masked, drafted
    uint8 [B, Lr]."""
    B, Hq, L, d = q.shape
    Lr = masked.shape[1]
    for t in (k_live, k_cache):
        if t.shape != k_live.shape or t.stride() != k_live.stride() or t.dtype != q.dtype:
            raise ValueError("k_live and k_cache need equal shape, strides and dtype")
    for t in (masked, drafted):
        if t.shape != (B, Lr) or t.dtype != torch.uint8 or not t.is_contiguous():
            raise ValueError("masked / drafted must be contiguous uint8 [B, Lr]")
    if lse.shape != (B, Hq, L) or lse.dtype != torch.float32 or not lse.is_contiguous():
        raise ValueError("lse must be contiguous fp32 [B, Hq, L]")
    max_seeds = 0 if seed_idx is None else seed_idx.shape[-1]
    dev = q.device
    d_in = torch.empty((B, Lr), device=dev, dtype=torch.float32)
    d_out = torch.empty((B, Lr), device=dev, dtype=torch.float32)
    need = attn_stats_workspace(B, Hq, Lr)
    if workspace is None:
        workspace = torch.empty(max(1, need), device=dev, dtype=torch.float32)
    elif (workspace.dtype != torch.float32 or not workspace.is_contiguous()
          or workspace.numel() < need or workspace.device != dev):
        raise ValueError(f"workspace must be a contiguous fp32 tensor of at least {need} floats "
                         f"on {dev}")
    desc = StatsDesc(attn_desc(q, k_live, max_seeds, scale), int(r0), int(Lr))
    st = lib().cover_attn_stats(_ptr(q), _ptr(k_live), _ptr(k_cache), _ptr(seed_idx),
                                _ptr(n_seed), _ptr(lse), _ptr(masked), _ptr(drafted), _ptr(d_in),
                                _ptr(d_out), _ptr(workspace), ctypes.byref(desc), _stream(stream))
    if st != COVER_OK:
        raise CoverError(st, "cover_attn_stats")
    return d_in, d_out


COVER_STATS_SCRATCH_FLOATS = 1 << 20


def cover_attn_stats_noalloc(q, k_live, k_cache, seed_idx, n_seed, lse, masked, drafted,
                             r0: int, d_in, d_out, scale: float = 0.0, stream=None):
    """cover_attn_stats with the library's own per-GPU workspace: nothing is allocated, so the
    outputs d_in, d_out (contiguous fp32 [B, Lr]) are the caller's."""
    B, Hq, L, d = q.shape
    Lr = masked.shape[1]
    for t in (k_live, k_cache):
        if t.shape != k_live.shape or t.stride() != k_live.stride() or t.dtype != q.dtype:
            raise ValueError("k_live and k_cache need equal shape, strides and dtype")
    for t in (masked, drafted):
        if t.shape != (B, Lr) or t.dtype != torch.uint8 or not t.is_contiguous():
            raise ValueError("masked / drafted must be contiguous uint8 [B, Lr]")
    if lse.shape != (B, Hq, L) or lse.dtype != torch.float32 or not lse.is_contiguous():
        raise ValueError("lse must be contiguous fp32 [B, Hq, L]")
    for t in (d_in, d_out):
        if t.shape != (B, Lr) or t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError("d_in / d_out must be contiguous fp32 [B, Lr]")
    max_seeds = 0 if seed_idx is None else seed_idx.shape[-1]
    desc = StatsDesc(attn_desc(q, k_live, max_seeds, scale), int(r0), int(Lr))
    st = lib().cover_attn_stats_noalloc(_ptr(q), _ptr(k_live), _ptr(k_cache), _ptr(seed_idx),
                                        _ptr(n_seed), _ptr(lse), _ptr(masked), _ptr(drafted),
                                        _ptr(d_in), _ptr(d_out), ctypes.byref(desc),
                                        _stream(stream))
    if st != COVER_OK:
        raise CoverError(st, "cover_attn_stats_noalloc")
    return d_in, d_out


def attn_flops(B: int, Hq: int, L: int, d: int) -> int:
    """Algorithmic flops of one call: QK^T plus PV, 2 flops per multiply-add, non-causal."""
    return 4 * B * Hq * L * L * d


def default_scale(d: int) -> float:
    return 1.0 / math.sqrt(d)


class PreparedAttn:
    """A cover_attn_fwd call with its arguments marshalled once, for tight loops: calling it
    re-launches the kernel on the same tensors (their contents may change between calls)."""

    def __init__(self, q, k_live, v_live, k_cache, v_cache, seed_idx=None, n_seed=None, out=None,
                 lse=None, scale: float = 0.0, stream=None):
        self.out, self.lse = cover_attn_fwd(q, k_live, v_live, k_cache, v_cache, seed_idx, n_seed,
                                            out=out, lse=lse, scale=scale, stream=stream)
        self._keep = (q, k_live, v_live, k_cache, v_cache, seed_idx, n_seed, self.out, self.lse)
        max_seeds = 0 if seed_idx is None else seed_idx.shape[-1]
        self._desc = attn_desc(q, k_live, max_seeds, scale)
        self._args = (_ptr(q), _ptr(k_live), _ptr(v_live), _ptr(k_cache), _ptr(v_cache),
                      _ptr(seed_idx), _ptr(n_seed), _ptr(self.out), _ptr(self.lse),
                      ctypes.byref(self._desc), _stream(stream))
        self._fn = lib().cover_attn_fwd

    def __call__(self):
        st = self._fn(*self._args)
        if st != COVER_OK:
            raise CoverError(st, "cover_attn_fwd")


class PreparedRect:
    """A cover_attn_rect call with its arguments marshalled once (see PreparedAttn)."""

    def __init__(self, q, k_live, v_live, k_cache, v_cache, q_off: int, seed_idx=None,
                 n_seed=None, out=None, lse=None, scale: float = 0.0, n_split=None, workspace=None,
                 stream=None):
        B, Hq, Lq, d = q.shape
        L = k_live.shape[2]
        if n_split is None:
            n_split = rect_splits(B, Hq, Lq, L)
        need = rect_workspace(B, Hq, Lq, n_split)
        if need and workspace is None:
            workspace = torch.empty(need, device=q.device, dtype=torch.float32)
        self.out, self.lse = cover_attn_rect(q, k_live, v_live, k_cache, v_cache, q_off, seed_idx,
                                             n_seed, out=out, lse=lse, scale=scale, n_split=n_split,
                                             workspace=workspace, stream=stream)
        self.n_split = n_split
        ws = workspace if need else None
        self._keep = (q, k_live, v_live, k_cache, v_cache, seed_idx, n_seed, self.out, self.lse, ws)
        max_seeds = 0 if seed_idx is None else seed_idx.shape[-1]
        ad = attn_desc(q, k_live, max_seeds, scale)
        ad.L = L
        self._desc = RectDesc(ad, q_off, Lq, n_split)
        self._args = (_ptr(q), _ptr(k_live), _ptr(v_live), _ptr(k_cache), _ptr(v_cache),
                      _ptr(seed_idx), _ptr(n_seed), _ptr(self.out), _ptr(self.lse), _ptr(ws),
                      ctypes.byref(self._desc), _stream(stream))
        self._fn = lib().cover_attn_rect

    def __call__(self):
        st = self._fn(*self._args)
        if st != COVER_OK:
            raise CoverError(st, "cover_attn_rect")


class PreparedSelect:
    """A cover_select_seeds call with its arguments marshalled once (see PreparedAttn)."""

    def __init__(self, logp, d_in, d_out, flags, max_seeds: int, pos_offset: int = 0,
                 seed_idx=None, n_seed=None, score=None, want_score: bool = True, stream=None):
        self.seed_idx, self.n_seed, self.score = cover_select_seeds(
            logp, d_in, d_out, flags, max_seeds, pos_offset, seed_idx=seed_idx, n_seed=n_seed,
            score=score, want_score=want_score, stream=stream)
        self._keep = (logp, d_in, d_out, flags, self.seed_idx, self.n_seed, self.score)
        self._desc = SelectDesc(logp.shape[0], logp.shape[1], max_seeds, pos_offset)
        self._args = (_ptr(logp), _ptr(d_in), _ptr(d_out), _ptr(flags), _ptr(self.seed_idx),
                      _ptr(self.n_seed), _ptr(self.score), ctypes.byref(self._desc),
                      _stream(stream))
        self._fn = lib().cover_select_seeds

    def __call__(self):
        st = self._fn(*self._args)
        if st != COVER_OK:
            raise CoverError(st, "cover_select_seeds")
