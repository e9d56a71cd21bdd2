"""Host-side checks of the C ABI (no GPU needed): the library loads, exports every function
``include/cover.h`` declares, and rejects bad descriptors before enqueuing anything (the
rejected calls below pass no valid device memory, so reaching a launch would fail)."""
import ctypes
import os
import re

import pytest

from paper_2602_06161_amd import cover

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cover.h")

pytestmark = pytest.mark.skipif(not os.path.exists(cover.LIB), reason="libcover.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(cover_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(cover.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = cover.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings_and_version():
    assert cover.status_str(cover.COVER_OK) == "COVER_OK"
    assert cover.status_str(cover.COVER_ERR_INVALID) == "COVER_ERR_INVALID"
    assert cover.status_str(cover.COVER_ERR_UNSUPPORTED) == "COVER_ERR_UNSUPPORTED"
    assert cover.status_str(cover.COVER_ERR_HIP) == "COVER_ERR_HIP"
    assert cover.version() == 100


FAKE = 0x100000  # 16-byte aligned, never dereferenced: every case below fails validation first


def _attn(desc, q=FAKE, k=FAKE, out=FAKE, si=FAKE, ns=FAKE, lse=None):
    lib = cover.lib()
    p = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.cover_attn_fwd(p(q), p(k), p(k), p(k), p(k), p(si), p(ns), p(out), p(lse),
                              None if desc is None else ctypes.byref(desc), None)


def _good(**kw):
    d = dict(B=1, Hq=4, Hkv=2, L=64, d=128, max_seeds=4, dtype=cover.COVER_BF16, scale=0.0,
             q_sb=4 * 64 * 128, q_sh=64 * 128, q_sl=128, kv_sb=2 * 64 * 128, kv_sh=64 * 128, kv_sl=128)
    d.update(kw)
    return cover.AttnDesc(**d)


@pytest.mark.parametrize("kw,expect", [
    (dict(B=-1), cover.COVER_ERR_INVALID),
    (dict(Hq=0), cover.COVER_ERR_INVALID),
    (dict(Hkv=3), cover.COVER_ERR_INVALID),            # 4 % 3 != 0
    (dict(L=-5), cover.COVER_ERR_INVALID),
    (dict(max_seeds=-1), cover.COVER_ERR_INVALID),
    (dict(dtype=7), cover.COVER_ERR_INVALID),
    (dict(scale=-1.0), cover.COVER_ERR_INVALID),
    (dict(scale=float("nan")), cover.COVER_ERR_INVALID),
    (dict(d=96), cover.COVER_ERR_UNSUPPORTED),
    (dict(d=0), cover.COVER_ERR_INVALID),
    (dict(L=cover.COVER_MAX_L + 1), cover.COVER_ERR_UNSUPPORTED),
    (dict(q_sl=100), cover.COVER_ERR_INVALID),          # not a multiple of 8 bf16 elements
    (dict(kv_sl=64), cover.COVER_ERR_INVALID),          # rows would overlap
    (dict(q_sh=-8), cover.COVER_ERR_INVALID),
])
def test_attn_descriptor_errors(kw, expect):
    assert _attn(_good(**kw)) == expect


def test_attn_pointer_errors():
    assert _attn(None) == cover.COVER_ERR_INVALID
    assert _attn(_good(), q=None) == cover.COVER_ERR_INVALID
    assert _attn(_good(), q=FAKE + 8) == cover.COVER_ERR_INVALID     # misaligned
    assert _attn(_good(), out=None) == cover.COVER_ERR_INVALID
    assert _attn(_good(), si=None) == cover.COVER_ERR_INVALID        # max_seeds > 0
    assert _attn(_good(), ns=FAKE + 2) == cover.COVER_ERR_INVALID
    assert _attn(_good(), lse=FAKE + 2) == cover.COVER_ERR_INVALID


def test_attn_empty_problems_are_no_ops():
    # nothing to compute: success without touching (invalid) memory
    assert _attn(_good(B=0), q=None, k=None, out=None) == cover.COVER_OK
    assert _attn(_good(L=0), q=None, k=None, out=None) == cover.COVER_OK


def _sel(desc, lp=FAKE, fl=FAKE, si=FAKE, ns=FAKE, sc=None):
    lib = cover.lib()
    p = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.cover_select_seeds(p(lp), p(lp), p(lp), p(fl), p(si), p(ns), p(sc),
                                  None if desc is None else ctypes.byref(desc), None)


def test_select_errors():
    good = dict(B=1, Lr=256, max_seeds=8, pos_offset=768)
    assert _sel(None) == cover.COVER_ERR_INVALID
    assert _sel(cover.SelectDesc(**{**good, "B": -1})) == cover.COVER_ERR_INVALID
    assert _sel(cover.SelectDesc(**{**good, "Lr": -1})) == cover.COVER_ERR_INVALID
    assert _sel(cover.SelectDesc(**{**good, "max_seeds": -2})) == cover.COVER_ERR_INVALID
    assert _sel(cover.SelectDesc(**{**good, "Lr": cover.COVER_MAX_LR + 1})) == cover.COVER_ERR_UNSUPPORTED
    assert _sel(cover.SelectDesc(**good), ns=None) == cover.COVER_ERR_INVALID
    assert _sel(cover.SelectDesc(**good), si=None) == cover.COVER_ERR_INVALID
    assert _sel(cover.SelectDesc(**good), lp=None) == cover.COVER_ERR_INVALID
    assert _sel(cover.SelectDesc(**good), lp=FAKE + 1) == cover.COVER_ERR_INVALID
    assert _sel(cover.SelectDesc(**good), sc=FAKE + 4) == cover.COVER_ERR_INVALID
    assert _sel(cover.SelectDesc(**{**good, "pos_offset": 0x7fffff00})) == cover.COVER_ERR_INVALID
    assert _sel(cover.SelectDesc(**{**good, "B": 0}), lp=None, fl=None, si=None, ns=None) == cover.COVER_OK


def _tok(desc, logits=FAKE, tokens=FAKE, logp=FAKE):
    p = lambda x: None if x is None else ctypes.c_void_p(x)
    return cover.lib().cover_token_stats(p(logits), p(tokens), p(logp), None, None,
                                         None if desc is None else ctypes.byref(desc), None)


@pytest.mark.parametrize("kw,expect", [
    (dict(R=-1), cover.COVER_ERR_INVALID),
    (dict(V=0), cover.COVER_ERR_INVALID),
    (dict(row_stride=100), cover.COVER_ERR_INVALID),       # < V
    (dict(row_stride=1004), cover.COVER_ERR_INVALID),      # 2008 bytes: not a multiple of 16
    (dict(dtype=7), cover.COVER_ERR_INVALID),
])
def test_token_stats_rejects_bad_descriptors(kw, expect):
    d = dict(R=4, V=1000, dtype=cover.COVER_BF16, row_stride=1008)
    d.update(kw)
    assert _tok(cover.TokenDesc(**d)) == expect


def test_token_stats_rejects_bad_pointers():
    good = cover.TokenDesc(4, 1000, cover.COVER_BF16, 1008)
    assert _tok(None) == cover.COVER_ERR_INVALID
    assert _tok(good, logits=None) == cover.COVER_ERR_INVALID
    assert _tok(good, logits=FAKE + 8) == cover.COVER_ERR_INVALID   # not 16-byte aligned
    assert _tok(good, tokens=None) == cover.COVER_ERR_INVALID       # logp wanted, no tokens
    assert _tok(cover.TokenDesc(0, 1000, cover.COVER_BF16, 1008), logits=None) == cover.COVER_OK


def _stats(desc, ws=FAKE, lse=FAKE):
    p = lambda x: None if x is None else ctypes.c_void_p(x)
    return cover.lib().cover_attn_stats(p(FAKE), p(FAKE), p(FAKE), p(FAKE), p(FAKE), p(lse),
                                        p(FAKE), p(FAKE), p(FAKE), p(FAKE), p(ws),
                                        None if desc is None else ctypes.byref(desc), None)


@pytest.mark.parametrize("kw,r0,Lr,expect", [
    (dict(), -1, 8, cover.COVER_ERR_INVALID),
    (dict(), 60, 8, cover.COVER_ERR_INVALID),               # r0 + Lr > L
    (dict(), 0, -1, cover.COVER_ERR_INVALID),
    (dict(dtype=cover.COVER_F32), 0, 8, cover.COVER_ERR_UNSUPPORTED),
    (dict(d=96), 0, 8, cover.COVER_ERR_UNSUPPORTED),
    (dict(Hkv=3), 0, 8, cover.COVER_ERR_INVALID),
    (dict(), 0, 0, cover.COVER_OK),                         # empty region: no-op
    (dict(L=4096), 0, 2049, cover.COVER_ERR_UNSUPPORTED),   # region longer than the LDS rows
])
def test_attn_stats_rejects_bad_descriptors(kw, r0, Lr, expect):
    assert _stats(cover.StatsDesc(_good(**kw), r0, Lr)) == expect


def _stats_na(desc, lse=FAKE, d_in=FAKE):
    p = lambda x: None if x is None else ctypes.c_void_p(x)
    return cover.lib().cover_attn_stats_noalloc(p(FAKE), p(FAKE), p(FAKE), p(FAKE), p(FAKE),
                                                p(lse), p(FAKE), p(FAKE), p(d_in), p(FAKE),
                                                None if desc is None else ctypes.byref(desc), None)


@pytest.mark.parametrize("kw,r0,Lr,expect", [
    (dict(), -1, 8, cover.COVER_ERR_INVALID),
    (dict(), 60, 8, cover.COVER_ERR_INVALID),
    (dict(dtype=cover.COVER_F32), 0, 8, cover.COVER_ERR_UNSUPPORTED),
    (dict(Hkv=3), 0, 8, cover.COVER_ERR_INVALID),
    (dict(), 0, 0, cover.COVER_OK),
    (dict(L=2048, Hq=257, Hkv=257), 0, 2048, cover.COVER_ERR_UNSUPPORTED),  # beyond its array
    (dict(L=512, Hq=1025, Hkv=1025), 0, 512, cover.COVER_ERR_UNSUPPORTED),
])
def test_attn_stats_noalloc_rejects_before_any_gpu_call(kw, r0, Lr, expect):
    # every one of these returns before the library touches the GPU (there is none here)
    assert _stats_na(cover.StatsDesc(_good(**kw), r0, Lr)) == expect


def test_attn_stats_noalloc_rejects_missing_buffers():
    good = cover.StatsDesc(_good(), 0, 8)
    assert _stats_na(None) == cover.COVER_ERR_INVALID
    assert _stats_na(good, lse=None) == cover.COVER_ERR_INVALID
    assert _stats_na(good, d_in=None) == cover.COVER_ERR_INVALID


def test_attn_stats_workspace_sizes():
    ws = cover.lib().cover_attn_stats_workspace
    assert ws(1, 32, 256) == 32 * 9 * 256        # 8 key tiles, one per group
    assert ws(2, 4, 1100) == 8 * 19 * 1100       # 35 tiles in 18 groups
    assert ws(1, 256, 2048) == cover.COVER_STATS_SCRATCH_FLOATS
    assert ws(0, 4, 100) == 0 and ws(-1, 4, 100) == -1
    for B, Hq, Lr in [(1, 1, 1), (3, 7, 2048), (8, 32, 512), (1, 300, 33)]:
        assert ws(B, Hq, Lr) <= B * Hq * (1 + (Lr + 31) // 32) * Lr  # the header's bound


def test_attn_stats_rejects_missing_buffers():
    good = cover.StatsDesc(_good(), 0, 8)
    assert _stats(None) == cover.COVER_ERR_INVALID
    assert _stats(good, ws=None) == cover.COVER_ERR_INVALID
    assert _stats(good, lse=None) == cover.COVER_ERR_INVALID
    assert cover.attn_stats_workspace(1, 32, 256) == 32 * 9 * 256


def _upd(desc, tok=FAKE, si=FAKE, ns=FAKE, counts=None, last=None, ff=None):
    p = lambda x: None if x is None else ctypes.c_void_p(x)
    return cover.lib().cover_decode_update(p(tok), p(FAKE), p(FAKE), p(si), p(ns), p(FAKE), None,
                                           None, p(counts), p(last), p(ff),
                                           None if desc is None else ctypes.byref(desc), None)


def test_decode_update_rejects_bad_arguments():
    good = dict(B=1, Lr=256, max_seeds=16, pos_offset=768, mask_id=126463, draft_cap=15,
                remask_budget=2, tau=0.9)
    d = lambda **kw: cover.UpdateDesc(**{**good, **kw})
    assert _upd(None) == cover.COVER_ERR_INVALID
    assert _upd(d(B=-1)) == cover.COVER_ERR_INVALID
    assert _upd(d(Lr=-1)) == cover.COVER_ERR_INVALID
    assert _upd(d(max_seeds=-1)) == cover.COVER_ERR_INVALID
    assert _upd(d(draft_cap=-1)) == cover.COVER_ERR_INVALID
    assert _upd(d(tau=float("nan"))) == cover.COVER_ERR_INVALID
    assert _upd(d(min_draft=-1)) == cover.COVER_ERR_INVALID
    assert _upd(d(min_draft=16)) == cover.COVER_ERR_INVALID          # above draft_cap
    assert _upd(d(Lr=cover.COVER_MAX_LR + 1)) == cover.COVER_ERR_UNSUPPORTED
    assert _upd(d(), tok=None) == cover.COVER_ERR_INVALID
    assert _upd(d(), tok=FAKE + 2) == cover.COVER_ERR_INVALID
    assert _upd(d(), si=None) == cover.COVER_ERR_INVALID
    assert _upd(d(), ns=FAKE + 1) == cover.COVER_ERR_INVALID
    assert _upd(d(), counts=FAKE + 2) == cover.COVER_ERR_INVALID
    assert _upd(d(), ff=FAKE) == cover.COVER_ERR_INVALID              # flip-flops need last_unmask
    assert _upd(d(), last=FAKE + 2, ff=FAKE) == cover.COVER_ERR_INVALID
    assert _upd(d(B=0), tok=None, si=None, ns=None) == cover.COVER_OK


def _rect(desc, ws=FAKE):
    p = lambda x: None if x is None else ctypes.c_void_p(x)
    return cover.lib().cover_attn_rect(p(FAKE), p(FAKE), p(FAKE), p(FAKE), p(FAKE), p(FAKE),
                                       p(FAKE), p(FAKE), None, p(ws),
                                       None if desc is None else ctypes.byref(desc), None)


@pytest.mark.parametrize("kw,q_off,Lq,n_split,expect", [
    (dict(), -1, 8, 1, cover.COVER_ERR_INVALID),
    (dict(), 60, 8, 1, cover.COVER_ERR_INVALID),            # q_off + Lq > L
    (dict(), 0, -1, 1, cover.COVER_ERR_INVALID),
    (dict(), 0, 8, 0, cover.COVER_ERR_INVALID),             # n_split < 1
    (dict(), 0, 8, 257, cover.COVER_ERR_INVALID),
    (dict(d=64), 0, 8, 1, cover.COVER_ERR_UNSUPPORTED),
    (dict(dtype=cover.COVER_F32, q_sl=128, kv_sl=128), 0, 8, 1, cover.COVER_ERR_UNSUPPORTED),
    (dict(), 0, 0, 1, cover.COVER_OK),                      # empty block: no-op
])
def test_attn_rect_rejects_bad_descriptors(kw, q_off, Lq, n_split, expect):
    assert _rect(cover.RectDesc(_good(**kw), q_off, Lq, n_split)) == expect


def test_attn_rect_workspace_rules():
    # key splits across workgroups need the caller's workspace; the single launch needs none
    assert _rect(None) == cover.COVER_ERR_INVALID
    assert _rect(cover.RectDesc(_good(), 0, 8, 2), ws=None) == cover.COVER_ERR_INVALID
    assert _rect(cover.RectDesc(_good(), 0, 8, 2), ws=FAKE + 4) == cover.COVER_ERR_INVALID
    assert cover.rect_workspace(1, 32, 256, 4) == 32 * 4 * 256 * cover.COVER_RECT_RECORD
    assert cover.rect_workspace(1, 32, 256, 1) == 0
    # single launch: a missing workspace passes validation (the stride limit is what fails)
    big = _good(kv_sl=1 << 26, kv_sh=64 << 26, kv_sb=128 << 26)
    assert _rect(cover.RectDesc(big, 0, 8, 1), ws=None) == cover.COVER_ERR_UNSUPPORTED


def test_attn_rect_grid_limits():
    # at most 2^32 work-items per launch: 2^23 - 8 workgroups of 512 for the single launch
    huge = _good(B=1 << 20, Hq=8, Hkv=8)
    assert _rect(cover.RectDesc(huge, 0, 64, 1), ws=None) == cover.COVER_ERR_UNSUPPORTED
    assert _rect(cover.RectDesc(huge, 0, 64, 2)) == cover.COVER_ERR_UNSUPPORTED


def test_token_sample_rejects_bad_arguments():
    p = lambda x: None if x is None else ctypes.c_void_p(x)
    lib = cover.lib()
    good = cover.TokenDesc(4, 1000, cover.COVER_BF16, 1008)
    call = lambda d, T=1.0, logits=FAKE, tok=FAKE: lib.cover_token_sample(
        p(logits), T, 1, 0, p(tok), None, None if d is None else ctypes.byref(d), None)
    assert call(None) == cover.COVER_ERR_INVALID
    assert call(good, T=0.0) == cover.COVER_ERR_INVALID
    assert call(good, T=-1.0) == cover.COVER_ERR_INVALID
    assert call(good, T=float("inf")) == cover.COVER_ERR_INVALID
    assert call(good, T=float("nan")) == cover.COVER_ERR_INVALID
    assert call(good, tok=None) == cover.COVER_ERR_INVALID
    assert call(good, logits=FAKE + 8) == cover.COVER_ERR_INVALID
    assert call(cover.TokenDesc(4, 1000, cover.COVER_BF16, 1004)) == cover.COVER_ERR_INVALID
    assert call(cover.TokenDesc(0, 1000, cover.COVER_BF16, 1008), logits=None, tok=None) == cover.COVER_OK


def test_rect_split_choice():
    # the single launch up to L = 2048, and past it whenever its workgroups fill the GPU
    assert cover.rect_splits(1, 32, 256, 1024) == 1
    assert cover.rect_splits(1, 32, 32, 2048) == 1
    assert cover.rect_splits(1, 32, 256, 4200) == 1          # 256 workgroups of 32 rows
    # long sequences with few rows: key splits across workgroups (at least 128 keys each)
    n = cover.rect_splits(1, 4, 32, 8192)
    assert 2 <= n <= 256 and -(-8192 // n) >= 128
    assert cover.rect_splits(1, 1, 1, 4096) == 32            # 4096 / 128 keys per split
    assert cover.rect_workspace(1, 4, 32, n) > 0 and cover.rect_workspace(1, 4, 32, 1) == 0
