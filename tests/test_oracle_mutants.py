"""The oracle's pins must catch plausible mistakes in it.

Each mutant below is one textual edit of ``oracle/cover_oracle.c`` (a dropped term, a
swapped operand, a wrong index or comparison).  The mutant is compiled on the CPU into a
scratch library and the compact pin set below -- library attention over views built from
the paper's definitions, the paper's closed-form route, and the hand-worked selection
examples plus exact brute force -- must fail for every one of them.
"""
import json
import math
import os
import subprocess
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

SRC = os.path.join(os.path.dirname(oracle.__file__), "cover_oracle.c")
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "select_examples.json")

MUTANTS = [
    ("override_source_swapped", "const double* src = is_seed[j] ? cache : live;",
     "const double* src = is_seed[j] ? live : cache;"),
    ("diag_key_not_restored", "memcpy(Kv + (size_t)i * d, k_live", "memcpy(Kv + (size_t)i * d, k_cache"),
    ("diag_value_not_restored", "memcpy(Vv + (size_t)i * d, v_live", "memcpy(Vv + (size_t)i * d, v_cache"),
    ("scale_dropped", "s[j] = scale * dot(qi, Kv", "s[j] = dot(qi, Kv"),
    ("normaliser_sign", "z += exp(s[j] - m);\n  for (int c = 0; c < d; ++c) o[c] = 0.0;",
     "z += exp(s[j] + m);\n  for (int c = 0; c < d; ++c) o[c] = 0.0;"),
    ("lse_without_max", "*lse = m + log(z);", "*lse = log(z);"),
    ("gqa_head_map", "int g = h / group;\n        const unsigned char* S",
     "int g = h % Hkv;\n        const unsigned char* S"),
    ("closed_form_alpha", "double alpha = exp(s[i] - lse_ovr);", "double alpha = exp(s[i]);"),
    ("closed_form_lse", "lse[row] = lse_ovr + log(r);", "lse[row] = lse_ovr;"),
    ("score_terms_swapped", "s[j] = (u * (1.0 + di)) / (1.0 + dv);", "s[j] = (u * (1.0 + dv)) / (1.0 + di);"),
    ("count_not_strict", "s[j] > mean) ++c;", "s[j] >= mean) ++c;"),
    ("budget_floor_sqrt", "while (r * r < c) ++r;", "while ((r + 1) * (r + 1) <= c) ++r;"),
    ("tie_break_reversed", "return ja < jb;", "return ja > jb;"),
    ("exclusion_ignored", "if ((flags[base + j] & 3u) != 1u || taken[j]) continue;",
     "if (!(flags[base + j] & 1u) || taken[j]) continue;"),
    ("pos_offset_dropped", "= j + pos_offset;", "= j;"),
    ("mean_over_eligible", "double mean = a[0] / (double)n;", "double mean = a[0] / (double)n_elig;"),
    ("capacity_ignored", "if (k > max_seeds) k = max_seeds;", ""),
]


def _build_mutant(tmp_path, name, find, repl):
    src = open(SRC).read()
    assert src.count(find) == 1, f"mutant {name}: anchor text not found exactly once"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(find, repl))
    lib = tmp_path / f"{name}.so"
    subprocess.run(["gcc", *oracle._CFLAGS, "-o", str(lib), str(path), "-lm"], check=True)
    return str(lib)


def _case(seed, B, Hq, Hkv, L, d, n):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, Hq, L, d))
    kv = [rng.standard_normal((B, Hkv, L, d)) for _ in range(4)]
    si = np.stack([np.sort(rng.choice(L, n, replace=False)) for _ in range(B)]).astype(np.int32)
    return (q, *kv, si, np.full(B, n, np.int32))


def _attn_pins_hold():
    for seed, dims in [(0, (2, 4, 2, 14, 8, 4)), (1, (1, 2, 2, 9, 4, 9))]:
        q, kl, vl, kc, vc, si, ns = _case(seed, *dims)
        B, Hq, L, d = q.shape
        grp = Hq // kl.shape[1]
        try:
            out, lse = oracle.attn(q, kl, vl, kc, vc, si, ns, mode="fast")
            out_l, _ = oracle.attn(q, kl, vl, kc, vc, si, ns, mode="literal")
            oc, lc = oracle.attn_closed_form(q, kl, vl, kc, vc, si, ns)
        except oracle.OracleError:
            return False
        if not np.array_equal(out, out_l):
            return False
        if not (np.allclose(oc, out, rtol=1e-9, atol=1e-11) and np.allclose(lc, lse, rtol=1e-11, atol=1e-11)):
            return False
        for b in range(B):
            mask = np.zeros(L, bool)
            mask[si[b, : ns[b]]] = True
            for h in range(Hq):
                g = h // grp
                Kp = np.where(mask[:, None], kc[b, g], kl[b, g])
                Vp = np.where(mask[:, None], vc[b, g], vl[b, g])
                for i in range(L):
                    Ki, Vi = Kp.copy(), Vp.copy()
                    if mask[i]:
                        Ki[i], Vi[i] = kl[b, g, i], vl[b, g, i]
                    t = lambda x: torch.from_numpy(np.ascontiguousarray(x))
                    ref = F.scaled_dot_product_attention(t(q[b, h, i])[None, None, None], t(Ki)[None, None],
                                                         t(Vi)[None, None], scale=1 / math.sqrt(d))[0, 0, 0].numpy()
                    ref_lse = torch.logsumexp(t(Ki) @ t(q[b, h, i]) / math.sqrt(d), 0).item()
                    if not (np.allclose(out[b, h, i], ref, rtol=1e-11, atol=1e-12)
                            and abs(lse[b, h, i] - ref_lse) < 1e-11):
                        return False
    return True


def _select_pins_hold():
    with open(GOLDEN) as f:
        g = json.load(f)
    f32 = lambda x: np.array([x], np.float32)
    for ex in g["examples"]:
        si, ns, score = oracle.select(f32(ex["logp"]), f32(ex["d_in"]), f32(ex["d_out"]),
                                      np.array([ex["flags"]], np.uint8), ex["max_seeds"], ex["pos_offset"])
        if si[0].tolist() != ex["seed_idx"] or score[0].tolist() != [float(v) for v in ex["score"]]:
            return False
    rng = np.random.default_rng(2)
    for _ in range(400):
        n = int(rng.integers(1, 11))
        logp = -rng.integers(0, 6, n).astype(np.float32)
        d_in = rng.choice([0.0, 0.5, 1.0, 3.0], n).astype(np.float32)
        d_out = rng.choice([0.0, 1.0, 3.0], n).astype(np.float32)
        flags = rng.choice([0, 1, 1, 1, 3], n).astype(np.uint8)
        ms = int(rng.integers(0, 5))
        si, ns, _ = oracle.select(logp[None], d_in[None], d_out[None], flags[None], ms)
        U = [j for j in range(n) if flags[j] & 1]
        s = {j: Fraction(-float(logp[j])) * (1 + Fraction(float(d_in[j]))) / (1 + Fraction(float(d_out[j])))
             for j in U}
        ref = []
        if U:
            mean = sum(s.values()) / len(U)
            c = sum(1 for j in U if s[j] > mean)
            k = math.isqrt(c) + (0 if math.isqrt(c) ** 2 == c else 1)
            E = [j for j in U if not flags[j] & 2]
            ref = sorted(sorted(E, key=lambda j: (-s[j], j))[: min(k, len(E), ms)])
        if si[0, : ns[0]].tolist() != ref:
            return False
    return True


def _with_lib(path, fn):
    """Run fn with the oracle's ctypes functions bound to the library at path."""
    saved, real_build = oracle._lib, oracle.build
    try:
        oracle._lib = None
        oracle.build = lambda force=False: path
        oracle._load()
        oracle.build = real_build
        return fn()
    finally:
        oracle._lib, oracle.build = saved, real_build


def test_unmutated_oracle_passes_compact_pins():
    assert _attn_pins_hold() and _select_pins_hold()


@pytest.mark.parametrize("name,find,repl", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, find, repl):
    lib = _build_mutant(tmp_path, name, find, repl)
    caught = not _with_lib(lib, lambda: _attn_pins_hold() and _select_pins_hold())
    assert caught, f"pins did not detect mutant {name}"
