"""Pins of the oracle's decode-step update (Sec. 5.2 drafting and revision, Sec. 3 state
update, Sec. 5.3 exclusion): hand-worked examples, and properties that follow from the rules
checked on random rows (the draft set is the top-cap of the qualifying positions by brute
force, the seeds split into Keep / Replace / ReMask, U_t = (U_{t-1} + D) - R, counters and
flags).  Each planted mistake below must be caught by these pins."""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "decode_examples.json")


def _run(e, fn=oracle.decode_update):
    a = lambda k, dt: np.array([e[k]], dtype=dt)
    si = np.array([e["seed_idx"]], np.int32).reshape(1, -1) if e["seed_idx"] else np.zeros((1, 0), np.int32)
    kw = {"last_unmask": a("last_unmask", np.int32)} if "last_unmask" in e else {}
    return fn(a("tokens", np.int32), a("argmax", np.int32), a("conf", np.float32), si,
              np.array([e["n_seed"]], np.int32), a("remask_count", np.int32), e["mask_id"],
              e["tau"], e["cap"], e["remask_budget"], e["pos_offset"], **kw)


def _golden_ok(fn):
    for e in json.load(open(GOLDEN))["examples"]:
        r = _run(e, fn)
        tok, cnt, flags, drafted, counts = r[:5]
        if "last_unmask" in e and not (r[5][0].tolist() == e["out_last_unmask"]
                                       and int(r[6][0]) == e["flipflops"]):
            return False
        if not (tok[0].tolist() == e["out_tokens"] and cnt[0].tolist() == e["out_remask_count"]
                and flags[0].tolist() == e["flags"] and drafted[0].tolist() == e["drafted"]
                and counts[0].tolist() == e["counts"]):
            return False
    return True


def test_hand_worked_examples():
    assert _golden_ok(oracle.decode_update)


def random_rows(seed, B=6, Lr=64, vocab=20, mask_id=19):
    rng = np.random.default_rng(seed)
    tok = rng.integers(0, vocab - 1, (B, Lr)).astype(np.int32)
    tok[rng.random((B, Lr)) < 0.5] = mask_id
    am = rng.integers(0, vocab - 1, (B, Lr)).astype(np.int32)
    keep = rng.random((B, Lr)) < 0.3
    am = np.where(keep & (tok != mask_id), tok, am)
    conf = rng.choice(np.float32([0.3, 0.6, 0.8, 0.85, 0.9, 0.95, 0.99]), (B, Lr)).astype(np.float32)
    ms = 8
    si = np.full((B, ms), -1, np.int32)
    ns = np.zeros(B, np.int32)
    for b in range(B):
        um = np.nonzero(tok[b] != mask_id)[0]
        k = min(ms, um.size, int(rng.integers(0, ms + 1)))
        si[b, :k] = 100 + rng.choice(um, k, replace=False)
        ns[b] = k
    cnt = rng.integers(0, 4, (B, Lr)).astype(np.int32)
    return tok, am, conf, si, ns, cnt, mask_id


def _properties(fn, seed, cap=5, tau=0.85, budget=3):
    tok, am, conf, si, ns, cnt, mask_id = random_rows(seed)
    out_tok, out_cnt, flags, drafted, counts = fn(tok, am, conf, si, ns, cnt, mask_id, tau, cap,
                                                  budget, 100)
    t32 = np.float32(tau)
    for b in range(tok.shape[0]):
        masked = tok[b] == mask_id
        seeds = {int(x) - 100 for x in si[b, :ns[b]]}
        qual = [i for i in np.nonzero(masked & (conf[b] > t32))[0]]
        D = set(np.nonzero(drafted[b])[0].tolist())
        # brute force: D is the lexicographically best set of size min(cap, |qual|) by (conf, -pos)
        ranked = sorted(qual, key=lambda i: (-conf[b, i], i))
        if D != set(ranked[:cap]):
            return False
        kept = [i for i in seeds if am[b, i] == tok[b, i]]
        repl = [i for i in seeds if am[b, i] != tok[b, i] and conf[b, i] > t32]
        R = [i for i in seeds if i not in kept and i not in repl]
        exp = tok[b].copy()
        for i in D | set(repl):
            exp[i] = am[b, i]
        for i in R:
            exp[i] = mask_id
        if not np.array_equal(out_tok[b], exp):
            return False
        U0 = set(np.nonzero(~masked)[0])
        U1 = set(np.nonzero(out_tok[b] != mask_id)[0])
        if U1 != (U0 | D) - set(R):
            return False
        dc = out_cnt[b] - cnt[b]
        if set(np.nonzero(dc)[0]) != set(R) or np.any(dc[list(R)] != 1):
            return False
        excl = np.array([(i in seeds) or out_cnt[b, i] >= budget for i in range(tok.shape[1])])
        if not np.array_equal(flags[b], ((out_tok[b] != mask_id) * 1 + excl * 2).astype(np.uint8)):
            return False
        if counts[b].tolist() != [len(D), len(kept), len(repl), len(R), int(np.sum(out_tok[b] == mask_id))]:
            return False
    return True


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("cap", [0, 1, 5, 64])
def test_rule_properties_on_random_rows(seed, cap):
    assert _properties(oracle.decode_update, seed, cap=cap)


def _mutant(old, new):
    import inspect
    src = inspect.getsource(oracle.decode_update)
    assert old in src, old
    ns = {"np": np}
    exec(src.replace(old, new), ns)
    return ns["decode_update"]


def _history_ok(fn, seed, steps=40, Lr=48):
    """Chained steps on one state with a small vocabulary (tokens recur): the flip-flops the
    update reports add up to F counted from the definition over the recorded unmask history,
    and every unmask event is a drafted position (sum of |D| = total unmask events)."""
    rng = np.random.default_rng(seed)
    mask_id = 5
    tok = np.full((1, Lr), mask_id, np.int32)
    cnt = np.zeros((1, Lr), np.int32)
    last = np.full((1, Lr), -1, np.int32)
    si, ns = np.full((1, 8), -1, np.int32), np.zeros(1, np.int32)
    hist = [[] for _ in range(Lr)]
    F = n_d = 0
    for _ in range(steps):
        am = rng.integers(0, mask_id, (1, Lr)).astype(np.int32)
        conf = rng.choice(np.float32([0.5, 0.92, 0.97]), (1, Lr))
        before = tok.copy()
        tok, cnt, flags, drafted, counts, last, ff = fn(tok, am, conf, si, ns, cnt, mask_id, 0.9,
                                                        6, 100, 0, last_unmask=last)
        for i in range(Lr):
            if before[0, i] == mask_id and tok[0, i] != mask_id:
                hist[i].append(int(tok[0, i]))
        F += int(ff[0])
        n_d += int(counts[0, 0])
        ok = np.nonzero(flags[0] & 1)[0]
        k = min(8, ok.size)
        si[0] = -1
        si[0, :k] = rng.choice(ok, k, replace=False) if k else []
        ns[0] = k
    F_def = sum(sum(1 for a, b in zip(h, h[1:]) if a == b) for h in hist)
    return F == F_def and n_d == sum(len(h) for h in hist) and F > 0


def test_min_draft_forces_progress_only_when_needed():
    # nothing above tau: the two most confident masked positions are drafted (ties by position)
    tok = np.array([[9, 9, 9, 1, 9]], np.int32)
    am = np.array([[4, 5, 6, 1, 7]], np.int32)
    conf = np.array([[0.3, 0.6, 0.6, 0.99, 0.1]], np.float32)
    none = (np.zeros((1, 0), np.int32), np.zeros(1, np.int32), np.zeros((1, 5), np.int32))
    r = oracle.decode_update(tok, am, conf, none[0], none[1], none[2], 9, 0.9, 15, 5, 0,
                             min_draft=2)
    assert r[3][0].tolist() == [0, 1, 1, 0, 0] and r[0][0].tolist() == [9, 5, 6, 1, 9]
    # enough above tau: min_draft changes nothing; 0 keeps the paper's rule
    conf2 = np.array([[0.95, 0.6, 0.6, 0.99, 0.97]], np.float32)
    a = oracle.decode_update(tok, am, conf2, *none, 9, 0.9, 15, 5, 0, min_draft=2)
    b = oracle.decode_update(tok, am, conf2, *none, 9, 0.9, 15, 5, 0)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    c = oracle.decode_update(tok, am, conf, *none, 9, 0.9, 15, 5, 0)
    assert not c[3].any()
    # fewer masked positions than min_draft: all of them
    d = oracle.decode_update(tok, am, conf, *none, 9, 0.9, 15, 5, 0, min_draft=10)
    assert d[3][0].tolist() == [1, 1, 1, 0, 1]


@pytest.mark.parametrize("seed", range(3))
def test_flip_flops_match_the_definition_over_a_history(seed):
    assert _history_ok(oracle.decode_update, seed)


MUTANTS = [
    ("draft_threshold_not_strict", "c[b, i] > t32]", "c[b, i] >= t32]"),
    ("draft_ties_larger_first", "(-float(c[b, i]), i)", "(-float(c[b, i]), -i)"),
    ("cap_ignored", "D = cand[:max(0, int(cap))]", "D = cand"),
    ("replace_not_strict", "elif c[b, i] > t32:", "elif c[b, i] >= t32:"),
    ("keep_compares_wrong", "if am[b, i] == tok[b, i]:", "if am[b, i] != tok[b, i]:"),
    ("counter_not_kept", "cnt[b, i] += 1", "cnt[b, i] += 0"),
    ("budget_off_by_one", "cnt[b, i] >= remask_budget", "cnt[b, i] > remask_budget"),
    ("seed_not_excluded", "excl = i in seeds or", "excl ="),
    ("offset_ignored", "i = int(si[b, t]) - pos_offset", "i = int(si[b, t])"),
    ("flip_flop_compares_wrong", "if last[b, i] == am[b, i]:", "if last[b, i] != am[b, i]:"),
    ("flip_flop_not_recorded", "last[b, i] = am[b, i]", "pass"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistakes(name, old, new):
    fn = _mutant(old, new)
    caught = not _golden_ok(fn) or not all(_properties(fn, s, cap=cap) for s in range(5)
                                           for cap in (5, 64)) or \
        not all(_history_ok(fn, s) for s in range(3))
    assert caught, name
