"""Pins of the oracle's temperature sampling (Gumbel-max over Philox4x32-10 uniforms): the
drawn tokens follow softmax(x / T) (chi-square over 20000 rows of the same logits, several
temperatures), a vanishing temperature gives the argmax, the uniforms are uniform on (0, 1)
and exact in fp32, draws depend on every counter component, and planted mistakes (x * T for
x / T, noise dropped, noise sign flipped, a counter component ignored) are caught.  The
generator itself is pinned by the three published Random123 known-answer vectors
(tests/golden/philox4x32_10_kat.json), which one-line mistakes in its multipliers, key
schedule, round count or output order all fail."""
import inspect
import json
import os

import numpy as np
import pytest

import oracle

X = np.array([1.0, 0.5, -0.3, 2.0, 0.0, 1.2, -1.0])


def _freq_ok(fn, T, seed=7):
    R = 20000
    tok, p, _ = fn(np.tile(X, (R, 1)), T, seed, 3)
    q = np.exp(X / T - np.max(X / T))
    q /= q.sum()
    obs = np.bincount(tok, minlength=X.size)
    exp = R * q
    keep = exp > 5
    chi2 = (((obs - exp) ** 2) / exp)[keep].sum()
    return chi2 < 35 and np.allclose(p, q[tok])  # 6 dof: p(chi2 > 35) ~ 4e-6


@pytest.mark.parametrize("T", [0.3, 1.0, 2.5])
def test_draws_follow_softmax_at_temperature(T):
    assert _freq_ok(oracle.token_sample, T)


def test_vanishing_temperature_is_argmax():
    rng = np.random.default_rng(0)
    x = rng.normal(size=(50, 300)) * 3
    tok, p, _ = oracle.token_sample(x, 1e-4, 11, 0)
    assert np.array_equal(tok, np.argmax(x, axis=1)) and np.allclose(p, 1.0)


def _uniform_ok(su):
    u = su(64, 4096, 123, 5)
    if not (0.0 < u.min() and u.max() < 1.0):
        return False
    if not np.array_equal(u.astype(np.float32).astype(np.float64), u):  # exact in fp32
        return False
    counts = np.histogram(u, bins=32, range=(0, 1))[0]
    e = u.size / 32
    if ((counts - e) ** 2 / e).sum() >= 70:  # 31 dof
        return False
    # every counter component and the key matter
    a = su(2, 16, 123, 5)
    return (not np.array_equal(a[0], a[1])
            and not np.array_equal(a, su(2, 16, 124, 5))
            and not np.array_equal(a, su(2, 16, 123, 6))
            and not np.array_equal(a, su(2, 16, 123 + (1 << 32), 5))
            and len(set(np.round(a[0], 12))) == 16)


def test_uniforms():
    assert _uniform_ok(oracle.sample_uniforms)


def _mutant(src_fn, old, new):
    src = inspect.getsource(src_fn)
    assert old in src
    ns = dict(vars(oracle))
    exec(src.replace(old, new), ns)
    return ns[src_fn.__name__]


@pytest.mark.parametrize("old,new", [
    ("y = x / temperature - np.log(-np.log(u))", "y = x * temperature - np.log(-np.log(u))"),
    ("y = x / temperature - np.log(-np.log(u))", "y = x / temperature"),
    ("y = x / temperature - np.log(-np.log(u))", "y = x / temperature + np.log(-np.log(u))"),
])
def test_planted_sampling_mistakes_are_caught(old, new):
    fn = _mutant(oracle.token_sample, old, new)
    assert not (_freq_ok(fn, 0.3) and _freq_ok(fn, 1.0))


@pytest.mark.parametrize("old,new", [
    ("r, np.uint64(step)", "r * np.uint64(0), np.uint64(step)"),          # row ignored
    ("r, np.uint64(step)", "r, np.uint64(0)"),                            # step ignored
    ("np.uint64(seed & 0xFFFFFFFF)", "np.uint64(0)"),                     # key ignored
    ("np.uint64(_PHILOX_W[1])", "np.uint64(0)"),                          # key schedule wrong
])
def test_planted_generator_mistakes_are_caught(old, new):
    if "PHILOX_W" in old:
        ph = _mutant(oracle.philox4x32_10, old, new)
        src = inspect.getsource(oracle.sample_uniforms)
        ns = dict(vars(oracle))
        ns["philox4x32_10"] = ph
        exec(src, ns)
        su = ns["sample_uniforms"]
        # a wrong key schedule still looks random: it is the GPU parity (an independent
        # implementation of the same definition) that catches it; here it must at least differ
        assert not np.array_equal(su(2, 16, 123, 5), oracle.sample_uniforms(2, 16, 123, 5))
        return
    assert not _uniform_ok(_mutant(oracle.sample_uniforms, old, new))


# ---- known answers of the generator itself ----------------------------------------------
_KAT = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.json")))


def _kat_ok(fn):
    for v in _KAT["vectors"]:
        c = [int(x, 16) for x in v["counter"]]
        k = [int(x, 16) for x in v["key"]]
        got = [int(w) for w in fn(*c, *k)]
        if got != [int(x, 16) for x in v["out"]]:
            return False
    return True


def test_philox_known_answers():
    # the published Random123 vectors pin the multipliers, the Weyl key schedule, the round
    # count and the output word order
    assert _kat_ok(oracle.philox4x32_10)


@pytest.mark.parametrize("old,new", [
    ("_PHILOX_M[0]) * c[0]", "_PHILOX_M[1]) * c[0]"),                     # multipliers swapped
    ("p1 = np.uint64(_PHILOX_M[1])", "p1 = np.uint64(_PHILOX_M[0])"),
    ("c = [hi1 ^ c[1] ^ k0, lo1, hi0 ^ c[3] ^ k1, lo0]",
     "c = [hi0 ^ c[1] ^ k0, lo0, hi1 ^ c[3] ^ k1, lo1]"),                  # products exchanged
    ("return c", "return [c[1], c[0], c[2], c[3]]"),                      # output words swapped
    ("return c", "return c[::-1]"),                                       # output order reversed
    ("        if r:\n", "        if r > 1:\n"),                           # a key bump missing
    ("k0 = (k0 + np.uint64(_PHILOX_W[0])) & _U32", "k0 = k0"),           # k0 never advanced
    ("k1 = (k1 + np.uint64(_PHILOX_W[1])) & _U32",
     "k1 = (k1 + np.uint64(_PHILOX_W[0])) & _U32"),                       # wrong Weyl constant
    ("for r in range(10):", "for r in range(9):"),                        # a round missing
    ("hi1 ^ c[1] ^ k0", "hi1 ^ c[1] ^ k1"),                               # keys exchanged
])
def test_planted_philox_mistakes_fail_the_known_answers(old, new):
    assert not _kat_ok(_mutant(oracle.philox4x32_10, old, new))
