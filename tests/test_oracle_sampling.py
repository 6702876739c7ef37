"""Pins for the temperature-sampling oracle (oracle/sampling.py).

- Philox4x32-10 against the published known-answer vectors (tests/golden).
- The noise transform against the Gumbel law: Kolmogorov-Smirnov distance of
  200k draws to F(g) = exp(-exp(-g)).
- Gumbel-max against its closed form: the sampled-token frequencies over many
  (request, position) counters match softmax(logits / T) for T = 1 and 0.5.
- Limits: as T -> 0 the sample is the greedy argmax; for T -> infinity it is
  the argmax of the noise alone, and every column is equally likely.
- Counter semantics: a (request, position) pair always gets the same noise,
  different pairs and different seeds get different noise.
"""
import json
import os

import numpy as np
import pytest

from oracle import sampling as osm

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.json")


def test_philox_known_answers():
    kat = json.load(open(GOLDEN))
    assert len(kat["vectors"]) == 3
    for v in kat["vectors"]:
        ctr = [np.uint32(int(h, 16)) for h in v["ctr"]]
        key = [int(h, 16) for h in v["key"]]
        out = osm.philox4x32_10(ctr, key)
        assert [f"{int(o):08x}" for o in out] == v["out"]


def test_gumbel_law():
    n_rows, V = 400, 500
    g = osm.gumbel(np.zeros(n_rows, np.int64), np.arange(n_rows), V, seed=7).ravel()
    g.sort()
    F = np.exp(-np.exp(-g))
    emp = np.arange(1, g.size + 1) / g.size
    ks = np.max(np.abs(F - emp))
    assert ks < 1.63 / np.sqrt(g.size)          # 99 % critical value
    assert abs(g.mean() - 0.5772156649) < 0.01   # Euler-Mascheroni constant
    u = osm.uniforms(np.zeros(4, np.int64), np.arange(4), 300, seed=1)
    assert u.min() > 0.0 and u.max() < 1.0


@pytest.mark.parametrize("T", [1.0, 0.5])
def test_gumbel_max_matches_softmax(T):
    logits = np.array([0.0, 1.0, 2.0, -1.0, 0.5])
    n = 40000
    L = np.broadcast_to(logits, (n, logits.size))
    tok = osm.sample_tokens(L, np.arange(n) % 7, np.arange(n) // 7, T, seed=1234)["token"]
    freq = np.bincount(tok, minlength=logits.size) / n
    p = np.exp(logits / T - np.max(logits / T))
    p /= p.sum()
    sigma = np.sqrt(p * (1 - p) / n)
    assert np.all(np.abs(freq - p) < 5 * sigma + 1e-4), (freq, p)


def test_limits():
    rng = np.random.default_rng(0)
    logits = rng.normal(size=(64, 300))
    greedy = np.argmax(logits, axis=1)
    cold = osm.sample_tokens(logits, np.arange(64), np.zeros(64, np.int64), 1e-9, seed=3)["token"]
    assert np.array_equal(cold, greedy)
    hot = osm.sample_tokens(logits, np.arange(64), np.zeros(64, np.int64), 1e30, seed=3)["token"]
    g = osm.gumbel(np.arange(64), np.zeros(64, np.int64), 300, seed=3)
    assert np.array_equal(hot, np.argmax(g, axis=1))
    n = 30000
    uni = osm.sample_tokens(np.zeros((n, 6)), np.arange(n), np.arange(n) % 5, 1.0, seed=9)["token"]
    freq = np.bincount(uni, minlength=6) / n
    assert np.all(np.abs(freq - 1 / 6) < 5 * np.sqrt(1 / 6 * 5 / 6 / n))


def test_counter_semantics():
    a = osm.uniforms([3, 3, 4], [10, 11, 10], 260, seed=5)
    b = osm.uniforms([4, 3], [10, 10], 260, seed=5)
    assert np.array_equal(a[0], b[1]) and np.array_equal(a[2], b[0])   # same pair, same noise
    assert not np.any(a[0] == a[1]) and not np.any(a[0] == a[2])        # other pairs differ
    c = osm.uniforms([3], [10], 260, seed=6)
    assert not np.any(c[0] == a[0])                                      # other seed differs
    assert np.unique(a[0]).size == 260                                   # columns differ


def test_rejects_bad_temperature():
    with pytest.raises(ValueError):
        osm.sample_tokens(np.zeros((1, 3)), [0], [0], 0.0, seed=0)
