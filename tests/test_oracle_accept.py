"""Pins for the acceptance oracle: brute-force prefix matching and the pruning invariant."""
import numpy as np
import pytest

from oracle import accept as oacc
from oracle import select as osel


def _brute_accept(draft_row, g_rows, n):
    """Largest m in [0, n] such that every j in 1..m matches (checked for every m)."""
    best = 0
    for m in range(n + 1):
        if all(draft_row[j] == g_rows[j - 1] for j in range(1, m + 1)):
            best = m
    return best


@pytest.mark.parametrize("seed", range(10))
def test_bruteforce(seed):
    rng = np.random.default_rng(seed)
    B, D, V = int(rng.integers(1, 20)), 15, 7        # tiny vocab -> frequent accidental matches
    draft = rng.integers(0, V, size=(B, D + 1)).astype(np.int32)
    g_full = rng.integers(0, V, size=(B, D + 1)).astype(np.int32)
    hit = rng.random((B, D)) < 0.8
    g_full[:, :D] = np.where(hit, draft[:, 1:], g_full[:, :D])
    keep = rng.integers(1, D + 2, size=B).astype(np.int32)
    cu = np.concatenate([[0], np.cumsum(keep)]).astype(np.int32)
    argmax = np.concatenate([g_full[i, :keep[i]] for i in range(B)]).astype(np.int32)
    out = oacc.accept(draft, keep, cu, argmax)
    for i in range(B):
        a = _brute_accept(draft[i], g_full[i], int(keep[i]) - 1)
        assert out["accept_len"][i] == a
        assert out["next_tok"][i] == g_full[i, a]
    assert int(out["total"][0]) == int((out["accept_len"] + 1).sum())


@pytest.mark.parametrize("seed", range(10))
def test_pruning_invariant(seed):
    """a_i(pruned) = min(a_i(full), n_i) when the target outputs do not depend on pruning."""
    rng = np.random.default_rng(100 + seed)
    B, D, V = 12, 15, 50
    draft = rng.integers(0, V, size=(B, D + 1)).astype(np.int32)
    g_full = rng.integers(0, V, size=(B, D + 1)).astype(np.int32)
    hit = rng.random((B, D)) < 0.85
    g_full[:, :D] = np.where(hit, draft[:, 1:], g_full[:, :D])
    full = np.full(B, D + 1, np.int32)
    cuf = np.concatenate([[0], np.cumsum(full)]).astype(np.int32)
    a_full = oacc.accept(draft, full, cuf, g_full.ravel())["accept_len"]
    conf = rng.random((B, D)).astype(np.float32)
    for K in [B, 2 * B + 3, 5 * B, B * (D + 1)]:
        sel = osel.select(conf, draft, np.zeros(B, np.int32), [K], [1.0])
        kl, cu = sel["keep_len"], sel["cu"]
        argmax = np.concatenate([g_full[i, :kl[i]] for i in range(B)]).astype(np.int32)
        out = oacc.accept(draft, kl, cu, argmax)
        assert (out["accept_len"] == np.minimum(a_full, kl - 1)).all()
        assert (out["next_tok"] == g_full[np.arange(B), out["accept_len"]]).all()


def test_edge_cases():
    draft = np.array([[5, 1, 2, 3]], np.int32)
    # keep only the bonus: nothing to accept, next token is the bonus row's argmax
    out = oacc.accept(draft, np.array([1], np.int32), np.array([0, 1], np.int32), np.array([9], np.int32))
    assert out["accept_len"].tolist() == [0] and out["next_tok"].tolist() == [9] and out["total"][0] == 1
    # full match: all drafts accepted, next token from the last row
    out = oacc.accept(draft, np.array([4], np.int32), np.array([0, 4], np.int32),
                      np.array([1, 2, 3, 7], np.int32))
    assert out["accept_len"].tolist() == [3] and out["next_tok"].tolist() == [7] and out["total"][0] == 4
    # first mismatch stops acceptance even if later drafts match
    out = oacc.accept(draft, np.array([4], np.int32), np.array([0, 4], np.int32),
                      np.array([1, 0, 3, 7], np.int32))
    assert out["accept_len"].tolist() == [1] and out["next_tok"].tolist() == [0]
