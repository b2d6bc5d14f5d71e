"""Pins for the oracle's draft assembly (Section 3.6 batch verification:
drafts as EOS-padded rows).  Hand-derived fixtures, properties that follow
from the definition (idempotence, rank order, no duplicates, EOS after the
first EOS), and a brute-force comparison with a set-based formulation."""
import json
import os

import numpy as np
import pytest

import oracle

FIX = os.path.join(os.path.dirname(__file__), "golden", "draft_packing.json")


def test_golden_draft_packing():
    for c in json.load(open(FIX))["cases"]:
        d, n = oracle.pack_drafts(np.asarray(c["tokens"]), c["r"], c["length"], c["eos"])
        assert d.tolist() == c["drafts"], c["name"]
        assert n.tolist() == c["count"], c["name"]


def _random_tokens(seed, B=6, k=40, L=7, vocab=4, eos=0):
    rng = np.random.default_rng(seed)
    return rng.integers(0, vocab, (B, k, L)).astype(np.int32)


def test_properties():
    for seed in range(5):
        t = _random_tokens(seed)
        d, n = oracle.pack_drafts(t, r=12, length=5, eos=0)
        for b in range(t.shape[0]):
            rows = [tuple(x) for x in d[b, : n[b]]]
            assert len(set(rows)) == len(rows)                       # no duplicates
            assert all(x[0] != 0 for x in rows)                      # no empty draft
            for x in rows:                                           # EOS pads the tail
                if 0 in x:
                    assert all(v == 0 for v in x[x.index(0):])
            assert (d[b, n[b]:] == 0).all()                          # missing rows are EOS
            # rank order: each kept draft's first source rank increases
            firsts = []
            for x in rows:
                for rank in range(t.shape[1]):
                    y = list(t[b, rank, :5])
                    if 0 in y:
                        y = y[: y.index(0)] + [0] * (5 - y.index(0))
                    if tuple(y) == x:
                        firsts.append(rank)
                        break
            assert firsts == sorted(firsts)


def test_against_set_formulation():
    """Kept drafts = the distinct non-empty normalised drafts, ordered by their
    first rank, truncated to r."""
    for seed in range(5):
        t = _random_tokens(100 + seed, vocab=3)
        r, ln = 9, 4
        d, n = oracle.pack_drafts(t, r, ln, eos=0)
        for b in range(t.shape[0]):
            norm = []
            for rank in range(t.shape[1]):
                y = t[b, rank, :ln].tolist()
                if 0 in y:
                    y = y[: y.index(0)] + [0] * (ln - y.index(0))
                norm.append(tuple(y))
            first = {}
            for rank, y in enumerate(norm):
                if y[0] != 0 and y not in first:
                    first[y] = rank
            want = [list(y) for y, _ in sorted(first.items(), key=lambda kv: kv[1])][:r]
            assert d[b, : n[b]].tolist() == want


def test_idempotent():
    t = _random_tokens(7)
    d, n = oracle.pack_drafts(t, r=10, length=6)
    d2, n2 = oracle.pack_drafts(d, r=10, length=6)
    assert np.array_equal(d, d2) and np.array_equal(n, n2)


def test_argument_errors():
    with pytest.raises(ValueError):
        oracle.pack_drafts(np.zeros((1, 2, 3), np.int32), 1, 4)
    with pytest.raises(ValueError):
        oracle.pack_drafts(np.zeros((1, 2, 3), np.int32), 0, 2)
