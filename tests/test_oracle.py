"""Pins for the CPU oracle (no GPU).

The oracle implements DReSD Section 3.5, Eq. 3 (argmax of cosine similarity
over unit-norm keys, Section 3.4, Eq. 2) as exact top-k.  None of these checks
re-types its arithmetic: they use hand-derived closed forms (tests/golden),
exact rational brute force, format definitions checked against numpy/torch
conversions, invariants, planted duplicates with the Eq. 4 self-retrieval MRR
in closed form, and structural continuations.  ``test_planted_mistakes``
shows each class of plausible mistake fails at least one of them.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from datagen import WORKLOADS, generate, to_numpy_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "closed_forms.json")
GOLDEN_FILTERED = os.path.join(os.path.dirname(__file__), "golden", "filtered_closed_forms.json")


def _identity_keys(n, dtype):
    e = np.eye(n, dtype=np.float32)
    if dtype == "f32":
        return e
    if dtype == "f16":
        return e.astype(np.float16).view(np.uint16)
    return torch.from_numpy(e).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


# --- pins -------------------------------------------------------------------

def pin_golden_closed_forms():
    cases = json.load(open(GOLDEN))["cases"]
    for c in cases:
        for dt in ("f32", "f16", "bf16"):
            keys = _identity_keys(c["N"], dt)
            q = np.zeros((1, c["d"]), np.float32)
            for j, v in c["query"].items():
                q[0, int(j)] = np.float32(v)
            idx, score, _, _ = oracle.topk(keys, dt, q, c["k"])
            assert idx[0].tolist() == c["idx"], (c["name"], dt, idx[0].tolist())
            assert np.array_equal(score[0], np.asarray(c["score"], np.float32)), (c["name"], dt)


def _exact_fp32_score(q_row, e_row):
    s = sum((Fraction(float(a)) * Fraction(float(b)) for a, b in zip(q_row, e_row)), Fraction(0))
    return np.float32(float(s))


def pin_exact_bruteforce():
    """Exact rational arithmetic on tiny inputs, ranked by (-score, index)."""
    rng = np.random.default_rng(12345)
    for dt in ("f32", "f16"):
        N, d, B, k = 37, 7, 3, 6
        x = rng.standard_normal((N, d))
        x /= np.linalg.norm(x, axis=1, keepdims=True)
        if dt == "f32":
            keys = x.astype(np.float32)
            vals = keys.astype(np.float64)
        else:
            h = x.astype(np.float16)
            keys = h.view(np.uint16)
            vals = h.astype(np.float64)
        keys = np.ascontiguousarray(keys)
        # plant an exact duplicate (row 20 = row 4) so the tie rule matters
        keys[20] = keys[4]
        vals[20] = vals[4]
        q = rng.standard_normal((B, d)).astype(np.float32)
        q[0] = vals[4].astype(np.float32)
        idx, score, _, nxt = oracle.topk(keys, dt, q, k)
        for b in range(B):
            s = [_exact_fp32_score(q[b], vals[i]) for i in range(N)]
            order = sorted(range(N), key=lambda i: (-float(s[i]), i))
            assert idx[b].tolist() == order[:k], (dt, b)
            assert [float(v) for v in score[b]] == [float(s[i]) for i in order[:k]]
            assert float(nxt[b]) == float(s[order[k]])
        r0 = idx[0].tolist()
        assert r0.index(4) < r0.index(20)


def pin_decode_f16_all_patterns():
    bits = np.arange(65536, dtype=np.uint16)
    vals = bits.view(np.float16)
    ok = np.isfinite(vals)
    keys = bits[ok].reshape(-1, 1)
    got = oracle.score_rows(keys, "f16", np.ones(1, np.float32), np.arange(keys.shape[0]))
    want = vals[ok].astype(np.float32)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32)) or np.array_equal(got, want)


def pin_decode_bf16_all_patterns():
    bits = np.arange(65536, dtype=np.uint16)
    t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float32).numpy()
    ok = np.isfinite(t)
    keys = bits[ok].reshape(-1, 1)
    got = oracle.score_rows(keys, "bf16", np.ones(1, np.float32), np.arange(keys.shape[0]))
    assert np.array_equal(got, t[ok])


def pin_decode_keys_all_patterns():
    """The fp64 decoder that feeds the k-means, partitioned and pipeline
    oracles, over every 16-bit pattern: f16 against numpy's binary16 (as bits
    and as float16 values), bf16 against torch's bfloat16, and both against
    the C decoder's scores of the same rows for a unit query."""
    bits = np.arange(65536, dtype=np.uint16)
    f16 = bits.view(np.float16).astype(np.float64)
    bf16 = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    for dt, want in (("f16", f16), ("bf16", bf16)):
        got = oracle.decode_keys(bits.reshape(-1, 1), dt).reshape(-1)
        assert got.dtype == np.float64
        assert np.array_equal(np.isnan(got), np.isnan(want)), dt
        ok = ~np.isnan(want)
        assert np.array_equal(got[ok], want[ok]), dt
        assert np.array_equal(np.signbit(got[ok]), np.signbit(want[ok])), dt  # -0.0 kept
        fin = np.isfinite(want)
        c = oracle.score_rows(bits[fin].reshape(-1, 1), dt, np.ones(1, np.float32),
                              np.arange(int(fin.sum())))
        assert np.array_equal(c.astype(np.float64), got[fin]), dt
    vals = bits.view(np.float16)
    assert np.array_equal(oracle.decode_keys(vals.reshape(-1, 1), "f16").reshape(-1)[~np.isnan(f16)],
                          f16[~np.isnan(f16)])
    x = np.random.default_rng(5).standard_normal((7, 3)).astype(np.float32)
    assert np.array_equal(oracle.decode_keys(x, "f32"), x.astype(np.float64))


def _c1_like(N=4096):
    w = WORKLOADS["flat16k_d256_f32"].scaled(N)
    return w, generate(w, "cpu")


def pin_invariants_and_self_match():
    w, g = _c1_like()
    keys, dt = to_numpy_bits(g["keys"])
    q = g["queries"].numpy()
    idx, score, _, nxt = oracle.topk(keys, dt, q, 32)
    assert np.all(np.diff(score.astype(np.float64), axis=1) <= 0)
    assert np.all(np.abs(score) <= 1 + 1e-6)
    assert np.all(nxt <= score[:, -1])
    # every row scored against itself (fp32 keys): within 1e-6 of 1
    rows = np.arange(w.N)
    s_self = np.array([oracle.score_rows(keys, dt, keys[i], [i])[0] for i in range(0, w.N, 7)])
    assert np.all(np.abs(s_self.astype(np.float64) - 1.0) <= 1e-6)
    # a query equal to a row returns that row at rank 1
    pick = rows[::97][:24]
    idx1, sc1, _, _ = oracle.topk(keys, dt, keys[pick].astype(np.float32), 1)
    assert np.array_equal(idx1[:, 0], pick)
    assert np.all(np.abs(sc1[:, 0].astype(np.float64) - 1.0) <= 1e-6)


def pin_self_match_16bit():
    """16-bit rows are not exactly unit norm after rounding: the self score is
    |x_hat|^2, which must be within 1e-5 of its fp64 value and within 2e-3 of 1."""
    for name in ("pca4m_d1024_f16", "hidden1m_d4096_bf16"):
        w = WORKLOADS[name].scaled(2048)
        g = generate(w, "cpu", with_queries=False)
        keys, dt = to_numpy_bits(g["keys"])
        full = g["keys"].to(torch.float64).numpy()
        for i in range(0, w.N, 61):
            s = oracle.score_rows(keys, dt, full[i].astype(np.float32), [i])[0]
            n2 = float(np.dot(full[i], full[i]))
            assert abs(float(s) - n2) <= 1e-5
            assert abs(float(s) - 1.0) <= 2e-3


def pin_duplicates_and_mrr():
    """Planted duplicates: the lower index wins the tie; self-retrieval MRR
    (Eq. 4) is 1 for unique rows and 1/2 for each later copy."""
    w = WORKLOADS["flat16k_d256_f32"].scaled(3000)
    g = generate(w, "cpu", with_queries=False, planted_duplicates=12)
    keys, dt = to_numpy_bits(g["keys"])
    dups = g["duplicates"]
    later = {t for _, t in dups}
    q_rows = sorted({s for s, _ in dups} | later | set(range(0, w.N, 211)))
    idx, score, _, _ = oracle.topk(keys, dt, keys[q_rows], 3)
    rr = []
    for r, i in enumerate(q_rows):
        ranks = idx[r].tolist()
        rr.append(1.0 / (ranks.index(i) + 1) if i in ranks else 0.0)
    expect = (len(q_rows) - len(later) + 0.5 * len(later)) / len(q_rows)
    assert abs(float(np.mean(rr)) - expect) < 1e-12
    for s, t in dups:
        row = q_rows.index(t)
        assert idx[row, 0] == s and idx[row, 1] == t and score[row, 0] == score[row, 1]


def pin_structural_continuations():
    w = WORKLOADS["zipf33m_d128_f16"].scaled(5000)
    g = generate(w, "cpu")
    keys, dt = to_numpy_bits(g["keys"])
    L = 10
    cont = (np.arange(w.N, dtype=np.int64)[:, None] * L + np.arange(L)).astype(np.int32)
    idx, _, tok, _ = oracle.topk(keys, dt, g["queries"][:4].numpy(), 20, cont)
    assert np.array_equal(tok, (idx[..., None] * L + np.arange(L)).astype(np.int32))


def pin_full_sort_permutation():
    w = WORKLOADS["batch10m_d256_f16"].scaled(300)
    g = generate(w, "cpu")
    keys, dt = to_numpy_bits(g["keys"])
    q = g["queries"][:2].numpy()
    idx, score, _, nxt = oracle.topk(keys, dt, q, w.N)
    for b in range(2):
        assert sorted(idx[b].tolist()) == list(range(w.N))
        assert np.isnan(nxt[b])
        # the last row of a full sort of q against -q-like rows: argmin
        s_all = oracle.score_rows(keys, dt, q[b], np.arange(w.N))
        assert idx[b, -1] == int(np.lexsort((-np.arange(w.N), s_all))[0])


# --- pins of the next-token filter (Section 3.5) ------------------------------

def _fval(v):
    return np.float32(-np.inf) if v == "-inf" else np.float32(v)


def pin_filtered_golden_closed_forms():
    g = json.load(open(GOLDEN_FILTERED))
    n = len(g["first_tokens"])
    cont = np.stack([np.asarray(g["first_tokens"], np.int32),
                     np.arange(n, dtype=np.int32) + 100], axis=1)
    q = np.asarray([g["query"]], np.float32)
    for c in g["cases"]:
        for dt in ("f32", "f16", "bf16"):
            keys = _identity_keys(n, dt)
            idx, score, tok, _ = oracle.topk(keys, dt, q, c["k"], cont, next_tok=[c["next_tok"]])
            assert idx[0].tolist() == c["idx"], (c["name"], dt, idx[0].tolist())
            want = np.asarray([_fval(v) for v in c["score"]], np.float32)
            assert np.array_equal(score[0], want), (c["name"], dt, score[0])
            for r, i in enumerate(c["idx"]):
                want_tok = cont[i] if i >= 0 else np.zeros(2, np.int32)
                assert np.array_equal(tok[0, r], want_tok), (c["name"], dt, r)


def pin_filtered_bruteforce():
    """Exact rational scores on tiny inputs; only rows whose continuation
    starts with the query's token compete, ranked by (-score, index); ranks
    past them are (-1, -inf, zeros)."""
    rng = np.random.default_rng(777)
    N, d, B, k, L = 41, 6, 4, 7, 3
    x = rng.standard_normal((N, d))
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    keys = x.astype(np.float32)
    q = rng.standard_normal((B, d)).astype(np.float32)
    cont = rng.integers(0, 4, (N, L)).astype(np.int32)
    nt = np.asarray([0, 1, 2, 9], np.int32)  # the last token matches no row
    idx, score, tok, nxt = oracle.topk(keys, "f32", q, k, cont, next_tok=nt)
    for b in range(B):
        rows = [i for i in range(N) if cont[i, 0] == nt[b]]
        s = {i: _exact_fp32_score(q[b], keys[i]) for i in rows}
        order = sorted(rows, key=lambda i: (-float(s[i]), i))
        for r in range(k):
            if r < len(order):
                assert idx[b, r] == order[r] and score[b, r] == s[order[r]], (b, r)
                assert np.array_equal(tok[b, r], cont[order[r]])
            else:
                assert idx[b, r] == -1 and score[b, r] == -np.inf and not tok[b, r].any()
        if len(order) > k:
            assert nxt[b] == s[order[k]]
        else:
            assert np.isnan(nxt[b])


def pin_filter_admitting_all_rows_is_unfiltered():
    """A token every continuation starts with filters nothing: the result is
    the unfiltered top-k, bit for bit."""
    w = WORKLOADS["flat16k_d256_f32"].scaled(3000)
    g = generate(w, "cpu")
    keys, dt = to_numpy_bits(g["keys"])
    cont = g["cont"].numpy().copy()
    cont[:, 0] = 31
    q = g["queries"][:5].numpy()
    a = oracle.topk(keys, dt, q, 12, cont)
    b = oracle.topk(keys, dt, q, 12, cont, next_tok=np.full(5, 31))
    for x, y in zip(a, b):
        assert np.array_equal(x, y, equal_nan=True)


FILTER_PINS = [pin_filtered_golden_closed_forms, pin_filtered_bruteforce,
               pin_filter_admitting_all_rows_is_unfiltered]


@pytest.mark.parametrize("pin", FILTER_PINS, ids=[p.__name__ for p in FILTER_PINS])
def test_filter_pin(pin):
    pin()


PINS = [pin_golden_closed_forms, pin_exact_bruteforce, pin_decode_f16_all_patterns,
        pin_decode_bf16_all_patterns, pin_decode_keys_all_patterns, pin_invariants_and_self_match, pin_self_match_16bit,
        pin_duplicates_and_mrr, pin_structural_continuations, pin_full_sort_permutation]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin()


def test_textbook_lexsort_agrees():
    """Special case reducing to library routines: fp64 matmul, one rounding to
    fp32, stable lexsort on (-score, index)."""
    w = WORKLOADS["pca4m_d1024_f16"].scaled(4096)
    g = generate(w, "cpu")
    keys, dt = to_numpy_bits(g["keys"])
    q = g["queries"][:6].numpy()
    idx, score, _, _ = oracle.topk(keys, dt, q, 40)
    vals = g["keys"].to(torch.float64).numpy()
    s = (q.astype(np.float64) @ vals.T).astype(np.float32)
    for b in range(q.shape[0]):
        order = np.lexsort((np.arange(w.N), -s[b]))[:40]
        assert np.array_equal(order, idx[b])
        assert np.allclose(score[b], s[b, order], rtol=0, atol=1e-7)


def test_argument_errors():
    keys = np.eye(4, dtype=np.float32)
    q = np.ones((1, 4), np.float32)
    with pytest.raises(ValueError):
        oracle.topk(keys, "f32", q, 0)
    with pytest.raises(ValueError):
        oracle.topk(keys, "f32", q, 5)
    with pytest.raises(TypeError):
        oracle.topk(keys.astype(np.float64), "f32", q, 1)


MUTATIONS = {
    1: "drops the last term of the dot product",
    2: "flips the sign of the first term",
    3: "reads key elements at mirrored dimensions",
    4: "breaks ties by highest index",
    5: "ranks ascending",
    6: "truncates scores to 16 bits",
    7: "gathers the continuation of the next row",
    8: "filters on the continuation's second token",
}


@pytest.mark.parametrize("m", sorted(MUTATIONS), ids=[MUTATIONS[m] for m in sorted(MUTATIONS)])
def test_planted_mistakes(m):
    failed = []
    with oracle.mutation(m):
        for pin in PINS + FILTER_PINS:
            try:
                pin()
            except AssertionError:
                failed.append(pin.__name__)
    assert failed, "planted mistake %d (%s) passed every pin" % (m, MUTATIONS[m])
