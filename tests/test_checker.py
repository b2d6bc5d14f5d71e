"""The parity checker must reject each kind of wrong device result (CPU only).

A correct result built from the oracle passes; each planted defect (a swapped
index, a score moved by 2*tol, a flipped token bit, a broken order, a
duplicate or out-of-range index) must raise ParityError.
"""
import numpy as np
import pytest

import oracle
from datagen import WORKLOADS, generate, to_numpy_bits
from parity import ParityError, TOL, check_batch


@pytest.fixture(scope="module")
def case():
    w = WORKLOADS["pca4m_d1024_f16"].scaled(3000)
    g = generate(w, "cpu")
    keys, dt = to_numpy_bits(g["keys"])
    q = g["queries"][:4].numpy()
    cont = g["cont"].numpy()
    k = 16
    idx, score, tok, nxt = oracle.topk(keys, dt, q, k, cont)

    def exact(b, rows):
        return oracle.score_rows(keys, dt, q[b], rows)

    return dict(keys=keys, dt=dt, q=q, cont=cont, idx=idx, score=score, tok=tok, nxt=nxt,
                exact=exact, N=w.N, tol=TOL[dt], k=k)


def _run(c, idx=None, score=None, tok=None, tol=None):
    return check_batch(c["idx"] if idx is None else idx, c["score"] if score is None else score,
                       c["tok"] if tok is None else tok, c["idx"], c["score"], c["nxt"],
                       c["exact"], c["N"], c["cont"], c["tol"] if tol is None else tol)


def test_oracle_result_passes(case):
    rep = _run(case)
    assert rep["exact_order_rate"] == 1.0


def test_swapped_in_outside_row_fails(case):
    idx = case["idx"].copy()
    outside = next(i for i in range(case["N"]) if i not in set(idx[0].tolist()))
    idx[0, 0] = outside
    with pytest.raises(ParityError):
        _run(case, idx=idx)


def test_score_moved_by_two_tol_fails(case):
    s = case["score"].copy()
    s[1, 3] -= 2 * case["tol"]
    with pytest.raises(ParityError):
        _run(case, score=s)


def test_flipped_token_bit_fails(case):
    t = case["tok"].copy()
    t[2, 5, 7] ^= 1
    with pytest.raises(ParityError):
        _run(case, tok=t)


def test_broken_order_fails(case):
    idx = case["idx"].copy()
    s = case["score"].copy()
    idx[0, [0, 5]] = idx[0, [5, 0]]
    s[0, [0, 5]] = s[0, [5, 0]]
    with pytest.raises(ParityError):
        _run(case, idx=idx, score=s, tol=1.0)


def test_duplicate_index_fails(case):
    idx = case["idx"].copy()
    idx[3, 2] = idx[3, 1]
    with pytest.raises(ParityError):
        _run(case, idx=idx, tol=1.0)


def test_out_of_range_fails(case):
    idx = case["idx"].copy()
    idx[0, -1] = case["N"]
    with pytest.raises(ParityError):
        _run(case, idx=idx, tol=1.0)


def test_near_tie_swap_at_boundary_is_allowed(case):
    """Within tol of the rank-k score, another row may take the last rank."""
    c = case
    b = 0
    # the oracle's (k+1)-th row
    idx_k1, sc_k1, _, _ = oracle.topk(c["keys"], c["dt"], c["q"][b:b + 1], c["k"] + 1)
    gap = float(c["score"][b, -1]) - float(sc_k1[0, -1])
    if gap >= c["tol"]:
        pytest.skip("no near tie at the boundary for this query")
    idx = c["idx"].copy()
    s = c["score"].copy()
    idx[b, -1] = idx_k1[0, -1]
    s[b, -1] = sc_k1[0, -1]
    tok = c["tok"].copy()
    tok[b, -1] = c["cont"][idx_k1[0, -1]]
    _run(c, idx=idx, score=s, tok=tok)
