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


# --- next-token-filtered searches -------------------------------------------

def _filtered_case():
    rng = np.random.default_rng(5)
    N, d, B, k = 300, 16, 3, 8
    x = rng.standard_normal((N, d))
    x = (x / np.linalg.norm(x, axis=1, keepdims=True)).astype(np.float32)
    q = rng.standard_normal((B, d)).astype(np.float32)
    cont = rng.integers(0, 6, (N, 2)).astype(np.int32)
    cont[:5, 0] = 40  # token 40: exactly five rows, fewer than k
    nt = np.asarray([1, 40, 77], np.int32)  # 77 matches no row
    o = oracle.topk(x, "f32", q, k, cont, next_tok=nt)
    ex = lambda b, rows: oracle.score_rows(x, "f32", q[b], rows)
    return x, cont, nt, o, ex, N


def test_filtered_oracle_result_passes():
    x, cont, nt, (oi, os_, ot, on), ex, N = _filtered_case()
    assert (oi[1, 5:] == -1).all() and (oi[2] == -1).all()
    check_batch(oi, os_, ot, oi, os_, on, ex, N, cont, 1e-5, next_tok=nt)


def test_filtered_unadmitted_row_fails():
    x, cont, nt, (oi, os_, ot, on), ex, N = _filtered_case()
    gi, gs, gt = oi.copy(), os_.copy(), ot.copy()
    bad = int(np.nonzero(cont[:, 0] != nt[0])[0][0])
    gi[0, -1] = bad  # score left as the oracle's: only the filter rule can reject it
    gt[0, -1] = cont[bad]
    with pytest.raises(ParityError):
        check_batch(gi, gs, gt, oi, os_, on, ex, N, cont, 1e-5, next_tok=nt)


def test_filtered_padding_must_match():
    x, cont, nt, (oi, os_, ot, on), ex, N = _filtered_case()
    gi, gs, gt = oi.copy(), os_.copy(), ot.copy()
    gi[1, 5], gs[1, 5] = 7, 0.0  # a real row where the oracle pads
    with pytest.raises(ParityError):
        check_batch(gi, gs, gt, oi, os_, on, ex, N, cont, 1e-5, next_tok=nt)
    gi, gs, gt = oi.copy(), os_.copy(), ot.copy()
    gt[2, 0, 0] = 1  # padding tokens must be zero
    with pytest.raises(ParityError):
        check_batch(gi, gs, gt, oi, os_, on, ex, N, cont, 1e-5, next_tok=nt)


def _partitioned_case():
    rng = np.random.default_rng(21)
    N, d, P = 600, 16, 6
    x = rng.standard_normal((N, d))
    x = (x / np.linalg.norm(x, axis=1, keepdims=True)).astype(np.float32)
    cont = rng.integers(0, 50, (N, 2)).astype(np.int32)
    assign = rng.integers(0, P, N).astype(np.int32)
    q = rng.standard_normal((3, d)).astype(np.float32)
    probes = np.array([[0, 1], [2, 2], [5, -1]], np.int32)
    o = oracle.topk_partitioned(x, "f32", q, 12, assign, P, probes, cont)
    sets = [set(p for p in row if 0 <= p < P) for row in probes]

    def ex(b, rows):
        return oracle.score_rows(x, "f32", q[b], rows)

    def adm(b, rows):
        return np.isin(assign[rows], list(sets[b]))
    return x, cont, assign, probes, o, ex, adm, N


def test_partitioned_oracle_result_passes():
    x, cont, assign, probes, (oi, os_, ot, on), ex, adm, N = _partitioned_case()
    check_batch(oi, os_, ot, oi, os_, on, ex, N, cont, 1e-5, admitted_b=adm)


def test_partitioned_row_outside_probes_fails():
    x, cont, assign, probes, (oi, os_, ot, on), ex, adm, N = _partitioned_case()
    gi, gs, gt = oi.copy(), os_.copy(), ot.copy()
    bad = int(np.nonzero(~np.isin(assign, [0, 1]))[0][0])
    gi[0, -1] = bad  # score left as the oracle's: only the partition rule can reject it
    gt[0, -1] = cont[bad]
    with pytest.raises(ParityError):
        check_batch(gi, gs, gt, oi, os_, on, ex, N, cont, 1e-5, admitted_b=adm)


# Operand model: a device that rounds the query as documented passes; one
# whose conversion truncates, or rounds twice (through bf16 first), fails.
def _model_case(dtype_name, B):
    w = WORKLOADS[dtype_name].scaled(4000)
    g = generate(w, "cpu")
    keys, dt = to_numpy_bits(g["keys"])
    q = g["queries"][:B].numpy()
    x = oracle.decode_keys(keys, dt)
    return keys, dt, q, x


def _scores(x, qeff, rows):
    # what a device computing exactly with operand qeff would return
    return (x[rows] @ qeff.astype(np.float64)).astype(np.float32)


def _f16_trunc(q):
    # round toward zero to f16 (a truncating conversion)
    r = q.astype(np.float16)
    over = np.abs(r.astype(np.float32)) > np.abs(q)
    step = np.nextafter(r, np.float16(0))
    return np.where(over, step, r).astype(np.float32)


@pytest.mark.parametrize("wl,B", [("batch10m_d256_f16", 64), ("zipf33m_d128_f16", 128),
                                  ("hidden1m_d4096_bf16", 8), ("pca4m_d1024_f16", 4)])
def test_operand_model_accepts_documented_rounding(wl, B):
    from parity import check_operand_model, operand_model
    keys, dt, q, x = _model_case(wl, min(B, 8))
    for b in range(q.shape[0]):
        rows = np.arange(0, 4000, 97)
        qm, _, _ = operand_model(q[b][None, :], dt, B)
        g = _scores(x, qm[0], rows)
        check_operand_model(rows, g, q[b], B, dt, lambda r: x[r],
                            lambda qq, r: oracle.score_rows(keys, dt, qq, r))


@pytest.mark.parametrize("bad", ["truncate", "twice"])
def test_operand_model_rejects_wrong_f16_rounding(bad):
    from parity import check_operand_model
    keys, dt, q, x = _model_case("zipf33m_d128_f16", 8)
    rows = np.arange(0, 4000, 7)
    failed = 0
    for b in range(q.shape[0]):
        if bad == "truncate":
            qe = _f16_trunc(q[b])
        else:  # through bf16 first, then f16
            import torch
            qb = torch.from_numpy(q[b]).to(torch.bfloat16).to(torch.float32).numpy()
            qe = qb.astype(np.float16).astype(np.float32)
        g = _scores(x, qe, rows)
        try:
            check_operand_model(rows, g, q[b], 128, dt, lambda r: x[r],
                                lambda qq, r: oracle.score_rows(keys, dt, qq, r))
        except ParityError:
            failed += 1
    assert failed == q.shape[0]
