"""Parity rules between the device path and the oracle (per query).

The rules follow the acceptance statement for exact top-k retrieval:
scores agree within ``tol`` (1e-5 for fp32 keys, 2e-3 for 16-bit keys);
index sets are identical except at ranks where the oracle's rank-k and
rank-(k+1) scores differ by less than ``tol``; gathered continuation tokens
are bit-exact for the returned indices.

  R1  |g_score[r] - o_score[r]| <= tol for every rank r
  R2  |g_score[r] - exact(g_idx[r])| <= tol (exact = oracle re-score of that row)
  R3  g_score non-increasing; equal g_score values have ascending g_idx
  R4  g_idx distinct and inside [0, N)
  R5  must-include M = {o_idx[r] : o_score[r] - o_next >= tol} is contained in
      set(g_idx), which is contained in A = {i : exact(i) > o_score[k-1] - tol}
      (identical sets whenever the rank-k / rank-(k+1) gap is >= tol)
  R7  tokens[r, :] == cont[g_idx[r], :] bit for bit
Also reported (not gating): exact-order agreement and max |g - exact|.

Operand model (``check_operand_model``), per returned element: the device
score lies within fp32 accumulation error of the exact inner product of the
row with the query *as the matrix cores take it* (the operand precision the
library documents for the batch size: the query itself, two bf16 parts, or
the query rounded once to f16), and within the documented rounding bound of
the exact inner product with the fp32 query.  This is much tighter than the
2e-3 tolerance and fails for a truncating or double-rounding conversion.

Searches over a subset of the rows -- next-token-filtered (Section 3.5) or
partitioned (the probed partitions) -- add: every returned row is in the
subset, and ranks past the subset's rows -- exactly where the oracle's are --
hold index -1, score -inf and zero tokens; the rules above apply to the ranks
before them.
"""
from __future__ import annotations

import numpy as np

TOL = {"f32": 1e-5, "f16": 2e-3, "bf16": 2e-3}


class ParityError(AssertionError):
    pass


def check_query(g_idx, g_score, g_tok, o_idx, o_score, o_next, exact_of, N, cont=None,
                tol=1e-5):
    """Check one query.  ``exact_of(rows) -> fp32 scores`` re-scores rows with
    the oracle.  Returns a small report dict; raises ParityError on failure."""
    g_idx = np.asarray(g_idx, np.int64)
    g_score = np.asarray(g_score, np.float32)
    o_idx = np.asarray(o_idx, np.int64)
    o_score = np.asarray(o_score, np.float32)
    k = o_idx.size
    if g_idx.shape != (k,) or g_score.shape != (k,):
        raise ParityError("shape mismatch")
    # R4
    if g_idx.min() < 0 or g_idx.max() >= N:
        raise ParityError("R4: index out of range")
    if np.unique(g_idx).size != k:
        raise ParityError("R4: duplicate indices")
    # R3
    ds = np.diff(g_score.astype(np.float64))
    if np.any(ds > 0):
        raise ParityError("R3: scores increase at rank %d" % int(np.argmax(ds > 0)))
    eq = ds == 0
    if np.any(eq & (np.diff(g_idx) < 0)):
        raise ParityError("R3: equal scores not in ascending index order")
    # R1
    d1 = np.abs(g_score.astype(np.float64) - o_score.astype(np.float64))
    if np.any(d1 > tol):
        r = int(np.argmax(d1))
        raise ParityError("R1: rank %d score %r vs oracle %r" % (r, g_score[r], o_score[r]))
    # R2
    ex = np.asarray(exact_of(g_idx), np.float32)
    d2 = np.abs(g_score.astype(np.float64) - ex.astype(np.float64))
    if np.any(d2 > tol):
        r = int(np.argmax(d2))
        raise ParityError("R2: rank %d row %d score %r vs exact %r" % (r, g_idx[r], g_score[r],
                                                                        ex[r]))
    # R5
    if o_next is None or np.isnan(o_next):
        must = set(o_idx.tolist())
    else:
        must = {int(i) for i, s in zip(o_idx, o_score) if float(s) - float(o_next) >= tol}
    gset = set(g_idx.tolist())
    if not must <= gset:
        raise ParityError("R5: missing must-include rows %s" % sorted(must - gset)[:8])
    floor = float(o_score[-1]) - tol
    if np.any(ex.astype(np.float64) <= floor):
        raise ParityError("R5: returned a row scoring <= rank-k score - tol")
    # R7
    if g_tok is not None and cont is not None:
        want = np.asarray(cont)[g_idx]
        if not np.array_equal(np.asarray(g_tok), want):
            raise ParityError("R7: gathered tokens differ")
    return {
        "exact_order": bool(np.array_equal(g_idx, o_idx)),
        "max_abs_vs_exact": float(d2.max()) if d2.size else 0.0,
        "max_abs_vs_oracle": float(d1.max()) if d1.size else 0.0,
    }


def check_query_padded(g_idx, g_score, g_tok, o_idx, o_score, o_next, exact_of, N, cont,
                       admitted, what, tol=1e-5):
    """One query of a search over a subset of the rows (next-token filter,
    probed partitions): ranks past the subset -- exactly where the oracle's
    are -- hold (-1, -inf, zero tokens); every returned row is in the subset
    (``admitted(rows) -> bool array``, ``what`` names the rule); the rules
    above apply to the ranks before the padding."""
    g_idx = np.asarray(g_idx, np.int64)
    g_score = np.asarray(g_score, np.float32)
    o_idx = np.asarray(o_idx, np.int64)
    k = o_idx.size
    pad = np.nonzero(o_idx < 0)[0]
    m = int(pad[0]) if pad.size else k
    if np.any(o_idx[m:] >= 0):
        raise ParityError("oracle padding is not a suffix")
    if g_idx.shape != (k,):
        raise ParityError("shape mismatch")
    if np.any(g_idx[m:] != -1) or np.any(g_score[m:] != -np.inf):
        raise ParityError("padding: ranks >= %d must be (-1, -inf)" % m)
    if g_tok is not None and np.any(np.asarray(g_tok)[m:] != 0):
        raise ParityError("padding: tokens of ranks >= %d must be zero" % m)
    if m == 0:
        return {"exact_order": True, "max_abs_vs_exact": 0.0, "max_abs_vs_oracle": 0.0}
    if np.any(g_idx[:m] < 0) or np.any(g_idx[:m] >= N):
        raise ParityError("R4: index out of range")
    if not np.all(admitted(g_idx[:m])):
        raise ParityError(what)
    return check_query(g_idx[:m], g_score[:m], None if g_tok is None else np.asarray(g_tok)[:m],
                       o_idx[:m], np.asarray(o_score)[:m], o_next, exact_of, N, cont, tol)


def check_query_filtered(g_idx, g_score, g_tok, o_idx, o_score, o_next, exact_of, N, cont,
                         first_token, tol=1e-5):
    """One query of a next-token-filtered search: ``first_token`` is the
    token its drafts must start with."""
    return check_query_padded(
        g_idx, g_score, g_tok, o_idx, o_score, o_next, exact_of, N, cont,
        lambda rows: np.asarray(cont)[rows, 0] == first_token,
        "filter: returned a row whose continuation does not start with %d" % first_token, tol)


def check_batch(g_idx, g_score, g_tok, o_idx, o_score, o_next, exact_of_b, N, cont=None,
                tol=1e-5, next_tok=None, admitted_b=None):
    """``exact_of_b(b, rows)`` re-scores rows for query b; ``next_tok`` [B]
    marks a next-token-filtered search; ``admitted_b(b, rows)`` a search over
    a per-query subset of the rows (probed partitions)."""
    reps = []
    for b in range(o_idx.shape[0]):
        try:
            args = (g_idx[b], g_score[b], None if g_tok is None else g_tok[b], o_idx[b],
                    o_score[b], None if o_next is None else o_next[b],
                    lambda rows, b=b: exact_of_b(b, rows), N, cont)
            if admitted_b is not None:
                reps.append(check_query_padded(*args, lambda rows, b=b: admitted_b(b, rows),
                                               "partitions: returned a row of a partition that "
                                               "was not probed", tol))
            elif next_tok is None:
                reps.append(check_query(*args, tol))
            else:
                reps.append(check_query_filtered(*args, int(next_tok[b]), tol))
        except ParityError as e:
            raise ParityError("query %d: %s" % (b, e)) from None
    return {
        "exact_order_rate": float(np.mean([r["exact_order"] for r in reps])) if reps else 1.0,
        "max_abs_vs_exact": max([r["max_abs_vs_exact"] for r in reps], default=0.0),
        "max_abs_vs_oracle": max([r["max_abs_vs_oracle"] for r in reps], default=0.0),
    }


def _bf16_rne(x: np.ndarray) -> np.ndarray:
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).to(
        torch.float32).numpy()


def operand_model(q, key_dtype: str, B: int):
    """The query as the matrix cores take it in a batch of B queries over keys
    of this storage type, as the library documents it: the query itself for
    fp32 keys and for 16-bit keys with B <= 4 (three 16-bit parts that sum to
    it exactly); for larger bf16 batches the high part (the query rounded to
    nearest-even bf16) plus the remainder rounded the same way; for larger
    f16 batches the query rounded once to nearest-even f16.  Returns
    (fp32 array, which it is, relative bound of its difference from q)."""
    q = np.asarray(q, np.float32)
    if key_dtype == "f32" or B <= 4:
        return q.copy(), "exact", 0.0
    if key_dtype == "f16":
        return q.astype(np.float16).astype(np.float32), "f16-rounded", 2.0 ** -11
    hi = _bf16_rne(q)
    lo = _bf16_rne(q - hi)  # q - hi is exact in fp32
    return (hi.astype(np.float64) + lo).astype(np.float32), "bf16-two-part", 2.0 ** -17


def check_operand_model(g_idx, g_score, q, B, key_dtype, decode_rows, score_with):
    """Check one query's returned elements against the operand model.

    ``decode_rows(rows) -> float64 [n, d]`` decodes key rows exactly;
    ``score_with(q_fp32, rows) -> fp32`` is the oracle's score of the rows for
    an arbitrary fp32 query.  For every returned row x (index >= 0):
      |g - model|  <= gam * sum_j |qm_j x_j|, qm the modelled query, gam =
                      (d + 4) 2^-23 (16-bit keys: products exact, at most d + 4
                      roundings of partial sums, each within 2^-23 of them),
                      (2 d + 4) 2^-23 for fp32 keys (products rounded too);
                      with f16 rounding, plus 2^-14 sum |x_j| over the
                      components below f16's normal range (in case such tiny
                      components do not keep their subnormal value);
      |g - exact|  <= rel * sum_j |q_j x_j| + 2^-25 sum_j |x_j| (f16 only)
                      + the first bound, rel the model's documented relative
                      error (2^-11 f16-rounded, 2^-17 bf16 two-part, 0 exact).
    Returns (max |g - model|, max |g - exact|, mode)."""
    g_idx = np.asarray(g_idx, np.int64)
    g_score = np.asarray(g_score, np.float32)
    keep = g_idx >= 0
    rows = g_idx[keep]
    if rows.size == 0:
        return 0.0, 0.0, "empty"
    q = np.asarray(q, np.float32).reshape(-1)
    d = q.size
    qm, mode, rel = operand_model(q[None, :], key_dtype, B)
    qm = qm[0]
    x = np.abs(decode_rows(rows))
    Sm = x @ np.abs(qm.astype(np.float64))
    Sq = x @ np.abs(q.astype(np.float64))
    A = x.sum(axis=1)
    gam = (2 * d + 4 if key_dtype == "f32" else d + 4) * 2.0 ** -23
    tiny = (np.abs(q) < 2.0 ** -14) if mode == "f16-rounded" else np.zeros(d, bool)
    bound_m = gam * Sm + 2.0 ** -14 * (x[:, tiny].sum(axis=1) if tiny.any() else 0.0)
    bound_e = rel * Sq + (2.0 ** -25 * A if mode == "f16-rounded" else 0.0) + bound_m
    g = g_score[keep].astype(np.float64)
    dm = np.abs(g - score_with(qm, rows).astype(np.float64))
    de = np.abs(g - score_with(q, rows).astype(np.float64))
    if np.any(dm > bound_m):
        r = int(np.argmax(dm - bound_m))
        raise ParityError("operand model (%s): row %d |g - model| %.3e > bound %.3e"
                          % (mode, int(rows[r]), dm[r], bound_m[r]))
    if np.any(de > bound_e):
        r = int(np.argmax(de - bound_e))
        raise ParityError("operand model (%s): row %d |g - exact| %.3e > bound %.3e"
                          % (mode, int(rows[r]), de[r], bound_e[r]))
    return float(dm.max()), float(de.max()), mode
