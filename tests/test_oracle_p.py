"""Pins for the oracle's chunked layout (the paper's own chunk structure,
Section 5, with the CPU converter of Section 5.2); runs without a GPU.

Checked against: the definition of the pattern order (every n-subset once,
adjacent patterns one position apart), hand-worked greedy runs
(tests/golden/chunked_greedy.json), the exact optimum of each chunk's
assignment problem (SciPy's linear_sum_assignment), exact invariants of the
layout, and a dense NumPy product.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
from scipy.optimize import linear_sum_assignment

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("m,n", [(4, 2), (4, 1), (8, 2), (6, 3), (5, 5), (10, 1), (7, 4), (9, 2)])
def test_pattern_order(m, n):
    pats = [tuple(int(v) for v in row) for row in oracle.p_patterns(m, n)]
    assert len(pats) == math.comb(m, n)
    assert sorted(pats) == sorted(itertools.combinations(range(m), n))   # every subset once, ascending
    for a, b in zip(pats, pats[1:]):
        assert len(set(a) & set(b)) == n - 1                            # one position changes
    assert pats[0] == tuple(range(n))


def test_hand_worked_greedy():
    gold = json.load(open(os.path.join(GOLDEN, "chunked_greedy.json")))
    for case in gold["cases"]:
        n, m, g = case["n"], case["m"], case["g"]
        assert oracle.p_patterns(m, n).tolist() == case["patterns"]
        W = np.array(case["W"], np.float32)
        values, index = oracle.p_compress(W, n, m, g)
        assert index[:, 0].tolist() == case["index_col0"], case["name"]
        assert values.tolist() == case["values"], case["name"]
        assert float(np.abs(values.astype(np.float64)).sum()) == case["kept"]
        assert chunk_optimum(W, n, m, g, 0, 0) == case["optimum"]


def chunk_scores(W, n, m, g, c, b):
    """|kept| of every (row, pattern) of chunk (c, b), in binary64."""
    pats = oracle.p_patterns(m, n)
    S = len(pats) * g
    rows = np.abs(W[c * S:(c + 1) * S, b * m:(b + 1) * m].astype(np.float64))
    return np.stack([rows[:, list(p)].sum(axis=1) for p in pats], axis=1)


def chunk_optimum(W, n, m, g, c, b):
    """The exact optimum: an assignment of S rows to S slots (each pattern g times)."""
    sc = np.repeat(chunk_scores(W, n, m, g, c, b), g, axis=1)
    ri, ci = linear_sum_assignment(-sc)
    return float(sc[ri, ci].sum())


LAYOUTS = [(2, 4, 1, 12, 8), (2, 4, 4, 48, 16), (1, 4, 8, 64, 12), (1, 2, 3, 12, 6),
           (3, 6, 2, 80, 12), (2, 5, 1, 20, 10)]


@pytest.mark.parametrize("n,m,g,M,K", LAYOUTS)
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_invariants_and_bounds(n, m, g, M, K, dtype):
    rng = np.random.default_rng(M + K + n)
    W = rng.standard_normal((M, K)).astype(dtype)
    values, index = oracle.p_compress(W, n, m, g)
    pats = oracle.p_patterns(m, n)
    P, S, B = len(pats), len(pats) * g, K // m
    dense, mask = oracle.p_densify(values, index, K, n, m, g)
    # densify gives W on the kept positions, +0 elsewhere (bits)
    assert np.array_equal(dense.view(np.uint8), np.where(mask, W, np.zeros_like(W)).view(np.uint8))
    for c in range(M // S):
        for b in range(B):
            col = index[c * S:(c + 1) * S, b]
            assert sorted(col.tolist()) == list(range(S))          # a permutation of the chunk rows
            for j in range(S):                                     # position j uses pattern j // g
                r = c * S + col[j]
                kept = np.flatnonzero(mask[r, b * m:(b + 1) * m])
                assert kept.tolist() == pats[j // g].tolist()
                for p in range(P):                                 # rows of a group ascending
                    grp = col[p * g:(p + 1) * g]
                    assert list(grp) == sorted(grp)
            kept_total = float(np.abs(values[c * S:(c + 1) * S, b * n:(b + 1) * n].astype(np.float64)).sum())
            opt = chunk_optimum(W, n, m, g, c, b)
            assert kept_total <= opt * (1 + 1e-12) + 1e-12
            assert kept_total >= 0.5 * opt - 1e-12                 # the greedy's guarantee


def test_greedy_is_optimal_on_separable_chunks():
    """Every row has its own dominant pattern and the dominants are balanced:
    the greedy then finds the (unique) optimum."""
    n, m, g = 2, 4, 2
    pats = oracle.p_patterns(m, n)
    P, S = len(pats), len(pats) * g
    rng = np.random.default_rng(3)
    order = rng.permutation(S)
    W = np.zeros((S, m), np.float32)
    for r in range(S):
        p = order[r] % P
        W[r, list(pats[p])] = 8 + r                      # dominant pattern
        W[r] += rng.uniform(0, 0.25, m).astype(np.float32)
    values, index = oracle.p_compress(W, n, m, g)
    kept = float(np.abs(values.astype(np.float64)).sum())
    assert kept == pytest.approx(chunk_optimum(W, n, m, g, 0, 0), rel=1e-12)


def test_ties_go_to_the_lower_pattern_then_row():
    n, m, g = 1, 4, 3
    W = np.zeros((12, 8), np.float32)
    values, index = oracle.p_compress(W, n, m, g)
    assert (index[:, 0] == np.arange(12)).all() and (index[:, 1] == np.arange(12)).all()


@pytest.mark.parametrize("n,m,g,M,K", LAYOUTS)
def test_product_is_the_dense_product(n, m, g, M, K):
    rng = np.random.default_rng(7 * M + K)
    W = rng.integers(-8, 9, (M, K)).astype(np.float32) / 8     # exact in binary64 sums
    X = rng.integers(-8, 9, (K, 5)).astype(np.float32) / 4
    values, index = oracle.p_compress(W, n, m, g)
    dense, _ = oracle.p_densify(values, index, K, n, m, g)
    Y, Bnd = oracle.p_spmm(values, index, X, K, n, m, g)
    assert np.array_equal(Y, dense.astype(np.float64) @ X.astype(np.float64))
    assert np.array_equal(Bnd, np.abs(dense.astype(np.float64)) @ np.abs(X.astype(np.float64)))


def test_rejections():
    W = np.zeros((24, 8), np.float32)
    with pytest.raises(oracle.OracleError) as e:
        oracle.p_compress(W[:, :7], 2, 4, 4)       # K % m != 0
    assert e.value.status == 2
    with pytest.raises(oracle.OracleError) as e:
        oracle.p_compress(W[:20], 2, 4, 4)         # M % (6 * 4) != 0
    assert e.value.status == 2
    with pytest.raises(oracle.OracleError) as e:
        oracle.p_compress(np.zeros((924, 12), np.float32), 6, 12, 1)   # C(12, 6) = 924 patterns
    assert e.value.status == 1
    values, index = oracle.p_compress(W, 2, 4, 4)
    bad = index.copy()
    bad[1, 0] = bad[0, 0]                          # not a permutation of the chunk rows
    with pytest.raises(oracle.OracleError) as e:
        oracle.p_densify(values, bad, 8, 2, 4, 4)
    assert e.value.status == 3


# ------------------------------------------------------------ swap search

def kept(values):
    return float(np.abs(values.astype(np.float64)).sum())


def test_refine_fixes_the_hand_example():
    """Golden case 2: the greedy keeps 3 of the optimum 5; one swap (gain
    2 + 3 - 3 - 0 = 2) reaches it."""
    gold = json.load(open(os.path.join(GOLDEN, "chunked_greedy.json")))["cases"][1]
    W = np.array(gold["W"], np.float32)
    values, index = oracle.p_compress(W, 1, 2, 1)
    rv, ridx, rounds = oracle.p_refine(W, index, 1, 2, 1)
    assert ridx[:, 0].tolist() == [1, 0] and rv.tolist() == [[3.0], [2.0]]
    assert kept(rv) == gold["optimum"] and rounds == 1


@pytest.mark.parametrize("n,m,g,M,K", LAYOUTS)
def test_refine_is_a_local_optimum_between_greedy_and_optimum(n, m, g, M, K):
    rng = np.random.default_rng(11 * M + K)
    W = rng.standard_normal((M, K)).astype(np.float32)
    values, index = oracle.p_compress(W, n, m, g)
    rv, ridx, rounds = oracle.p_refine(W, index, n, m, g)
    pats = oracle.p_patterns(m, n)
    P, S, B = len(pats), len(pats) * g, K // m
    assert rounds < 8 * S
    dense, mask = oracle.p_densify(rv, ridx, K, n, m, g)      # a valid packing of W
    assert np.array_equal(dense.view(np.uint8), np.where(mask, W, np.zeros_like(W)).view(np.uint8))
    for c in range(M // S):
        for b in range(B):
            sl = slice(c * S, (c + 1) * S)
            before, after = kept(values[sl, b * n:(b + 1) * n]), kept(rv[sl, b * n:(b + 1) * n])
            assert after >= before
            assert after <= chunk_optimum(W, n, m, g, c, b) * (1 + 1e-12)
            # no pair swap improves (binary64 sums of the binary32 magnitudes)
            sc = chunk_scores_f32(W, n, m, g, c, b)
            pa = np.empty(S, int)
            pa[ridx[sl, b]] = np.arange(S) // g
            for r in range(S):
                for q in range(S):
                    if pa[r] != pa[q]:
                        gain = (sc[r, pa[q]] + sc[q, pa[r]]) - (sc[r, pa[r]] + sc[q, pa[q]])
                        assert gain <= 0


def chunk_scores_f32(W, n, m, g, c, b):
    """The layout's scores: binary32 sums of |w| over each pattern's offsets in
    ascending order, from +0; returned as binary64."""
    pats = oracle.p_patterns(m, n)
    S = len(pats) * g
    rows = np.abs(W[c * S:(c + 1) * S, b * m:(b + 1) * m].astype(np.float32))
    out = np.zeros((S, len(pats)), np.float64)
    for p, offs in enumerate(pats):
        acc = np.zeros(S, np.float32)
        for o in offs:
            acc = (acc + rows[:, o]).astype(np.float32)
        out[:, p] = acc
    return out
