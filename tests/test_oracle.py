"""Pins for the CPU oracle (runs without a GPU).

The oracle is checked against things other than itself: hand-worked examples
(tests/golden), brute-force enumeration of every admissible pattern on tiny
inputs, special cases that reduce to library routines (g = 1 -> a per-row sort;
n = m -> a dense matmul), exact invariants of the definition, and NumPy / SciPy
implementations of the binary16 conversions and of erf.

Paper: STen (arXiv 2304.07613) Section 5 (layout), 5.1 (product), 5.2
(converter objective and conversion back to dense), 6.1 (energy).
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def chunk_width(K, m, c):
    return min(m, K - c * m)


# --------------------------------------------------------------- golden cases

def test_hand_example_2_4_2():
    gd = load_golden("hand_2_4_2.json")
    W = np.array(gd["W"], dtype=np.float32)
    n, m, g = gd["n"], gd["m"], gd["g"]
    values, indices = oracle.compress(W, n, m, g)
    assert indices.tolist() == gd["indices"]
    assert values.tolist() == gd["values"]
    Y, B = oracle.spmm(values, indices, np.ones((8, 1), np.float32), 8, n, m, g)
    assert Y[:, 0].tolist() == gd["Y_ones"]
    assert oracle.energy(W, values) == gd["energy_num"] / gd["energy_den"]
    _, idx1 = oracle.compress(W, n, m, 1)
    assert idx1.tolist() == gd["indices_g1"]


def test_score_is_binary32_in_ascending_row_order():
    gd = load_golden("score_rounding.json")
    W = np.array(gd["W"], dtype=np.float32)
    assert W[1, 0] == np.float32(2.0 ** -24) and W[0, 1] == np.float32(1 + 2.0 ** -23)
    _, indices = oracle.compress(W, gd["n"], gd["m"], gd["g"])
    assert indices.tolist() == gd["indices"]


# ----------------------------------------------------------------- brute force

def brute_force_indices(W, n, m, g):
    """Enumerate every n-subset of every (group, chunk); keep the one with the
    largest exact kept L1 mass, the lexicographically smallest on ties."""
    M, K = W.shape
    C = -(-K // m)
    out = np.zeros((M // g, C * n), np.uint8)
    for G in range(M // g):
        for c in range(C):
            w = chunk_width(K, m, c)
            score = [sum(Fraction(abs(float(W[G * g + i, c * m + j]))) for i in range(g))
                     for j in range(w)]
            best = None
            for sub in itertools.combinations(range(w), n):
                mass = sum(score[j] for j in sub)
                if best is None or mass > best[0]:
                    best = (mass, sub)
            out[G, c * n:(c + 1) * n] = best[1]
    return out


def dyadic(rng, shape, dtype=np.float32):
    """Multiples of 1/16 in [-1, 1]: binary32 (and binary16) sums of a few of
    them are exact, and many scores tie."""
    return (rng.integers(-16, 17, size=shape) / 16.0).astype(dtype)


@pytest.mark.parametrize("seed", range(40))
def test_bruteforce_selection_and_product(seed):
    rng = np.random.default_rng(seed)
    m = int(rng.integers(1, 7))
    n = int(rng.integers(1, m + 1))
    g = int(rng.choice([1, 2, 4]))
    M = g * int(rng.integers(1, 8 // g + 1))
    # K with a tail chunk of width >= n
    C = int(rng.integers(1, 4))
    tail = int(rng.integers(n, m + 1))
    K = (C - 1) * m + tail
    dtype = np.float16 if seed % 3 == 0 else np.float32
    W = dyadic(rng, (M, K), dtype)
    values, indices = oracle.compress(W, n, m, g)
    assert np.array_equal(indices, brute_force_indices(W, n, m, g))
    # product: naive triple loop, exact in rationals (dyadic data)
    N = int(rng.integers(1, 6))
    X = dyadic(rng, (K, N), dtype)
    Y, B = oracle.spmm(values, indices, X, K, n, m, g)
    Wd, mask = oracle.densify(values, indices, K, n, m, g)
    for r in range(M):
        for t in range(N):
            exact = sum(Fraction(float(Wd[r, k])) * Fraction(float(X[k, t])) for k in range(K))
            scale = sum(abs(Fraction(float(Wd[r, k])) * Fraction(float(X[k, t]))) for k in range(K))
            assert Fraction(Y[r, t]) == exact
            assert Fraction(B[r, t]) == scale


@pytest.mark.parametrize("seed", range(10))
def test_bruteforce_selection_continuous(seed):
    """Normal draws (no ties): exact-rational brute force agrees with the
    binary32 scores whenever no two exact scores fall within rounding."""
    rng = np.random.default_rng(100 + seed)
    n, m, g = [(1, 4, 2), (2, 4, 4), (2, 6, 1), (3, 5, 2), (1, 3, 8)][seed % 5]
    M, K = 8, 2 * m + n
    W = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    _, indices = oracle.compress(W, n, m, g)
    assert np.array_equal(indices, brute_force_indices(W, n, m, g))


# -------------------------------------------------------------- special cases

@pytest.mark.parametrize("n,m,K", [(1, 4, 64), (2, 4, 66), (2, 8, 70), (1, 10, 72), (3, 7, 40)])
def test_g1_is_per_row_sort(n, m, K):
    """g = 1 is per-row n:m magnitude pruning: compare with a NumPy stable sort
    by (-|w|, offset)."""
    rng = np.random.default_rng(K)
    W = dyadic(rng, (12, K))  # many ties
    W[::3] = (rng.standard_normal((4, K)) * 0.02).astype(np.float32)
    values, indices = oracle.compress(W, n, m, 1)
    C = -(-K // m)
    for r in range(12):
        for c in range(C):
            w = chunk_width(K, m, c)
            a = np.abs(W[r, c * m:c * m + w])
            order = np.lexsort((np.arange(w), -a))  # primary -|w|, then offset
            expect = np.sort(order[:n])
            assert indices[r, c * n:(c + 1) * n].tolist() == expect.tolist()
            assert values[r, c * n:(c + 1) * n].tolist() == W[r, c * m + expect].tolist()


def test_n_equals_m_is_dense_matmul():
    rng = np.random.default_rng(7)
    M, K, N, m = 32, 40, 17, 4
    W = rng.standard_normal((M, K)).astype(np.float32)
    X = rng.standard_normal((K, N)).astype(np.float32)
    for g in (1, 4, 32):
        values, indices = oracle.compress(W, m, m, g)
        assert np.array_equal(indices, np.tile(np.arange(K) % m, (M // g, 1)))
        assert np.array_equal(values, W)
        Y, B = oracle.spmm(values, indices, X, K, m, m, g)
        ref = W.astype(np.float64) @ X.astype(np.float64)
        assert np.all(np.abs(Y - ref) <= 1e-13 * B)
        assert np.allclose(B, np.abs(W.astype(np.float64)) @ np.abs(X.astype(np.float64)),
                           rtol=1e-13, atol=0)


def test_g_equals_M_single_group():
    rng = np.random.default_rng(11)
    M, K, n, m = 16, 24, 2, 6
    W = rng.standard_normal((M, K)).astype(np.float32)
    values, indices = oracle.compress(W, n, m, M)
    assert indices.shape == (1, (K // m) * n)
    score = np.abs(W).sum(axis=0)  # exactness not needed: no near ties here
    for c in range(K // m):
        expect = np.sort(np.argsort(-score[c * m:(c + 1) * m], kind="stable")[:n])
        assert indices[0, c * n:(c + 1) * n].tolist() == expect.tolist()


# ----------------------------------------------------------------- invariants

CASES = [(2, 4, 4, 64, 40), (1, 4, 8, 64, 42), (1, 10, 16, 32, 92), (2, 8, 8, 48, 64),
         (1, 20, 32, 64, 48), (3, 5, 2, 10, 23), (4, 4, 1, 8, 16), (5, 9, 3, 9, 41)]


@pytest.mark.parametrize("n,m,g,M,K", CASES)
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_definition_invariants(n, m, g, M, K, dtype):
    rng = np.random.default_rng(M * K + n)
    W = (rng.standard_normal((M, K)) * 0.02).astype(dtype)
    W[0, :3] = 0.0
    W[1 % M, 1] = -0.0
    values, indices = oracle.compress(W, n, m, g)
    C = -(-K // m)
    Wd, mask = oracle.densify(values, indices, K, n, m, g)
    # densify(compress(W)) == W masked, bit for bit (sign of zeros included)
    assert np.array_equal(Wd.view(np.uint16 if dtype == np.float16 else np.uint32),
                          np.where(mask, W, np.zeros_like(W)).view(
                              np.uint16 if dtype == np.float16 else np.uint32))
    W32 = W.astype(np.float32)
    for G in range(M // g):
        rows = slice(G * g, G * g + g)
        # every row of a group has the same mask
        assert (mask[rows] == mask[G * g]).all()
        for c in range(C):
            w = chunk_width(K, m, c)
            cols = mask[G * g, c * m:c * m + w]
            assert cols.sum() == n  # exactly n kept per (row, chunk)
            off = indices[G, c * n:(c + 1) * n]
            assert (np.diff(off.astype(int)) > 0).all()
            s = np.zeros(w, np.float32)
            for i in range(g):
                s = s + np.abs(W32[G * g + i, c * m:c * m + w])
            kept, dropped = np.flatnonzero(cols), np.flatnonzero(~cols)
            for a in kept:
                for b in dropped:
                    assert s[a] > s[b] or (s[a] == s[b] and a < b)
    # values are the kept W entries in ascending column order
    for r in range(M):
        assert np.array_equal(values[r].view(np.uint8), W[r][mask[r]].view(np.uint8))


def test_sign_of_zero_and_ties_with_negative_zero():
    W = np.array([[-0.0, 0.0, 0.0, -0.0]], np.float32)
    values, indices = oracle.compress(W, 2, 4, 1)
    assert indices.tolist() == [[0, 1]]
    assert np.signbit(values[0, 0]) and not np.signbit(values[0, 1])


def test_nan_orders_above_every_number():
    W = np.array([[1.0, np.nan, np.inf, 2.0, np.nan, 0.5]], np.float32)
    _, indices = oracle.compress(W, 2, 6, 1)
    assert indices.tolist() == [[1, 4]]
    _, indices = oracle.compress(W, 3, 6, 1)
    assert indices.tolist() == [[1, 2, 4]]


# -------------------------------------------------------------------- energy

@pytest.mark.parametrize("n,m", [(2, 4), (1, 4), (2, 8), (1, 10)])
def test_energy_bounds_and_nesting(n, m):
    rng = np.random.default_rng(n * 100 + m)
    M, K = 64, 8 * m
    W = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    energies = {}
    for g in (1, 2, 4, 8, 16, 32, 64):
        values, indices = oracle.compress(W, n, m, g)
        energies[g] = oracle.energy(W, values)
        # per (group, chunk) the top n keep at least n/m of the group mass
        Wd, mask = oracle.densify(values, indices, K, n, m, g)
        A = np.abs(W.astype(np.float64))
        for G in range(M // g):
            for c in range(K // m):
                blk = (slice(G * g, G * g + g), slice(c * m, c * m + m))
                assert A[blk][mask[blk]].sum() >= n / m * A[blk].sum() * (1 - 1e-12)
    # the pattern chosen for g' is admissible for every g dividing g'
    gs = sorted(energies)
    for a, b in zip(gs, gs[1:]):
        assert energies[a] >= energies[b] - 1e-12
    assert energies[1] <= 1.0 and energies[64] >= n / m - 1e-12


# -------------------------------------------------------------- rejections

def test_rejections():
    W = np.zeros((8, 10), np.float32)
    with pytest.raises(oracle.OracleError) as e:
        oracle.compress(W, 3, 4, 1)  # tail width 2 < n = 3
    assert e.value.status == 2
    with pytest.raises(oracle.OracleError) as e:
        oracle.compress(W, 1, 4, 3)  # 8 rows not a multiple of g
    assert e.value.status == 2
    with pytest.raises(oracle.OracleError) as e:
        oracle.compress(W, 5, 4, 1)  # n > m
    assert e.value.status == 1
    with pytest.raises(oracle.OracleError) as e:
        oracle.compress(np.zeros((1, 300), np.float32), 1, 256, 1)  # m > 255
    assert e.value.status == 1
    values, indices = oracle.compress(W, 1, 4, 2)
    bad = indices.copy()
    bad[0, 2] = 2  # tail chunk has width 2: offset 2 is outside it
    with pytest.raises(oracle.OracleError) as e:
        oracle.densify(values, bad, 10, 1, 4, 2)
    assert e.value.status == 3
    values, indices = oracle.compress(W, 2, 4, 2)
    bad = indices.copy()
    bad[0, 0], bad[0, 1] = 1, 1  # not strictly ascending
    with pytest.raises(oracle.OracleError):
        oracle.spmm(values, bad, np.zeros((10, 3), np.float32), 10, 2, 4, 2)


# --------------------------------------------------------------- spmm parts

def test_spmm_points_match_full_product():
    rng = np.random.default_rng(5)
    M, K, N, n, m, g = 48, 70, 33, 2, 8, 8
    W = rng.standard_normal((M, K)).astype(np.float32)
    X = rng.standard_normal((K, N)).astype(np.float32)
    values, indices = oracle.compress(W, n, m, g)
    Y, B = oracle.spmm(values, indices, X, K, n, m, g, nthreads=2)
    rows = rng.integers(0, M, 50)
    cols = rng.integers(0, N, 50)
    yp, bp = oracle.spmm_points(values, indices, X, K, n, m, g, rows, cols)
    assert np.array_equal(yp, Y[rows, cols]) and np.array_equal(bp, B[rows, cols])
    Wd, _ = oracle.densify(values, indices, K, n, m, g)
    ref = Wd.astype(np.float64) @ X.astype(np.float64)
    assert np.all(np.abs(Y - ref) <= 1e-13 * B)


def test_spmm_thread_count_does_not_change_results():
    rng = np.random.default_rng(6)
    M, K, N = 64, 96, 40
    W = rng.standard_normal((M, K)).astype(np.float32)
    X = rng.standard_normal((K, N)).astype(np.float32)
    values, indices = oracle.compress(W, 1, 4, 8)
    Y1, B1 = oracle.spmm(values, indices, X, K, 1, 4, 8, nthreads=1)
    Y4, B4 = oracle.spmm(values, indices, X, K, 1, 4, 8, nthreads=4)
    assert np.array_equal(Y1, Y4) and np.array_equal(B1, B4)


# --------------------------------------------------------- binary16 helpers

def test_half_to_float_every_encoding():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float32)
    got = np.array([oracle.half_to_float(int(b)) for b in bits], np.float32)
    finite = np.isfinite(ref)
    assert np.array_equal(got[finite].view(np.uint32), ref[finite].view(np.uint32))
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    assert np.array_equal(got[np.isinf(ref)], ref[np.isinf(ref)])


def test_double_to_half_rounding():
    rng = np.random.default_rng(3)
    x = np.concatenate([
        rng.standard_normal(20000) * 10.0 ** rng.integers(-9, 6, 20000),
        # exact midpoints between neighbouring binary16 values (ties)
        (np.arange(0, 4096, dtype=np.float64) + 0.5) * 2.0 ** -24,
        (np.arange(1024, 2048, dtype=np.float64) + 0.5) * 2.0 ** -5,
        [65504.0, 65519.99, 65520.0, 1e6, -65520.0, 2.0 ** -25, 2.0 ** -26, 3 * 2.0 ** -26,
         -0.0, 0.0, np.inf, -np.inf],
    ])
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    got = oracle.round_to_half(x).view(np.uint16)
    assert np.array_equal(got, ref)
    f = x.astype(np.float32)
    with np.errstate(over="ignore"):
        f16 = f[:3000].astype(np.float16).view(np.uint16)
    assert all(oracle.float_to_half(float(v)) == int(r)
               for v, r in zip(f[:3000], f16))


def test_gelu_f16_matches_scipy_erf():
    from scipy.special import erf
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    x = bits.view(np.float16)
    x = x[np.isfinite(x)]
    got = oracle.gelu_f16(x)
    xd = x.astype(np.float64)
    ref64 = 0.5 * xd * (1.0 + erf(xd / math.sqrt(2.0)))
    ref = ref64.astype(np.float16)
    # scipy's erf and libm's erf may differ in the last binary64 bits; that can
    # only flip the binary16 rounding when the value sits on a midpoint
    differ = got.view(np.uint16) != ref.view(np.uint16)
    if differ.any():
        lo = np.minimum(got[differ], ref[differ]).astype(np.float64)
        hi = np.maximum(got[differ], ref[differ]).astype(np.float64)
        mid = (lo + hi) / 2
        assert np.all(np.abs(ref64[differ] - mid) <= 1e-12 * np.abs(mid) + 1e-300)
    assert got[x == 0].astype(np.float64).tolist() == [0.0] * int((x == 0).sum())


def test_add_f16_is_correctly_rounded():
    rng = np.random.default_rng(9)
    a = (rng.standard_normal(50000) * 10.0 ** rng.integers(-4, 4, 50000)).astype(np.float16)
    b = (rng.standard_normal(50000) * 10.0 ** rng.integers(-4, 4, 50000)).astype(np.float16)
    ref = (a.astype(np.float64) + b.astype(np.float64)).astype(np.float16)
    assert np.array_equal(oracle.add_f16(a, b).view(np.uint16), ref.view(np.uint16))


def test_linear_stack_layer_dense_control():
    """With n = m the stack layer is dense: compare with NumPy matmuls, SciPy's
    erf and NumPy's binary16 rounding."""
    from scipy.special import erf
    rng = np.random.default_rng(12)
    d, f, T, m = 16, 32, 8, 4
    x = rng.standard_normal((d, T)).astype(np.float16)
    Ws = {k: (rng.standard_normal(s) * 0.02).astype(np.float16)
          for k, s in (("qkv", (3 * d, d)), ("ao", (d, d)), ("up", (f, d)), ("down", (d, f)))}
    packed = {}
    for k, W in Ws.items():
        v, idx = oracle.compress(W, m, m, 4)
        packed[k] = (v, idx, W.shape[1])
    got = oracle.linear_stack_layer(x, packed, m, m, 4)

    def lin(W, inp):
        return (W.astype(np.float64) @ inp.astype(np.float64)).astype(np.float16)

    qkv = lin(Ws["qkv"], x)
    h = (x.astype(np.float64) + lin(Ws["ao"], qkv[2 * d:]).astype(np.float64)).astype(np.float16)
    u = lin(Ws["up"], h).astype(np.float64)
    gl = (0.5 * u * (1 + erf(u / math.sqrt(2)))).astype(np.float16)
    ref = (h.astype(np.float64) + lin(Ws["down"], gl).astype(np.float64)).astype(np.float16)
    # binary64 sums in a different order may flip a binary16 rounding by 1 ulp
    diff = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    ulp = np.spacing(np.abs(ref).astype(np.float16)).astype(np.float64)
    assert np.all(diff <= ulp)


# --------------------------------------------------------- fixed-mask repack

def test_repack_hand_example():
    gold = load_golden("repack_2_4_2.json")
    W2 = np.array(gold["W2"], np.float32)
    idx = np.array(gold["indices"], np.uint8)
    got = oracle.repack(W2, idx, gold["n"], gold["m"], gold["g"])
    want = np.array(gold["values"], np.float32)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))  # -0 kept


@pytest.mark.parametrize("n,m,g,M,K,dtype", [
    (2, 4, 4, 16, 22, np.float32), (1, 10, 8, 16, 33, np.float16), (3, 8, 2, 6, 21, np.float32),
    (4, 4, 1, 5, 12, np.float16), (1, 1, 3, 9, 7, np.float32)])
def test_repack_agrees_with_compress_and_densify(n, m, g, M, K, dtype):
    """Against two independently pinned parts of the oracle: re-packing W into
    its own pattern gives the converter's values, and any other weight packed
    into that pattern densifies to that weight masked by the pattern."""
    rng = np.random.default_rng(M * K + n)
    W = rng.standard_normal((M, K)).astype(dtype)
    values, indices = oracle.compress(W, n, m, g)
    assert np.array_equal(oracle.repack(W, indices, n, m, g).view(np.uint8), values.view(np.uint8))
    W2 = rng.standard_normal((M, K)).astype(dtype)
    W2[0, 0] = -0.0
    v2 = oracle.repack(W2, indices, n, m, g)
    dense, mask = oracle.densify(v2, indices, K, n, m, g)
    want = np.where(mask, W2, np.zeros_like(W2))
    assert np.array_equal(dense.view(np.uint8), want.view(np.uint8))
    assert mask.sum() == M * n * n_chunks_of(K, m)


def n_chunks_of(K, m):
    return -(-K // m)


def test_repack_rejects_invalid_indices():
    W = np.zeros((4, 10), np.float32)
    values, indices = oracle.compress(W, 1, 4, 2)
    bad = indices.copy()
    bad[1, 2] = 3  # tail chunk of width 2
    with pytest.raises(oracle.OracleError) as e:
        oracle.repack(W, bad, 1, 4, 2)
    assert e.value.status == 3
