"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bars (written out in each check):
  - indices, masks, values, densified weights: bit-exact;
  - binary32 products: |Y - Y_ref| <= 1e-5 * (|W_s| |X|) elementwise;
  - binary16 in / binary32 accumulate: |Y - Y_ref| <= 2e-2 * (|W_s| |X|), and
    the tighter bound of exact binary16 products summed in binary32 and
    rounded once to binary16 (tight_f16_bound), which one dropped or
    misplaced k-slot exceeds;
  - residual add: bit-exact (binary32 holds the binary16 sum exactly enough
    for one correct rounding); GELU: within one binary16 ulp.
Y_ref and |W_s| |X| come from the oracle in binary64 on the same inputs.

Paper: STen (arXiv 2304.07613) Section 5 (layout), 5.1 (product), 5.2
(converter, conversion back to dense).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2304_07613_amd import build, synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = {torch.float32: 1e-5, torch.float16: 2e-2}


@pytest.fixture(scope="module")
def nmg():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2304_07613_amd import nmg as binding
    binding.lib()  # raises if the library is not built: no fallback
    return binding


def np_of(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


def bits(a: np.ndarray) -> np.ndarray:
    return a.view(np.uint16 if a.dtype == np.float16 else np.uint32)


def check_compress(nmg, W, n, m, g, tag=""):
    """GPU compress == oracle compress, bit for bit; returns both packings."""
    print(f"[compress] {tag} W{tuple(W.shape)} {W.dtype} {n}:{m}:{g}", flush=True)
    v, idx, L = nmg.compress(W.to(DEV), n, m, g)
    torch.cuda.synchronize()
    rv, ridx = oracle.compress(np_of(W), n, m, g)
    gv, gidx = np_of(v), np_of(idx)
    assert np.array_equal(gidx, ridx), f"indices differ at {np.argwhere(gidx != ridx)[:5]}"
    assert np.array_equal(bits(gv), bits(rv)), "values differ"
    return v, idx, L, rv, ridx


def tight_f16_bound(Yref, B, keff):
    """A binary16 bound that one dropped or misplaced k-slot exceeds.

    Binary16 products are exact in binary32, so the binary32 sum of k_eff of
    them is within k_eff * 2^-24 * B of the exact sum (B = |W_s| |X|; factor 2
    of slack for the instruction's internal order), and rounding that sum to
    binary16 adds at most 2^-11 of its magnitude, or 2^-25 below binary16's
    normal range."""
    acc = 2.0 * keff * 2.0 ** -24 * B
    return 2.0 ** -11 * (np.abs(Yref) + acc) + acc + 2.0 ** -25


def check_product(Y, Yref, B, dtype, what="", keff=None):
    """|Y - Y_ref| within the contract bound (1e-5 B in binary32, 2e-2 B in
    binary16) and, for binary16, also within tight_f16_bound; returns the
    worst |Y - Y_ref| / B."""
    Yg = np_of(Y).astype(np.float64)
    err = np.abs(Yg - Yref)
    bounds = [("contract", TOL[dtype] * B)]
    if dtype == torch.float16:
        assert keff is not None, "binary16 checks need k_eff"
        bounds.append(("tight binary16", tight_f16_bound(Yref, B, keff)))
    for name, bound in bounds:
        bad = err > bound
        if bad.any():
            i = np.argwhere(bad)[0]
            raise AssertionError(f"{what}: {bad.sum()} outputs out of the {name} bound; first "
                                 f"{tuple(i)}: gpu {Yg[tuple(i)]!r} ref {Yref[tuple(i)]!r} "
                                 f"bound {bound[tuple(i)]!r}")
    nz = B > 0
    return float((err[nz] / B[nz]).max()) if nz.any() else 0.0


def spmm_full(nmg, v, idx, L, X, rv, ridx, kernel, tag=""):
    """Full comparison; returns None when `kernel` does not take this layout."""
    print(f"[spmm] {tag} {L} N={X.shape[1]} kernel={kernel}", flush=True)
    try:
        Y = nmg.spmm(v, idx, X.to(DEV), L, kernel)
    except nmg.NmgError as e:
        if e.status == nmg.ERR_UNSUPPORTED and kernel not in ("auto", "valu"):
            return None
        raise
    torch.cuda.synchronize()
    Yref, B = oracle.spmm(rv, ridx, np_of(X), L.K, L.n, L.m, L.g)
    return check_product(Y, Yref, B, L.dtype, f"{tag} {kernel}", L.C * L.n)


# every kernel family; the matrix-core ones decline layouts they cannot take
KERNELS = ["auto", "valu", "mfma_general", "mfma_scalar", "mfma_f16", "mfma_direct", "smfmac_f16",
           "valu_staged", "mfma_wide", "mfma_split", "mfma_expand"]


def kernels_for(nmg, L, N):
    return KERNELS


# ------------------------------------------------------ small, multi-tile

SMALL = [
    # M,   K,   N,   n, m,   g,   dtype
    (256, 64, 64, 2, 4, 4, torch.float32),      # exactly one workgroup tile
    (264, 70, 200, 2, 4, 8, torch.float32),     # ragged rows, K tail 2, ragged N
    (520, 100, 130, 1, 10, 8, torch.float32),   # 1:10 windows, M % 256 != 0
    (384, 96, 1000, 1, 4, 32, torch.float32),   # g = 32, many token tiles
    (128, 96, 77, 2, 8, 16, torch.float16),     # binary16, ragged N
    (64, 68, 65, 1, 20, 4, torch.float32),      # 1:20, tail chunk of 8
    (96, 64, 33, 3, 5, 3, torch.float32),       # n = 3, g = 3: vector kernel only
    (48, 40, 9, 4, 4, 1, torch.float32),        # dense control, g = 1
    (32, 33, 5, 1, 1, 2, torch.float32),        # m = 1: every column kept
    (8, 255, 3, 7, 255, 8, torch.float32),      # m = 255, one chunk
    (4, 4, 1, 1, 4, 4, torch.float32),          # one group, one chunk, N = 1
    (768, 64, 40, 2, 4, 768, torch.float32),    # g = M
    (96, 48, 300, 2, 4, 12, torch.float16),     # g = 12 (unit of 4 rows)
    (512, 128, 260, 4, 8, 8, torch.float32),    # n = 4
    # binary16 matrix cores (N % 8 == 0): ragged row and token tiles, one
    # ragged window with unaligned value rows (C*n = 18)
    (264, 72, 264, 2, 8, 8, torch.float16),
    (512, 200, 520, 1, 4, 8, torch.float16),    # two windows, the last one ragged
    (384, 768, 1024, 2, 8, 16, torch.float16),  # units of 16 rows, 6 windows
    (192, 100, 136, 1, 10, 4, torch.float16),   # 1:10, windows of 8 k-slots, units of 4
    (96, 48, 304, 2, 4, 12, torch.float16),     # g = 12
    (64, 40, 8, 4, 4, 1, torch.float16),        # dense control, N = 8
    (128, 84, 40, 1, 20, 32, torch.float16),    # 1:20, windows of 4 k-slots, tail 4
    # gathering kernel: many windows split unevenly over waves, n above the
    # window, a last window past the k-slots
    (272, 3000, 70, 1, 10, 16, torch.float32),
    (64, 40, 21, 16, 20, 4, torch.float32),     # n = 16 > 8 k-slots per window
    (1024, 300, 1, 2, 4, 8, torch.float32),     # one token, 150 k-slots
    # binary16 on the sparse matrix instruction (n <= 2, m in {4, 8, 16},
    # C * n % 8 == 0): ragged row and token tiles, g = 1, a tail chunk and a
    # partial last step of 64 columns
    (200, 256, 136, 2, 8, 1, torch.float16),
    (72, 192, 24, 1, 4, 2, torch.float16),
    (128, 92, 64, 2, 8, 8, torch.float16),      # tail chunk of 4, 92 % 64 != 0
    (16, 128, 8, 1, 16, 16, torch.float16),
    (512, 256, 512, 2, 4, 4, torch.float16),
    (32, 1024, 264, 2, 16, 32, torch.float16),
    # the LDS-staged vector kernel: g = 1 and 3, n = 3 and 5, chunks of 32,
    # ragged rows and tokens, a last window past the chunks
    (200, 256, 516, 1, 4, 1, torch.float32),
    (96, 100, 260, 3, 8, 3, torch.float32),
    (70, 90, 64, 5, 32, 1, torch.float32),
    (64, 770, 1028, 2, 10, 2, torch.float32),
    # binary16 with 4 tokens per lane (enough rows x tokens for 8 waves of
    # 256-token tiles per CU): swizzled staging, a ragged last token tile
    (2048, 64, 4096, 2, 8, 8, torch.float16),
    (2048, 72, 4104, 1, 4, 16, torch.float16),
    (2048, 64, 4096, 4, 8, 8, torch.float16),   # n = 4: k-groups of one chunk
    (2048, 36, 4096, 2, 4, 4, torch.float16),   # C * n = 18: unaligned rows, a part-filled chunk block
    # binary16 staging by chunk class: n above 2, a window past the chunks
    (128, 96, 136, 4, 8, 8, torch.float16),
    (64, 128, 72, 8, 16, 4, torch.float16),
    (96, 200, 264, 2, 8, 8, torch.float16),     # 25 chunks in one window of 32
]


@pytest.mark.parametrize("M,K,N,n,m,g,dtype", SMALL,
                         ids=[f"{c[0]}x{c[1]}x{c[2]}-{c[3]}:{c[4]}:{c[5]}-{str(c[6])[6:]}"
                              for c in SMALL])
def test_small_shapes(nmg, M, K, N, n, m, g, dtype):
    W = synth.normal((M, K), 11 + M + K, 0.02, dtype)
    X = synth.normal((K, N), 12 + N, 1.0, dtype)
    v, idx, L, rv, ridx = check_compress(nmg, W, n, m, g, "small")
    dense = nmg.densify(v, idx, L)
    rd, _ = oracle.densify(rv, ridx, K, n, m, g)
    assert np.array_equal(bits(np_of(dense)), bits(rd))
    for kernel in kernels_for(nmg, L, N):
        spmm_full(nmg, v, idx, L, X, rv, ridx, kernel, "small")


def random_layouts(count=100, seed=2304):
    """Seeded random layouts across the whole parameter space the product
    takes (n and m of every size class, any g, a ragged tail chunk, ragged
    token counts, both element types), each small enough for the oracle."""
    rng = np.random.RandomState(seed)
    out = []
    while len(out) < count:
        m = int(rng.choice([1, 2, 3, 4, 5, 6, 8, 10, 12, 16, 20, 24, 32, 40]))
        n = min(m, int(rng.choice([1, 1, 2, 2, 3, 4, 8, 16])))
        g = int(rng.choice([1, 2, 3, 4, 8, 12, 16, 32]))
        C = int(rng.randint(1, 41))
        r = m if rng.rand() < 0.5 else int(rng.randint(n, m + 1))   # tail width, >= n
        K = (C - 1) * m + r
        M = g * int(rng.randint(1, max(2, 512 // g)))
        dtype = torch.float16 if rng.rand() < 0.5 else torch.float32
        N = 8 * int(rng.randint(1, 40)) if rng.rand() < 0.6 else int(rng.randint(1, 300))
        if M * C * n * N > 20_000_000:
            continue
        out.append((M, K, N, n, m, g, dtype))
    return out


RANDOM = random_layouts()


@pytest.mark.parametrize("M,K,N,n,m,g,dtype", RANDOM,
                         ids=[f"r{i}-{c[0]}x{c[1]}x{c[2]}-{c[3]}:{c[4]}:{c[5]}-{str(c[6])[6:]}"
                              for i, c in enumerate(RANDOM)])
def test_random_layouts(nmg, M, K, N, n, m, g, dtype):
    W = synth.normal((M, K), 21 + M + 7 * K, 0.02, dtype)
    X = synth.normal((K, N), 22 + N + 3 * K, 1.0, dtype)
    v, idx, L, rv, ridx = check_compress(nmg, W, n, m, g, "random")
    dense = nmg.densify(v, idx, L)
    rd, _ = oracle.densify(rv, ridx, K, n, m, g)
    assert np.array_equal(bits(np_of(dense)), bits(rd))
    for kernel in kernels_for(nmg, L, N):
        spmm_full(nmg, v, idx, L, X, rv, ridx, kernel, "random")


def random_x16(count=40, seed=2308):
    """Seeded random layouts the 16 x 16 x 32 products take (n of 1 or 2, g a
    multiple of 8, binary16 m % 4 == 0 up to 12, binary32 m up to 4 / 8),
    ragged tail chunks, rows and token tiles, with weight and X scales spread
    over six decades (binary32: the split products' per-unit weight scaling;
    X kept at |x| >= 1e-3 standard deviation, where their error bound is well
    inside 1e-5 B)."""
    rng = np.random.RandomState(seed)
    out = []
    while len(out) < count:
        dtype = torch.float16 if rng.rand() < 0.5 else torch.float32
        n = int(rng.choice([1, 2]))
        if dtype == torch.float16:
            m = 4 if n == 1 else int(rng.choice([4, 8, 12]))
        else:
            m = int(rng.randint(n, (4 if n == 1 else 8) + 1))
        g = int(rng.choice([8, 8, 16, 24, 32, 64]))
        C = int(rng.randint(1, 60))
        r = m if rng.rand() < 0.5 else int(rng.randint(n, m + 1))
        K = (C - 1) * m + r
        M = g * int(rng.randint(1, max(2, 1024 // g)))
        N = (8 if dtype == torch.float16 else 4) * int(rng.randint(1, 80))
        wscale = 10.0 ** rng.uniform(-3, 3) if dtype == torch.float32 else 1.0
        xscale = 10.0 ** rng.uniform(-3, 3) if dtype == torch.float32 else 10.0 ** rng.uniform(-2, 1)
        if M * C * n * N > 30_000_000:
            continue
        out.append((M, K, N, n, m, g, dtype, wscale, xscale))
    return out


X16_RANDOM = random_x16()


@pytest.mark.parametrize("M,K,N,n,m,g,dtype,wscale,xscale", X16_RANDOM,
                         ids=[f"x{i}-{c[0]}x{c[1]}x{c[2]}-{c[3]}:{c[4]}:{c[5]}-{str(c[6])[6:]}"
                              for i, c in enumerate(X16_RANDOM)])
def test_x16_random(nmg, M, K, N, n, m, g, dtype, wscale, xscale):
    """The 16 x 16 x 32 product on operands prepared once, against the
    oracle in full (binary16: the contract and the tight bound; binary32
    through binary16 parts: 1e-5 B), and the per-call path bit for bit."""
    W = synth.normal((M, K), 41 + M + 5 * K, 0.02 * wscale, dtype)
    X = synth.normal((K, N), 42 + N + 3 * K, xscale, dtype)
    if dtype == torch.float32 and M >= 16:
        W[:8] *= 1e-20      # a unit of tiny weights and one of large ones:
        W[8:16] *= 1e20     # the per-unit scaling keeps both exact enough
    v, idx, L, rv, ridx = check_compress(nmg, W, n, m, g, "x16")
    kernel = "mfma_wide" if dtype == torch.float16 else "mfma_split"
    print(f"[x16] {L} N={N} wscale={wscale:.3g} xscale={xscale:.3g}", flush=True)
    prepared = nmg.x16_prepare(v, idx, L)
    Xd = X.to(DEV)
    Y = nmg.spmm_x16_epilogue(L, prepared, Xd)
    Y2 = nmg.spmm(v, idx, Xd, L, kernel)
    torch.cuda.synchronize()
    assert torch.equal(Y.view(torch.uint8), Y2.view(torch.uint8))
    Yref, B = oracle.spmm(rv, ridx, np_of(X), K, n, m, g)
    check_product(Y, Yref, B, dtype, f"x16 {kernel}", L.C * L.n)


@pytest.mark.parametrize("M,N", [(3072, 4096), (3072, 3960), (2304, 4096), (2304, 3960)])
def test_x16_two_tiles(nmg, M, N):
    """Layers whose one-tile grid takes two rounds of workgroups (FFN up and
    QKV shapes, 2:8:8 binary16) run two token tiles per workgroup, the second
    tile's windows staged while the first tile's outputs drain; 3960 tokens
    leave the last workgroup one ragged tile.  Every output is bit for bit
    what the one-tile launch gives on column blocks of 1024 tokens (its grid
    fits one round), also with the residual sum and on row-strided operands,
    and sampled outputs meet the bound against the oracle."""
    K, n, m, g = 768, 2, 8, 8
    W = synth.normal((M, K), 51 + M, 0.02, torch.float16)
    X = synth.normal((K, N), 52 + N, 1.0, torch.float16)
    R = synth.normal((M, N), 53 + N, 1.0, torch.float16).to(DEV)
    v, idx, L, rv, ridx = check_compress(nmg, W, n, m, g, "two tiles")
    print(f"[x16 two tiles] {L} N={N}", flush=True)
    prepared = nmg.x16_prepare(v, idx, L)
    Xd = X.to(DEV)
    Y = nmg.spmm_x16_epilogue(L, prepared, Xd)
    Ya = nmg.spmm_x16_epilogue(L, prepared, Xd, "add", R)
    Yb = torch.full_like(Y, 7.0)
    Yab = torch.full_like(Y, 7.0)
    for c0 in range(0, N, 1024):
        c1 = min(N, c0 + 1024)
        nmg.spmm_x16_epilogue(L, prepared, Xd[:, c0:c1], Y=Yb[:, c0:c1])
        nmg.spmm_x16_epilogue(L, prepared, Xd[:, c0:c1], "add", R[:, c0:c1], Y=Yab[:, c0:c1])
    # the two-tile launch on row-strided X, R and Y (views of wider buffers)
    Xw = torch.zeros((K, N + 64), dtype=torch.float16, device=DEV)
    Rw = torch.zeros((M, N + 72), dtype=torch.float16, device=DEV)
    Yw = torch.full((M, N + 40), 7.0, dtype=torch.float16, device=DEV)
    Xw[:, :N] = Xd
    Rw[:, 8:N + 8] = R
    nmg.spmm_x16_epilogue(L, prepared, Xw[:, :N], "add", Rw[:, 8:N + 8], Y=Yw[:, :N])
    torch.cuda.synchronize()
    assert torch.equal(Y.view(torch.int16), Yb.view(torch.int16))
    assert torch.equal(Ya.view(torch.int16), Yab.view(torch.int16))
    assert torch.equal(Yw[:, :N].view(torch.int16), Ya.view(torch.int16))
    assert bool((Yw[:, N:] == 7.0).all())
    check_sampled(nmg, v, idx, L, X, Y, rv, ridx, what="x16 two tiles")


def random_large(count=12, seed=2306):
    """Seeded random layouts at the workloads' scale (the launch shapes small
    cases never reach: 4 tokens per lane, several rounds of workgroups,
    k-splits), checked on sampled outputs."""
    rng = np.random.RandomState(seed)
    out = []
    for _ in range(count):
        n, m = [(2, 4), (1, 4), (2, 8), (1, 10), (1, 20), (4, 8), (1, 2)][rng.randint(7)]
        g = int(rng.choice([1, 4, 8, 16, 32]))
        M = g * int(rng.randint(max(1, 512 // g), 3072 // g + 1))
        K = int(rng.choice([384, 768, 1000, 2048, 3072]))
        N = int(rng.choice([512, 1024, 2048, 4096, 4104, 3000]))
        dtype = torch.float16 if rng.rand() < 0.5 else torch.float32
        out.append((M, K, N, n, m, g, dtype))
    return out


LARGE = random_large()


@pytest.mark.parametrize("M,K,N,n,m,g,dtype", LARGE,
                         ids=[f"L{i}-{c[0]}x{c[1]}x{c[2]}-{c[3]}:{c[4]}:{c[5]}-{str(c[6])[6:]}"
                              for i, c in enumerate(LARGE)])
def test_random_large(nmg, M, K, N, n, m, g, dtype):
    """Compress compared in full; every kernel family's product on 30000
    sampled outputs (every token tile and row tile hit) against the oracle."""
    W = synth.normal((M, K), 31 + M + K, 0.02, dtype)
    X = synth.normal((K, N), 32 + N, 1.0, dtype)
    v, idx, L, rv, ridx = check_compress(nmg, W, n, m, g, "large")
    rng = np.random.RandomState(M * 7 + N)
    rows = rng.randint(0, M, 30000)
    cols = rng.randint(0, N, 30000)
    Yref, B = oracle.spmm_points(rv, ridx, np_of(X), K, n, m, g, rows, cols)
    Xd = X.to(DEV)
    for kernel in kernels_for(nmg, L, N):
        print(f"[spmm] large {L} N={N} kernel={kernel}", flush=True)
        try:
            Y = nmg.spmm(v, idx, Xd, L, kernel)
        except nmg.NmgError as e:
            if e.status == nmg.ERR_UNSUPPORTED and kernel not in ("auto", "valu"):
                continue
            raise
        torch.cuda.synchronize()
        check_product(Y[torch.as_tensor(rows, device=Y.device),
                        torch.as_tensor(cols, device=Y.device)], Yref, B, dtype,
                      f"large {kernel}", L.C * L.n)


@pytest.mark.parametrize("M,K,N,n,m,g,xoff", [
    (3072, 768, 1030, 1, 10, 4, 0), (3056, 768, 1030, 1, 20, 8, 0),
    (768, 3072, 2046, 1, 10, 16, 0), (3072, 768, 1024, 1, 20, 4, 1),
    (768, 768, 130, 2, 4, 4, 0), (768, 768, 127, 1, 10, 16, 0), (1536, 768, 200, 1, 20, 8, 1)])
def test_gather_shapes(nmg, M, K, N, n, m, g, xoff):
    """The gathering kernel in both its shapes (4 tokens a lane when the
    256-token tiles cover the CUs, else the k-split one): ragged token tiles,
    N % 4 != 0 and X rows off 16-byte alignment (element loads), a partial
    row tile, against the oracle on sampled outputs."""
    W = synth.normal((M, K), 51 + M + K, 0.02, torch.float32)
    X = synth.normal((K, N), 52 + N, 1.0, torch.float32)
    v, idx, L, rv, ridx = check_compress(nmg, W, n, m, g, "gather")
    Xb = torch.zeros((K, N + 4), dtype=torch.float32, device=DEV)
    Xd = Xb[:, xoff:xoff + N]
    Xd.copy_(X.to(DEV))
    print(f"[spmm] gather {L} N={N} xoff={xoff}", flush=True)
    Y = nmg.spmm(v, idx, Xd, L, "mfma_direct")
    torch.cuda.synchronize()
    check_sampled(nmg, v, idx, L, X, Y, rv, ridx, count=8192, seed=M + N, what="gather")


# ------------------------------------------------------ fixed-mask repack

def random_patterns(rng, groups, K, n, m):
    """Valid index rows drawn at random (not from the converter)."""
    C = -(-K // m)
    idx = np.empty((groups, C * n), np.uint8)
    for G in range(groups):
        for c in range(C):
            w = min(m, K - c * m)
            idx[G, c * n:(c + 1) * n] = np.sort(rng.choice(w, n, replace=False))
    return idx


@pytest.mark.parametrize("M,K,n,m,g,dtype", [
    (64, 70, 2, 4, 8, torch.float32), (96, 300, 1, 10, 16, torch.float16),
    (40, 35, 3, 8, 4, torch.float32), (3072, 768, 1, 4, 8, torch.float32),
    (2304, 768, 2, 8, 8, torch.float16), (8, 255, 7, 255, 2, torch.float16)])
def test_repack(nmg, M, K, n, m, g, dtype):
    rng = np.random.default_rng(M + K)
    W = synth.normal((M, K), 61 + M, 0.02, dtype)
    idx = random_patterns(rng, M // g, K, n, m)
    print(f"[repack] {M}x{K} {n}:{m}:{g} {dtype}", flush=True)
    L = nmg.Layout(M, K, n, m, g, dtype)
    v = nmg.repack(W.to(DEV), torch.from_numpy(idx).to(DEV), L)
    torch.cuda.synchronize()
    rv = oracle.repack(np_of(W), idx, n, m, g)
    assert np.array_equal(bits(np_of(v)), bits(rv))
    # a weight re-packed into its own pattern gives the converter's values
    v2, idx2, L2 = nmg.compress(W.to(DEV), n, m, g)
    assert torch.equal(nmg.repack(W.to(DEV), idx2, L2).view(torch.uint8), v2.view(torch.uint8))


# --------------------------------------------------------- fused epilogues

@pytest.mark.parametrize("M,K,N,n,m,g,dtype", [
    (264, 72, 264, 2, 8, 8, torch.float16), (768, 768, 4096, 2, 8, 8, torch.float16),
    (3072, 768, 512, 2, 8, 8, torch.float16), (96, 48, 77, 2, 4, 12, torch.float16),
    (128, 100, 136, 1, 10, 4, torch.float32), (64, 40, 33, 3, 8, 2, torch.float32),
    (200, 64, 96, 1, 4, 8, torch.float16), (272, 96, 136, 2, 4, 16, torch.float32),
    (136, 40, 260, 1, 4, 8, torch.float32)])
def test_spmm_epilogue_equals_composition(nmg, M, K, N, n, m, g, dtype):
    """GELU / residual folded into the product give the bits of the product
    followed by nmg_gelu / nmg_add, for every kernel family that takes the
    layout; the pieces themselves are checked against the oracle elsewhere."""
    W = synth.normal((M, K), 71 + M, 0.02, dtype).to(DEV)
    X = synth.normal((K, N), 72 + N, 1.0, dtype).to(DEV)
    R = synth.normal((M, N), 73 + N, 1.0, dtype).to(DEV)
    v, idx, L = nmg.compress(W, n, m, g)
    for kernel in KERNELS:
        print(f"[epilogue] {M}x{K}x{N} {n}:{m}:{g} {dtype} kernel={kernel}", flush=True)
        try:
            P = nmg.spmm(v, idx, X, L, kernel)
        except nmg.NmgError as e:
            assert e.status == nmg.ERR_UNSUPPORTED and kernel not in ("auto", "valu")
            continue
        Yg = nmg.spmm_epilogue(v, idx, X, L, "gelu", kernel=kernel)
        Ya = nmg.spmm_epilogue(v, idx, X, L, "add", R, kernel=kernel)
        Yn = nmg.spmm_epilogue(v, idx, X, L, "none", kernel=kernel)
        torch.cuda.synchronize()
        assert torch.equal(Yn.view(torch.uint8), P.view(torch.uint8))
        assert torch.equal(Yg.view(torch.uint8), nmg.gelu(P).view(torch.uint8)), kernel
        assert torch.equal(Ya.view(torch.uint8), nmg.add(P, R).view(torch.uint8)), kernel
    # strided Y and R (the second pass runs row by row on the unfused families)
    Yb = torch.zeros((M, N + 8), dtype=dtype, device=DEV)
    Rb = torch.zeros((M, N + 8), dtype=dtype, device=DEV)
    Rb[:, :N] = R
    Ys = nmg.spmm_epilogue(v, idx, X, L, "add", Rb[:, :N], Y=Yb[:, :N])
    torch.cuda.synchronize()
    assert torch.equal(Ys.view(torch.uint8), nmg.add(nmg.spmm(v, idx, X, L), R).view(torch.uint8))
    assert (Yb[:, N:] == 0).all()
    # the same through prepared operands, when these products take the layout
    x16 = "mfma_wide" if dtype == torch.float16 else "mfma_split"
    try:
        prepared = nmg.x16_prepare(v, idx, L)
    except nmg.NmgError as e:
        assert e.status == nmg.ERR_UNSUPPORTED
        return
    if N % (8 if dtype == torch.float16 else 4):
        return
    Yb.zero_()
    Ys = nmg.spmm_x16_epilogue(L, prepared, X, "add", Rb[:, :N], Y=Yb[:, :N])
    torch.cuda.synchronize()
    P = nmg.spmm(v, idx, X, L, x16)
    assert torch.equal(Ys.view(torch.uint8), nmg.add(P, R).view(torch.uint8))
    assert (Yb[:, N:] == 0).all()
    Yb.zero_()
    Ys = nmg.spmm_x16_epilogue(L, prepared, X, "gelu", Y=Yb[:, :N])
    torch.cuda.synchronize()
    assert torch.equal(Ys.view(torch.uint8), nmg.gelu(P).view(torch.uint8))
    assert (Yb[:, N:] == 0).all()


def test_x16_gelu_every_input(nmg):
    """GELU folded into the 16 x 16 x 32 product against the product followed
    by nmg_gelu, on a product that reproduces every binary16 bit pattern
    (except -0): each 8-row group keeps weight 1 at one X row of its own that
    holds 256 of the patterns, every other kept weight is 0 on finite X."""
    C, N, groups = 43, 256, 256
    M, K = 8 * groups, 8 * C
    W = torch.zeros((M, K), dtype=torch.float16)
    sel = []
    for G in range(groups):
        col = 8 * (G % C) + 2 + G // C     # offsets 2..7: no other group keeps it
        W[8 * G:8 * G + 8, col] = 1.0
        sel.append(col)
    X = synth.normal((K, N), 808, 1.0, torch.float16)
    patt = torch.arange(65536, dtype=torch.int32).to(torch.int16).view(torch.float16)
    for G, col in enumerate(sel):
        X[col] = patt[G * N:(G + 1) * N]
    v, idx, L = nmg.compress(W.to(DEV), 2, 8, 8)
    Xd = X.to(DEV)
    prepared = nmg.x16_prepare(v, idx, L)
    P = nmg.spmm_x16_epilogue(L, prepared, Xd)
    Yg = nmg.spmm_x16_epilogue(L, prepared, Xd, "gelu")
    torch.cuda.synchronize()
    Pb = np_of(P).view(np.uint16)
    want = np_of(X).view(np.uint16)[sel].repeat(8, axis=0)
    want = np.where(want == 0x8000, 0, want)       # -0 + (+0 products) = +0
    nan = (want & 0x7c00) == 0x7c00
    nan &= (want & 0x03ff) != 0
    assert np.array_equal(Pb[~nan], want[~nan]) and ((Pb[nan] & 0x7c00) == 0x7c00).all()
    assert torch.equal(Yg.view(torch.uint8), nmg.gelu(P).view(torch.uint8))


def test_stack_graph_replay(nmg):
    """Two BERT layers captured in a HIP graph: every replay, with eager work
    and synchronisations between the replays, gives the eager forward's bits,
    also after the input changes."""
    from paper_2304_07613_amd.stack import LinearStack
    stack = LinearStack.from_workload(4, nmg, n_layers=2, keep_dense=False)
    x = synth.normal((synth.BERT_HIDDEN, synth.BERT_TOKENS), synth.seed_for(4, 0, "X"), 1.0,
                     torch.float16).to(DEV)
    graph, y = stack.capture(x)
    for rep in range(4):
        if rep == 2:   # new input, written in place
            x.copy_(synth.normal(tuple(x.shape), 4321, 1.0, torch.float16).to(DEV))
        eager = stack.forward(x)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), eager.view(torch.int16)), f"replay {rep}"


def test_stack_fused_equals_stepwise(nmg):
    """One BERT layer: the fused forward gives the bits of the step-by-step
    forward whose every step the stack test checks against the oracle."""
    from paper_2304_07613_amd.stack import LinearStack
    stack = LinearStack.from_workload(4, nmg, n_layers=2, keep_dense=False)
    x = synth.normal((synth.BERT_HIDDEN, synth.BERT_TOKENS), synth.seed_for(4, 0, "X"), 1.0,
                     torch.float16).to(DEV)
    for layer in stack.layers:
        fused = stack.forward_layer(layer, x)
        stepwise = stack.forward_layer(layer, x, trace={})
        torch.cuda.synchronize()
        assert torch.equal(fused.view(torch.uint8), stepwise.view(torch.uint8))
        x = fused


# ----------------------------------------------------------- edge cases

def test_ties_signed_zeros_and_nan(nmg):
    rng = np.random.default_rng(1)
    W = (rng.integers(-4, 5, size=(64, 96)) / 4.0).astype(np.float32)  # many ties
    W[0, :8] = -0.0
    W[3, 10] = np.nan
    W[9, 20] = np.inf
    W[17, 30:34] = np.nan
    Wt = torch.from_numpy(W)
    for n, m, g in [(2, 4, 4), (1, 4, 8), (2, 8, 16), (3, 8, 1), (1, 10, 2)]:
        check_compress(nmg, Wt, n, m, g, "ties/nan")
    v, idx, L, rv, ridx = check_compress(nmg, Wt, 2, 4, 4, "signed zeros")
    assert np.signbit(np_of(v)[0, :4]).all()


def test_subnormal_scores(nmg):
    rng = np.random.default_rng(2)
    W = (rng.standard_normal((64, 64)) * 1e-39).astype(np.float32)  # binary32 subnormals
    check_compress(nmg, torch.from_numpy(W), 1, 4, 8, "f32 subnormal")
    H = (rng.standard_normal((64, 64)) * 1e-6).astype(np.float16)   # binary16 subnormals
    check_compress(nmg, torch.from_numpy(H), 2, 8, 4, "f16 subnormal")


def test_all_zero_weight(nmg):
    W = torch.zeros(32, 40)
    v, idx, L, rv, ridx = check_compress(nmg, W, 2, 8, 8, "zeros")
    assert (np_of(idx).reshape(-1, 2) == [0, 1]).all()
    X = synth.normal((40, 70), 5)
    for kernel in kernels_for(nmg, L, 70):
        try:
            Y = nmg.spmm(v, idx, X.to(DEV), L, kernel)
        except nmg.NmgError as e:
            assert e.status == nmg.ERR_UNSUPPORTED
            continue
        assert (np_of(Y) == 0).all()


def test_strided_inputs_and_outputs(nmg):
    """Leading dimensions larger than the row length (views of wider tensors)."""
    Wb = synth.normal((128, 100), 21, 0.02)
    Xb = synth.normal((96, 140), 22)
    W, X = Wb[:, :96], Xb[:, :128]
    v, idx, L, rv, ridx = check_compress(nmg, W, 1, 4, 8, "strided W")
    Ybig = torch.full((128, 136), 7.0, device=DEV)
    Y = Ybig[:, :128]
    nmg.spmm_into(L, v, idx, X.to(DEV), Y)
    torch.cuda.synchronize()
    Yref, B = oracle.spmm(rv, ridx, np.ascontiguousarray(np_of(X)), 96, 1, 4, 8)
    check_product(Y, Yref, B, torch.float32, "strided")
    assert (np_of(Ybig)[:, 128:] == 7.0).all()  # nothing written outside Y


@pytest.mark.parametrize("dtype", [torch.float32, torch.float16])
def test_unaligned_x_rows(nmg, dtype):
    """X starting one element past a 16-byte boundary, with an odd leading
    dimension: the element-wise load path."""
    Wt = synth.normal((64, 40), 3, 0.02, dtype)
    Xb = synth.normal((40 * 37 + 1,), 4, 1.0, dtype)
    X = Xb[1:].view(40, 37)
    v, idx, L, rv, ridx = check_compress(nmg, Wt, 1, 4, 8, "unaligned X")
    Xd = Xb.to(DEV)[1:].view(40, 37)
    for kernel in kernels_for(nmg, L, 37):
        try:
            Y = nmg.spmm(v, idx, Xd, L, kernel)
        except nmg.NmgError as e:
            assert e.status == nmg.ERR_UNSUPPORTED
            continue
        torch.cuda.synchronize()
        Yref, B = oracle.spmm(rv, ridx, np.ascontiguousarray(np_of(X)), 40, 1, 4, 8)
        check_product(Y, Yref, B, dtype, f"unaligned {kernel}", L.C * L.n)


def test_element_misaligned_pointer_is_rejected(nmg):
    import ctypes
    W = synth.normal((32, 32), 3, 0.02).to(DEV)
    v, idx, L = nmg.compress(W, 1, 4, 8)
    X = torch.zeros(32, 32, device=DEV)
    Y = torch.empty(32, 32, device=DEV)
    st = nmg.lib().nmg_spmm(ctypes.byref(L.c), ctypes.c_void_p(v.data_ptr()),
                            ctypes.c_void_p(idx.data_ptr()), ctypes.c_void_p(X.data_ptr() + 2),
                            32, 32, ctypes.c_void_p(Y.data_ptr()), 32, ctypes.c_void_p(0))
    assert st == nmg.ERR_ALIGN


def test_repeatable(nmg):
    W = synth.normal((512, 768), 31, 0.02).to(DEV)
    X = synth.normal((768, 512), 32).to(DEV)
    v, idx, L = nmg.compress(W, 1, 4, 8)
    Y1 = nmg.spmm(v, idx, X, L)
    Y2 = nmg.spmm(v, idx, X, L)
    assert torch.equal(Y1, Y2)


# ------------------------------------------------------ the five workloads

def sample_points(M, N, count, seed):
    rng = np.random.default_rng(seed)
    rows = np.concatenate([rng.integers(0, M, count), [0, M - 1, M - 1]])
    cols = np.concatenate([rng.integers(0, N, count), [0, N - 1, 0]])
    return rows, cols


def check_sampled(nmg, v, idx, L, X, Y, rv, ridx, count=4096, seed=0, what=""):
    rows, cols = sample_points(L.M, X.shape[1], count, seed)
    Yref, B = oracle.spmm_points(rv, ridx, np_of(X), L.K, L.n, L.m, L.g, rows, cols)
    Ys = Y[torch.as_tensor(rows, device=Y.device), torch.as_tensor(cols, device=Y.device)]
    return check_product(Ys, Yref, B, L.dtype, what, L.C * L.n)


@pytest.mark.parametrize("workload", [1, 2, 3])
def test_workload_single_layer(nmg, workload):
    wl = synth.WORKLOADS[workload]
    lin = wl.layers[0]
    W, X = synth.layer_inputs(workload, 0, lin)
    v, idx, L, rv, ridx = check_compress(nmg, W, lin.n, lin.m, lin.g, wl.key)
    dense = nmg.densify(v, idx, L)
    rd, _ = oracle.densify(rv, ridx, lin.K, lin.n, lin.m, lin.g)
    assert np.array_equal(bits(np_of(dense)), bits(rd))
    for kernel in KERNELS:
        worst = spmm_full(nmg, v, idx, L, X, rv, ridx, kernel, wl.key)
        if worst is not None:
            print(f"[{wl.key}] {kernel}: worst |Y-Yref|/B = {worst:.3e}", flush=True)


def test_workload_sweep(nmg):
    wl = synth.WORKLOADS[5]
    for j, lin in enumerate(wl.layers):
        W, X = synth.layer_inputs(5, j, lin)
        v, idx, L, rv, ridx = check_compress(nmg, W, lin.n, lin.m, lin.g, lin.name)
        Xd = X.to(DEV)
        for kernel in kernels_for(nmg, L, lin.N):
            print(f"[spmm] sweep {lin.name} kernel={kernel}", flush=True)
            try:
                Y = nmg.spmm(v, idx, Xd, L, kernel)
            except nmg.NmgError as e:
                assert e.status == nmg.ERR_UNSUPPORTED
                continue
            torch.cuda.synchronize()
            check_sampled(nmg, v, idx, L, X, Y, rv, ridx, 2048, j, f"{lin.name} {kernel}")


def test_workload_bert_stack(nmg):
    """12 layers of the fp16 linear stack, chained on the GPU; every product,
    GELU and residual sum is checked against the oracle on the GPU's own input
    to that step."""
    from paper_2304_07613_amd.stack import LinearStack
    layers = synth.WORKLOADS[4].layers
    stack = LinearStack.from_workload(4, nmg, n=2, m=8, g=8)
    x = synth.normal((synth.BERT_HIDDEN, synth.BERT_TOKENS), synth.seed_for(4, 0, "X"), 1.0,
                     torch.float16).to(DEV)
    for li, layer in enumerate(stack.layers):
        trace = {}
        x_next = stack.forward_layer(layer, x, trace)
        torch.cuda.synchronize()
        # packed weights equal the oracle's packing of the same dense weight
        for lin in layers:
            W = layer.dense[lin.name]
            rv, ridx = oracle.compress(np_of(W), lin.n, lin.m, lin.g)
            v, idx, _ = layer.packed[lin.name]
            assert np.array_equal(np_of(idx), ridx) and np.array_equal(bits(np_of(v)), bits(rv))
        for name, (inp, out) in trace["linear"].items():
            v, idx, L = layer.packed[name]
            rv, ridx = np_of(v), np_of(idx)
            print(f"[stack] layer {li} {name}", flush=True)
            check_sampled(nmg, v, idx, L, inp.cpu(), out, rv, ridx, 2048, li, f"L{li} {name}")
        u, gl = trace["gelu"]
        ref = oracle.gelu_f16(np_of(u))
        diff = np.abs(np_of(gl).astype(np.float64) - ref.astype(np.float64))
        with np.errstate(over="ignore"):
            ulp = np.spacing(np.abs(ref)).astype(np.float64)
        assert (diff <= ulp).all(), f"gelu layer {li}"
        for a, b, s in trace["add"]:
            assert np.array_equal(bits(np_of(s)), bits(oracle.add_f16(np_of(a), np_of(b)))), \
                f"residual layer {li}"
        x = x_next
    assert torch.isfinite(x.float()).all()
    assert 0.1 < float(x.float().std()) < 100.0


def test_elementwise_glue(nmg):
    bits16 = torch.arange(65536, dtype=torch.int32).to(torch.int16).view(torch.float16)
    h = bits16[torch.isfinite(bits16)].contiguous()
    g = nmg.gelu(h.to(DEV))
    ref = oracle.gelu_f16(np_of(h))
    got = np_of(g)
    hx = np_of(h)
    with np.errstate(over="ignore"):
        ulp = np.spacing(np.abs(ref)).astype(np.float64)
    diff = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    bad = np.isfinite(ref) & ~(diff <= ulp)
    assert not bad.any(), (f"{bad.sum()} GELU outputs beyond one binary16 ulp, e.g. "
                           f"x={hx[bad][:4]} gpu={got[bad][:4]} ref={ref[bad][:4]}")
    a = synth.normal((1 << 16,), 41, 30.0, torch.float16)
    b = synth.normal((1 << 16,), 42, 0.01, torch.float16)
    s = nmg.add(a.to(DEV), b.to(DEV))
    assert np.array_equal(bits(np_of(s)), bits(oracle.add_f16(np_of(a), np_of(b))))
    x32 = synth.normal((4099,), 43, 3.0)
    g32 = np_of(nmg.gelu(x32.to(DEV))).astype(np.float64)
    from scipy.special import erf
    xd = np_of(x32).astype(np.float64)
    assert np.allclose(g32, 0.5 * xd * (1 + erf(xd / np.sqrt(2))), rtol=1e-6, atol=1e-7)


# ------------------------------------------- the paper's chunked layout

P_SHAPES = [
    # M,    K,   N,    n, m, g,  dtype
    (48, 16, 100, 2, 4, 2, torch.float32),
    (96, 40, 256, 1, 4, 8, torch.float16),
    (120, 60, 77, 3, 6, 1, torch.float32),      # ragged N
    (192, 48, 64, 2, 4, 32, torch.float32),     # S = 192
    (256, 32, 40, 1, 4, 64, torch.float16),     # S = 256, one chunk row-set
    (224, 16, 33, 2, 8, 8, torch.float32),      # 28 patterns, S = 224
    (768, 768, 128, 2, 4, 4, torch.float32),    # the single-layer shape
    # m = 4 with whole 8-block windows: the matrix-core kernel's row path
    (96, 64, 300, 3, 4, 8, torch.float32),      # n = 3, ragged N
    (192, 64, 70, 2, 4, 16, torch.float16),     # S = 96: tiles straddle two chunks
    (384, 128, 513, 1, 4, 48, torch.float32),   # S = 192, N past a whole tile
]


@pytest.mark.parametrize("M,K,N,n,m,g,dtype", P_SHAPES,
                         ids=[f"{c[0]}x{c[1]}x{c[2]}-{c[3]}:{c[4]}:{c[5]}-{str(c[6])[6:]}"
                              for c in P_SHAPES])
def test_chunked_layout(nmg, M, K, N, n, m, g, dtype):
    W = synth.normal((M, K), 81 + M, 0.02, dtype)
    X = synth.normal((K, N), 82 + N, 1.0, dtype)
    print(f"[chunked] {M}x{K}x{N} {n}:{m}:{g} {dtype}", flush=True)
    v, idx, L = nmg.p_compress(W.to(DEV), n, m, g)
    torch.cuda.synchronize()
    rv, ridx = oracle.p_compress(np_of(W), n, m, g)
    assert np.array_equal(np_of(idx), ridx), f"index differs at {np.argwhere(np_of(idx) != ridx)[:5]}"
    assert np.array_equal(bits(np_of(v)), bits(rv))
    dense = nmg.p_densify(v, idx, L)
    rd, _ = oracle.p_densify(rv, ridx, K, n, m, g)
    assert np.array_equal(bits(np_of(dense)), bits(rd))
    Yref, B = oracle.p_spmm(rv, ridx, np_of(X), K, n, m, g)
    Xd = X.to(DEV)
    for kernel in ("auto", "valu", "mfma"):
        if kernel == "mfma" and m > 32:
            continue
        print(f"[chunked spmm] {kernel}", flush=True)
        Y = nmg.p_spmm(v, idx, Xd, L, kernel)
        torch.cuda.synchronize()
        check_product(Y, Yref, B, dtype, f"chunked {kernel}", (K // m) * n)


def random_chunked(count=30, seed=2305):
    """Seeded random shapes of the chunked layout: K % m == 0, M a multiple
    of S = C(m, n) * g <= 256, within the kernels' LDS limits (S P <= 8192,
    S m <= 8192, P n <= 4096; beyond them the library reports
    NMG_ERR_UNSUPPORTED)."""
    from math import comb
    rng = np.random.RandomState(seed)
    out = []
    while len(out) < count:
        m = int(rng.randint(1, 9))
        n = int(rng.randint(1, m + 1))
        P = comb(m, n)
        gs = [g for g in (1, 2, 3, 4, 8, 16, 32, 64)
              if P * g <= 256 and P * g * P <= 8192 and P * g * m <= 8192 and P * n <= 4096]
        if not gs:
            continue
        g = int(rng.choice(gs))
        S = P * g
        M = S * int(rng.randint(1, max(2, 512 // S)))
        K = m * int(rng.randint(1, 25))
        N = int(rng.randint(1, 200))
        dtype = torch.float16 if rng.rand() < 0.5 else torch.float32
        out.append((M, K, N, n, m, g, dtype))
    return out


P_RANDOM = random_chunked()


@pytest.mark.parametrize("M,K,N,n,m,g,dtype", P_RANDOM,
                         ids=[f"p{i}-{c[0]}x{c[1]}x{c[2]}-{c[3]}:{c[4]}:{c[5]}-{str(c[6])[6:]}"
                              for i, c in enumerate(P_RANDOM)])
def test_chunked_random(nmg, M, K, N, n, m, g, dtype):
    """Converter, densify, product and swap search of the chunked layout on
    random shapes, against the oracle."""
    test_chunked_layout(nmg, M, K, N, n, m, g, dtype)
    W = synth.normal((M, K), 81 + M, 0.02, dtype)
    Wd = W.to(DEV)
    v, idx, L = nmg.p_compress(Wd, n, m, g)
    rv_g, ridx_g = nmg.p_refine(Wd, idx, L)
    torch.cuda.synchronize()
    rv, ridx, rounds = oracle.p_refine(np_of(W), np_of(idx), n, m, g)
    assert np.array_equal(np_of(ridx_g), ridx)
    assert np.array_equal(bits(np_of(rv_g)), bits(rv))


def test_chunked_layout_ties_and_nan(nmg):
    rng = np.random.default_rng(5)
    W = (rng.integers(-3, 4, size=(96, 24)) / 2.0).astype(np.float32)   # many equal magnitudes
    W[5, 3] = np.nan
    W[40:50, 8:12] = -0.0
    for n, m, g in [(2, 4, 4), (1, 4, 8), (1, 2, 6), (3, 6, 1)]:
        if 96 % (math_comb(m, n) * g) or 24 % m:
            continue
        print(f"[chunked ties] {n}:{m}:{g}", flush=True)
        v, idx, L = nmg.p_compress(torch.from_numpy(W).to(DEV), n, m, g)
        torch.cuda.synchronize()
        rv, ridx = oracle.p_compress(W, n, m, g)
        assert np.array_equal(np_of(idx), ridx)
        assert np.array_equal(bits(np_of(v)), bits(rv))


def math_comb(m, n):
    import math
    return math.comb(m, n)


def test_chunked_layout_ffn_shape(nmg):
    """The FFN up-projection shape (3072 x 768, 1:4:8 -> chunks of 32 rows) with
    4096 tokens: packing bit-exact, products checked on 192 whole rows."""
    lin = synth.WORKLOADS[2].layers[0]
    W, X = synth.layer_inputs(2, 0, lin)
    v, idx, L = nmg.p_compress(W.to(DEV), 1, 4, 8)
    torch.cuda.synchronize()
    rv, ridx = oracle.p_compress(np_of(W), 1, 4, 8)
    assert np.array_equal(np_of(idx), ridx) and np.array_equal(bits(np_of(v)), bits(rv))
    rd, _ = oracle.p_densify(rv, ridx, lin.K, 1, 4, 8)
    rows = np.random.default_rng(9).choice(lin.M, 192, replace=False)
    Xd = np_of(X).astype(np.float64)
    Yref = rd[rows].astype(np.float64) @ Xd
    B = np.abs(rd[rows].astype(np.float64)) @ np.abs(Xd)
    for kernel in ("valu", "mfma"):
        print(f"[chunked ffn] {kernel}", flush=True)
        Y = nmg.p_spmm(v, idx, X.to(DEV), L, kernel)
        torch.cuda.synchronize()
        check_product(Y[torch.as_tensor(rows, device=Y.device)], Yref, B, torch.float32,
                      f"chunked ffn {kernel}")



@pytest.mark.parametrize("M,K,N,n,m,g,dtype", P_SHAPES[:6],
                         ids=[f"{c[0]}x{c[1]}-{c[3]}:{c[4]}:{c[5]}-{str(c[6])[6:]}" for c in P_SHAPES[:6]])
def test_chunked_swap_search(nmg, M, K, N, n, m, g, dtype):
    """The swap search from the greedy packing and from the identity packing
    (every chunk's rows in order), bit-exact against the oracle's."""
    W = synth.normal((M, K), 91 + M, 0.02, dtype)
    Wd = W.to(DEV)
    v, idx, L = nmg.p_compress(Wd, n, m, g)
    ident = torch.from_numpy(np.tile(np.arange(L.S, dtype=np.uint8), M // L.S)[:, None]
                             .repeat(L.B, axis=1)).to(DEV)
    for start, name in ((idx, "greedy"), (ident, "identity")):
        print(f"[swap] {M}x{K} {n}:{m}:{g} {dtype} from {name}", flush=True)
        rv_g, ridx_g = nmg.p_refine(Wd, start, L)
        torch.cuda.synchronize()
        rv, ridx, rounds = oracle.p_refine(np_of(W), np_of(start), n, m, g)
        assert np.array_equal(np_of(ridx_g), ridx), name
        assert np.array_equal(bits(np_of(rv_g)), bits(rv)), name
