"""nmg_spmm_epilogue_noalloc against nmg_spmm_epilogue, through the C ABI.

The allocation-free entry point keeps the scratch memory of the families that
have some (the 16 x 16 x 32 products' prepared operands, the expanded
product's dense weight, also when AUTO picks it) in the library's fixed
per-GPU array; its results must equal the
allocating entry point's bit for bit (same kernels), on consecutive calls
that reuse the array, the second with a smaller layout (whatever the first
left in the array must not leak into it).
"""
import numpy as np
import pytest
import torch

from paper_2304_07613_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def nmg():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2304_07613_amd import nmg as binding
    binding.lib()  # raises if the library is not built: no fallback
    return binding


def make(nmg, M, K, N, n, m, g, dtype, seed):
    W = synth.normal((M, K), seed, 0.02, dtype).to(DEV)
    X = synth.normal((K, N), seed + 1, 1.0, dtype).to(DEV)
    R = synth.normal((M, N), seed + 2, 1.0, dtype).to(DEV)
    v, idx, L = nmg.compress(W, n, m, g)
    return v, idx, L, X, R


def same_bits(a, b):
    return torch.equal(a.view(torch.uint8), b.view(torch.uint8))


# (first call, second call): the second smaller, so that it runs on a region
# of the array the first one filled with other operands
CASES = [
    ("mfma_wide", torch.float16, (3072, 768, 4096, 2, 8, 8), (264, 72, 264, 2, 8, 8)),
    ("mfma_wide", torch.float16, (768, 3072, 1024, 1, 4, 16), (200, 64, 96, 1, 4, 8)),
    ("mfma_split", torch.float32, (768, 3072, 2048, 1, 4, 8), (136, 40, 260, 1, 4, 8)),
    ("mfma_split", torch.float32, (1024, 512, 512, 2, 4, 16), (272, 96, 136, 2, 4, 16)),
    ("mfma_expand", torch.float32, (3072, 768, 1024, 2, 4, 1), (200, 64, 96, 1, 4, 2)),
    ("auto", torch.float32, (1024, 768, 512, 3, 8, 8), (64, 40, 33, 3, 8, 2)),
]


@pytest.mark.parametrize("kernel,dtype,big,small", CASES)
@pytest.mark.parametrize("epilogue", ["none", "add", "gelu"])
def test_noalloc_equals_allocating(nmg, kernel, dtype, big, small, epilogue):
    for call, shape in enumerate((big, small)):
        M, K, N, n, m, g = shape
        print(f"[noalloc] call {call} {kernel} {M}x{K}x{N} {n}:{m}:{g} {epilogue}", flush=True)
        v, idx, L, X, R = make(nmg, M, K, N, n, m, g, dtype, 500 + 10 * call + M)
        r = R if epilogue == "add" else None
        Y0 = torch.full((M, N), float("nan"), dtype=dtype, device=DEV)
        Y1 = torch.full((M, N), float("nan"), dtype=dtype, device=DEV)
        nmg.spmm_epilogue_noalloc(v, idx, X, L, epilogue, r, kernel, Y=Y1)
        nmg.spmm_epilogue(v, idx, X, L, epilogue, r, kernel, Y=Y0)
        torch.cuda.synchronize()
        assert same_bits(Y1, Y0), f"call {call}: no-alloc result differs"
        assert torch.isfinite(Y1.float()).all()


def test_noalloc_strided_and_repeated(nmg):
    """Strided X, Y and R; the same call three times gives the same bits."""
    v, idx, L, X, R = make(nmg, 512, 256, 384, 2, 8, 8, torch.float16, 91)
    Xb = torch.zeros((256, 400), dtype=torch.float16, device=DEV)
    Xb[:, :384] = X
    Rb = torch.zeros((512, 392), dtype=torch.float16, device=DEV)
    Rb[:, :384] = R
    ref = nmg.spmm_epilogue(v, idx, X, L, "add", R, "mfma_wide")
    for rep in range(3):
        Yb = torch.zeros((512, 392), dtype=torch.float16, device=DEV)
        nmg.spmm_epilogue_noalloc(v, idx, Xb[:, :384], L, "add", Rb[:, :384], "mfma_wide",
                                  Y=Yb[:, :384])
        torch.cuda.synchronize()
        assert same_bits(Yb[:, :384].contiguous(), ref), f"repeat {rep}"
        assert (Yb[:, 384:] == 0).all()


def test_noalloc_other_families_unchanged(nmg):
    """Families without scratch memory run as nmg_spmm_epilogue runs them."""
    v, idx, L, X, R = make(nmg, 256, 128, 256, 1, 4, 8, torch.float32, 77)
    for kernel in ("auto", "mfma_scalar", "valu"):
        a = nmg.spmm_epilogue_noalloc(v, idx, X, L, "add", R, kernel)
        b = nmg.spmm_epilogue(v, idx, X, L, "add", R, kernel)
        torch.cuda.synchronize()
        assert same_bits(a, b), kernel


def test_noalloc_capacity(nmg):
    """A layout whose prepared operands exceed the array is refused before
    any launch, and the array still serves the next call."""
    import ctypes
    big = nmg.Layout(32768, 8192, 2, 8, 8, torch.float16)
    assert nmg.lib().nmg_x16_prepared_bytes(ctypes.byref(big.c)) > 16 << 20
    p = ctypes.c_void_p(1 << 20)   # never dereferenced: refused on the host
    st = nmg.lib().nmg_spmm_epilogue_noalloc(ctypes.byref(big.c), nmg.KERNELS["mfma_wide"], 0, p, p, p,
                                              4096, 4096, None, 0, p, 4096, None)
    assert st == nmg.ERR_CAPACITY
    v, idx, L, X, R = make(nmg, 264, 72, 264, 2, 8, 8, torch.float16, 33)
    a = nmg.spmm_epilogue_noalloc(v, idx, X, L, "none", None, "mfma_wide")
    b = nmg.spmm_epilogue(v, idx, X, L, "none", None, "mfma_wide")
    torch.cuda.synchronize()
    assert same_bits(a, b)
    assert np.isfinite(a.float().cpu().numpy()).all()
