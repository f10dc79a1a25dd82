"""The C ABI without a GPU: the library loads, exports every function
``include/nmg.h`` declares, and validates arguments on the host (no call here
reaches a kernel launch)."""
import ctypes

import pytest
import torch

from paper_2304_07613_amd import build, nmg


@pytest.fixture(scope="module")
def lib():
    if build.is_stale():
        build.build()
    return nmg.lib()


def test_every_declared_symbol_is_exported(lib):
    names = nmg.header_functions()
    assert len(names) >= 12
    for name in names:
        assert hasattr(lib, name), f"{name} declared in nmg.h but not exported"
    assert nmg.version().startswith("nmg ")


def test_layout_init_validation(lib):
    L = nmg._Layout()
    init = lambda *a: lib.nmg_layout_init(ctypes.byref(L), *a)
    assert init(3072, 768, 1, 4, 8, nmg.F32) == nmg.OK and L.C == 192
    assert init(768, 3072, 1, 10, 16, nmg.F32) == nmg.OK and L.C == 308
    assert lib.nmg_values_numel(ctypes.byref(L)) == 768 * 308
    assert lib.nmg_indices_numel(ctypes.byref(L)) == 48 * 308
    assert init(768, 768, 2, 4, 4, 7) == nmg.ERR_DTYPE
    assert init(768, 768, 5, 4, 4, nmg.F32) == nmg.ERR_PARAM      # n > m
    assert init(768, 768, 0, 4, 4, nmg.F32) == nmg.ERR_PARAM      # n < 1
    assert init(768, 768, 1, 256, 4, nmg.F32) == nmg.ERR_PARAM    # m > 255
    assert init(768, 768, 1, 4, 0, nmg.F32) == nmg.ERR_PARAM      # g < 1
    assert init(0, 768, 1, 4, 1, nmg.F32) == nmg.ERR_PARAM        # M < 1
    assert init(770, 768, 1, 4, 4, nmg.F32) == nmg.ERR_SHAPE      # M % g
    assert init(8, 10, 3, 4, 1, nmg.F32) == nmg.ERR_SHAPE         # tail 2 < n
    assert init(8, 10, 2, 4, 1, nmg.F32) == nmg.OK
    assert lib.nmg_layout_init(None, 8, 8, 1, 4, 1, nmg.F32) == nmg.ERR_NULL


def test_calls_reject_bad_arguments_before_launch(lib):
    L = nmg._Layout()
    assert lib.nmg_layout_init(ctypes.byref(L), 64, 64, 1, 4, 8, nmg.F32) == nmg.OK
    p = ctypes.c_void_p(1 << 20)          # never dereferenced: validation fails first
    odd = ctypes.c_void_p((1 << 20) + 2)  # not aligned to a binary32 element
    s = ctypes.c_void_p(0)
    assert lib.nmg_compress(ctypes.byref(L), None, 64, p, p, s) == nmg.ERR_NULL
    assert lib.nmg_compress(ctypes.byref(L), p, 63, p, p, s) == nmg.ERR_PARAM
    assert lib.nmg_spmm(ctypes.byref(L), p, p, p, 32, 33, p, 33, s) == nmg.ERR_PARAM  # ldx < N
    assert lib.nmg_spmm(ctypes.byref(L), p, p, p, 32, 0, p, 32, s) == nmg.ERR_PARAM   # N = 0
    assert lib.nmg_spmm(ctypes.byref(L), p, p, odd, 32, 32, p, 32, s) == nmg.ERR_ALIGN
    assert lib.nmg_spmm(ctypes.byref(L), p, p, p, 32, 32, odd, 32, s) == nmg.ERR_ALIGN
    assert lib.nmg_spmm(ctypes.byref(L), None, p, p, 32, 32, p, 32, s) == nmg.ERR_NULL
    assert lib.nmg_densify(ctypes.byref(L), p, p, p, 60, s) == nmg.ERR_PARAM
    assert lib.nmg_repack(ctypes.byref(L), p, 60, p, p, s) == nmg.ERR_PARAM    # ldw < K
    assert lib.nmg_repack(ctypes.byref(L), p, 64, None, p, s) == nmg.ERR_NULL
    assert lib.nmg_repack(ctypes.byref(L), odd, 64, p, p, s) == nmg.ERR_ALIGN
    ep = lib.nmg_spmm_epilogue
    big = ctypes.c_void_p(1 << 30)  # far from p: no overlap
    assert ep(ctypes.byref(L), 0, 7, p, p, p, 32, 32, None, 0, p, 32, s) == nmg.ERR_PARAM  # epilogue
    assert ep(ctypes.byref(L), 0, 2, p, p, p, 32, 32, None, 32, p, 32, s) == nmg.ERR_NULL  # no R
    assert ep(ctypes.byref(L), 0, 2, p, p, p, 32, 32, big, 16, p, 32, s) == nmg.ERR_PARAM  # ldr < N
    assert ep(ctypes.byref(L), 0, 2, p, p, p, 32, 32, odd, 32, p, 32, s) == nmg.ERR_ALIGN
    assert ep(ctypes.byref(L), 0, 2, p, p, p, 32, 32, p, 32, p, 32, s) == nmg.ERR_PARAM   # R == Y
    assert lib.nmg_gelu(9, p, p, 10, s) == nmg.ERR_DTYPE
    assert lib.nmg_add(nmg.F16, p, None, p, 10, s) == nmg.ERR_NULL
    assert lib.nmg_gelu(nmg.F32, p, p, 0, s) == nmg.OK   # empty input: nothing to launch
    bad = nmg._Layout(64, 64, 1, 4, 8, 17, nmg.F32)    # inconsistent C
    assert lib.nmg_compress(ctypes.byref(bad), p, 64, p, p, s) == nmg.ERR_PARAM
    # g % 4 != 0: the grouped matrix-core kernels decline; at m <= 8 n the
    # expanded dense weight on the matrix cores is the choice
    assert lib.nmg_layout_init(ctypes.byref(L), 64, 64, 1, 4, 2, nmg.F32) == nmg.OK
    for fam in ("mfma", "mfma_general", "mfma_scalar", "mfma_f16", "mfma_direct", "smfmac_f16"):
        assert lib.nmg_spmm_with(ctypes.byref(L), nmg.KERNELS[fam], p, p, p, 32, 32, p, 32,
                                 s) == nmg.ERR_UNSUPPORTED
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 32) == nmg.KERNELS["mfma_expand"]
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 30) == nmg.KERNELS["mfma_expand"]
    # M % 4 != 0: no expanded product either
    assert lib.nmg_layout_init(ctypes.byref(L), 66, 64, 1, 4, 2, nmg.F32) == nmg.OK
    assert lib.nmg_spmm_with(ctypes.byref(L), nmg.KERNELS["mfma_expand"], p, p, p, 32, 32, p, 32,
                             s) == nmg.ERR_UNSUPPORTED
    # above m = 8 n a vector kernel is the choice (the LDS-staged one when X
    # rows can be copied 16 bytes at a time)
    assert lib.nmg_layout_init(ctypes.byref(L), 64, 640, 1, 10, 2, nmg.F32) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 32) == nmg.KERNELS["valu_staged"]
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 30) == nmg.KERNELS["valu"]    # N % 4 != 0
    assert lib.nmg_layout_init(ctypes.byref(L), 64, 660, 1, 33, 1, nmg.F32) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 32) == nmg.KERNELS["valu"]    # m > 32
    assert lib.nmg_spmm_with(ctypes.byref(L), nmg.KERNELS["valu_staged"], p, p, p, 32, 32, p, 32,
                             s) == nmg.ERR_UNSUPPORTED
    # 1:20, g = 1: a 32 KB window holds one chunk, so the staged kernel takes
    # its wide shape (64 KB windows of 3 chunks), faster than gathering
    assert lib.nmg_layout_init(ctypes.byref(L), 3072, 768, 1, 20, 1, nmg.F32) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) == nmg.KERNELS["valu_staged"]
    assert lib.nmg_layout_init(ctypes.byref(L), 3072, 768, 1, 10, 1, nmg.F32) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) == nmg.KERNELS["valu_staged"]
    assert lib.nmg_layout_init(ctypes.byref(L), 3072, 768, 1, 4, 8, nmg.F32) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) == nmg.KERNELS["mfma_scalar"]
    # 1:10 with groups of 16: gathering the selected rows reads less than
    # staging whole windows
    assert lib.nmg_layout_init(ctypes.byref(L), 768, 3072, 1, 10, 16, nmg.F32) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) == nmg.KERNELS["mfma_direct"]
    # with 256-token tiles that cover the CUs, units of 8 or 16 rows gather up
    # to 1.75 times the staged kernel's rows: 1:10:8 (1.6 times) gathers,
    # 1:4:16 (2 times) stages; units of 4 rows up to 3.5 times: 1:10:4 (3.2
    # times) gathers, 2:8:4 (8 times) stages
    for (n_, m_, g_), fam in (((1, 10, 8), "mfma_direct"), ((1, 4, 16), "mfma_scalar"),
                              ((1, 20, 4), "mfma_direct"), ((1, 10, 4), "mfma_direct"),
                              ((2, 8, 4), "mfma_scalar")):
        assert lib.nmg_layout_init(ctypes.byref(L), 3072, 768, n_, m_, g_, nmg.F32) == nmg.OK
        assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) == nmg.KERNELS[fam], (n_, m_, g_)
    # a layer too small to fill the GPU without splitting its k-slots
    assert lib.nmg_layout_init(ctypes.byref(L), 768, 768, 2, 4, 4, nmg.F32) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 128) == nmg.KERNELS["mfma_direct"]
    # n = 3 is not a power of two: the general matrix-core kernel declines too,
    # the expanded product takes it
    assert lib.nmg_layout_init(ctypes.byref(L), 3072, 768, 3, 8, 8, nmg.F32) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) == nmg.KERNELS["mfma_expand"]
    # binary32 g = 1 sweep points: expanded at 2:4, 1:4, 2:8; staged vector FMAs at 1:10
    for n_, m_ in ((2, 4), (1, 4), (2, 8)):
        assert lib.nmg_layout_init(ctypes.byref(L), 3072, 768, n_, m_, 1, nmg.F32) == nmg.OK
        assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) == nmg.KERNELS["mfma_expand"]
    # n = m (dense) with g = 1: one group, so the matrix cores take it
    assert lib.nmg_layout_init(ctypes.byref(L), 3072, 768, 4, 4, 1, nmg.F32) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) == nmg.KERNELS["mfma_scalar"]
    # binary16: the binary16 matrix cores when X can be staged 16 bytes at a
    # time (N % 8 == 0), else the binary32 matrix-core kernel on widened X
    assert lib.nmg_layout_init(ctypes.byref(L), 3072, 768, 2, 8, 8, nmg.F16) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) == nmg.KERNELS["mfma_f16"]
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4100) == nmg.KERNELS["mfma_scalar"]
    assert lib.nmg_layout_init(ctypes.byref(L), 768, 3072, 1, 10, 16, nmg.F16) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) == nmg.KERNELS["mfma_f16"]
    # a window of 4 k-slots at 1:255 needs 1020 staged rows: declined
    assert lib.nmg_layout_init(ctypes.byref(L), 64, 510, 1, 255, 8, nmg.F16) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) != nmg.KERNELS["mfma_f16"]
    assert lib.nmg_layout_init(ctypes.byref(L), 64, 64, 1, 4, 2, nmg.F16) == nmg.OK
    assert lib.nmg_spmm_with(ctypes.byref(L), nmg.KERNELS["mfma_f16"], p, p, p, 32, 32, p, 32,
                             s) == nmg.ERR_UNSUPPORTED
    # g = 2: no quads of rows, but the sparse matrix instruction takes any g
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) == nmg.KERNELS["smfmac_f16"]
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4100) == nmg.KERNELS["valu"]
    assert lib.nmg_layout_init(ctypes.byref(L), 64, 96, 1, 3, 2, nmg.F16) == nmg.OK
    assert lib.nmg_spmm_auto_kernel(ctypes.byref(L), 4096) == nmg.KERNELS["valu"]  # m = 3
    assert lib.nmg_layout_init(ctypes.byref(L), 64, 40, 2, 8, 1, nmg.F16) == nmg.OK   # C n = 10
    assert lib.nmg_spmm_with(ctypes.byref(L), nmg.KERNELS["smfmac_f16"], p, p, p, 32, 32, p, 32,
                             s) == nmg.ERR_UNSUPPORTED
    # the gathering kernel is binary32 only
    assert lib.nmg_layout_init(ctypes.byref(L), 64, 64, 1, 4, 8, nmg.F16) == nmg.OK
    assert lib.nmg_spmm_with(ctypes.byref(L), nmg.KERNELS["mfma_direct"], p, p, p, 32, 32, p, 32,
                             s) == nmg.ERR_UNSUPPORTED


def test_status_strings(lib):
    for st in range(9):
        assert nmg.status_str(st)
    assert nmg.status_str(99) == "unknown status"


def test_binding_refuses_cpu_tensors(lib):
    W = torch.zeros(8, 8)
    with pytest.raises(ValueError):
        nmg.compress(W, 1, 4, 4)


def test_chunked_layout_validation(lib):
    import ctypes
    L = nmg._PLayout()
    assert lib.nmg_p_layout_init(ctypes.byref(L), 3072, 768, 1, 4, 8, nmg.F32) == nmg.OK
    assert (L.P, L.S, L.B) == (4, 32, 192)
    assert lib.nmg_p_layout_init(ctypes.byref(L), 3072, 768, 2, 8, 8, nmg.F32) == nmg.ERR_SHAPE  # 224 rows
    assert lib.nmg_p_layout_init(ctypes.byref(L), 768, 770, 2, 4, 4, nmg.F32) == nmg.ERR_SHAPE   # K % m
    assert lib.nmg_p_layout_init(ctypes.byref(L), 924, 12, 6, 12, 1, nmg.F32) == nmg.ERR_PARAM   # 924 patterns
    assert lib.nmg_p_layout_init(ctypes.byref(L), 512, 8, 1, 4, 128, nmg.F32) == nmg.ERR_SHAPE  # S = 512
    assert lib.nmg_p_layout_init(None, 8, 8, 1, 4, 2, nmg.F32) == nmg.ERR_NULL
    assert lib.nmg_p_layout_init(ctypes.byref(L), 48, 16, 2, 4, 2, nmg.F16) == nmg.OK
    p, s = ctypes.c_void_p(1 << 20), ctypes.c_void_p(0)
    odd = ctypes.c_void_p((1 << 20) + 1)
    assert lib.nmg_p_compress(ctypes.byref(L), p, 15, p, p, s) == nmg.ERR_PARAM     # ldw < K
    assert lib.nmg_p_compress(ctypes.byref(L), None, 16, p, p, s) == nmg.ERR_NULL
    assert lib.nmg_p_compress(ctypes.byref(L), odd, 16, p, p, s) == nmg.ERR_ALIGN
    assert lib.nmg_p_spmm(ctypes.byref(L), p, p, p, 8, 16, p, 16, s) == nmg.ERR_PARAM  # ldx < N
    assert lib.nmg_p_spmm_with(ctypes.byref(L), nmg.KERNELS["mfma_f16"], p, p, p, 16, 16, p, 16,
                               s) == nmg.ERR_UNSUPPORTED   # not a chunked-layout kernel
    assert lib.nmg_p_spmm_with(ctypes.byref(L), nmg.KERNELS["mfma"], p, p, p, 8, 16, p, 16,
                               s) == nmg.ERR_PARAM          # ldx < N
    assert lib.nmg_p_spmm_with(ctypes.byref(L), nmg.KERNELS["valu"], p, p, None, 16, 16, p, 16,
                               s) == nmg.ERR_NULL
    assert lib.nmg_p_densify(ctypes.byref(L), p, None, p, 16, s) == nmg.ERR_NULL
    assert lib.nmg_p_refine(ctypes.byref(L), p, 8, p, p, s) == nmg.ERR_PARAM       # ldw < K
    assert lib.nmg_p_refine(ctypes.byref(L), p, 16, p, None, s) == nmg.ERR_NULL
    bad = nmg._PLayout(48, 16, 2, 4, 2, 6, 10, 4, nmg.F16)   # S inconsistent with P * g
    assert lib.nmg_p_compress(ctypes.byref(bad), p, 16, p, p, s) == nmg.ERR_PARAM


def test_x16_validation(lib):
    L = nmg._Layout()
    p, s = ctypes.c_void_p(1 << 20), ctypes.c_void_p(0)
    big = ctypes.c_void_p(1 << 30)
    assert lib.nmg_layout_init(ctypes.byref(L), 3072, 768, 2, 8, 8, nmg.F16) == nmg.OK
    nbytes = lib.nmg_x16_prepared_bytes(ctypes.byref(L))
    assert nbytes > 0 and nbytes % 16 == 0
    assert lib.nmg_x16_prepare(ctypes.byref(L), p, None, p, s) == nmg.ERR_NULL
    assert lib.nmg_x16_prepare(ctypes.byref(L), p, p, ctypes.c_void_p((1 << 20) + 8),
                               s) == nmg.ERR_ALIGN
    # the binary32 family declines binary16; N % 8 != 0 is declined (before
    # any allocation)
    assert lib.nmg_spmm_with(ctypes.byref(L), nmg.KERNELS["mfma_split"], p, p, p, 32, 32, big,
                             32, s) == nmg.ERR_UNSUPPORTED
    assert lib.nmg_spmm_with(ctypes.byref(L), nmg.KERNELS["mfma_wide"], p, p, p, 36, 36, big,
                             36, s) == nmg.ERR_UNSUPPORTED
    ep = lib.nmg_spmm_x16_epilogue
    assert ep(ctypes.byref(L), p, 7, p, 64, 64, None, 0, big, 64, s) == nmg.ERR_PARAM   # epilogue
    assert ep(ctypes.byref(L), p, 1, p, 64, 60, None, 0, big, 64, s) == nmg.ERR_UNSUPPORTED  # N % 8
    assert ep(ctypes.byref(L), p, 2, p, 64, 64, None, 64, big, 64, s) == nmg.ERR_NULL   # no R
    assert ep(ctypes.byref(L), p, 2, p, 64, 64, big, 32, big, 64, s) == nmg.ERR_PARAM   # ldr < N
    assert ep(ctypes.byref(L), p, 2, p, 64, 64, ctypes.c_void_p((1 << 30) + 8), 64,
              p, 64, s) == nmg.ERR_UNSUPPORTED                                             # R 8-aligned
    assert ep(ctypes.byref(L), p, 2, p, 64, 64, big, 64, big, 64, s) == nmg.ERR_PARAM   # R == Y
    assert ep(ctypes.byref(L), p, 0, p, 64, 60, None, 0, big, 64, s) == nmg.ERR_UNSUPPORTED  # N % 8
    assert lib.nmg_spmm_x16(ctypes.byref(L), p, p, 32, 64, big, 64, s) == nmg.ERR_PARAM  # ldx < N
    # n = 3 and g % 8 != 0: not taken
    assert lib.nmg_layout_init(ctypes.byref(L), 3072, 768, 3, 8, 8, nmg.F16) == nmg.OK
    assert lib.nmg_x16_prepared_bytes(ctypes.byref(L)) == -1
    assert lib.nmg_x16_prepare(ctypes.byref(L), p, p, p, s) == nmg.ERR_UNSUPPORTED
    assert lib.nmg_layout_init(ctypes.byref(L), 3072, 768, 2, 8, 4, nmg.F32) == nmg.OK
    assert lib.nmg_x16_prepared_bytes(ctypes.byref(L)) == -1


def test_noalloc_refuses_before_launch(lib):
    """The allocation-free product refuses a layout whose prepared operands
    exceed its fixed array, and bad arguments, on the host."""
    L = nmg._Layout()
    p, s = ctypes.c_void_p(1 << 20), ctypes.c_void_p(0)
    assert lib.nmg_layout_init(ctypes.byref(L), 32768, 8192, 2, 8, 8, nmg.F16) == nmg.OK
    assert lib.nmg_x16_prepared_bytes(ctypes.byref(L)) > 16 << 20
    na = lib.nmg_spmm_epilogue_noalloc
    assert na(ctypes.byref(L), nmg.KERNELS["mfma_wide"], 0, p, p, p, 4096, 4096, None, 0, p,
              4096, s) == nmg.ERR_CAPACITY
    assert na(ctypes.byref(L), nmg.KERNELS["mfma_wide"], 0, None, p, p, 4096, 4096, None, 0, p,
              4096, s) == nmg.ERR_NULL
    assert lib.nmg_layout_init(ctypes.byref(L), 3072, 768, 3, 8, 8, nmg.F16) == nmg.OK
    assert na(ctypes.byref(L), nmg.KERNELS["mfma_wide"], 0, p, p, p, 64, 64, None, 0, p, 64,
              s) == nmg.ERR_UNSUPPORTED
    # the other families take nmg_spmm_epilogue's path and its checks
    assert na(ctypes.byref(L), 0, 7, p, p, p, 64, 64, None, 0, p, 64, s) == nmg.ERR_PARAM


def test_gelu_table_rules(tmp_path):
    """The binary16 GELU table is its own input from NMG_GELU_F16_IDENTITY_FROM
    up (+inf included), -0 for finite negative inputs from
    NMG_GELU_F16_NEGZERO_FROM, NMG_GELU_F16_NAN_OUT for NaN and -inf: the rules
    the 16 x 16 x 32 product's fused GELU applies instead of those entries."""
    import re
    import subprocess
    import sys

    import numpy as np
    from paper_2304_07613_amd import build
    out = tmp_path / "gelu_f16_table.inc"
    subprocess.run([sys.executable, build.GENERATORS[0], str(out)], check=True)
    t = np.array([int(v, 16) for v in re.findall(r"0x([0-9a-f]{4})", out.read_text())],
                 dtype=np.uint16)
    assert t.size == 65536
    bounds = dict(re.findall(r"#define (\w+) (0x[0-9a-f]+)", (tmp_path / "gelu_f16_bounds.inc").read_text()))
    ident = int(bounds["NMG_GELU_F16_IDENTITY_FROM"], 16)
    negz = int(bounds["NMG_GELU_F16_NEGZERO_FROM"], 16)
    nan_out = int(bounds["NMG_GELU_F16_NAN_OUT"], 16)
    b = np.arange(65536, dtype=np.uint32)
    rule_pos = (b < 0x8000) & (b >= ident)
    rule_neg = (b >= 0x8000) & (b >= negz)
    assert (t[rule_pos & (b <= 0x7c00)] == b[rule_pos & (b <= 0x7c00)]).all()
    assert (t[rule_pos & (b > 0x7c00)] == nan_out).all()
    assert (t[rule_neg & (b < 0xfc00)] == 0x8000).all()
    assert (t[rule_neg & (b >= 0xfc00)] == nan_out).all()
    # the rules cover what they should: GELU(x) = x from about 3.45, -0 below
    # about -5.72, and the entries kept are under 36 KB on each side
    x = b.astype(np.uint16).view(np.float16)
    assert 3.0 < float(x[ident]) < 4.0 and -6.0 < float(x[negz]) < -5.0
    assert 2 * ident <= 36 * 1024 and 2 * (negz - 0x8000) <= 36 * 1024
