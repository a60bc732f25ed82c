"""Host-side checks of the C ABI: the library loads without a GPU, exports every
symbol declared in include/sol_attn.h, and rejects invalid arguments with the
documented codes before making any GPU call."""
import ctypes
import math
import os
import re

import pytest

from paper_2607_24027_amd import binding as sb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sol_attn.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sol_attn_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = sb.lib()
    names = header_functions()
    assert len(names) == 12
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(sb.SIGNATURES)


def test_header_constants_match_binding():
    text = open(HEADER).read()
    for name, val in [("SOL_DENSE", 0), ("SOL_SPARSE", 1), ("SOL_SPARSE_NO_CORRECTION", 2), ("SOL_BF16", 0),
                      ("SOL_THRESHOLD_DIAGONAL", 0x100), ("SOL_ROUTE_TOPK", 0), ("SOL_ROUTE_TOPP", 1),
                      ("SOL_F32", 1), ("SOL_ERR_INVALID_ARG", -1), ("SOL_ERR_UNSUPPORTED", -2),
                      ("SOL_ERR_HIP", -3), ("SOL_ERR_WORKSPACE", -4), ("SOL_ERR_NO_DATA", -5)]:
        m = re.search(rf"\b{name}\s*=\s*(-?(?:0x[0-9a-fA-F]+|\d+))", text)
        assert m and int(m.group(1), 0) == val
        assert getattr(sb, name) == val


P = ctypes.c_void_p
FAKE = [P(0x1000), P(0x2000), P(0x3000), P(0x4000)]  # never dereferenced: validation fails first


def fwd(*, B=1, H=2, N=1000, d=128, bq=128, bk=64, tau=0.5, mode=1, dtype=0, keep=0, ptrs=FAKE):
    return sb.lib().sol_attn_forward_ex(*ptrs, B, H, N, d, bq, bk, tau, mode, dtype, keep, None, 0, None, None, None)


@pytest.mark.parametrize("kwargs,code", [
    (dict(ptrs=[None] + FAKE[1:]), sb.SOL_ERR_INVALID_ARG),
    (dict(N=0), sb.SOL_ERR_INVALID_ARG),
    (dict(B=-1), sb.SOL_ERR_INVALID_ARG),
    (dict(mode=7), sb.SOL_ERR_INVALID_ARG),
    (dict(mode=sb.SOL_SPARSE | 0x200), sb.SOL_ERR_INVALID_ARG),
    (dict(mode=3 | sb.SOL_THRESHOLD_DIAGONAL), sb.SOL_ERR_INVALID_ARG),
    (dict(dtype=5), sb.SOL_ERR_INVALID_ARG),
    (dict(tau=float("nan")), sb.SOL_ERR_INVALID_ARG),
    (dict(keep=30), sb.SOL_ERR_INVALID_ARG),
    (dict(keep=1024), sb.SOL_ERR_INVALID_ARG),
    (dict(ptrs=[FAKE[0], FAKE[1], FAKE[2], FAKE[0]]), sb.SOL_ERR_INVALID_ARG),
    (dict(d=96), sb.SOL_ERR_UNSUPPORTED),
    (dict(bk=32), sb.SOL_ERR_UNSUPPORTED),
    (dict(bq=256), sb.SOL_ERR_UNSUPPORTED),
    (dict(N=64 * 60000), sb.SOL_ERR_UNSUPPORTED),
])
def test_forward_validation(kwargs, code):
    assert fwd(**kwargs) == code
    assert sb.last_error() != ""


def fwdc(*, B=1, H=2, N=1000, d=128, bq=128, bk=64, tau=0.5, mode=1, dtype=0, granule=1, ptrs=FAKE):
    return sb.lib().sol_attn_forward_causal(*ptrs, B, H, N, d, bq, bk, tau, mode, dtype, granule, None, 0, None, None,
                                            None)


@pytest.mark.parametrize("kwargs,code", [
    (dict(granule=0), sb.SOL_ERR_INVALID_ARG),
    (dict(granule=-3), sb.SOL_ERR_INVALID_ARG),
    (dict(mode=sb.SOL_SPARSE | sb.SOL_THRESHOLD_DIAGONAL), sb.SOL_ERR_INVALID_ARG),
    (dict(mode=5), sb.SOL_ERR_INVALID_ARG),
    (dict(tau=float("nan")), sb.SOL_ERR_INVALID_ARG),
    (dict(ptrs=[FAKE[0], None, FAKE[2], FAKE[3]]), sb.SOL_ERR_INVALID_ARG),
    (dict(d=96), sb.SOL_ERR_UNSUPPORTED),
    (dict(bq=32), sb.SOL_ERR_UNSUPPORTED),
    # the per-row proxies of a causal row live in LDS: 15000 key blocks fit without a mask only
    (dict(N=64 * 15000), sb.SOL_ERR_UNSUPPORTED),
])
def test_causal_forward_validation(kwargs, code):
    assert fwdc(**kwargs) == code
    assert sb.last_error() != ""


def test_causal_sizes_accepted_without_mask():
    # same size as the rejected causal case passes validation without the mask (fails only
    # later, at the fake pointers, which validation never reaches here: use the workspace query)
    assert sb.workspace_bytes(1, 2, 64 * 15000, 128, 128, 64, "sparse") > 0


def test_other_entry_points_validate():
    lib = sb.lib()
    assert lib.sol_attn_forward(None, None, None, None, 1, 1, 64, 64, 64, 64, 0.0, 1) == sb.SOL_ERR_INVALID_ARG
    assert lib.sol_attn_pool_blocks(*FAKE[:3], None, None, None, 1, 1, 64, 64, 64, 64, 0, None) == sb.SOL_ERR_INVALID_ARG
    assert lib.sol_attn_pool_blocks(None, *FAKE[1:3], FAKE[3], None, None, 1, 1, 64, 64, 64, 64, 0, None) == sb.SOL_ERR_INVALID_ARG
    assert lib.sol_attn_pool_blocks(*FAKE[:3], FAKE[3], None, None, 1, 1, 64, 80, 64, 64, 0, None) == sb.SOL_ERR_UNSUPPORTED
    assert lib.sol_attn_thresholds(FAKE[0], FAKE[1], FAKE[2], None, None, 1, 1, 4, 8, 9, 64, 0.0, 0, None) == sb.SOL_ERR_INVALID_ARG
    assert lib.sol_attn_thresholds(FAKE[0], FAKE[1], FAKE[2], None, None, 1, 1, 4, 8, 8, 64, math.nan, 0, None) == sb.SOL_ERR_INVALID_ARG
    assert lib.sol_attn_thresholds(FAKE[0], FAKE[1], FAKE[2], None, None, 1, 1, 4, 8, 8, 64, 0.0, 1, None) == sb.SOL_ERR_INVALID_ARG
    rm = lib.sol_attn_route_materialized
    assert rm(FAKE[0], FAKE[1], FAKE[2], None, 1, 1, 4, 8, 8, 64, 0, 2.0, None) == sb.SOL_ERR_INVALID_ARG
    assert rm(FAKE[0], FAKE[1], FAKE[2], FAKE[3], 1, 1, 4, 8, 8, 64, 0, 9.0, None) == sb.SOL_ERR_INVALID_ARG
    assert rm(FAKE[0], FAKE[1], FAKE[2], FAKE[3], 1, 1, 4, 8, 8, 64, 0, 2.5, None) == sb.SOL_ERR_INVALID_ARG
    assert rm(FAKE[0], FAKE[1], FAKE[2], FAKE[3], 1, 1, 4, 8, 8, 64, 1, 0.0, None) == sb.SOL_ERR_INVALID_ARG
    assert rm(FAKE[0], FAKE[1], FAKE[2], FAKE[3], 1, 1, 4, 8, 8, 64, 2, 0.5, None) == sb.SOL_ERR_INVALID_ARG
    assert rm(FAKE[0], FAKE[1], FAKE[2], FAKE[3], 1, 1, 4, 5000, 5000, 64, 1, 0.5, None) == sb.SOL_ERR_UNSUPPORTED
    assert rm(FAKE[0], FAKE[1], FAKE[2], FAKE[3], 1, 1, 4, 8, 8, 80, 0, 2.0, None) == sb.SOL_ERR_UNSUPPORTED
    arr = (ctypes.c_float * 4)()
    assert lib.sol_attn_stats(ctypes.cast(arr, P), 2, 2) == sb.SOL_ERR_NO_DATA
    assert lib.sol_attn_stats(None, 2, 2) == sb.SOL_ERR_INVALID_ARG


def test_workspace_bytes_accepts_the_threshold_flag():
    ws = sb.workspace_bytes
    assert ws(1, 2, 1000, 128, 128, 64, sb.SOL_SPARSE | sb.SOL_THRESHOLD_DIAGONAL) == ws(1, 2, 1000, 128, 128, 64, "sparse")
    assert ws(1, 2, 1000, 128, 128, 64, sb.SOL_SPARSE | 0x400) == 0


def test_workspace_bytes():
    ws = sb.workspace_bytes
    assert ws(1, 2, 1000, 128, 128, 64, "sparse") > 0
    assert ws(1, 2, 1000, 96, 128, 64, "sparse") == 0
    # the dense bf16 path needs only the transposed f16 values (+ per-block counts)
    dense = ws(1, 40, 75600, 128, 128, 64, "dense")
    assert dense >= 40 * 128 * 1182 * 64 * 2
    assert ws(1, 40, 75600, 128, 128, 64, "sparse") > dense
    assert ws(1, 2, 2048, 64, 64, 64, "sparse", sb.SOL_F32) > 0
