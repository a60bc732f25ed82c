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
    assert len(names) == 13
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
    # the routing state of a block lives in LDS: at d = 128 the last supported length is 1,478,656
    # tokens (23,104 key blocks), at d = 64 1,971,200 (30,800 key blocks)
    (dict(N=1478656 + 64), sb.SOL_ERR_UNSUPPORTED),
    (dict(N=1971200 + 64, d=64), sb.SOL_ERR_UNSUPPORTED),
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
    # a causal row's proxies live in the tile stages while they fit there (16384 key blocks at
    # d = 128), and past that beside the lists, which no longer fit: 16385 key blocks fit without
    # a mask only
    (dict(N=64 * 16385), sb.SOL_ERR_UNSUPPORTED),
    (dict(N=1015808 + 64, d=64, bq=128), sb.SOL_ERR_UNSUPPORTED),
])
def test_causal_forward_validation(kwargs, code):
    assert fwdc(**kwargs) == code
    assert sb.last_error() != ""


def test_causal_sizes_accepted_without_mask():
    # same size as the rejected causal case passes validation without the mask (fails only
    # later, at the fake pointers, which validation never reaches here: use the workspace query)
    assert sb.workspace_bytes(1, 2, 64 * 16385, 128, 128, 64, "sparse") > 0


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
    assert lib.sol_attn_stats(None, 2, 2, None) == sb.SOL_ERR_INVALID_ARG
    assert lib.sol_attn_stats(ctypes.cast(arr, P), 0, 2, None) == sb.SOL_ERR_INVALID_ARG


def test_noalloc_entry_point_validates_before_any_gpu_call():
    lib = sb.lib()
    na = lib.sol_attn_forward_noalloc
    # counts are required (the library's own counts buffer would need an allocation)
    assert na(*FAKE, 1, 2, 1000, 128, 128, 64, 0.5, 1, 0, 0, None, None, None) == sb.SOL_ERR_INVALID_ARG
    assert "counts" in sb.last_error()
    # a shape whose workspace exceeds the built-in scratch: a clear error, no GPU call
    assert sb.workspace_bytes(1, 40, 75600, 128, 128, 64, "sparse") > 64 << 20
    assert na(*FAKE, 1, 40, 75600, 128, 128, 64, 0.5, 1, 0, 0, P(0x5000), None, None) == sb.SOL_ERR_WORKSPACE
    assert "built-in scratch" in sb.last_error()
    # the usual validation runs first
    assert na(*FAKE, 1, 2, 1000, 96, 128, 64, 0.5, 1, 0, 0, P(0x5000), None, None) == sb.SOL_ERR_UNSUPPORTED


def test_stats_without_a_forward_has_no_data():
    # No forward has run on this thread (CPU tests never launch one): with counts = NULL there
    # is no record; a counts buffer no forward wrote has none either.  Both fail before any HIP
    # call.
    import threading
    lib = sb.lib()
    arr = (ctypes.c_float * 4)()
    res = {}

    def probe():
        res["null"] = lib.sol_attn_stats(ctypes.cast(arr, P), 2, 2, None)
        res["null_msg"] = sb.last_error()
        res["foreign"] = lib.sol_attn_stats(ctypes.cast(arr, P), 2, 2, P(0x5000))
        res["foreign_msg"] = sb.last_error()

    t = threading.Thread(target=probe)   # a fresh thread: no last forward of its own
    t.start()
    t.join()
    assert res["null"] == sb.SOL_ERR_NO_DATA and "thread" in res["null_msg"]
    assert res["foreign"] == sb.SOL_ERR_NO_DATA and "not written" in res["foreign_msg"]


# --------------------------------------------------------------------------- binding argument checks
# The Python binding checks every tensor it hands to the library (shape, dtype, device, layout)
# before the call, so a mismatched tensor never reaches a kernel.  CPU tensors get through the
# shape/dtype/buffer checks and stop at the GPU check, which comes last.

def _qkv(B=1, H=2, N=300, d=64, dtype=None):
    import torch
    dtype = dtype or torch.bfloat16
    return tuple(torch.zeros((B, H, N, d), dtype=dtype) for _ in range(3))


def test_binding_rejects_mismatched_inputs():
    import torch
    q, k, v = _qkv()
    with pytest.raises(ValueError, match="one shape"):
        sb.forward(q, k[:, :, :299].contiguous(), v, 64, 64, 0.5)
    with pytest.raises(ValueError, match="one shape"):
        sb.forward(q, k, torch.zeros((1, 2, 300, 128), dtype=torch.bfloat16), 64, 64, 0.5)
    with pytest.raises(ValueError, match="one dtype"):
        sb.forward(q, k.float(), v, 64, 64, 0.5)
    with pytest.raises(ValueError, match="one device"):
        sb.forward(q, k, torch.empty_like(v, device="meta"), 64, 64, 0.5)
    with pytest.raises(ValueError, match="contiguous"):
        sb.forward(q, k.transpose(2, 3).contiguous().transpose(2, 3), v, 64, 64, 0.5)
    with pytest.raises(TypeError):
        sb.forward(*(t.half() for t in (q, k, v)), 64, 64, 0.5)
    with pytest.raises(ValueError, match="GPU"):
        sb.forward(q, k, v, 64, 64, 0.5)   # every check passes but the device


@pytest.mark.parametrize("what,bad", [
    ("out", lambda q: torch_zeros((1, 2, 299, 64), "bfloat16")),
    ("out", lambda q: torch_zeros((1, 2, 300, 64), "float32")),
    ("out", lambda q: torch_zeros((1, 2, 300, 64), "bfloat16", device="meta")),
    ("counts", lambda q: torch_zeros((2, 1), "int32")),
    ("counts", lambda q: torch_zeros((1, 2), "int64")),
    ("counts", lambda q: torch_zeros((1, 2), "float32")),
    ("mask_out", lambda q: torch_zeros((1, 2, 5, 2), "int32")),     # 300 rows: NQ = NK = 5, one mask word
    ("mask_out", lambda q: torch_zeros((1, 2, 4, 1), "int32")),
    ("mask_out", lambda q: torch_zeros((1, 2, 5, 1), "int64")),
    ("workspace", lambda q: torch_zeros((16,), "int32")),
    ("workspace", lambda q: torch_zeros((4, 4), "uint8")),
])
def test_binding_rejects_bad_buffers(what, bad):
    q, k, v = _qkv()
    with pytest.raises(ValueError, match=what):
        sb.forward(q, k, v, 64, 64, 0.5, **{what: bad(q)})


def test_binding_accepts_matching_buffers_up_to_the_gpu_check():
    q, k, v = _qkv()
    bufs = dict(out=torch_zeros((1, 2, 300, 64), "bfloat16"), counts=torch_zeros((1, 2), "int32"),
                mask_out=torch_zeros((1, 2, 5, 1), "int32"), workspace=torch_zeros((1024,), "uint8"))
    with pytest.raises(ValueError, match="GPU"):
        sb.forward(q, k, v, 64, 64, 0.5, **bufs)
    # 64 forced tail tokens leave 4 routable key blocks: still one mask word
    with pytest.raises(ValueError, match="GPU"):
        sb.forward(q, k, v, 64, 64, 0.5, keep_tail_tokens=64, **bufs)


def test_binding_short_form_and_other_calls_check_arguments():
    import torch
    q, k, v = _qkv()
    with pytest.raises(ValueError, match="bf16"):
        sb.forward_short(q.float(), k.float(), v.float(), torch.zeros_like(q.float()), 64, 64, 0.5)
    with pytest.raises(ValueError, match="out"):
        sb.forward_short(q, k, v, torch_zeros((1, 2, 300, 32), "bfloat16"), 64, 64, 0.5)
    with pytest.raises(ValueError, match="one shape"):
        sb.pool_blocks(q, k[:, :1].contiguous(), v, 64, 64)
    with pytest.raises(ValueError, match="counts"):
        sb.stats(1, 2, counts=torch_zeros((2, 2), "int32"))
    with pytest.raises(ValueError, match="32-bit"):
        sb.stats(1, 2, counts=torch_zeros((1, 2), "int64"))
    qbar, kbar = torch_zeros((1, 2, 5, 64), "float32"), torch_zeros((1, 2, 5, 64), "float32")
    with pytest.raises(ValueError, match="disagree"):
        sb.thresholds(qbar, torch_zeros((1, 3, 5, 64), "float32"), 0.5)
    with pytest.raises(ValueError, match="float32"):
        sb.route_materialized(qbar.double(), kbar, "topk", 2)
    with pytest.raises(ValueError, match="proxies"):
        sb.route_materialized(qbar, kbar, "topk", 2, proxies=torch_zeros((1, 2, 5, 4), "float32"))


def torch_zeros(shape, dtype, device="cpu"):
    import torch
    return torch.zeros(shape, dtype=getattr(torch, dtype), device=device)


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
