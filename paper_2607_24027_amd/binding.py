"""ctypes binding of libsolattn.so (C ABI in include/sol_attn.h).

Argument marshalling only: torch tensors supply device memory and the current
stream; every step of the computation runs in the library's HIP kernels.  The
library must be built (``python -m paper_2607_24027_amd.build``); loading fails
loudly otherwise.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsolattn.so")

SOL_DENSE, SOL_SPARSE, SOL_SPARSE_NO_CORRECTION = 0, 1, 2
SOL_BF16, SOL_F32 = 0, 1
SOL_THRESHOLD_DIAGONAL = 0x100
THRESHOLD_MODES = {"exact": 0, "diagonal": SOL_THRESHOLD_DIAGONAL}
SOL_OK, SOL_ERR_INVALID_ARG, SOL_ERR_UNSUPPORTED, SOL_ERR_HIP, SOL_ERR_WORKSPACE, SOL_ERR_NO_DATA = 0, -1, -2, -3, -4, -5
MODES = {"dense": SOL_DENSE, "sparse": SOL_SPARSE, "sparse_no_correction": SOL_SPARSE_NO_CORRECTION}

# (name, restype, argtypes) for every symbol of include/sol_attn.h
_P, _I, _F, _S = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
SIGNATURES = {
    "sol_attn_pool_blocks": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _P]),
    "sol_attn_thresholds": (_I, [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _P]),
    "sol_attn_forward": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I]),
    "sol_attn_forward_ex": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _I, _I, _P, _S, _P, _P, _P]),
    "sol_attn_forward_causal": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _I, _I, _P, _S, _P, _P, _P]),
    "sol_attn_forward_noalloc": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _I, _I, _P, _P, _P]),
    "sol_attn_workspace_bytes": (_S, [_I, _I, _I, _I, _I, _I, _I, _I, _I]),
    "sol_attn_stats": (_I, [_P, _I, _I, _P]),
    "sol_attn_timing_enable": (_I, [_I]),
    "sol_attn_kernel_timing": (_I, [_P, _P]),
    "sol_attn_route_materialized": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _F, _P]),
    "sol_attn_last_error": (ctypes.c_char_p, []),
    "sol_attn_release": (_I, []),
}

_lib = None


class SolAttnError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"sol_attn error {code}: {msg}")
        self.code = code


def lib() -> ctypes.CDLL:
    """Load libsolattn.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_24027_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def last_error() -> str:
    return lib().sol_attn_last_error().decode()


def _check(rc: int):
    if rc != SOL_OK:
        raise SolAttnError(rc, last_error())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(device) -> int:
    import torch
    return torch.cuda.current_stream(device).cuda_stream


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return SOL_BF16
    if t.dtype == torch.float32:
        return SOL_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _check_qkv(*ts):
    """q, k, v (any may be None): contiguous 4-D tensors of one shape, dtype and GPU device."""
    present = [t for t in ts if t is not None]
    if not present:
        raise ValueError("no input tensors given")
    ref = present[0]
    for t in present:
        if t.dim() != 4 or not t.is_contiguous():
            raise ValueError("q, k and v must be contiguous 4-D [B,H,N,d] tensors")
        if tuple(t.shape) != tuple(ref.shape):
            raise ValueError(f"q, k and v must have one shape (got {tuple(ref.shape)} and {tuple(t.shape)})")
        if t.dtype != ref.dtype:
            raise ValueError(f"q, k and v must have one dtype (got {ref.dtype} and {t.dtype})")
        if t.device != ref.device:
            raise ValueError(f"q, k and v must be on one device (got {ref.device} and {t.device})")
    _dtype_code(ref)


def _require_gpu(t):
    if t.device.type != "cuda":
        raise ValueError(f"tensors must be on a GPU (got device {t.device})")


def _check_buffer(name, t, shape, dtypes, device):
    """An output/scratch tensor handed to the library: exact shape, dtype and device, contiguous."""
    if t is None:
        return
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} must have dtype {' or '.join(str(d) for d in dtypes)} (got {t.dtype})")
    if t.device != device:
        raise ValueError(f"{name} must be on {device} (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _check_forward_buffers(q, block_q, nkr, out=None, counts=None, mask_out=None, workspace=None):
    """out like q; counts [B,H] 32-bit ints; mask_out [B,H,NQ,ceil(NKr/32)] int32; workspace a 1-D
    uint8 tensor (its size is checked by the library against sol_attn_workspace_bytes)."""
    import torch
    B, H, N, d = q.shape
    _check_buffer("out", out, q.shape, (q.dtype,), q.device)
    int32_like = tuple({torch.int32, getattr(torch, "uint32", torch.int32)})
    _check_buffer("counts", counts, (B, H), int32_like, q.device)
    if block_q > 0:
        _check_buffer("mask_out", mask_out, (B, H, -(-N // block_q), mask_words(nkr)), (torch.int32,), q.device)
    if workspace is not None:
        if workspace.dim() != 1:
            raise ValueError("workspace must be a 1-D uint8 tensor")
        _check_buffer("workspace", workspace, workspace.shape, (torch.uint8,), q.device)


def _check_pooled(qbar, kbar):
    """Pooled queries [B,H,NQ,d] and keys [B,H,NK,d]: f32, same B, H, d and GPU device."""
    import torch
    for name, t in (("qbar", qbar), ("kbar", kbar)):
        if t.dim() != 4 or t.dtype != torch.float32:
            raise ValueError(f"{name} must be a 4-D float32 tensor")
    if qbar.shape[:2] != kbar.shape[:2] or qbar.shape[3] != kbar.shape[3]:
        raise ValueError(f"qbar {tuple(qbar.shape)} and kbar {tuple(kbar.shape)} disagree in B, H or d")
    if qbar.device != kbar.device:
        raise ValueError("qbar and kbar must be on one device")


def pool_blocks(q, k, v, block_q: int, block_k: int):
    """Block means (Qbar [B,H,NQ,d], Kbar, Vbar [B,H,NK,d], f32) of q, k, v."""
    import torch
    _check_qkv(q, k, v)
    B, H, N, d = q.shape
    if block_q <= 0 or block_k <= 0:
        raise ValueError("block sizes must be positive")
    _require_gpu(next(t for t in (q, k, v) if t is not None))
    nq, nk = -(-N // block_q), -(-N // block_k)
    qbar = torch.empty((B, H, nq, d), device=q.device, dtype=torch.float32)
    kbar = torch.empty((B, H, nk, d), device=q.device, dtype=torch.float32)
    vbar = torch.empty((B, H, nk, d), device=q.device, dtype=torch.float32)
    _check(lib().sol_attn_pool_blocks(_ptr(q), _ptr(k), _ptr(v), _ptr(qbar), _ptr(kbar), _ptr(vbar),
                                      B, H, N, d, block_q, block_k, _dtype_code(q), _stream(q.device)))
    return qbar, kbar, vbar


def thresholds(qbar, kbar, beta: float, nk_routable: Optional[int] = None, threshold_mode: str = "exact"):
    """(tau, mu, sigma) [B,H,NQ] f32 from pooled queries/keys (moment form, or the
    diagonal estimator with threshold_mode="diagonal")."""
    import torch
    _check_pooled(qbar, kbar)
    B, H, NQ, d = qbar.shape
    NK = kbar.shape[2]
    nkr = NK if nk_routable is None else nk_routable
    _require_gpu(qbar)
    tau = torch.empty((B, H, NQ), device=qbar.device, dtype=torch.float32)
    mu = torch.empty_like(tau)
    sigma = torch.empty_like(tau)
    _check(lib().sol_attn_thresholds(_ptr(qbar.contiguous()), _ptr(kbar.contiguous()), _ptr(tau), _ptr(mu),
                                     _ptr(sigma), B, H, NQ, NK, nkr, d, float(beta),
                                     THRESHOLD_MODES[threshold_mode], _stream(qbar.device)))
    return tau, mu, sigma


def _mode_code(mode, threshold_mode="exact") -> int:
    return (MODES[mode] if isinstance(mode, str) else int(mode)) | THRESHOLD_MODES[threshold_mode]


SOL_ROUTE_TOPK, SOL_ROUTE_TOPP = 0, 1


def route_materialized(qbar, kbar, rule: str, param: float, nk_routable: Optional[int] = None, proxies=None,
                       mask_out=None):
    """Baseline routing through a materialised proxy map: rule "topk" (param = k) or "topp"
    (param = p).  Returns (proxies [B,H,NQ,NKr] f32, mask [B,H,NQ,MW] int32) device tensors."""
    import torch
    _check_pooled(qbar, kbar)
    B, H, NQ, d = qbar.shape
    NK = kbar.shape[2]
    nkr = NK if nk_routable is None else nk_routable
    _check_buffer("proxies", proxies, (B, H, NQ, nkr), (torch.float32,), qbar.device)
    _check_buffer("mask_out", mask_out, (B, H, NQ, mask_words(nkr)), (torch.int32,), qbar.device)
    _require_gpu(qbar)
    if proxies is None:
        proxies = torch.empty((B, H, NQ, nkr), device=qbar.device, dtype=torch.float32)
    if mask_out is None:
        mask_out = torch.empty((B, H, NQ, mask_words(nkr)), device=qbar.device, dtype=torch.int32)
    code = {"topk": SOL_ROUTE_TOPK, "topp": SOL_ROUTE_TOPP}[rule]
    _check(lib().sol_attn_route_materialized(_ptr(qbar.contiguous()), _ptr(kbar.contiguous()), _ptr(proxies),
                                             _ptr(mask_out), B, H, NQ, NK, nkr, d, code, float(param),
                                             _stream(qbar.device)))
    return proxies, mask_out


def workspace_bytes(B, H, N, d, block_q, block_k, mode, dtype=SOL_BF16, keep_tail_tokens=0) -> int:
    return int(lib().sol_attn_workspace_bytes(B, H, N, d, block_q, block_k, MODES.get(mode, mode), dtype,
                                              keep_tail_tokens))


def forward(q, k, v, block_q: int, block_k: int, tau: float, mode="sparse", keep_tail_tokens: int = 0,
            out=None, workspace=None, counts=None, mask_out=None, threshold_mode: str = "exact",
            causal_granule: int = 0):
    """Routed attention forward through sol_attn_forward_ex, or sol_attn_forward_causal when
    causal_granule > 0.  Returns out.  threshold_mode "diagonal" ORs SOL_THRESHOLD_DIAGONAL
    into the mode.  Every tensor is checked for shape, dtype and device before the call."""
    import torch
    _check_qkv(q, k, v)
    B, H, N, d = q.shape
    nkr = -(-N // block_k) - keep_tail_tokens // block_k if block_k > 0 else 0
    _check_forward_buffers(q, block_q, nkr, out, counts, mask_out, workspace)
    _require_gpu(q)
    if out is None:
        out = torch.empty_like(q)
    m = _mode_code(mode, threshold_mode)
    ws_ptr, ws_bytes = (None, 0) if workspace is None else (workspace.data_ptr(), workspace.numel() * workspace.element_size())
    if causal_granule:
        if keep_tail_tokens:
            raise ValueError("causal masks take no forced tail")
        _check(lib().sol_attn_forward_causal(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, N, d, block_q, block_k,
                                             float(tau), m, _dtype_code(q), int(causal_granule), ws_ptr, ws_bytes,
                                             _ptr(counts), _ptr(mask_out), _stream(q.device)))
        return out
    _check(lib().sol_attn_forward_ex(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, N, d, block_q, block_k,
                                     float(tau), m, _dtype_code(q), keep_tail_tokens, ws_ptr, ws_bytes,
                                     _ptr(counts), _ptr(mask_out), _stream(q.device)))
    return out


def forward_noalloc(q, k, v, out, counts, block_q: int, block_k: int, tau: float, mode="sparse",
                    keep_tail_tokens: int = 0, mask_out=None, threshold_mode: str = "exact"):
    """sol_attn_forward_noalloc: the forward with the library's built-in scratch (no device
    allocation by the library; out and counts are caller-owned and required)."""
    _check_qkv(q, k, v)
    if out is None or counts is None:
        raise ValueError("out and counts must be given")
    B, H, N, d = q.shape
    nkr = -(-N // block_k) - keep_tail_tokens // block_k if block_k > 0 else 0
    _check_forward_buffers(q, block_q, nkr, out, counts, mask_out)
    _require_gpu(q)
    _check(lib().sol_attn_forward_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, N, d, block_q, block_k,
                                          float(tau), _mode_code(mode, threshold_mode), _dtype_code(q),
                                          keep_tail_tokens, _ptr(counts), _ptr(mask_out), _stream(q.device)))
    return out


def forward_short(q, k, v, out, block_q: int, block_k: int, tau: float, mode="sparse"):
    """The 12-argument sol_attn_forward (bf16, default stream, library workspace)."""
    import torch
    _check_qkv(q, k, v)
    if q.dtype != torch.bfloat16:
        raise ValueError("sol_attn_forward takes bf16 tensors")
    if out is None:
        raise ValueError("out must be given")
    _check_forward_buffers(q, block_q, 0, out)
    _require_gpu(q)
    B, H, N, d = q.shape
    m = MODES[mode] if isinstance(mode, str) else int(mode)
    _check(lib().sol_attn_forward(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, N, d, block_q, block_k,
                                  float(tau), m))
    return out


def stats(B: int, H: int, counts=None):
    """Per-head selected fraction (host list, synchronising) of the forward that wrote `counts`
    (a [B,H] device tensor passed to forward()), or with counts=None of the last forward on this
    thread that used the library's own counts buffer."""
    if counts is not None:
        _check_buffer("counts", counts, (B, H), (counts.dtype,), counts.device)
        if counts.element_size() != 4 or counts.dtype.is_floating_point:
            raise ValueError("counts must be a 32-bit integer tensor")
        _require_gpu(counts)
    arr = (ctypes.c_float * (B * H))()
    _check(lib().sol_attn_stats(ctypes.cast(arr, ctypes.c_void_p), B, H, _ptr(counts)))
    return [float(x) for x in arr]


def mask_words(NKr: int) -> int:
    return -(-NKr // 32)


def unpack_mask(words, NKr: int):
    """[..., MW] int32/uint32 words -> [..., NKr] bool (bit j%32 of word j//32)."""
    import numpy as np
    w = np.asarray(words).astype(np.uint32)
    bits = ((w[..., :, None] >> np.arange(32, dtype=np.uint32)) & 1).astype(bool)
    return bits.reshape(w.shape[:-1] + (w.shape[-1] * 32,))[..., :NKr]


def timing_enable(enable: bool = True):
    _check(lib().sol_attn_timing_enable(1 if enable else 0))


def kernel_timing():
    """(total_ms, launches) of the fused attention kernel since the last call."""
    ms = ctypes.c_float()
    n = ctypes.c_int()
    _check(lib().sol_attn_kernel_timing(ctypes.cast(ctypes.pointer(ms), ctypes.c_void_p),
                                        ctypes.cast(ctypes.pointer(n), ctypes.c_void_p)))
    return float(ms.value), int(n.value)


def release():
    _check(lib().sol_attn_release())


NEG_INF = -math.inf
