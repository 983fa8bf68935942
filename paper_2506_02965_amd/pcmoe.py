"""ctypes binding of libpcmoe.so: the C ABI's calls under the same names, argument marshalling only.

Tensors are torch tensors on the GPU; their data pointers and the current HIP stream are handed
to the library. Every step of the layer runs in the library's HIP kernels. If the library is not
built, loading fails loudly: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libpcmoe.so")

MOE_OK, MOE_ERR_INVALID_ARGUMENT, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE_TOO_SMALL, MOE_ERR_HIP = range(5)
MOE_F32, MOE_BF16 = 0, 1
MOE_WS_PERMUTE, MOE_WS_FFN_SAVED, MOE_WS_FFN_FWD, MOE_WS_FFN_BWD, MOE_WS_ROUTE_BWD = range(5)

# every symbol include/pcmoe.h declares
EXPORTS = ("moe_workspace_size", "moe_route", "moe_permute", "moe_permute_noalloc", "moe_expert_ffn_fwd", "moe_combine", "moe_combine_bwd",
           "moe_expert_ffn_bwd", "moe_route_bwd", "moe_permute_bwd", "moe_expert_update", "moe_kernel_timing",
           "moe_kernel_timing_select", "moe_kernel_timing_report", "moe_status_string", "moe_last_error")
MOE_OPT_SGD, MOE_OPT_ADAMW = 0, 1


class moe_desc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("d_model", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32), ("local_begin", ctypes.c_int32),
                ("local_count", ctypes.c_int32), ("n_shared", ctypes.c_int32), ("renormalize", ctypes.c_int32),
                ("dtype", ctypes.c_int32)]


class moe_opt(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("lr", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("step", ctypes.c_int32)]


def make_opt(kind="adamw", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, step=1) -> moe_opt:
    return moe_opt(MOE_OPT_ADAMW if kind == "adamw" else MOE_OPT_SGD, lr, beta1, beta2, eps, weight_decay, step)


class MoeError(RuntimeError):
    def __init__(self, fn, status, detail):
        super().__init__(f"{fn}: {status_string(status)}: {detail}")
        self.status = status


_lib = None
_VP, _SZ, _I32, _INT = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int


def lib():
    """The loaded library (raises if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2506_02965_amd.build_lib`")
        L = ctypes.CDLL(LIB_PATH)
        D = ctypes.POINTER(moe_desc)
        sig = {
            "moe_workspace_size": (_SZ, [D, _INT]),
            "moe_route": (_INT, [D, _VP, _VP, _VP, _I32, _VP, _VP, _VP, _VP]),
            "moe_permute": (_INT, [D, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _SZ, _VP]),
            "moe_permute_noalloc": (_INT, [D, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP]),
            "moe_expert_ffn_fwd": (_INT, [D, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _SZ, _VP]),
            "moe_combine": (_INT, [D, _VP, _VP, _VP, _VP, _VP]),
            "moe_combine_bwd": (_INT, [D, _VP, _VP, _VP, _VP, _VP, _VP, _VP]),
            "moe_expert_ffn_bwd": (_INT, [D] + [_VP] * 14 + [_SZ, _VP]),
            "moe_route_bwd": (_INT, [D, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _SZ, _VP]),
            "moe_permute_bwd": (_INT, [D, _VP, _VP, _VP, _VP, _VP, _VP]),
            "moe_expert_update": (_INT, [D, ctypes.POINTER(moe_opt)] + [_VP] * 9 + [_VP]),
            "moe_kernel_timing": (_INT, [_INT]),
            "moe_kernel_timing_select": (_INT, [ctypes.c_char_p]),
            "moe_kernel_timing_report": (_SZ, [ctypes.c_char_p, _SZ]),
            "moe_status_string": (ctypes.c_char_p, [_INT]),
            "moe_last_error": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _lib = L
    return _lib


def status_string(st: int) -> str:
    return lib().moe_status_string(st).decode()


def last_error() -> str:
    return lib().moe_last_error().decode()


def _ptr(t) -> Optional[int]:
    """Device address of a tensor (or a raw integer address, passed through). A host tensor or a strided view
    would be read as if it were a dense device buffer, so both are refused here."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError(f"expected a GPU tensor, got one on {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"expected a contiguous tensor, got shape {tuple(t.shape)} strides {t.stride()}")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _check(fn, st):
    if st != MOE_OK:
        raise MoeError(fn, st, last_error())


def make_desc(T, d_model, d_ff, n_experts, top_k, local_begin=0, local_count=None, n_shared=0, renormalize=True,
              dtype="bf16") -> moe_desc:
    return moe_desc(T, d_model, d_ff, n_experts, top_k, local_begin,
                    n_experts if local_count is None else local_count, n_shared, int(bool(renormalize)),
                    MOE_BF16 if dtype == "bf16" else MOE_F32)


def moe_workspace_size(desc: moe_desc, which: int) -> int:
    return int(lib().moe_workspace_size(ctypes.byref(desc), which))


def moe_route(desc, x, w_router, logit_bias, bias_groups, logits, topk_idx, topk_w, stream=None):
    _check("moe_route", lib().moe_route(ctypes.byref(desc), _ptr(x), _ptr(w_router), _ptr(logit_bias), bias_groups,
                                        _ptr(logits), _ptr(topk_idx), _ptr(topk_w), _stream(stream)))


def moe_permute(desc, topk_idx, x, counts, offsets, row_to_slot, slot_to_row, x_perm, ws, ws_bytes, stream=None):
    _check("moe_permute", lib().moe_permute(ctypes.byref(desc), _ptr(topk_idx), _ptr(x), _ptr(counts), _ptr(offsets),
                                            _ptr(row_to_slot), _ptr(slot_to_row), _ptr(x_perm), _ptr(ws), ws_bytes,
                                            _stream(stream)))


def moe_permute_noalloc(desc, topk_idx, x, counts, offsets, row_to_slot, slot_to_row, x_perm, stream=None):
    _check("moe_permute_noalloc", lib().moe_permute_noalloc(
        ctypes.byref(desc), _ptr(topk_idx), _ptr(x), _ptr(counts), _ptr(offsets), _ptr(row_to_slot),
        _ptr(slot_to_row), _ptr(x_perm), _stream(stream)))


def moe_expert_ffn_fwd(desc, x, x_perm, offsets, w_gate, w_up, w_down, y_perm, saved, ws, ws_bytes, stream=None):
    _check("moe_expert_ffn_fwd", lib().moe_expert_ffn_fwd(
        ctypes.byref(desc), _ptr(x), _ptr(x_perm), _ptr(offsets), _ptr(w_gate), _ptr(w_up), _ptr(w_down),
        _ptr(y_perm), _ptr(saved), _ptr(ws), ws_bytes, _stream(stream)))


def moe_combine(desc, y_perm, slot_to_row, topk_w, y, stream=None):
    _check("moe_combine", lib().moe_combine(ctypes.byref(desc), _ptr(y_perm), _ptr(slot_to_row), _ptr(topk_w), _ptr(y),
                                            _stream(stream)))


def moe_combine_bwd(desc, dy, y_perm, slot_to_row, topk_w, dy_perm, dgate, stream=None):
    _check("moe_combine_bwd", lib().moe_combine_bwd(ctypes.byref(desc), _ptr(dy), _ptr(y_perm), _ptr(slot_to_row),
                                                    _ptr(topk_w), _ptr(dy_perm), _ptr(dgate), _stream(stream)))


def moe_expert_ffn_bwd(desc, x, x_perm, dy, dy_perm, offsets, w_gate, w_up, w_down, saved, dx_perm, dw_gate, dw_up,
                       dw_down, ws, ws_bytes, stream=None):
    _check("moe_expert_ffn_bwd", lib().moe_expert_ffn_bwd(
        ctypes.byref(desc), _ptr(x), _ptr(x_perm), _ptr(dy), _ptr(dy_perm), _ptr(offsets), _ptr(w_gate), _ptr(w_up),
        _ptr(w_down), _ptr(saved), _ptr(dx_perm), _ptr(dw_gate), _ptr(dw_up), _ptr(dw_down), _ptr(ws), ws_bytes,
        _stream(stream)))


def moe_route_bwd(desc, x, logits, topk_idx, topk_w, dgate, dlogits, dw_router, ws, ws_bytes, stream=None):
    _check("moe_route_bwd", lib().moe_route_bwd(ctypes.byref(desc), _ptr(x), _ptr(logits), _ptr(topk_idx),
                                                _ptr(topk_w), _ptr(dgate), _ptr(dlogits), _ptr(dw_router), _ptr(ws),
                                                ws_bytes, _stream(stream)))


def moe_permute_bwd(desc, dx_perm, slot_to_row, dlogits, w_router, dx, stream=None):
    _check("moe_permute_bwd", lib().moe_permute_bwd(ctypes.byref(desc), _ptr(dx_perm), _ptr(slot_to_row),
                                                    _ptr(dlogits), _ptr(w_router), _ptr(dx), _stream(stream)))


def moe_expert_update(desc, opt, w_gate, w_up, w_down, dw_gate, dw_up, dw_down, master=None, m=None, v=None,
                      stream=None):
    _check("moe_expert_update", lib().moe_expert_update(
        ctypes.byref(desc), ctypes.byref(opt), _ptr(w_gate), _ptr(w_up), _ptr(w_down), _ptr(dw_gate), _ptr(dw_up),
        _ptr(dw_down), _ptr(master), _ptr(m), _ptr(v), _stream(stream)))


def moe_kernel_timing(enable: bool):
    _check("moe_kernel_timing", lib().moe_kernel_timing(int(bool(enable))))


def moe_kernel_timing_select(name: Optional[str]):
    """Record only the launches of kernel `name` (None: all kernels)."""
    _check("moe_kernel_timing_select", lib().moe_kernel_timing_select(None if name is None else name.encode()))


def moe_kernel_timing_report() -> dict:
    """{kernel name: (launches, total ms)} of the launches recorded since timing was enabled."""
    n = lib().moe_kernel_timing_report(None, 0)
    buf = ctypes.create_string_buffer(int(n))
    lib().moe_kernel_timing_report(buf, n)
    out = {}
    for line in buf.value.decode().splitlines():
        name, cnt, ms = line.split()
        out[name] = (int(cnt), float(ms))
    return out
