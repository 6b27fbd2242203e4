"""Python binding of libsnn's C ABI (argument marshalling only).

Every function below has the name of the C entry point it calls and takes torch tensors in
place of device pointers; all computation happens in the HIP kernels of libsnn.so. Tensors
must be CUDA(HIP) tensors on the current device, contiguous, with the dtype the header
states. Work is enqueued on torch's current stream and nothing is synchronised, except in
the convenience helpers that say so.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsnn.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "snn.h")

SNN_OK, SNN_ERR_INVALID_ARG, SNN_ERR_UNSUPPORTED, SNN_ERR_HIP = 0, -1, -2, -3

_P = ctypes.c_void_p
_I = ctypes.c_int
_F = ctypes.c_float
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t

_SIGNATURES = {
    "snn_status_string": (ctypes.c_char_p, [_I]),
    "snn_lif_forward": (_I, [_P, _P, _I, _I, _I, _I, _F, _F, _P, _P, _P, _P]),
    "snn_active_compact_workspace": (_SZ, [_I, _I, _I]),
    "snn_active_compact": (_I, [_P, _I, _I, _I, _F, _F, _F, _P, _P, _P, _I64, _P, _P, _SZ, _P]),
    "snn_sparse_backward_workspace": (_SZ, [_I, _I, _I, _I, _I64]),
    "snn_sparse_backward": (_I, [_P, _P, _I, _I, _I, _I, _F, _P, _P, _P, _P, _I64, _P, _P, _I64, _P, _P, _P, _SZ,
                                 _P, _P]),
    "snn_active_bits_words": (_SZ, [_I, _I, _I]),
    "snn_lif_forward_active": (_I, [_P, _P, _I, _I, _I, _I, _F, _F, _F, _P, _P, _P, _P, _P]),
    "snn_lif_forward_traces": (_I, [_P, _P, _I, _I, _I, _I, _F, _F, _F, _P, _P, _P, _P, _F, _P, _P]),
    "snn_active_compact_bits_workspace": (_SZ, [_I, _I, _I]),
    "snn_active_compact_bits": (_I, [_P, _P, _I, _I, _I, _F, _F, _P, _P, _P, _I64, _P, _P, _SZ, _P]),
    "snn_active_compact_bits_noalloc": (_I, [_P, _P, _I, _I, _I, _F, _F, _P, _P, _P, _I64, _P, _P]),
    "snn_sparse_dw_workspace": (_SZ, [_I, _I, _I, _I, _I64]),
    "snn_sparse_dw": (_I, [_P, _I, _I, _I, _I, _P, _P, _P, _P, _I64, _P, _P, _SZ, _P]),
    "snn_sparse_dw_layout": (_I, [_I, _I, _I, _I, _P, _P, _I64, _P, _SZ, _P]),
    "snn_sparse_dw_prepared": (_I, [_P, _I, _I, _I, _I, _P, _P, _P, _P, _I64, _P, _P, _SZ, _P]),
    "snn_trace_checkpoint_count": (_I64, [_I, _I]),
    "snn_trace_checkpoints": (_I, [_P, _I, _I, _I, _F, _I, _P, _P]),
    "snn_sparse_dw_spikes_workspace": (_SZ, [_I, _I, _I, _I, _I64, _I]),
    "snn_sparse_dw_spikes": (_I, [_P, _P, _I, _F, _I, _I, _I, _I, _P, _P, _P, _P, _I64, _P, _P, _SZ, _P]),
    "snn_sparse_grad_in_workspace": (_SZ, [_I, _I, _I]),
    "snn_sparse_grad_in": (_I, [_P, _I, _I, _I, _I, _F, _P, _P, _P, _P, _I64, _P, _P, _I64, _P, _I, _P, _SZ, _P]),
    "snn_dense_backward_workspace": (_SZ, [_I, _I, _I, _I]),
    "snn_dense_backward_ref": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _F, _F, _F, _F, _P, _P, _P, _SZ, _P]),
    "snn_readout_ce_workspace": (_SZ, [_I, _I, _I, _I]),
    "snn_readout_ce": (_I, [_P, _P, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "snn_activity_reg_workspace": (_SZ, [_I, _I, _I]),
    "snn_activity_reg": (_I, [_P, _I, _I, _I, _F, _F, _F, _F, _P, _P, _P, _P, _SZ, _P]),
    "snn_activity_reg_grad": (_I, [_P, _I, _I, _I, _P, _P, _I64, _P, _P]),
    "snn_adam_step": (_I, [_P, _P, _P, _P, _I64, _F, _F, _F, _F, _I, _P]),
    "snn_conv_lif_forward": (_I, [_P, _P, _I, _I, _I, _I, _I, _I, _F, _F, _F, _P, _P, _P, _P, _P]),
    "snn_maxpool_spikes": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P]),
    "snn_pool_route_bits": (_I, [_P, _P, _I, _I, _I, _I, _I, _P, _P]),
    "snn_pool_scatter_eps": (_I, [_I, _I, _I, _I, _I, _P, _P, _I64, _P, _P, _P, _P, _I64, _P, _P]),
    "snn_pool_scatter_eps_dense": (_I, [_P, _P, _I, _I, _I, _I, _I, _P, _P]),
    "snn_conv_sparse_dw_workspace": (_SZ, [_I, _I, _I, _I, _I, _I]),
    "snn_conv_sparse_dw": (_I, [_P, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _I64, _P, _P, _SZ, _P]),
    "snn_conv_sparse_dw_pooled": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _F, _F, _P, _P, _P, _I64, _P, _P, _SZ,
                                       _P]),
    "snn_conv_dense_dw_workspace": (_SZ, [_I, _I, _I, _I, _I, _I]),
    "snn_conv_dense_dw": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _F, _F, _P, _P, _SZ, _P]),
}

_lib = None


class SnnError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {status_string(status)} ({status})")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libsnn.so (raises if it has not been built: there is no fallback path)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing; build it with `python -m paper_2105_08810_amd.build`")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(l, name)
            fn.restype = res
            fn.argtypes = args
        _lib = l
    return _lib


def status_string(status: int) -> str:
    return lib().snn_status_string(int(status)).decode()


def _ptr(t: Optional[torch.Tensor], dtype=None, name="tensor") -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream=None) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _check(fn: str, status: int):
    if status != SNN_OK:
        raise SnnError(fn, status)


def workspace(nbytes: int, device=None) -> torch.Tensor:
    """Device workspace of at least nbytes (256-byte aligned by the caching allocator)."""
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device or "cuda")


# ------------------------------------------------------------------ entry points

def snn_lif_forward(s_in, W, T, B, N_in, N_out, alpha, theta, V, s_out, trace_in=None, stream=None):
    _check("snn_lif_forward", lib().snn_lif_forward(
        _ptr(s_in, torch.uint8, "s_in"), _ptr(W, torch.float32, "W"), T, B, N_in, N_out, float(alpha), float(theta),
        _ptr(V, torch.float32, "V"), _ptr(s_out, torch.uint8, "s_out"), _ptr(trace_in, torch.float32, "trace_in"),
        _stream(stream)))


def snn_active_bits_words(T, B, N) -> int:
    return int(lib().snn_active_bits_words(T, B, N))


def snn_lif_forward_active(s_in, W, T, B, N_in, N_out, alpha, theta, b_th, V, s_out, trace_in, active_bits,
                           stream=None):
    _check("snn_lif_forward_active", lib().snn_lif_forward_active(
        _ptr(s_in, torch.uint8, "s_in"), _ptr(W, torch.float32, "W"), T, B, N_in, N_out, float(alpha), float(theta),
        float(b_th), _ptr(V, torch.float32, "V"), _ptr(s_out, torch.uint8, "s_out"),
        _ptr(trace_in, torch.float32, "trace_in"), _ptr(active_bits, torch.int64, "active_bits"), _stream(stream)))


def snn_lif_forward_traces(s_in, W, T, B, N_in, N_out, alpha, theta, b_th, V, s_out, trace_in, trace_out,
                           alpha_next, active_bits=None, stream=None):
    _check("snn_lif_forward_traces", lib().snn_lif_forward_traces(
        _ptr(s_in, torch.uint8, "s_in"), _ptr(W, torch.float32, "W"), T, B, N_in, N_out, float(alpha), float(theta),
        float(b_th), _ptr(V, torch.float32, "V"), _ptr(s_out, torch.uint8, "s_out"),
        _ptr(trace_in, torch.float32, "trace_in"), _ptr(trace_out, torch.float32, "trace_out"), float(alpha_next),
        _ptr(active_bits, torch.int64, "active_bits"), _stream(stream)))


def snn_active_compact_bits_workspace(T, B, N) -> int:
    return int(lib().snn_active_compact_bits_workspace(T, B, N))


def snn_active_compact_bits(active_bits, V, T, B, N, theta, beta, row_ptr, col_idx, g_act, capacity, nnz_dev, ws,
                            stream=None):
    _check("snn_active_compact_bits", lib().snn_active_compact_bits(
        _ptr(active_bits, torch.int64, "active_bits"), _ptr(V, torch.float32, "V"), T, B, N, float(theta),
        float(beta), _ptr(row_ptr, torch.int32, "row_ptr"), _ptr(col_idx, torch.int32, "col_idx"),
        _ptr(g_act, torch.float32, "g_act"), int(capacity), _ptr(nnz_dev, torch.int64, "nnz"),
        _ptr(ws, None, "workspace"), 0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def snn_active_compact_bits_noalloc(active_bits, V, T, B, N, theta, beta, row_ptr, col_idx, g_act, capacity,
                                    nnz_dev, stream=None):
    _check("snn_active_compact_bits_noalloc", lib().snn_active_compact_bits_noalloc(
        _ptr(active_bits, torch.int64, "active_bits"), _ptr(V, torch.float32, "V"), T, B, N, float(theta),
        float(beta), _ptr(row_ptr, torch.int32, "row_ptr"), _ptr(col_idx, torch.int32, "col_idx"),
        _ptr(g_act, torch.float32, "g_act"), int(capacity), _ptr(nnz_dev, torch.int64, "nnz"), _stream(stream)))


def snn_active_compact_workspace(T, B, N) -> int:
    return int(lib().snn_active_compact_workspace(T, B, N))


def snn_active_compact(V, T, B, N, theta, b_th, beta, row_ptr, col_idx, g_act, capacity, nnz_dev, ws,
                       stream=None):
    _check("snn_active_compact", lib().snn_active_compact(
        _ptr(V, torch.float32, "V"), T, B, N, float(theta), float(b_th), float(beta),
        _ptr(row_ptr, torch.int32, "row_ptr"), _ptr(col_idx, torch.int32, "col_idx"),
        _ptr(g_act, torch.float32, "g_act"), int(capacity), _ptr(nnz_dev, torch.int64, "nnz_dev"),
        _ptr(ws, None, "workspace"), ws.numel() * ws.element_size(), _stream(stream)))


def snn_sparse_backward_workspace(T, B, N_in, N_out, out_cap) -> int:
    return int(lib().snn_sparse_backward_workspace(T, B, N_in, N_out, int(out_cap)))


def snn_sparse_backward(W, trace_in, T, B, N_in, N_out, alpha, out_row_ptr, out_col_idx, out_g, eps_out, out_cap,
                        in_row_ptr, in_col_idx, in_cap, eps_in, dW, ws, stream=None, aux_stream=None):
    _check("snn_sparse_backward", lib().snn_sparse_backward(
        _ptr(W, torch.float32, "W"), _ptr(trace_in, torch.float32, "trace_in"), T, B, N_in, N_out, float(alpha),
        _ptr(out_row_ptr, torch.int32, "out_row_ptr"), _ptr(out_col_idx, torch.int32, "out_col_idx"),
        _ptr(out_g, torch.float32, "out_g"), _ptr(eps_out, torch.float32, "eps_out"), int(out_cap),
        _ptr(in_row_ptr, torch.int32, "in_row_ptr"), _ptr(in_col_idx, torch.int32, "in_col_idx"), int(in_cap),
        _ptr(eps_in, torch.float32, "eps_in"), _ptr(dW, torch.float32, "dW"),
        _ptr(ws, None, "workspace"), 0 if ws is None else ws.numel() * ws.element_size(), _stream(stream),
        None if aux_stream is None else aux_stream.cuda_stream))


def snn_sparse_dw_workspace(T, B, N_in, N_out, out_cap) -> int:
    return int(lib().snn_sparse_dw_workspace(T, B, N_in, N_out, int(out_cap)))


def snn_sparse_dw(trace_in, T, B, N_in, N_out, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, dW, ws,
                  stream=None):
    _check("snn_sparse_dw", lib().snn_sparse_dw(
        _ptr(trace_in, torch.float32, "trace_in"), T, B, N_in, N_out, _ptr(out_row_ptr, torch.int32, "out_row_ptr"),
        _ptr(out_col_idx, torch.int32, "out_col_idx"), _ptr(out_g, torch.float32, "out_g"),
        _ptr(eps_out, torch.float32, "eps_out"), int(out_cap), _ptr(dW, torch.float32, "dW"),
        _ptr(ws, None, "workspace"), 0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def snn_sparse_dw_layout(T, B, N_in, N_out, out_row_ptr, out_col_idx, out_cap, ws, stream=None):
    _check("snn_sparse_dw_layout", lib().snn_sparse_dw_layout(
        T, B, N_in, N_out, _ptr(out_row_ptr, torch.int32, "out_row_ptr"), _ptr(out_col_idx, torch.int32, "out_col_idx"),
        int(out_cap), _ptr(ws, None, "workspace"), 0 if ws is None else ws.numel() * ws.element_size(),
        _stream(stream)))


def snn_sparse_dw_prepared(trace_in, T, B, N_in, N_out, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, dW, ws,
                           stream=None):
    _check("snn_sparse_dw_prepared", lib().snn_sparse_dw_prepared(
        _ptr(trace_in, torch.float32, "trace_in"), T, B, N_in, N_out, _ptr(out_row_ptr, torch.int32, "out_row_ptr"),
        _ptr(out_col_idx, torch.int32, "out_col_idx"), _ptr(out_g, torch.float32, "out_g"),
        _ptr(eps_out, torch.float32, "eps_out"), int(out_cap), _ptr(dW, torch.float32, "dW"),
        _ptr(ws, None, "workspace"), 0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def sparse_dw_layout(trace_shape, out: "Csr", N_out, ws, stream=None):
    """Run snn_sparse_dw_layout for a layer whose input trace has shape [T, B, N_in] into ws."""
    T, B, N_in = trace_shape
    snn_sparse_dw_layout(T, B, N_in, N_out, out.row_ptr, out.col_idx, out.capacity, ws, stream)


def sparse_dw_prepared(trace_in, out: "Csr", eps_out, N_out, ws, stream=None, dW=None):
    """Run snn_sparse_dw_prepared (after sparse_dw_layout on ws). Returns dW [N_in, N_out]."""
    T, B, N_in = trace_in.shape
    if dW is None:
        dW = torch.empty((N_in, N_out), dtype=torch.float32, device=trace_in.device)
    snn_sparse_dw_prepared(trace_in, T, B, N_in, N_out, out.row_ptr, out.col_idx, out.g, eps_out, out.capacity, dW,
                           ws, stream)
    return dW


def snn_trace_checkpoint_count(T, K) -> int:
    return int(lib().snn_trace_checkpoint_count(T, K))


def snn_trace_checkpoints(s_in, T, B, N_in, alpha, K, ck, stream=None):
    _check("snn_trace_checkpoints", lib().snn_trace_checkpoints(
        _ptr(s_in, torch.uint8, "s_in"), T, B, N_in, float(alpha), K, _ptr(ck, torch.float32, "ck"), _stream(stream)))


def snn_sparse_dw_spikes_workspace(T, B, N_in, N_out, out_cap, K) -> int:
    return int(lib().snn_sparse_dw_spikes_workspace(T, B, N_in, N_out, int(out_cap), K))


def snn_sparse_dw_spikes(s_in, ck, K, alpha, T, B, N_in, N_out, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, dW,
                         ws, stream=None):
    _check("snn_sparse_dw_spikes", lib().snn_sparse_dw_spikes(
        _ptr(s_in, torch.uint8, "s_in"), _ptr(ck, torch.float32, "ck"), K, float(alpha), T, B, N_in, N_out,
        _ptr(out_row_ptr, torch.int32, "out_row_ptr"), _ptr(out_col_idx, torch.int32, "out_col_idx"),
        _ptr(out_g, torch.float32, "out_g"), _ptr(eps_out, torch.float32, "eps_out"), int(out_cap),
        _ptr(dW, torch.float32, "dW"), _ptr(ws, None, "workspace"),
        0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def snn_sparse_grad_in_workspace(T, B, N_out) -> int:
    return int(lib().snn_sparse_grad_in_workspace(T, B, N_out))


def snn_sparse_grad_in(W, T, B, N_in, N_out, alpha, out_row_ptr, out_col_idx, out_g, eps_out, out_cap, in_row_ptr,
                       in_col_idx, in_cap, eps_in, share_cu, ws, stream=None):
    _check("snn_sparse_grad_in", lib().snn_sparse_grad_in(
        _ptr(W, torch.float32, "W"), T, B, N_in, N_out, float(alpha), _ptr(out_row_ptr, torch.int32, "out_row_ptr"),
        _ptr(out_col_idx, torch.int32, "out_col_idx"), _ptr(out_g, torch.float32, "out_g"),
        _ptr(eps_out, torch.float32, "eps_out"), int(out_cap), _ptr(in_row_ptr, torch.int32, "in_row_ptr"),
        _ptr(in_col_idx, torch.int32, "in_col_idx"), int(in_cap), _ptr(eps_in, torch.float32, "eps_in"),
        int(share_cu), _ptr(ws, None, "workspace"), 0 if ws is None else ws.numel() * ws.element_size(),
        _stream(stream)))


def snn_dense_backward_workspace(T, B, N_in, N_out) -> int:
    return int(lib().snn_dense_backward_workspace(T, B, N_in, N_out))


def snn_dense_backward_ref(W, trace_in, V, eps_out, T, B, N_in, N_out, alpha, theta, b_th, beta, grad_in, dW, ws,
                           stream=None):
    _check("snn_dense_backward_ref", lib().snn_dense_backward_ref(
        _ptr(W, torch.float32, "W"), _ptr(trace_in, torch.float32, "trace_in"), _ptr(V, torch.float32, "V"),
        _ptr(eps_out, torch.float32, "eps_out"), T, B, N_in, N_out, float(alpha), float(theta), float(b_th),
        float(beta), _ptr(grad_in, torch.float32, "grad_in"), _ptr(dW, torch.float32, "dW"),
        _ptr(ws, None, "workspace"), ws.numel() * ws.element_size(), _stream(stream)))


def snn_readout_ce_workspace(T, B, C, mode) -> int:
    return int(lib().snn_readout_ce_workspace(T, B, C, mode))


def snn_readout_ce(V_out, labels, T, B, C, mode, row_ptr, col_idx, eps, loss, eps_dense, ws, stream=None):
    _check("snn_readout_ce", lib().snn_readout_ce(
        _ptr(V_out, torch.float32, "V_out"), _ptr(labels, torch.int32, "labels"), T, B, C, int(mode),
        _ptr(row_ptr, torch.int32, "row_ptr"), _ptr(col_idx, torch.int32, "col_idx"),
        _ptr(eps, torch.float32, "eps"), _ptr(loss, torch.float32, "loss"),
        _ptr(eps_dense, torch.float32, "eps_dense"), _ptr(ws, None, "workspace"), ws.numel() * ws.element_size(), _stream(stream)))


def snn_activity_reg_workspace(T, B, N) -> int:
    return int(lib().snn_activity_reg_workspace(T, B, N))


def snn_activity_reg(S, T, B, N, lam_low, nu_low, lam_up, nu_up, zeta, coef, penalty, ws, stream=None):
    _check("snn_activity_reg", lib().snn_activity_reg(
        _ptr(S, torch.uint8, "S"), T, B, N, float(lam_low), float(nu_low), float(lam_up), float(nu_up),
        _ptr(zeta, torch.int32, "zeta"), _ptr(coef, torch.float32, "coef"), _ptr(penalty, torch.float32, "penalty"),
        _ptr(ws, None, "workspace"), 0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def snn_activity_reg_grad(coef, T, B, N, row_ptr, col_idx, capacity, eps, stream=None):
    _check("snn_activity_reg_grad", lib().snn_activity_reg_grad(
        _ptr(coef, torch.float32, "coef"), T, B, N, _ptr(row_ptr, torch.int32, "row_ptr"),
        _ptr(col_idx, torch.int32, "col_idx"), int(capacity), _ptr(eps, torch.float32, "eps"), _stream(stream)))


def snn_adam_step(W, grad, m, v, n, lr, beta1, beta2, eps, step, stream=None):
    _check("snn_adam_step", lib().snn_adam_step(
        _ptr(W, torch.float32, "W"), _ptr(grad, torch.float32, "grad"), _ptr(m, torch.float32, "m"),
        _ptr(v, torch.float32, "v"), int(n), float(lr), float(beta1), float(beta2), float(eps), int(step),
        _stream(stream)))


def _nbytes(ws):
    return 0 if ws is None else ws.numel() * ws.element_size()


def snn_conv_lif_forward(s_in, Wc, T, B, H, W, C, F, alpha, theta, b_th, V, s_out, trace_in=None, active_bits=None,
                         stream=None):
    _check("snn_conv_lif_forward", lib().snn_conv_lif_forward(
        _ptr(s_in, torch.uint8, "s_in"), _ptr(Wc, torch.float32, "Wc"), T, B, H, W, C, F, float(alpha), float(theta),
        float(b_th), _ptr(V, torch.float32, "V"), _ptr(s_out, torch.uint8, "s_out"),
        _ptr(trace_in, torch.float32, "trace_in"), _ptr(active_bits, torch.int64, "active_bits"), _stream(stream)))


def snn_maxpool_spikes(S, T, B, H, W, F, P, arg, stream=None):
    _check("snn_maxpool_spikes", lib().snn_maxpool_spikes(
        _ptr(S, torch.uint8, "S"), T, B, H, W, F, _ptr(P, torch.uint8, "P"), _ptr(arg, torch.uint8, "arg"),
        _stream(stream)))


def snn_pool_route_bits(conv_bits, arg, T, B, H, W, F, pool_bits, stream=None):
    _check("snn_pool_route_bits", lib().snn_pool_route_bits(
        _ptr(conv_bits, torch.int64, "conv_bits"), _ptr(arg, torch.uint8, "arg"), T, B, H, W, F,
        _ptr(pool_bits, torch.int64, "pool_bits"), _stream(stream)))


def snn_pool_scatter_eps(T, B, H, W, F, pool_row_ptr, pool_col_idx, pool_cap, eps_pool, arg, conv_row_ptr,
                         conv_col_idx, conv_cap, eps_conv, stream=None):
    _check("snn_pool_scatter_eps", lib().snn_pool_scatter_eps(
        T, B, H, W, F, _ptr(pool_row_ptr, torch.int32, "pool_row_ptr"), _ptr(pool_col_idx, torch.int32, "pool_col_idx"),
        int(pool_cap), _ptr(eps_pool, torch.float32, "eps_pool"), _ptr(arg, torch.uint8, "arg"),
        _ptr(conv_row_ptr, torch.int32, "conv_row_ptr"), _ptr(conv_col_idx, torch.int32, "conv_col_idx"),
        int(conv_cap), _ptr(eps_conv, torch.float32, "eps_conv"), _stream(stream)))


def snn_pool_scatter_eps_dense(eps_pool, arg, T, B, H, W, F, eps_conv, stream=None):
    _check("snn_pool_scatter_eps_dense", lib().snn_pool_scatter_eps_dense(
        _ptr(eps_pool, torch.float32, "eps_pool"), _ptr(arg, torch.uint8, "arg"), T, B, H, W, F,
        _ptr(eps_conv, torch.float32, "eps_conv"), _stream(stream)))


def snn_conv_sparse_dw_workspace(T, B, H, W, C, F) -> int:
    return int(lib().snn_conv_sparse_dw_workspace(T, B, H, W, C, F))


def snn_conv_sparse_dw(trace_in, T, B, H, W, C, F, conv_row_ptr, conv_col_idx, conv_g, eps_conv, conv_cap, dWc, ws,
                       stream=None):
    _check("snn_conv_sparse_dw", lib().snn_conv_sparse_dw(
        _ptr(trace_in, torch.float32, "trace_in"), T, B, H, W, C, F, _ptr(conv_row_ptr, torch.int32, "conv_row_ptr"),
        _ptr(conv_col_idx, torch.int32, "conv_col_idx"), _ptr(conv_g, torch.float32, "conv_g"),
        _ptr(eps_conv, torch.float32, "eps_conv"), int(conv_cap), _ptr(dWc, torch.float32, "dWc"),
        _ptr(ws, None, "workspace"), _nbytes(ws), _stream(stream)))


def snn_conv_sparse_dw_pooled(trace_in, V, arg, T, B, H, W, C, F, theta, b_th, beta, pool_row_ptr, pool_col_idx,
                              eps_pool, pool_cap, dWc, ws, stream=None):
    _check("snn_conv_sparse_dw_pooled", lib().snn_conv_sparse_dw_pooled(
        _ptr(trace_in, torch.float32, "trace_in"), _ptr(V, torch.float32, "V"), _ptr(arg, torch.uint8, "arg"),
        T, B, H, W, C, F, float(theta), float(b_th), float(beta), _ptr(pool_row_ptr, torch.int32, "pool_row_ptr"),
        _ptr(pool_col_idx, torch.int32, "pool_col_idx"), _ptr(eps_pool, torch.float32, "eps_pool"), int(pool_cap),
        _ptr(dWc, torch.float32, "dWc"), _ptr(ws, None, "workspace"), _nbytes(ws), _stream(stream)))


def snn_conv_dense_dw_workspace(T, B, H, W, C, F) -> int:
    return int(lib().snn_conv_dense_dw_workspace(T, B, H, W, C, F))


def snn_conv_dense_dw(trace_in, V, eps_conv, T, B, H, W, C, F, theta, b_th, beta, dWc, ws, stream=None):
    _check("snn_conv_dense_dw", lib().snn_conv_dense_dw(
        _ptr(trace_in, torch.float32, "trace_in"), _ptr(V, torch.float32, "V"), _ptr(eps_conv, torch.float32, "eps_conv"),
        T, B, H, W, C, F, float(theta), float(b_th), float(beta), _ptr(dWc, torch.float32, "dWc"),
        _ptr(ws, None, "workspace"), _nbytes(ws), _stream(stream)))


# ------------------------------------------------------------------ allocation helpers

def lif_forward(s_in: torch.Tensor, W: torch.Tensor, alpha, theta, want_trace=True):
    """Allocate outputs and run snn_lif_forward. Returns (V, s_out, trace or None)."""
    T, B, N_in = s_in.shape
    N_out = W.shape[1]
    V = torch.empty((T, B, N_out), dtype=torch.float32, device=s_in.device)
    S = torch.empty((T, B, N_out), dtype=torch.uint8, device=s_in.device)
    tr = torch.empty((T, B, N_in), dtype=torch.float32, device=s_in.device) if want_trace else None
    snn_lif_forward(s_in, W, T, B, N_in, N_out, alpha, theta, V, S, tr)
    return V, S, tr


class Csr:
    """Device CSR of an active set: row_ptr [T*B+1], col_idx / g [capacity], nnz (int64 device scalar)."""

    def __init__(self, row_ptr, col_idx, g, nnz_dev, capacity):
        self.row_ptr, self.col_idx, self.g, self.nnz_dev, self.capacity = row_ptr, col_idx, g, nnz_dev, capacity

    def nnz(self) -> int:
        return int(self.nnz_dev.item())

    def record_stream(self, stream) -> None:
        """Mark every buffer as used on stream (for the caching allocator, when the CSR was made on
        another stream)."""
        for t in (self.row_ptr, self.col_idx, self.g, self.nnz_dev):
            if t is not None:
                t.record_stream(stream)


def active_compact(V: torch.Tensor, theta, b_th, beta, capacity: Optional[int] = None, with_g=True) -> Csr:
    """Allocate and run snn_active_compact. Without a capacity it first counts (one host sync)."""
    T, B, N = V.shape
    dev = V.device
    ws = workspace(snn_active_compact_workspace(T, B, N), dev)
    row_ptr = torch.empty(T * B + 1, dtype=torch.int32, device=dev)
    nnz = torch.empty(1, dtype=torch.int64, device=dev)
    if capacity is None:
        snn_active_compact(V, T, B, N, theta, b_th, beta, row_ptr, None, None, 0, nnz, ws)
        capacity = int(nnz.item())
    cap = max(int(capacity), 1)
    col = torch.empty(cap, dtype=torch.int32, device=dev)
    g = torch.empty(cap, dtype=torch.float32, device=dev) if with_g else None
    snn_active_compact(V, T, B, N, theta, b_th, beta, row_ptr, col, g, cap, nnz, ws)
    return Csr(row_ptr, col, g, nnz, cap)


def active_compact_bits(bits: torch.Tensor, V: Optional[torch.Tensor], theta, beta, capacity: Optional[int] = None,
                        with_g=True, shape=None) -> Csr:
    """Allocate and run snn_active_compact_bits. Without a capacity it first counts (one host sync).
    shape = (T, B, N) when V is None (then with_g must be False)."""
    T, B, N = V.shape if V is not None else shape
    dev = bits.device
    ws = workspace(snn_active_compact_bits_workspace(T, B, N), dev)
    row_ptr = torch.empty(T * B + 1, dtype=torch.int32, device=dev)
    nnz = torch.empty(1, dtype=torch.int64, device=dev)
    if capacity is None:
        snn_active_compact_bits(bits, V, T, B, N, theta, beta, row_ptr, None, None, 0, nnz, ws)
        capacity = int(nnz.item())
    cap = max(int(capacity), 1)
    col = torch.empty(cap, dtype=torch.int32, device=dev)
    g = torch.empty(cap, dtype=torch.float32, device=dev) if with_g else None
    snn_active_compact_bits(bits, V, T, B, N, theta, beta, row_ptr, col, g, cap, nnz, ws)
    return Csr(row_ptr, col, g, nnz, cap)


def readout_ce(V_out: torch.Tensor, labels: torch.Tensor, mode: int, dense=False):
    """Allocate and run snn_readout_ce. Returns (Csr with g=None, eps, loss, eps_dense or None)."""
    T, B, C = V_out.shape
    dev = V_out.device
    nnz = B * C if mode == 0 else T * B * C
    row_ptr = torch.empty(T * B + 1, dtype=torch.int32, device=dev)
    col = torch.empty(nnz, dtype=torch.int32, device=dev)
    eps = torch.empty(nnz, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    ed = torch.empty((T, B, C), dtype=torch.float32, device=dev) if dense else None
    ws = workspace(snn_readout_ce_workspace(T, B, C, mode), dev)
    snn_readout_ce(V_out, labels, T, B, C, mode, row_ptr, col, eps, loss, ed, ws)
    nnz_dev = torch.full((1,), nnz, dtype=torch.int64, device=dev)
    return Csr(row_ptr, col, None, nnz_dev, nnz), eps, loss, ed


def sparse_backward(W, trace_in, alpha, out: Csr, eps_out, inp: Optional[Csr] = None, ws=None, aux_stream=None):
    """Allocate outputs and run snn_sparse_backward. Returns (dW, eps_in or None).
    aux_stream (a torch.cuda.Stream) lets the spike-gradient part run beside dW."""
    T, B, N_in = trace_in.shape
    N_out = W.shape[1]
    dev = W.device
    dW = torch.empty((N_in, N_out), dtype=torch.float32, device=dev)
    eps_in = torch.empty(inp.capacity, dtype=torch.float32, device=dev) if inp is not None else None
    if ws is None:
        ws = workspace(snn_sparse_backward_workspace(T, B, N_in, N_out, out.capacity), dev)
    snn_sparse_backward(W, trace_in, T, B, N_in, N_out, alpha, out.row_ptr, out.col_idx, out.g, eps_out,
                        out.capacity, None if inp is None else inp.row_ptr, None if inp is None else inp.col_idx,
                        0 if inp is None else inp.capacity, eps_in, dW, ws, aux_stream=aux_stream)
    return dW, eps_in


def sparse_dw(trace_in, out: Csr, eps_out, N_out, ws=None, stream=None, dW=None):
    """Run snn_sparse_dw (dW only). Returns dW [N_in, N_out]."""
    T, B, N_in = trace_in.shape
    dev = trace_in.device
    if dW is None:
        dW = torch.empty((N_in, N_out), dtype=torch.float32, device=dev)
    if ws is None:
        ws = workspace(snn_sparse_dw_workspace(T, B, N_in, N_out, out.capacity), dev)
    snn_sparse_dw(trace_in, T, B, N_in, N_out, out.row_ptr, out.col_idx, out.g, eps_out, out.capacity, dW, ws,
                  stream)
    return dW


def trace_checkpoints(s_in: torch.Tensor, alpha, K: int, ck=None, stream=None):
    """Run snn_trace_checkpoints on s_in [T, B, N_in]. Returns ck [ceil(T/K), B, N_in]."""
    T, B, N_in = s_in.shape
    if ck is None:
        ck = torch.empty((snn_trace_checkpoint_count(T, K), B, N_in), dtype=torch.float32, device=s_in.device)
    snn_trace_checkpoints(s_in, T, B, N_in, alpha, K, ck, stream)
    return ck


def sparse_dw_spikes(s_in, ck, K, alpha, out: Csr, eps_out, N_out, ws=None, stream=None, dW=None):
    """Run snn_sparse_dw_spikes (dW with the trace rebuilt from s_in and checkpoints ck)."""
    T, B, N_in = s_in.shape
    dev = s_in.device
    if dW is None:
        dW = torch.empty((N_in, N_out), dtype=torch.float32, device=dev)
    if ws is None:
        ws = workspace(snn_sparse_dw_spikes_workspace(T, B, N_in, N_out, out.capacity, K), dev)
    snn_sparse_dw_spikes(s_in, ck, K, alpha, T, B, N_in, N_out, out.row_ptr, out.col_idx, out.g, eps_out,
                         out.capacity, dW, ws, stream)
    return dW


def sparse_grad_in(W, alpha, T, B, out: Csr, eps_out, inp: Csr, share_cu=False, ws=None, stream=None,
                   eps_in=None):
    """Run snn_sparse_grad_in. Returns eps_in aligned with inp."""
    N_in, N_out = W.shape
    dev = W.device
    if eps_in is None:
        eps_in = torch.empty(inp.capacity, dtype=torch.float32, device=dev)
    if ws is None:
        ws = workspace(snn_sparse_grad_in_workspace(T, B, N_out), dev)
    snn_sparse_grad_in(W, T, B, N_in, N_out, alpha, out.row_ptr, out.col_idx, out.g, eps_out, out.capacity,
                       inp.row_ptr, inp.col_idx, inp.capacity, eps_in, share_cu, ws, stream)
    return eps_in


def dense_backward_ref(W, trace_in, V, eps_out, alpha, theta, b_th, beta, grad_in=True, ws=None):
    """Allocate outputs and run snn_dense_backward_ref. Returns (dW, grad_in or None)."""
    T, B, N_in = trace_in.shape
    N_out = W.shape[1]
    dev = W.device
    dW = torch.empty((N_in, N_out), dtype=torch.float32, device=dev)
    gi = torch.empty((T, B, N_in), dtype=torch.float32, device=dev) if grad_in else None
    if ws is None:
        ws = workspace(snn_dense_backward_workspace(T, B, N_in, N_out), dev)
    snn_dense_backward_ref(W, trace_in, V, eps_out, T, B, N_in, N_out, alpha, theta, b_th, beta, gi, dW, ws)
    return dW, gi


def activity_reg(S: torch.Tensor, lam_low, nu_low, lam_up, nu_up, want_zeta=False, ws=None, stream=None):
    """Allocate and run snn_activity_reg on S [T, B, N]. Returns (coef [B, N], penalty [1], zeta or None)."""
    T, B, N = S.shape
    dev = S.device
    coef = torch.empty((B, N), dtype=torch.float32, device=dev)
    pen = torch.empty(1, dtype=torch.float32, device=dev)
    zeta = torch.empty((B, N), dtype=torch.int32, device=dev) if want_zeta else None
    if ws is None:
        ws = workspace(snn_activity_reg_workspace(T, B, N), dev)
    snn_activity_reg(S, T, B, N, lam_low, nu_low, lam_up, nu_up, zeta, coef, pen, ws, stream)
    return coef, pen, zeta


def activity_reg_grad(coef: torch.Tensor, T: int, eps: torch.Tensor, csr: Optional["Csr"] = None, stream=None):
    """Run snn_activity_reg_grad: eps at csr's entries (or dense [T, B, N] when csr is None) += coef."""
    B, N = coef.shape
    if csr is None:
        snn_activity_reg_grad(coef, T, B, N, None, None, 0, eps, stream)
    else:
        snn_activity_reg_grad(coef, T, B, N, csr.row_ptr, csr.col_idx, min(csr.capacity, eps.numel()), eps, stream)
    return eps


def adam_step(W, grad, m, v, step, lr, betas=(0.9, 0.999), eps=1e-8, stream=None):
    """Run snn_adam_step on W in place (m and v are its float32 moment buffers)."""
    n = W.numel()
    if grad.numel() != n or m.numel() != n or v.numel() != n:
        raise ValueError("adam_step: W, grad, m and v must have the same size")
    snn_adam_step(W, grad, m, v, n, lr, betas[0], betas[1], eps, step, stream)
    return W


INF = math.inf
