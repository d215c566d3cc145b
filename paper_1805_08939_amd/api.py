"""Thin Python binding of the C ABI: the same names as include/ard.h.

Argument marshalling only. Device buffers are torch tensors (memory and
streams come from PyTorch); every step runs inside libard.so. Errors raise
ArdError carrying the status code and the library's message.
"""

import ctypes

import numpy as np

from . import _ffi
from ._ffi import (ARD_ACT_NONE, ARD_ACT_RELU, ARD_BF16, ARD_DROPPED_SKIP, ARD_DROPPED_ZERO,  # noqa: F401
                   ARD_ERR_INVALID_ARG, ARD_ERR_NOT_CONVERGED, ARD_F32, ARD_SEARCH_MIRROR, ARD_SEARCH_PLAIN,
                   ARD_WEIGHTS_COMPACT, ARD_WEIGHTS_COMPACT_GRAD, ARD_WEIGHTS_FULL, ARD_WEIGHTS_INPUT_MAJOR,
                   ard_fc_desc, ard_lstm_desc, ard_lstm_tile_desc, ard_row_plan, ard_search_info, ard_search_opts,
                   ard_tile_desc, ard_tile_plan)


class ArdError(RuntimeError):
    def __init__(self, status, name, message):
        super().__init__(f"{name}: {message}")
        self.status = status
        self.name = name
        self.message = message


def _check(status):
    if status != 0:
        L = _ffi.lib()
        raise ArdError(status, L.ard_status_string(status).decode(), L.ard_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        if torch.cuda.is_available():
            return torch.cuda.current_stream().cuda_stream
        return None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _plan_ptr(plan):
    return ctypes.pointer(plan) if plan is not None else None


# --------------------------------------------------------------------------- host

def ard_version():
    return _ffi.lib().ard_version()


def ard_status_string(status):
    return _ffi.lib().ard_status_string(status).decode()


def ard_last_error():
    return _ffi.lib().ard_last_error().decode()


def ard_search_opts_default():
    o = ard_search_opts()
    _ffi.lib().ard_search_opts_default(ctypes.byref(o))
    return o


def ard_search_distribution(p, opts=None):
    """Returns (K as a numpy array, ard_search_info). ARD_ERR_NOT_CONVERGED raises
    ArdError with the last iterate attached as .K and .info."""
    o = opts if opts is not None else ard_search_opts_default()
    K = np.zeros(o.n_max, dtype=np.float64)
    info = ard_search_info()
    st = _ffi.lib().ard_search_distribution(
        float(p), ctypes.byref(o), K.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), ctypes.byref(info))
    if st == ARD_ERR_NOT_CONVERGED:
        err = ArdError(st, ard_status_string(st), ard_last_error())
        err.K, err.info = K, info
        raise err
    _check(st)
    return K, info


def ard_sample_row_pattern(K, seed, stream, iteration):
    """Returns (period, offset)."""
    K = np.ascontiguousarray(K, dtype=np.float64)
    out = _ffi.ard_row_pattern()
    _check(_ffi.lib().ard_sample_row_pattern(
        K.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), K.size, seed, stream, iteration,
        ctypes.byref(out)))
    return out.period, out.offset


def ard_row_kept(n, period, offset):
    return _ffi.lib().ard_row_kept(n, period, offset)


def _bitmap_buffer(tiles_n, tiles_k):
    return np.zeros((tiles_n * tiles_k + 31) // 32, dtype=np.uint32)


def ard_tile_bitmap_tdp(tiles_n, tiles_k, period, offset):
    bits = _bitmap_buffer(tiles_n, tiles_k)
    _check(_ffi.lib().ard_tile_bitmap_tdp(tiles_n, tiles_k, period, offset,
                                          bits.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))))
    return bits


def ard_tile_bitmap_bernoulli(tiles_n, tiles_k, p, seed, stream, iteration):
    bits = _bitmap_buffer(tiles_n, tiles_k)
    _check(_ffi.lib().ard_tile_bitmap_bernoulli(tiles_n, tiles_k, float(p), seed, stream, iteration,
                                                bits.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))))
    return bits


def ard_bitmap_popcount(bits, total):
    bits = np.ascontiguousarray(bits, dtype=np.uint32)
    return _ffi.lib().ard_bitmap_popcount(bits.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)), total)


# --------------------------------------------------------------------------- compaction

def ard_plan_rows(n, period, offset, d_idx, stream=None, plan=None):
    """Fills the int32 device tensor d_idx with the kept list (d_idx None: a
    list-free plan, nothing launched); returns the plan (``plan`` if given,
    refilled in place). The plan keeps a reference to d_idx."""
    plan = ard_row_plan() if plan is None else plan
    _check(_ffi.lib().ard_plan_rows(n, period, offset, _ptr(d_idx), ctypes.byref(plan), _stream(stream)))
    plan._keep = d_idx
    return plan


def ard_tile_plan_workspace_bytes(tiles_n, tiles_k):
    return _ffi.lib().ard_tile_plan_workspace_bytes(tiles_n, tiles_k)


def ard_plan_tiles(n, k, tile, d_bits, nnz, ws, stream=None):
    """d_bits: device uint32/int32 bitmap; ws: device buffer of the queried size."""
    plan = ard_tile_plan()
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(_ffi.lib().ard_plan_tiles(n, k, tile, _ptr(d_bits), nnz, _ptr(ws), nbytes,
                                     ctypes.byref(plan), _stream(stream)))
    plan._keep = (d_bits, ws)
    return plan


def ard_plan_tiles_bernoulli(n, k, tile, p, seed, stream_id, iteration, d_bits, ws, stream=None):
    """Samples the Bernoulli tile bitmap into d_bits on the device and plans from
    it (plan.nnz = -1: the kept count stays on the device)."""
    plan = ard_tile_plan()
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(_ffi.lib().ard_plan_tiles_bernoulli(n, k, tile, float(p), seed, stream_id, iteration, _ptr(d_bits),
                                               _ptr(ws), nbytes, ctypes.byref(plan), _stream(stream)))
    plan._keep = (d_bits, ws)
    return plan


# --------------------------------------------------------------------------- FC layer

def fc_desc(dtype, batch, in_features, out_features, in_plan=None, out_plan=None, scale=1.0,
            act=ARD_ACT_NONE, dropped=ARD_DROPPED_ZERO, weight_layout=ARD_WEIGHTS_FULL):
    d = ard_fc_desc(dtype, batch, in_features, out_features, _plan_ptr(in_plan), _plan_ptr(out_plan),
                    scale, act, dropped, weight_layout)
    d._keep = (in_plan, out_plan)
    return d


def _ws(ws):
    """(pointer, bytes) of a workspace tensor, or of a (pointer, bytes) pair."""
    if ws is None:
        return None, 0
    if isinstance(ws, tuple):
        return ws
    return ws.data_ptr(), ws.numel() * ws.element_size()


def ard_fc_compact_ld(desc):
    return _ffi.lib().ard_fc_compact_ld(ctypes.byref(desc))


def ard_fc_compact_bytes(desc):
    return _ffi.lib().ard_fc_compact_bytes(ctypes.byref(desc))


def ard_fc_compact_weights(desc, W, Wc, stream=None):
    _check(_ffi.lib().ard_fc_compact_weights(ctypes.byref(desc), _ptr(W), _ptr(Wc), _stream(stream)))


class CompactBatch:
    """Marshalled arguments of ard_fc_compact_weights_batch, built once and
    reused (the descriptors are read at each call, so their plans may change)."""

    def __init__(self, descs, Ws, Wcs):
        n = len(descs)
        self.descs = list(descs)
        self.count = n
        self.d = (ctypes.POINTER(ard_fc_desc) * n)(*[ctypes.pointer(x) for x in descs])
        self.w = (ctypes.c_void_p * n)(*[_ptr(x) for x in Ws])
        self.wc = (ctypes.c_void_p * n)(*[_ptr(x) for x in Wcs])


def ard_fc_compact_weights_batch(batch, stream=None):
    """Gathers the compact weights of up to 4 layers in one launch (a CompactBatch)."""
    _check(_ffi.lib().ard_fc_compact_weights_batch(batch.count, batch.d, batch.w, batch.wc, _stream(stream)))


def ard_fc_workspace_bytes(desc):
    return _ffi.lib().ard_fc_workspace_bytes(ctypes.byref(desc))


def ard_fc_fwd(desc, Xt, W, bias, Yt, ws=None, stream=None):
    p, n = _ws(ws)
    _check(_ffi.lib().ard_fc_fwd(ctypes.byref(desc), _ptr(Xt), _ptr(W), _ptr(bias), _ptr(Yt), p, n,
                                 _stream(stream)))


def ard_fc_fwd_noalloc(desc, Xt, W, bias, Yt, stream=None):
    """ard_fc_fwd with the library's static per-GPU scratch instead of a workspace."""
    _check(_ffi.lib().ard_fc_fwd_noalloc(ctypes.byref(desc), _ptr(Xt), _ptr(W), _ptr(bias), _ptr(Yt),
                                         _stream(stream)))


def ard_fc_bwd_data(desc, dYt, Yt, W, dXt, ws=None, stream=None, Xgate=None):
    p, n = _ws(ws)
    _check(_ffi.lib().ard_fc_bwd_data(ctypes.byref(desc), _ptr(dYt), _ptr(Yt), _ptr(W), _ptr(dXt),
                                      _ptr(Xgate), p, n, _stream(stream)))


def ard_fc_bwd_weight(desc, Xt, dYt, Yt, dW, dbias, ws=None, stream=None):
    p, n = _ws(ws)
    _check(_ffi.lib().ard_fc_bwd_weight(ctypes.byref(desc), _ptr(Xt), _ptr(dYt), _ptr(Yt), _ptr(dW),
                                        _ptr(dbias), p, n, _stream(stream)))


def ard_fc_bwd(desc, Xt, dYt, Yt, W, dXt, dW, dbias, ws=None, stream=None, Xgate=None):
    """bwd_data then bwd_weight of one layer (one launch where both are small)."""
    p, n = _ws(ws)
    _check(_ffi.lib().ard_fc_bwd(ctypes.byref(desc), _ptr(Xt), _ptr(dYt), _ptr(Yt), _ptr(W), _ptr(dXt),
                                 _ptr(Xgate), _ptr(dW), _ptr(dbias), p, n, _stream(stream)))


def ard_fc_sgd_momentum(desc, W, V, dW, bias, Vb, dbias, lr, momentum, stream=None):
    """Momentum SGD on the kept weights (and kept bias entries) of the descriptor's patterns."""
    _check(_ffi.lib().ard_fc_sgd_momentum(ctypes.byref(desc), _ptr(W), _ptr(V), _ptr(dW), _ptr(bias), _ptr(Vb),
                                          _ptr(dbias), lr, momentum, _stream(stream)))


# --------------------------------------------------------------------------- conventional dropout

def ard_dropout_fwd(dtype, n, batch, p, scale, seed, stream_id, iteration, Yt, mask, stream=None):
    """Bernoulli dropout of Yt[n][batch] in place; mask receives the keep bits."""
    _check(_ffi.lib().ard_dropout_fwd(dtype, n, batch, p, scale, seed, stream_id, iteration, _ptr(Yt), _ptr(mask),
                                      _stream(stream)))


def ard_dropout_bwd(dtype, n, batch, scale, mask, dYt, stream=None):
    _check(_ffi.lib().ard_dropout_bwd(dtype, n, batch, scale, _ptr(mask), _ptr(dYt), _stream(stream)))


# --------------------------------------------------------------------------- tile layer

def tile_desc(dtype, batch, in_features, out_features, scale=1.0, dropped=ARD_DROPPED_ZERO):
    return ard_tile_desc(dtype, batch, in_features, out_features, scale, dropped)


def ard_tile_fwd(desc, plan, Xt, W, Yt, stream=None):
    _check(_ffi.lib().ard_tile_fwd(ctypes.byref(desc), ctypes.byref(plan), _ptr(Xt), _ptr(W), _ptr(Yt),
                                   _stream(stream)))


def ard_tile_bwd_data(desc, plan, dYt, W, dXt, stream=None):
    _check(_ffi.lib().ard_tile_bwd_data(ctypes.byref(desc), ctypes.byref(plan), _ptr(dYt), _ptr(W),
                                        _ptr(dXt), _stream(stream)))


def ard_tile_bwd_weight(desc, plan, Xt, dYt, dW, stream=None):
    _check(_ffi.lib().ard_tile_bwd_weight(ctypes.byref(desc), ctypes.byref(plan), _ptr(Xt), _ptr(dYt),
                                          _ptr(dW), _stream(stream)))


def ard_tile_bwd(desc, plan, Xt, dYt, W, dXt, dW, stream=None):
    """ard_tile_bwd_data and ard_tile_bwd_weight in one call (one launch on the fast path)."""
    _check(_ffi.lib().ard_tile_bwd(ctypes.byref(desc), ctypes.byref(plan), _ptr(Xt), _ptr(dYt), _ptr(W),
                                   _ptr(dXt), _ptr(dW), _stream(stream)))


# --------------------------------------------------------------------------- LSTM layer

def lstm_desc(dtype, seq_len, batch, input_size, hidden_size, hidden_plan=None, input_plan=None):
    d = ard_lstm_desc(dtype, seq_len, batch, input_size, hidden_size, 0, _plan_ptr(hidden_plan),
                      _plan_ptr(input_plan))
    d._keep = (hidden_plan, input_plan)
    return d


def ard_lstm_workspace_bytes(desc):
    return _ffi.lib().ard_lstm_workspace_bytes(ctypes.byref(desc))


def ard_lstm_fwd(desc, X, W, bias, h0, c0, Hs, hT, cT, ws, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(_ffi.lib().ard_lstm_fwd(ctypes.byref(desc), _ptr(X), _ptr(W), _ptr(bias), _ptr(h0), _ptr(c0),
                                   _ptr(Hs), _ptr(hT), _ptr(cT), _ptr(ws), nbytes, _stream(stream)))


def ard_lstm_bwd(desc, X, dHs, dhT, dcT, ws, dX, dW, dbias, dh0, dc0, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(_ffi.lib().ard_lstm_bwd(ctypes.byref(desc), _ptr(X), _ptr(dHs), _ptr(dhT), _ptr(dcT),
                                   _ptr(ws), nbytes, _ptr(dX), _ptr(dW), _ptr(dbias), _ptr(dh0),
                                   _ptr(dc0), _stream(stream)))


# --------------------------------------------------------------------------- LSTM under a tile pattern

def lstm_tile_desc(dtype, seq_len, batch, input_size, hidden_size, weight_plan):
    d = ard_lstm_tile_desc(dtype, seq_len, batch, input_size, hidden_size, 0, ctypes.pointer(weight_plan))
    d._keep = weight_plan
    return d


def ard_lstm_tile_workspace_bytes(desc):
    return _ffi.lib().ard_lstm_tile_workspace_bytes(ctypes.byref(desc))


def ard_lstm_tile_fwd(desc, X, W, bias, h0, c0, Hs, hT, cT, ws, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(_ffi.lib().ard_lstm_tile_fwd(ctypes.byref(desc), _ptr(X), _ptr(W), _ptr(bias), _ptr(h0), _ptr(c0),
                                        _ptr(Hs), _ptr(hT), _ptr(cT), _ptr(ws), nbytes, _stream(stream)))


def ard_lstm_tile_bwd(desc, W, dHs, dhT, dcT, ws, dX, dW, dbias, dh0, dc0, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(_ffi.lib().ard_lstm_tile_bwd(ctypes.byref(desc), _ptr(W), _ptr(dHs), _ptr(dhT), _ptr(dcT), _ptr(ws),
                                        nbytes, _ptr(dX), _ptr(dW), _ptr(dbias), _ptr(dh0), _ptr(dc0),
                                        _stream(stream)))
