"""Python binding of libshardconv (the shard halo-convolution hot path on MI355X).

Argument marshalling only: every function forwards to the C-ABI entry point of
the same name in ``libshardconv.so`` (see ``include/shardconv.h`` for the
semantics, layouts and error behaviour), passing raw device pointers of torch
tensors and torch's current HIP stream. Every step of the hot path runs in the
library's HIP kernels; there is no fallback: if the library is not built,
importing this package raises.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libshardconv.so")

SHARD_OK, SHARD_ERR_INVALID, SHARD_ERR_UNSUPPORTED, SHARD_ERR_HIP = 0, 1, 2, 3
SHARD_F32, SHARD_BF16 = 0, 1

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it first (python -m paper_2605_11111_amd.build)")

_lib = ctypes.CDLL(LIB_PATH)
_i64p = ctypes.POINTER(ctypes.c_int64)
_vp = ctypes.c_void_p


SHARD_REGION_ALL, SHARD_REGION_INTERIOR, SHARD_REGION_BOUNDARY = 0, 1, 2
SHARD_KERNELS_FASTEST, SHARD_KERNELS_TILED, SHARD_KERNELS_DIRECT = 0, 1, 2


class shard_call_opts_t(ctypes.Structure):
    _fields_ = [("kernels", ctypes.c_int32), ("wait_polls", ctypes.c_uint32)]


class shard_halo_src_t(ctypes.Structure):
    _fields_ = [("slab", (ctypes.c_void_p * 2) * 3)]


class shard_tile_t(ctypes.Structure):
    _fields_ = [
        ("ndim", ctypes.c_int32),
        ("n", ctypes.c_int64),
        ("c", ctypes.c_int64),
        ("ext", ctypes.c_int64 * 3),
        ("halo_lo", ctypes.c_int64 * 3),
        ("halo_hi", ctypes.c_int64 * 3),
    ]


_tp = ctypes.POINTER(shard_tile_t)

_SIGS = {
    "shard_conv_geometry": (ctypes.c_int, [ctypes.c_int32] + [_i64p] * 11),
    "shard_halo_slab_shape": (ctypes.c_int, [_tp, ctypes.c_int32, ctypes.c_int64, _i64p]),
    "shard_halo_pack": (ctypes.c_int, [_tp, ctypes.c_int, _vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64, _vp, _vp]),
    "shard_halo_unpack": (ctypes.c_int, [_tp, ctypes.c_int, _vp, ctypes.c_int32, ctypes.c_int32, _vp, _vp]),
    "shard_conv_fwd": (ctypes.c_int, [_tp, ctypes.c_int, _vp, _vp, ctypes.c_int64, _i64p, _i64p, _i64p, _i64p, _vp,
                                      _vp, ctypes.c_size_t, _vp]),
    "shard_conv_wgrad": (ctypes.c_int, [_tp, ctypes.c_int, _vp, _vp, ctypes.c_int64, _i64p, _i64p, _i64p, _i64p,
                                        _vp, _vp, ctypes.c_size_t, _vp]),
    "shard_conv_dgrad": (ctypes.c_int, [_tp, ctypes.c_int, _vp, _vp, ctypes.c_int64, _i64p, _i64p, _i64p, _i64p,
                                        _vp, _vp, ctypes.c_size_t, _vp]),
    "shard_halo_pack_margin": (ctypes.c_int, [_tp, ctypes.c_int, _vp, ctypes.c_int32, ctypes.c_int32, _vp, _vp]),
    "shard_halo_accumulate": (ctypes.c_int, [_tp, ctypes.c_int, _vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                             _vp, _vp]),
    "shard_norm_workspace_bytes": (ctypes.c_size_t, [_tp, ctypes.c_int, ctypes.c_int64]),
    "shard_norm_stats": (ctypes.c_int, [_tp, ctypes.c_int, _vp, ctypes.c_int64, _vp, _vp, ctypes.c_size_t, _vp]),
    "shard_norm_apply": (ctypes.c_int, [_tp, ctypes.c_int, _vp, _vp, ctypes.c_double, ctypes.c_double, ctypes.c_int64,
                                        _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "shard_conv_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int32, _tp, ctypes.c_int, ctypes.c_int64, _i64p,
                                                     _i64p, _i64p]),
    "shard_conv_interior": (ctypes.c_int, [_tp, _i64p, _i64p, _i64p, _i64p, _i64p, _i64p]),
    "shard_conv_fwd_folded": (ctypes.c_int, [_tp, ctypes.c_int, _vp, ctypes.c_void_p, ctypes.c_int32, _vp,
                                             ctypes.c_int64, _i64p, _i64p, _i64p, _i64p, _vp, _vp, ctypes.c_size_t,
                                             _vp]),
    "shard_attn_block": (ctypes.c_int, [ctypes.c_int64] * 5 + [ctypes.c_int, ctypes.c_float, _vp, _vp, _vp, _vp, _vp,
                                                                 ctypes.c_int32, _vp]),
    "shard_halo_pack_pair": (ctypes.c_int, [_tp, ctypes.c_int, _vp, ctypes.c_int32, ctypes.c_int64, _vp,
                                            ctypes.c_int64, _vp, _vp]),
    "shard_halo_unpack_pair": (ctypes.c_int, [_tp, ctypes.c_int, _vp, ctypes.c_int32, _vp, _vp, _vp]),
    "shard_conv_wgrad_folded": (ctypes.c_int, [_tp, ctypes.c_int, _vp, ctypes.c_void_p, _vp, ctypes.c_int64, _i64p,
                                               _i64p, _i64p, _i64p, _vp, _vp, ctypes.c_size_t, _vp]),
    "shard_halo_pack_margin_pair": (ctypes.c_int, [_tp, ctypes.c_int, _vp, ctypes.c_int32, _vp, _vp, _vp]),
    "shard_halo_accumulate_pair": (ctypes.c_int, [_tp, ctypes.c_int, _vp, ctypes.c_int32, ctypes.c_int64, _vp,
                                                  ctypes.c_int64, _vp, _vp]),
    "shard_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "shard_set_call_opts": (ctypes.c_int, [ctypes.c_void_p]),
    "shard_conv_fwd_noalloc": (ctypes.c_int, [_tp, ctypes.c_int, _vp, _vp, ctypes.c_int64, _i64p, _i64p, _i64p,
                                              _i64p, _vp, _vp]),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTED = tuple(_SIGS)


class ShardError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn}: {shard_status_string(status)} (status {status})")
        self.status = status


def _check(fn: str, status: int):
    if status != SHARD_OK:
        raise ShardError(fn, status)


def _arr(vals, n=3):
    v = [int(x) for x in vals] + [0] * (n - len(vals))
    return (ctypes.c_int64 * n)(*v)


def tile_desc(n, c, ext, halo_lo=None, halo_hi=None) -> shard_tile_t:
    """Descriptor of a padded tile; ext/halo_lo/halo_hi are per spatial axis."""
    nd = len(ext)
    d = shard_tile_t()
    d.ndim = nd
    d.n, d.c = int(n), int(c)
    for a in range(nd):
        d.ext[a] = int(ext[a])
        d.halo_lo[a] = int(halo_lo[a]) if halo_lo is not None else 0
        d.halo_hi[a] = int(halo_hi[a]) if halo_hi is not None else 0
    return d


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return SHARD_F32
    if t.dtype == torch.bfloat16:
        return SHARD_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("device tensor required")
    if not t.is_contiguous():
        raise ValueError("contiguous tensor required")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(int(stream))
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def shard_status_string(status: int) -> str:
    return _lib.shard_status_string(int(status)).decode()


def shard_set_call_opts(kernels=SHARD_KERNELS_FASTEST, wait_polls=0):
    """Options of the calling host thread (None-like defaults restore them)."""
    o = shard_call_opts_t(int(kernels), int(wait_polls))
    _check("shard_set_call_opts", _lib.shard_set_call_opts(ctypes.byref(o)))


class call_opts:
    """Context manager: the calling thread's options inside the block, the
    defaults after it."""

    def __init__(self, kernels=SHARD_KERNELS_FASTEST, wait_polls=0):
        self.kernels, self.wait_polls = kernels, wait_polls

    def __enter__(self):
        shard_set_call_opts(self.kernels, self.wait_polls)
        return self

    def __exit__(self, *exc):
        _check("shard_set_call_opts", _lib.shard_set_call_opts(None))
        return False


def shard_conv_geometry(global_ext, shard_off, shard_ext, kernel, stride, sharded_mask) -> dict:
    nd = len(global_ext)
    outs = [_arr([0] * nd) for _ in range(5)]
    st = _lib.shard_conv_geometry(nd, _arr(global_ext), _arr(shard_off), _arr(shard_ext), _arr(kernel), _arr(stride),
                                  _arr(sharded_mask), *outs)
    _check("shard_conv_geometry", st)
    keys = ("halo_lo", "halo_hi", "pad_lo", "out_off", "out_ext")
    return {k: list(o)[:nd] for k, o in zip(keys, outs)}


def shard_halo_slab_shape(desc: shard_tile_t, axis: int, width: int) -> list:
    out = _arr([0] * 5, 5)
    _check("shard_halo_slab_shape", _lib.shard_halo_slab_shape(ctypes.byref(desc), axis, width, out))
    return list(out)


def shard_halo_pack(desc, tile, axis, side, width, slab, stream=None):
    _check("shard_halo_pack", _lib.shard_halo_pack(ctypes.byref(desc), _dtype_code(tile), _ptr(tile), axis, side,
                                                   width, _ptr(slab), _stream(stream)))


def shard_halo_unpack(desc, tile, axis, side, slab=None, stream=None):
    _check("shard_halo_unpack", _lib.shard_halo_unpack(ctypes.byref(desc), _dtype_code(tile), _ptr(tile), axis, side,
                                                       _ptr(slab), _stream(stream)))


def shard_conv_workspace_bytes(op, desc, dtype_code, c_out, kernel, stride, out_ext) -> int:
    n = _lib.shard_conv_workspace_bytes(op, ctypes.byref(desc), dtype_code, c_out, _arr(kernel), _arr(stride),
                                        _arr(out_ext))
    if n == ctypes.c_size_t(-1).value:
        raise ShardError("shard_conv_workspace_bytes", SHARD_ERR_INVALID)
    return int(n)


def shard_conv_fwd(desc, tile, w, c_out, kernel, stride, pad_lo, out_ext, y, ws, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check("shard_conv_fwd", _lib.shard_conv_fwd(ctypes.byref(desc), _dtype_code(tile), _ptr(tile), _ptr(w), c_out,
                                                 _arr(kernel), _arr(stride), _arr(pad_lo), _arr(out_ext), _ptr(y),
                                                 _ptr(ws), nbytes, _stream(stream)))


def shard_conv_fwd_noalloc(desc, tile, w, c_out, kernel, stride, pad_lo, out_ext, y, stream=None):
    _check("shard_conv_fwd_noalloc", _lib.shard_conv_fwd_noalloc(ctypes.byref(desc), _dtype_code(tile), _ptr(tile),
                                                                 _ptr(w), c_out, _arr(kernel), _arr(stride),
                                                                 _arr(pad_lo), _arr(out_ext), _ptr(y),
                                                                 _stream(stream)))


def shard_conv_wgrad(desc, tile, dy, c_out, kernel, stride, pad_lo, out_ext, dw, ws, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check("shard_conv_wgrad", _lib.shard_conv_wgrad(ctypes.byref(desc), _dtype_code(tile), _ptr(tile), _ptr(dy),
                                                     c_out, _arr(kernel), _arr(stride), _arr(pad_lo), _arr(out_ext),
                                                     _ptr(dw), _ptr(ws), nbytes, _stream(stream)))


def shard_conv_dgrad(desc, dy, w, c_out, kernel, stride, pad_lo, out_ext, dtile, ws, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check("shard_conv_dgrad", _lib.shard_conv_dgrad(ctypes.byref(desc), _dtype_code(dtile), _ptr(dy), _ptr(w), c_out,
                                                     _arr(kernel), _arr(stride), _arr(pad_lo), _arr(out_ext),
                                                     _ptr(dtile), _ptr(ws), nbytes, _stream(stream)))


def shard_halo_pack_margin(desc, tile, axis, side, slab, stream=None):
    _check("shard_halo_pack_margin", _lib.shard_halo_pack_margin(ctypes.byref(desc), _dtype_code(tile), _ptr(tile),
                                                                 axis, side, _ptr(slab), _stream(stream)))


def shard_halo_accumulate(desc, tile, axis, side, width, slab, stream=None):
    _check("shard_halo_accumulate", _lib.shard_halo_accumulate(ctypes.byref(desc), _dtype_code(tile), _ptr(tile),
                                                               axis, side, width, _ptr(slab), _stream(stream)))


def shard_halo_pack_margin_pair(desc, tile, axis, slab_lo=None, slab_hi=None, stream=None):
    _check("shard_halo_pack_margin_pair",
           _lib.shard_halo_pack_margin_pair(ctypes.byref(desc), _dtype_code(tile), _ptr(tile), axis, _ptr(slab_lo),
                                            _ptr(slab_hi), _stream(stream)))


def shard_halo_accumulate_pair(desc, tile, axis, width_lo, slab_lo, width_hi, slab_hi, stream=None):
    _check("shard_halo_accumulate_pair",
           _lib.shard_halo_accumulate_pair(ctypes.byref(desc), _dtype_code(tile), _ptr(tile), axis, width_lo,
                                           _ptr(slab_lo), width_hi, _ptr(slab_hi), _stream(stream)))


def shard_norm_workspace_bytes(desc, dtype_code, groups) -> int:
    n = _lib.shard_norm_workspace_bytes(ctypes.byref(desc), dtype_code, groups)
    if n == ctypes.c_size_t(-1).value:
        raise ShardError("shard_norm_workspace_bytes", SHARD_ERR_INVALID)
    return int(n)


def shard_norm_stats(desc, tile, groups, sums, ws, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check("shard_norm_stats", _lib.shard_norm_stats(ctypes.byref(desc), _dtype_code(tile), _ptr(tile), groups,
                                                     _ptr(sums), _ptr(ws), nbytes, _stream(stream)))


def shard_norm_apply(desc, tile, sums, count, eps, groups, gamma, beta, out, ws, stream=None):
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check("shard_norm_apply", _lib.shard_norm_apply(ctypes.byref(desc), _dtype_code(tile), _ptr(tile), _ptr(sums),
                                                     float(count), float(eps), groups, _ptr(gamma), _ptr(beta),
                                                     _ptr(out), _ptr(ws), nbytes, _stream(stream)))


def shard_conv_interior(desc, kernel, stride, pad_lo, out_ext) -> tuple:
    """(int_lo, int_hi): per axis, the outputs that read no margin."""
    nd = desc.ndim
    lo, hi = _arr([0] * nd), _arr([0] * nd)
    _check("shard_conv_interior", _lib.shard_conv_interior(ctypes.byref(desc), _arr(kernel), _arr(stride),
                                                           _arr(pad_lo), _arr(out_ext), lo, hi))
    return list(lo)[:nd], list(hi)[:nd]


def halo_src(slabs) -> shard_halo_src_t:
    """shard_halo_src_t from {(axis, side): tensor or None}."""
    h = shard_halo_src_t()
    for (axis, side), t in slabs.items():
        p = _ptr(t)
        h.slab[axis][side] = None if p is None else p.value
    return h


def shard_conv_fwd_folded(desc, tile, slabs, region, w, c_out, kernel, stride, pad_lo, out_ext, y, ws,
                          stream=None):
    """Forward with the halo read from the received slabs ({(axis, side): tensor
    or None}, or None for no slabs) for the outputs of `region`."""
    h = None if slabs is None else halo_src(slabs)
    st = _lib.shard_conv_fwd_folded(ctypes.byref(desc), _dtype_code(tile), _ptr(tile),
                                    None if h is None else ctypes.cast(ctypes.byref(h), ctypes.c_void_p),
                                    region, _ptr(w), c_out, _arr(kernel), _arr(stride), _arr(pad_lo), _arr(out_ext),
                                    _ptr(y), _ptr(ws), ws.numel() * ws.element_size() if ws is not None else 0,
                                    _stream(stream))
    _check("shard_conv_fwd_folded", st)


def shard_attn_block(q, k, v, o, lse, scale, first, stream=None):
    """One ring-attention block step: q [B][H][Sq][D], k/v [B][H][Sk][D] (bf16),
    merged into o [B][H][Sq][D] and lse [B][H][Sq] (float32)."""
    B, H, Sq, D = q.shape
    Sk = k.shape[2]
    st = _lib.shard_attn_block(B, H, Sq, Sk, D, _dtype_code(q), float(scale), _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                               _ptr(lse), 1 if first else 0, _stream(stream))
    _check("shard_attn_block", st)


def shard_halo_pack_pair(desc, tile, axis, width_lo, slab_lo, width_hi, slab_hi, stream=None):
    _check("shard_halo_pack_pair", _lib.shard_halo_pack_pair(ctypes.byref(desc), _dtype_code(tile), _ptr(tile), axis,
                                                             width_lo, _ptr(slab_lo), width_hi, _ptr(slab_hi),
                                                             _stream(stream)))


def shard_halo_unpack_pair(desc, tile, axis, slab_lo=None, slab_hi=None, stream=None):
    _check("shard_halo_unpack_pair", _lib.shard_halo_unpack_pair(ctypes.byref(desc), _dtype_code(tile), _ptr(tile),
                                                                 axis, _ptr(slab_lo), _ptr(slab_hi),
                                                                 _stream(stream)))


def shard_conv_wgrad_folded(desc, tile, slabs, dy, c_out, kernel, stride, pad_lo, out_ext, dw, ws, stream=None):
    """Weight gradient with the halo read from the received slabs ({(axis, side):
    tensor or None}, or None for no slabs)."""
    h = None if slabs is None else halo_src(slabs)
    st = _lib.shard_conv_wgrad_folded(ctypes.byref(desc), _dtype_code(tile), _ptr(tile),
                                      None if h is None else ctypes.cast(ctypes.byref(h), ctypes.c_void_p), _ptr(dy),
                                      c_out, _arr(kernel), _arr(stride), _arr(pad_lo), _arr(out_ext), _ptr(dw),
                                      _ptr(ws), ws.numel() * ws.element_size() if ws is not None else 0,
                                      _stream(stream))
    _check("shard_conv_wgrad_folded", st)
