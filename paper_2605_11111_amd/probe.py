"""Binding of libshardprobe.so (include/shardprobe.h): measurement aids that
sit beside the shard path. Argument marshalling only."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libshardprobe.so")
if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it first (python -m paper_2605_11111_amd.build)")
_lib = ctypes.CDLL(LIB_PATH)
_lib.shard_probe_mfma_bf16.restype = ctypes.c_int
_lib.shard_probe_mfma_bf16.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p]

EXPORTED = ("shard_probe_mfma_bf16",)


def shard_probe_mfma_bf16(iters: int, blocks: int, random: bool, out, clk) -> None:
    """Launch the MFMA-only kernel on the current stream (constant or random
    operands); `out` is a float32 CUDA tensor of blocks*256 elements, `clk` an
    int64 CUDA tensor of 2*blocks."""
    import torch
    assert out.is_cuda and out.dtype == torch.float32 and out.numel() >= blocks * 256
    assert clk.is_cuda and clk.dtype == torch.int64 and clk.numel() >= 2 * blocks
    rc = _lib.shard_probe_mfma_bf16(int(iters), int(blocks), int(bool(random)), ctypes.c_void_p(out.data_ptr()),
                                    ctypes.c_void_p(clk.data_ptr()),
                                    ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    if rc != 0:
        raise RuntimeError(f"shard_probe_mfma_bf16 failed ({rc})")
