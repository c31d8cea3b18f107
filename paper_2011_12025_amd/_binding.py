"""ctypes binding of libsegblocks.so (include/segblocks.h).

Argument marshalling only: every step of the block-conv path runs in the HIP
kernels of the library.  torch supplies device memory and the current
stream.  The library must be built (``python -m paper_2011_12025_amd.build``
or ``__graft_entry__.build()``); there is no fallback of any kind.
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  -- load torch's HIP runtime first so that the library shares it

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsegblocks.so")

SB_F32, SB_F16, SB_BF16 = 0, 1, 2
SB_NCHW, SB_NHWC = 0, 1
SB_FLAG_RELU, SB_FLAG_PAD_STRIDED, SB_FLAG_PAD_ZERO = 1, 2, 4
SB_PAD_AVG, SB_PAD_STRIDED, SB_PAD_ZERO = 0, 1, 2

EXPORTS = ["segblocks_count", "segblocks_split", "segblocks_pad", "segblocks_pad_ex", "segblocks_conv3x3", "segblocks_combine",
           "segblocks_block_conv3x3", "segblocks_layer", "segblocks_block_conv_ex", "segblocks_conv2d",
           "segblocks_maxpool", "segblocks_block_conv3x3_workspace_size", "segblocks_block_conv_ex_workspace_size",
           "segblocks_layer_workspace_size", "segblocks_block_conv_ex_noalloc", "segblocks_block_conv_chain",
           "segblocks_block_conv_chain_workspace_size", "segblocks_block_conv_chain_reads_half",
           "segblocks_policy_heuristic",
           "segblocks_combine_backward", "segblocks_split_backward", "segblocks_pad_backward",
           "segblocks_conv3x3_backward_data", "segblocks_conv3x3_backward_data_workspace_size",
           "segblocks_conv3x3_backward_weight", "segblocks_conv3x3_backward_weight_workspace_size",
           "segblocks_pad_halo", "segblocks_conv_halo", "segblocks_maxpool_halo", "segblocks_last_error"]

SB_OK, SB_EINVAL, SB_ESHAPE, SB_EHIP, SB_ENOMEM = 0, -1, -2, -3, -4

_P = ctypes.c_void_p
_I = ctypes.c_int
_Z = ctypes.c_size_t
_ZP = ctypes.POINTER(ctypes.c_size_t)
_SIGS = {
    "segblocks_count": [_P, _I, _I, _I, ctypes.POINTER(_I), ctypes.POINTER(_I), _P],
    "segblocks_split": [_P, _I, _I, _I, _I, _I, _I, _P, _I, _P, _I, _P, _I, _P],
    "segblocks_pad": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _P, _P, _I, _I, _P],
    "segblocks_pad_ex": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _P, _P, _I, _I, _I, _P],
    "segblocks_conv3x3": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _P, _P, _I, _P, _P, _I, _I, _P],
    "segblocks_combine": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _I, _I, _P, _P],
    "segblocks_block_conv3x3": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _P, _P, _I, _I, _P, _P, _P, _P, _I, _I,
                                _P, _Z, _P],
    "segblocks_layer": [_P, _I, _I, _I, _I, _I, _I, _P, _I, _P, _P, _I, _I, _P, _P, _Z, _P],
    "segblocks_block_conv_ex": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _P, _P, _I, _I, _I, _I, _P, _P, _P, _P,
                                _I, _I, _P, _Z, _P],
    "segblocks_block_conv_ex_noalloc": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _P, _P, _I, _I, _I, _I, _P, _P, _P,
                                        _P, _I, _I, _P],
    "segblocks_block_conv_chain": [_P, _P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _P, _P, _I, _I, _I, _I, _P, _P, _P,
                                   _P, _P, _I, _I, _P, _Z, _P],
    "segblocks_block_conv_chain_workspace_size": [_I] * 12 + [_ZP],
    "segblocks_block_conv_chain_reads_half": [_I] * 13 + [ctypes.POINTER(_I)],
    "segblocks_policy_heuristic": [_P, _I, _I, _I, _I, _I, _I, _I, ctypes.c_double, _P, _P, _P],
    "segblocks_combine_backward": [_P, _I, _I, _I, _I, _I, _I, _P, _I, _P, _I, _P, _I, _P],
    "segblocks_split_backward": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _I, _I, _P, _P],
    "segblocks_pad_backward": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _I, _P, _P, _I, _I, _P],
    "segblocks_conv3x3_backward_data": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _P, _I, _P, _P, _I, _I, _P, _Z,
                                        _P],
    "segblocks_conv3x3_backward_data_workspace_size": [_I] * 10 + [_ZP],
    "segblocks_conv3x3_backward_weight": [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _I, _P, _P, _I, _I, _P,
                                          _Z, _P],
    "segblocks_conv3x3_backward_weight_workspace_size": [_I] * 11 + [_ZP],
    "segblocks_pad_halo": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _I, _I, _P, _P, _I, _I, _P],
    "segblocks_conv_halo": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _I, _P, _P, _I, _I, _I, _I, _I, _P, _P, _I, _I,
                            _P],
    "segblocks_maxpool_halo": [_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _I, _I, _I, _P, _P, _I, _I, _P],
    "segblocks_block_conv3x3_workspace_size": [_I] * 10 + [_ZP],
    "segblocks_block_conv_ex_workspace_size": [_I] * 12 + [_ZP],
    "segblocks_layer_workspace_size": [_I] * 8 + [_ZP],
    "segblocks_conv2d": [_P, _I, _I, _I, _I, _I, _I, _P, _P, _I, _I, _I, _I, _I, _P, _P],
    "segblocks_maxpool": [_P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P],
}

_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2011_12025_amd.build`")
        l = ctypes.CDLL(LIB_PATH)
        for name, args in _SIGS.items():
            f = getattr(l, name)
            f.argtypes = args
            f.restype = _I
        l.segblocks_last_error.argtypes = []
        l.segblocks_last_error.restype = ctypes.c_char_p
        _lib = l
    return _lib


class SegBlocksError(RuntimeError):
    def __init__(self, fn: str, code: int, msg: str):
        super().__init__(f"{fn} failed with status {code}: {msg}")
        self.code = code


def check(fn: str, code: int) -> None:
    if code != 0:
        raise SegBlocksError(fn, code, lib().segblocks_last_error().decode())


def call(fn: str, *args) -> None:
    check(fn, getattr(lib(), fn)(*args))
