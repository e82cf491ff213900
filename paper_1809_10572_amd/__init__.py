"""SAMD b-bit quantized convolution for MI355X (gfx950): Python binding of libsamd.so.

The binding only marshals arguments: torch tensors supply device memory and the current
HIP stream, and every step runs in the HIP library.  Importing works without a GPU; any
call that would launch work raises if the library is missing or no GPU is visible.

Packed words are held in torch.int32 tensors (bit patterns of the library's uint32
words).  See include/samd.h for the storage format and the semantics of every call.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence, Tuple

import torch

__all__ = ["Fmt", "Conv2dDesc", "Conv1dPlan", "Conv2dPlan", "SamdError", "lib", "row_words", "pack", "unpack", "conv1d",
           "conv1d_plan", "conv2d_plan", "conv2d_candidates", "conv2d_tune_workspace", "conv2d_tune", "conv2d_untune",
           "conv2d_use_plan", "plan_key",
           "conv2d_workspace", "conv2d", "conv2d_noalloc", "conv2d_prepare", "conv2d_prepared",
           "conv2d_stage", "conv2d_accumulate",
           "conv2d_int8_prepare", "conv2d_int8_prepared", "conv2d_int8_workspace", "conv2d_int8", "conv2d_int8_plan",
           "conv2d_int8_candidates", "conv2d_int8_use_plan",
           "SpacedLayout", "conv2d_spaced_layout", "conv2d_spaced_plan", "conv2d_spaced_workspace", "conv2d_spaced_prepare",
           "conv2d_spaced_pack", "conv2d_spaced_from_packed", "conv2d_spaced", "relu_requant_spaced", "conv2d_spaced_tune", "max_i32",
           "relu_requant_pack", "relu_requant_nhwc_u8", "out_hw", "peak_launch", "peak_work", "LIB_PATH"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsamd.so")

SAMD_OK, SAMD_EINVAL, SAMD_EALIGN, SAMD_EUNSUPPORTED, SAMD_EOVERFLOW, SAMD_EHIP, SAMD_ENOSPC = 0, -1, -2, -3, -4, -5, -6


class Fmt(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_int32), ("is_signed", ctypes.c_int32)]

    def __init__(self, bits: int, is_signed: bool):
        super().__init__(int(bits), int(bool(is_signed)))

    def __repr__(self):
        return f"Fmt({self.bits}, {'s' if self.is_signed else 'u'})"


_DESC_FIELDS = ["N", "C", "H", "W", "M", "KH", "KW", "stride_h", "stride_w", "pad_h", "pad_w"]


class Conv2dDesc(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in _DESC_FIELDS]

    @classmethod
    def of(cls, shape) -> "Conv2dDesc":
        if isinstance(shape, cls):
            return shape
        vals = shape.as_tuple() if hasattr(shape, "as_tuple") else tuple(shape)
        return cls(*[int(v) for v in vals])


class Conv2dPlan(ctypes.Structure):
    _fields_ = [("lane_bits", ctypes.c_int32), ("lanes", ctypes.c_int32), ("taps_max", ctypes.c_int32),
                ("words_per_row", ctypes.c_int32), ("flush_channels", ctypes.c_int32),
                ("out_lanes", ctypes.c_int32), ("tap_words", ctypes.c_int32), ("phase", ctypes.c_int32 * 16), ("tap0", ctypes.c_int32 * 16),
                ("ntaps", ctypes.c_int32 * 16), ("rows_per_block", ctypes.c_int32), ("mblock", ctypes.c_int32),
                ("split_waves", ctypes.c_int32), ("chunk_channels", ctypes.c_int32), ("x_offset", ctypes.c_int32),
                ("col_segments", ctypes.c_int32), ("segment_columns", ctypes.c_int32),
                ("macs_per_mad", ctypes.c_double), ("rows_per_thread", ctypes.c_int32),
                ("shared_rows", ctypes.c_int32), ("model_cost", ctypes.c_double),
                ("layout_spaced", ctypes.c_int32), ("spacer_msb", ctypes.c_int32)]


class SpacedLayout(ctypes.Structure):
    _fields_ = [("lane_bits", ctypes.c_int32), ("lanes", ctypes.c_int32), ("words_per_row", ctypes.c_int32),
                ("tap_words", ctypes.c_int32), ("padded_rows", ctypes.c_int32), ("x_offset", ctypes.c_int32),
                ("spacer_msb", ctypes.c_int32), ("words", ctypes.c_int64)]


class Conv2dInt8Plan(ctypes.Structure):
    _fields_ = [("halo", ctypes.c_int32), ("mtile", ctypes.c_int32), ("positions", ctypes.c_int32),
                ("row_segments", ctypes.c_int32), ("lds_bytes", ctypes.c_int32), ("waves", ctypes.c_int32),
                ("workgroups", ctypes.c_int64)]


class Conv1dPlan(ctypes.Structure):
    _fields_ = [("lane_bits", ctypes.c_int32), ("lanes", ctypes.c_int32), ("groups", ctypes.c_int32),
                ("extra", ctypes.c_int32), ("out_lanes", ctypes.c_int32), ("tap0", ctypes.c_int32 * 16),
                ("ntaps", ctypes.c_int32 * 16)]


class SamdError(RuntimeError):
    def __init__(self, status: int, name: str, detail: str):
        super().__init__(f"{name} ({detail})" if detail else name)
        self.status = status


_lib = None
_p, _i64, _i32, _sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t


def lib():
    """The loaded libsamd.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_1809_10572_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        sigs = {
            "samd_status_str": (ctypes.c_char_p, [ctypes.c_int]),
            "samd_last_error": (ctypes.c_char_p, []),
            "samd_row_words": (_i64, [_i64, Fmt]),
            "samd_pack": (ctypes.c_int, [_p, _i64, _i64, Fmt, _p, _p, _p]),
            "samd_unpack": (ctypes.c_int, [_p, _i64, _i64, Fmt, _p, _p]),
            "samd_conv1d": (ctypes.c_int, [_p, _i64, Fmt, _p, _i32, Fmt, _p, _p]),
            "samd_conv1d_plan_query": (ctypes.c_int, [_i64, Fmt, _p, _i32, Fmt, ctypes.POINTER(Conv1dPlan)]),
            "samd_conv2d_plan_query": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt,
                                                      ctypes.POINTER(Conv2dPlan)]),
            "samd_conv2d_workspace": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt, ctypes.POINTER(_sz)]),
            "samd_conv2d": (ctypes.c_int, [_p, Fmt, _p, Fmt, ctypes.POINTER(Conv2dDesc), _p, _p, _sz, _p]),
            "samd_conv2d_prepare": (ctypes.c_int, [_p, Fmt, ctypes.POINTER(Conv2dDesc), Fmt, _p, _sz, _p]),
            "samd_conv2d_prepared": (ctypes.c_int, [_p, Fmt, Fmt, ctypes.POINTER(Conv2dDesc), _p, _p, _sz, _p]),
            "samd_conv2d_stage": (ctypes.c_int, [_p, Fmt, Fmt, ctypes.POINTER(Conv2dDesc), _p, _sz, _p]),
            "samd_conv2d_accumulate": (ctypes.c_int, [Fmt, Fmt, ctypes.POINTER(Conv2dDesc), _p, _p, _sz, _p]),
            "samd_conv2d_int8_prepare": (ctypes.c_int, [_p, Fmt, ctypes.POINTER(Conv2dDesc), Fmt, _p, _sz, _p]),
            "samd_conv2d_int8_prepared": (ctypes.c_int, [_p, Fmt, Fmt, ctypes.POINTER(Conv2dDesc), _p, _p, _sz,
                                                         _p]),
            "samd_conv2d_int8_workspace": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, ctypes.POINTER(_sz)]),
            "samd_conv2d_int8_plan_query": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt,
                                                           ctypes.POINTER(Conv2dInt8Plan)]),
            "samd_conv2d_int8_candidates": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt, _i32,
                                                           ctypes.POINTER(Conv2dInt8Plan), ctypes.POINTER(_i32)]),
            "samd_conv2d_int8_use_plan": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt,
                                                         ctypes.POINTER(Conv2dInt8Plan)]),
            "samd_conv2d_int8": (ctypes.c_int, [_p, Fmt, _p, Fmt, ctypes.POINTER(Conv2dDesc), _p, _p, _sz, _p]),
            "samd_max_i32": (ctypes.c_int, [_p, _i64, _p, _p]),
            "samd_relu_requant_pack": (ctypes.c_int, [_p, _i64, _i64, _p, Fmt, _p, _p, _p]),
            "samd_relu_requant_nhwc_u8": (ctypes.c_int, [_p, _i32, _i32, _i32, _i32, _p, Fmt, _p, _p]),
            "samd_relu_requant_stage": (ctypes.c_int, [_p, _p, Fmt, Fmt, ctypes.POINTER(Conv2dDesc), _p, _sz, _p,
                                                       _p]),
            "samd_lanewise": (ctypes.c_int, [ctypes.c_int, _p, _p, _i64, Fmt, _p, _p]),
            "samd_scale": (ctypes.c_int, [_p, _i64, Fmt, _i32, _p, _p]),
            "samd_conv2d_candidates": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt, _i32,
                                                      ctypes.POINTER(Conv2dPlan), ctypes.POINTER(_i32)]),
            "samd_conv2d_tune_workspace": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt, _i32,
                                                          ctypes.POINTER(_sz)]),
            "samd_conv2d_tune": (ctypes.c_int, [_p, Fmt, _p, Fmt, ctypes.POINTER(Conv2dDesc), _p, _p, _sz, _i32, _i32,
                                                ctypes.POINTER(Conv2dPlan), _p]),
            "samd_conv2d_untune": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt]),
            "samd_conv2d_use_plan": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt,
                                                    ctypes.POINTER(Conv2dPlan)]),
            "samd_conv2d_noalloc": (ctypes.c_int, [_p, Fmt, _p, Fmt, ctypes.POINTER(Conv2dDesc), _p, _p]),
            "samd_conv2d_spaced_layout": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt,
                                                         ctypes.POINTER(SpacedLayout)]),
            "samd_conv2d_spaced_plan_query": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt,
                                                             ctypes.POINTER(Conv2dPlan)]),
            "samd_conv2d_spaced_workspace": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt,
                                                            ctypes.POINTER(_sz)]),
            "samd_conv2d_spaced_prepare": (ctypes.c_int, [_p, Fmt, ctypes.POINTER(Conv2dDesc), Fmt, _p, _sz, _p]),
            "samd_conv2d_spaced_pack": (ctypes.c_int, [_p, Fmt, Fmt, ctypes.POINTER(Conv2dDesc), _p, _p]),
            "samd_conv2d_spaced_from_packed": (ctypes.c_int, [_p, Fmt, Fmt, ctypes.POINTER(Conv2dDesc), _p, _p]),
            "samd_conv2d_spaced": (ctypes.c_int, [_p, Fmt, Fmt, ctypes.POINTER(Conv2dDesc), _p, _p, _sz, _p]),
            "samd_relu_requant_spaced": (ctypes.c_int, [_p, _p, Fmt, Fmt, ctypes.POINTER(Conv2dDesc), _p, _p, _p]),
            "samd_conv2d_spaced_tune_workspace": (ctypes.c_int, [ctypes.POINTER(Conv2dDesc), Fmt, Fmt, _i32,
                                                                 ctypes.POINTER(_sz)]),
            "samd_conv2d_spaced_tune": (ctypes.c_int, [_p, Fmt, _p, Fmt, ctypes.POINTER(Conv2dDesc), _p, _p, _sz, _i32,
                                                       _i32, ctypes.POINTER(Conv2dPlan), _p]),
            "samd_peak_launch": (ctypes.c_int, [ctypes.c_int, _i64, _i32, _p, _p, _i64, _p]),
            "samd_peak_work": (ctypes.c_double, [ctypes.c_int, _i64, _i32, _i64]),
        }
        for name, (res, args) in sigs.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != SAMD_OK:
        L = lib()
        raise SamdError(status, L.samd_status_str(status).decode(), L.samd_last_error().decode())


def _stream(t: torch.Tensor) -> int:
    return torch.cuda.current_stream(t.device).cuda_stream


def _on_gpu(t: torch.Tensor) -> bool:
    return t.is_cuda


def _dev(t: torch.Tensor, dtype=None, name="tensor") -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not _on_gpu(t):
        raise ValueError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype not in (dtype if isinstance(dtype, tuple) else (dtype,)):
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _out(t: torch.Tensor, numel: int) -> torch.Tensor:
    _dev(t, torch.int32, "out")
    if t.numel() != numel:
        raise ValueError(f"out must hold {numel} int32 values, got {t.numel()}")
    return t


# The library cannot see how large a device buffer is: every tensor handed to it is
# checked here, so that a short or host-side tensor raises instead of being read or
# written past its end by a kernel.
def _min(t: torch.Tensor, dtype, numel: int, name: str) -> torch.Tensor:
    _dev(t, dtype, name)
    if t.numel() < numel:
        raise ValueError(f"{name} must hold at least {numel} {t.dtype} values, got {t.numel()}")
    return t


def _opt(t: Optional[torch.Tensor], name: str) -> Optional[int]:
    """Pointer of an optional one-value int32 device tensor (None stays NULL)."""
    return None if t is None else _min(t, torch.int32, 1, name).data_ptr()


def _ws_bytes(ws: torch.Tensor) -> int:
    _dev(ws, None, "ws")
    return ws.numel() * ws.element_size()


def _x_words(xp: torch.Tensor, shape, xfmt: Fmt, name: str = "xp") -> torch.Tensor:
    d = Conv2dDesc.of(shape)
    return _min(xp, torch.int32, d.N * d.C * d.H * row_words(d.W, xfmt.bits), name)


def _w_words(wp: torch.Tensor, shape, wfmt: Fmt, name: str = "wp") -> torch.Tensor:
    d = Conv2dDesc.of(shape)
    return _min(wp, torch.int32, d.M * d.C * d.KH * row_words(d.KW, wfmt.bits), name)


def out_hw(shape) -> Tuple[int, int]:
    d = Conv2dDesc.of(shape)
    return (d.H + 2 * d.pad_h - d.KH) // d.stride_h + 1, (d.W + 2 * d.pad_w - d.KW) // d.stride_w + 1


def row_words(length: int, bits: int) -> int:
    r = lib().samd_row_words(length, Fmt(bits, False))
    if r < 0:
        _check(int(r))
    return int(r)


def pack(values: torch.Tensor, bits: int, signed: bool, oor: Optional[torch.Tensor] = None,
         out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Pack the last axis of an int8 (signed) / uint8 (unsigned) GPU tensor."""
    _dev(values, torch.int8 if signed else torch.uint8, "values")
    length = values.shape[-1]
    rows = values.numel() // length if length else 0
    shape = values.shape[:-1] + (row_words(length, bits),)
    if out is None:
        out = torch.empty(shape, dtype=torch.int32, device=values.device)
    elif _dev(out, torch.int32, "out").shape != shape:
        raise ValueError(f"out must be a contiguous int32 tensor of shape {tuple(shape)}")
    _check(lib().samd_pack(values.data_ptr(), rows, length, Fmt(bits, signed), out.data_ptr(), _opt(oor, "oor"),
                           _stream(values)))
    return out


def unpack(words: torch.Tensor, length: int, bits: int, signed: bool) -> torch.Tensor:
    _dev(words, torch.int32, "words")
    if words.dim() == 0 or words.shape[-1] != row_words(length, bits):
        raise ValueError(f"words must have rows of {row_words(length, bits)} words for length {length}")
    rows = words.numel() // words.shape[-1] if words.shape[-1] else 0
    out = torch.empty(words.shape[:-1] + (length,), dtype=torch.int8 if signed else torch.uint8, device=words.device)
    _check(lib().samd_unpack(words.data_ptr(), rows, length, Fmt(bits, signed), out.data_ptr(), _stream(words)))
    return out


def conv1d(xp: torch.Tensor, n: int, bits: int, taps: Sequence[int], kbits: int,
           out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Valid-mode true convolution of one packed unsigned row with host taps."""
    _min(xp, torch.int32, row_words(n, bits) if n > 0 else 0, "xp")
    K = len(taps)
    arr = (ctypes.c_int32 * K)(*[int(t) for t in taps])
    if out is None:
        out = torch.empty(max(n - K + 1, 0), dtype=torch.int32, device=xp.device)
    _out(out, max(n - K + 1, 0))
    _check(lib().samd_conv1d(xp.data_ptr(), n, Fmt(bits, False), arr, K, Fmt(kbits, False), out.data_ptr(),
                             _stream(xp)))
    return out


def conv1d_plan(n: int, bits: int, taps: Sequence[int], kbits: int) -> Conv1dPlan:
    K = len(taps)
    arr = (ctypes.c_int32 * K)(*[int(t) for t in taps])
    plan = Conv1dPlan()
    _check(lib().samd_conv1d_plan_query(n, Fmt(bits, False), arr, K, Fmt(kbits, False), ctypes.byref(plan)))
    return plan


def conv2d_plan(shape, xfmt: Fmt, wfmt: Fmt) -> Conv2dPlan:
    plan = Conv2dPlan()
    _check(lib().samd_conv2d_plan_query(ctypes.byref(Conv2dDesc.of(shape)), xfmt, wfmt, ctypes.byref(plan)))
    return plan


def conv2d_workspace(shape, xfmt: Fmt, wfmt: Fmt) -> int:
    n = _sz(0)
    _check(lib().samd_conv2d_workspace(ctypes.byref(Conv2dDesc.of(shape)), xfmt, wfmt, ctypes.byref(n)))
    return int(n.value)


MAX_CANDIDATES = 64


def conv2d_candidates(shape, xfmt: Fmt, wfmt: Fmt, max_count: int = 16) -> List[Conv2dPlan]:
    """Candidate plans ranked by the planner's cost model, its own choice first."""
    arr = (Conv2dPlan * max(1, min(max_count, MAX_CANDIDATES)))()
    n = _i32(0)
    _check(lib().samd_conv2d_candidates(ctypes.byref(Conv2dDesc.of(shape)), xfmt, wfmt, max_count, arr,
                                        ctypes.byref(n)))
    return [arr[i] for i in range(n.value)]


def conv2d_tune_workspace(shape, xfmt: Fmt, wfmt: Fmt, candidates: int = 16) -> int:
    n = _sz(0)
    _check(lib().samd_conv2d_tune_workspace(ctypes.byref(Conv2dDesc.of(shape)), xfmt, wfmt, candidates,
                                            ctypes.byref(n)))
    return int(n.value)


def conv2d_tune(xp: torch.Tensor, xfmt: Fmt, wp: torch.Tensor, wfmt: Fmt, shape, candidates: int = 16,
                reps: int = 5, ws: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None) -> Conv2dPlan:
    """Time the first `candidates` plans on these inputs and keep the fastest for the shape
    (blocks until the timings are read).  Workspaces prepared for the shape earlier must
    be sized and prepared again afterwards."""
    _x_words(xp, shape, xfmt)
    _w_words(wp, shape, wfmt)
    d = Conv2dDesc.of(shape)
    Ho, Wo = out_hw(shape)
    if ws is None:
        ws = _workspace(conv2d_tune_workspace(shape, xfmt, wfmt, candidates), xp.device)
    if out is None:
        out = torch.empty((d.N, d.M, Ho, Wo), dtype=torch.int32, device=xp.device)
    _out(out, d.N * d.M * Ho * Wo)
    plan = Conv2dPlan()
    _check(lib().samd_conv2d_tune(xp.data_ptr(), xfmt, wp.data_ptr(), wfmt, ctypes.byref(d), out.data_ptr(),
                                  ws.data_ptr(), _ws_bytes(ws), candidates, reps, ctypes.byref(plan), _stream(xp)))
    return plan


PLAN_KEY_FIELDS = ("lane_bits", "lanes", "x_offset", "shared_rows", "rows_per_thread", "rows_per_block", "mblock",
                   "split_waves", "layout_spaced", "spacer_msb")


def plan_key(plan: Conv2dPlan) -> dict:
    """The fields that identify a plan among a shape's candidates (for conv2d_use_plan)."""
    return {f: int(getattr(plan, f)) for f in PLAN_KEY_FIELDS}


def conv2d_use_plan(shape, xfmt: Fmt, wfmt: Fmt, plan) -> None:
    """Make a plan (a Conv2dPlan, or a plan_key dict) the shape's plan, as if tuned."""
    if isinstance(plan, dict):
        p = Conv2dPlan()
        for f in PLAN_KEY_FIELDS:
            setattr(p, f, int(plan.get(f, 0)))
        plan = p
    _check(lib().samd_conv2d_use_plan(ctypes.byref(Conv2dDesc.of(shape)), xfmt, wfmt, ctypes.byref(plan)))


def conv2d_untune(shape=None, xfmt: Optional[Fmt] = None, wfmt: Optional[Fmt] = None) -> None:
    """Forget the tuned plan of one shape, or of every shape (shape None)."""
    if shape is None:
        _check(lib().samd_conv2d_untune(None, Fmt(1, False), Fmt(1, False)))
    else:
        _check(lib().samd_conv2d_untune(ctypes.byref(Conv2dDesc.of(shape)), xfmt, wfmt))


def _workspace(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator returns blocks aligned to at least 512 bytes
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def conv2d(xp: torch.Tensor, xfmt: Fmt, wp: torch.Tensor, wfmt: Fmt, shape, ws: Optional[torch.Tensor] = None,
           out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """SAMD conv2d of packed activations (N*C*H rows of W) and packed weights
    (M*C*KH rows of KW); returns int32 N x M x Ho x Wo."""
    _x_words(xp, shape, xfmt)
    _w_words(wp, shape, wfmt)
    d = Conv2dDesc.of(shape)
    Ho, Wo = out_hw(shape)
    if ws is None:
        ws = _workspace(conv2d_workspace(shape, xfmt, wfmt), xp.device)
    if out is None:
        out = torch.empty((d.N, d.M, Ho, Wo), dtype=torch.int32, device=xp.device)
    _out(out, d.N * d.M * Ho * Wo)
    _check(lib().samd_conv2d(xp.data_ptr(), xfmt, wp.data_ptr(), wfmt, ctypes.byref(d), out.data_ptr(),
                             ws.data_ptr(), _ws_bytes(ws), _stream(xp)))
    return out


NOALLOC_SCRATCH_BYTES = 64 << 20


def conv2d_noalloc(xp: torch.Tensor, xfmt: Fmt, wp: torch.Tensor, wfmt: Fmt, shape, out: torch.Tensor) -> torch.Tensor:
    """conv2d with the library's own scratch array as the workspace (the call allocates no
    device memory; `out` must be given).  Calls that may overlap on one GPU race."""
    _x_words(xp, shape, xfmt)
    _w_words(wp, shape, wfmt)
    d = Conv2dDesc.of(shape)
    Ho, Wo = out_hw(shape)
    _out(out, d.N * d.M * Ho * Wo)
    _check(lib().samd_conv2d_noalloc(xp.data_ptr(), xfmt, wp.data_ptr(), wfmt, ctypes.byref(d), out.data_ptr(),
                                     _stream(xp)))
    return out


def conv2d_prepare(wp: torch.Tensor, wfmt: Fmt, shape, xfmt: Fmt, ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Kernel words of one layer, for any number of conv2d_prepared calls."""
    _w_words(wp, shape, wfmt)
    if ws is None:
        ws = _workspace(conv2d_workspace(shape, xfmt, wfmt), wp.device)
    _check(lib().samd_conv2d_prepare(wp.data_ptr(), wfmt, ctypes.byref(Conv2dDesc.of(shape)), xfmt, ws.data_ptr(),
                                     _ws_bytes(ws), _stream(wp)))
    return ws


def conv2d_prepared(xp: torch.Tensor, xfmt: Fmt, wfmt: Fmt, shape, ws: torch.Tensor,
                    out: Optional[torch.Tensor] = None) -> torch.Tensor:
    _x_words(xp, shape, xfmt)
    d = Conv2dDesc.of(shape)
    Ho, Wo = out_hw(shape)
    if out is None:
        out = torch.empty((d.N, d.M, Ho, Wo), dtype=torch.int32, device=xp.device)
    _out(out, d.N * d.M * Ho * Wo)
    _check(lib().samd_conv2d_prepared(xp.data_ptr(), xfmt, wfmt, ctypes.byref(d), out.data_ptr(), ws.data_ptr(),
                                      _ws_bytes(ws), _stream(xp)))
    return out


def conv2d_stage(xp: torch.Tensor, xfmt: Fmt, wfmt: Fmt, shape, ws: torch.Tensor) -> torch.Tensor:
    """Spread the packed input into the workspace's operand words (first half of conv2d_prepared)."""
    _x_words(xp, shape, xfmt)
    _check(lib().samd_conv2d_stage(xp.data_ptr(), xfmt, wfmt, ctypes.byref(Conv2dDesc.of(shape)), ws.data_ptr(),
                                   _ws_bytes(ws), _stream(xp)))
    return ws


def conv2d_accumulate(xfmt: Fmt, wfmt: Fmt, shape, ws: torch.Tensor,
                      out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Multiply, accumulate, decode and store from a prepared and staged workspace."""
    ws_bytes = _ws_bytes(ws)
    d = Conv2dDesc.of(shape)
    Ho, Wo = out_hw(shape)
    if out is None:
        out = torch.empty((d.N, d.M, Ho, Wo), dtype=torch.int32, device=ws.device)
    _out(out, d.N * d.M * Ho * Wo)
    _check(lib().samd_conv2d_accumulate(xfmt, wfmt, ctypes.byref(d), out.data_ptr(), ws.data_ptr(), ws_bytes,
                                        _stream(ws)))
    return out


def conv2d_int8_prepare(w: torch.Tensor, wfmt: Fmt, shape, xfmt: Fmt, ws: Optional[torch.Tensor] = None):
    d = Conv2dDesc.of(shape)
    _min(w, torch.int8, d.M * d.C * d.KH * d.KW, "w")
    if ws is None:
        ws = _workspace(conv2d_int8_workspace(shape, xfmt), w.device)
    _check(lib().samd_conv2d_int8_prepare(w.data_ptr(), wfmt, ctypes.byref(d), xfmt, ws.data_ptr(), _ws_bytes(ws),
                                          _stream(w)))
    return ws


def conv2d_int8_prepared(x_nhwc: torch.Tensor, xfmt: Fmt, wfmt: Fmt, shape, ws: torch.Tensor,
                         out: Optional[torch.Tensor] = None) -> torch.Tensor:
    d = Conv2dDesc.of(shape)
    _min(x_nhwc, (torch.int8, torch.uint8), d.N * d.H * d.W * d.C, "x_nhwc")
    Ho, Wo = out_hw(shape)
    if out is None:
        out = torch.empty((d.N, d.M, Ho, Wo), dtype=torch.int32, device=x_nhwc.device)
    _out(out, d.N * d.M * Ho * Wo)
    _check(lib().samd_conv2d_int8_prepared(x_nhwc.data_ptr(), xfmt, wfmt, ctypes.byref(d), out.data_ptr(),
                                           ws.data_ptr(), _ws_bytes(ws), _stream(x_nhwc)))
    return out


def conv2d_int8_plan(shape, xfmt: Fmt, wfmt: Fmt) -> Conv2dInt8Plan:
    """The kernel and tile conv2d_int8 uses for this layer (16-byte aligned activations)."""
    plan = Conv2dInt8Plan()
    _check(lib().samd_conv2d_int8_plan_query(ctypes.byref(Conv2dDesc.of(shape)), xfmt, wfmt, ctypes.byref(plan)))
    return plan


def conv2d_int8_candidates(shape, xfmt: Fmt, wfmt: Fmt) -> List[Conv2dInt8Plan]:
    """Every launch conv2d_int8 can make for this layer (halo tiles, weight-resident runs, then im2col)."""
    arr = (Conv2dInt8Plan * MAX_CANDIDATES)()
    n = _i32(0)
    _check(lib().samd_conv2d_int8_candidates(ctypes.byref(Conv2dDesc.of(shape)), xfmt, wfmt, MAX_CANDIDATES, arr,
                                             ctypes.byref(n)))
    return [arr[i] for i in range(n.value)]


def conv2d_int8_use_plan(shape, xfmt: Fmt, wfmt: Fmt, plan: Optional[Conv2dInt8Plan]) -> None:
    """Make one of the layer's int8 candidates its launch (None: the library's own choice)."""
    _check(lib().samd_conv2d_int8_use_plan(ctypes.byref(Conv2dDesc.of(shape)), xfmt, wfmt,
                                           None if plan is None else ctypes.byref(plan)))


def conv2d_int8_workspace(shape, xfmt: Fmt) -> int:
    n = _sz(0)
    _check(lib().samd_conv2d_int8_workspace(ctypes.byref(Conv2dDesc.of(shape)), xfmt, ctypes.byref(n)))
    return int(n.value)


def conv2d_int8(x_nhwc: torch.Tensor, xfmt: Fmt, w: torch.Tensor, wfmt: Fmt, shape,
                ws: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Native 8-bit baseline: x is N x H x W x C int8/uint8, w is M x C x KH x KW int8."""
    d = Conv2dDesc.of(shape)
    _min(x_nhwc, (torch.int8, torch.uint8), d.N * d.H * d.W * d.C, "x_nhwc")
    _min(w, torch.int8, d.M * d.C * d.KH * d.KW, "w")
    Ho, Wo = out_hw(shape)
    if ws is None:
        ws = _workspace(conv2d_int8_workspace(shape, xfmt), x_nhwc.device)
    if out is None:
        out = torch.empty((d.N, d.M, Ho, Wo), dtype=torch.int32, device=x_nhwc.device)
    _out(out, d.N * d.M * Ho * Wo)
    _check(lib().samd_conv2d_int8(x_nhwc.data_ptr(), xfmt, w.data_ptr(), wfmt, ctypes.byref(d), out.data_ptr(),
                                  ws.data_ptr(), _ws_bytes(ws), _stream(x_nhwc)))
    return out


def max_i32(t: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    _dev(t, torch.int32, "t")
    if out is None:
        out = torch.empty(1, dtype=torch.int32, device=t.device)
    _check(lib().samd_max_i32(t.data_ptr(), t.numel(), _opt(out, "out"), _stream(t)))
    return out


def relu_requant_pack(acc: torch.Tensor, dev_max: torch.Tensor, bits: int,
                      shift_out: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """ReLU + requantise an int32 tensor's rows (last axis) to packed unsigned b bits."""
    _dev(acc, torch.int32, "acc")
    length = acc.shape[-1]
    rows = acc.numel() // length
    if out is None:
        out = torch.empty(acc.shape[:-1] + (row_words(length, bits),), dtype=torch.int32, device=acc.device)
    _min(out, torch.int32, rows * row_words(length, bits), "out")
    _check(lib().samd_relu_requant_pack(acc.data_ptr(), rows, length, _opt(dev_max, "dev_max"), Fmt(bits, False),
                                        out.data_ptr(), _opt(shift_out, "shift_out"), _stream(acc)))
    return out


def relu_requant_nhwc_u8(acc: torch.Tensor, dev_max: torch.Tensor, bits: int,
                         out: Optional[torch.Tensor] = None) -> torch.Tensor:
    _dev(acc, torch.int32, "acc")
    N, C, H, W = acc.shape
    if out is None:
        out = torch.empty((N, H, W, C), dtype=torch.uint8, device=acc.device)
    _min(out, torch.uint8, N * H * W * C, "out")
    _check(lib().samd_relu_requant_nhwc_u8(acc.data_ptr(), N, C, H, W, _opt(dev_max, "dev_max"), Fmt(bits, False),
                                           out.data_ptr(), _stream(acc)))
    return out


LANE_ADD, LANE_SUB, LANE_MUL = 0, 1, 2


def lanewise(op: int, a: torch.Tensor, b: torch.Tensor, bits: int, signed: bool,
             out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Lane-wise add, subtract or multiply (LANE_ADD / LANE_SUB / LANE_MUL) of two packed
    int32 word tensors of the same shape; lanes wrap modulo 2**bits."""
    a = _dev(a, torch.int32, "a")
    b = _dev(b, torch.int32, "b")
    if a.shape != b.shape:
        raise ValueError("a and b must have the same shape")
    out = _out(out, a.numel()) if out is not None else torch.empty_like(a)
    _check(lib().samd_lanewise(op, a.data_ptr(), b.data_ptr(), a.numel(), Fmt(bits, signed), out.data_ptr(),
                               _stream(a)))
    return out


def scale(a: torch.Tensor, scalar: int, bits: int, signed: bool, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Every lane of the packed words a times one scalar, modulo 2**bits."""
    a = _dev(a, torch.int32, "a")
    out = _out(out, a.numel()) if out is not None else torch.empty_like(a)
    _check(lib().samd_scale(a.data_ptr(), a.numel(), Fmt(bits, signed), int(scalar), out.data_ptr(), _stream(a)))
    return out


def relu_requant_stage(acc: torch.Tensor, dev_max: torch.Tensor, bits: int, wfmt: Fmt, shape, ws: torch.Tensor,
                       dev_shift: Optional[torch.Tensor] = None) -> torch.Tensor:
    """ReLU + requantisation of acc to unsigned `bits`, written as the operand words of the
    next layer (descriptor `shape`, weight format `wfmt`) into its workspace `ws`; follow
    with conv2d_accumulate.  Returns ws."""
    d = Conv2dDesc.of(shape)
    _min(acc, torch.int32, d.N * d.C * d.H * d.W, "acc")
    _check(lib().samd_relu_requant_stage(acc.data_ptr(), _opt(dev_max, "dev_max"), Fmt(bits, False), wfmt,
                                         ctypes.byref(d), ws.data_ptr(), _ws_bytes(ws), _opt(dev_shift, "dev_shift"),
                                         _stream(acc)))
    return ws


PEAK_MAD_I64_I32, PEAK_VALU_I32, PEAK_MFMA_I8, PEAK_COPY, PEAK_READ, PEAK_LDS, PEAK_WRITE = 0, 1, 2, 3, 4, 5, 6


def peak_work(kind: int, iters: int, blocks: int, nbytes: int = 0) -> float:
    """Work (lane ops, multiply-adds or bytes) of one peak_launch with these arguments."""
    w = lib().samd_peak_work(kind, iters, blocks, nbytes)
    if w < 0:
        raise ValueError("bad peak microbenchmark arguments")
    return w


def peak_launch(kind: int, iters: int, blocks: int, dst: torch.Tensor, src: Optional[torch.Tensor] = None,
                nbytes: int = 0) -> None:
    """Enqueue one ceiling microbenchmark (include/samd_peaks.h) on the current stream."""
    if kind == PEAK_WRITE:
        need = nbytes
    elif kind in (PEAK_COPY, PEAK_READ):
        if src is None:
            raise ValueError("copy and read need src")
        _min(src, None, 0, "src")
        if src.numel() * src.element_size() < nbytes:
            raise ValueError("src is shorter than nbytes")
        need = nbytes if kind == PEAK_COPY else 4 * blocks
    else:
        need = 4 * 256 * blocks
    _dev(dst, None, "dst")
    if dst.numel() * dst.element_size() < need:
        raise ValueError(f"dst must hold {need} bytes")
    _check(lib().samd_peak_launch(kind, iters, blocks, None if src is None else src.data_ptr(), dst.data_ptr(),
                                  nbytes, _stream(dst)))


# --- permanent-spacer layout (include/samd.h, "Permanent-spacer activations") -----------

def conv2d_spaced_layout(shape, xfmt: Fmt, wfmt: Fmt) -> SpacedLayout:
    out = SpacedLayout()
    _check(lib().samd_conv2d_spaced_layout(ctypes.byref(Conv2dDesc.of(shape)), xfmt, wfmt, ctypes.byref(out)))
    return out


def conv2d_spaced_plan(shape, xfmt: Fmt, wfmt: Fmt) -> Conv2dPlan:
    plan = Conv2dPlan()
    _check(lib().samd_conv2d_spaced_plan_query(ctypes.byref(Conv2dDesc.of(shape)), xfmt, wfmt, ctypes.byref(plan)))
    return plan


def conv2d_spaced_workspace(shape, xfmt: Fmt, wfmt: Fmt) -> int:
    n = _sz(0)
    _check(lib().samd_conv2d_spaced_workspace(ctypes.byref(Conv2dDesc.of(shape)), xfmt, wfmt, ctypes.byref(n)))
    return int(n.value)


def _spaced_out(out: Optional[torch.Tensor], shape, xfmt: Fmt, wfmt: Fmt, device) -> torch.Tensor:
    words = conv2d_spaced_layout(shape, xfmt, wfmt).words
    if out is None:
        return torch.empty(words, dtype=torch.int32, device=device)
    return _min(out, torch.int32, words, "out")


def conv2d_spaced_prepare(wp: torch.Tensor, wfmt: Fmt, shape, xfmt: Fmt, ws: Optional[torch.Tensor] = None):
    """Kernel words of one layer for the permanent-spacer convolution."""
    _w_words(wp, shape, wfmt)
    if ws is None:
        ws = _workspace(conv2d_spaced_workspace(shape, xfmt, wfmt), wp.device)
    _check(lib().samd_conv2d_spaced_prepare(wp.data_ptr(), wfmt, ctypes.byref(Conv2dDesc.of(shape)), xfmt,
                                            ws.data_ptr(), _ws_bytes(ws), _stream(wp)))
    return ws


def conv2d_spaced_pack(values: torch.Tensor, xfmt: Fmt, wfmt: Fmt, shape,
                       out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """8-bit activations (N x C x H x W, int8 when xfmt is signed, else uint8) written in
    the layer's permanent-spacer layout."""
    d = Conv2dDesc.of(shape)
    _min(values, torch.int8 if xfmt.is_signed else torch.uint8, d.N * d.C * d.H * d.W, "values")
    out = _spaced_out(out, shape, xfmt, wfmt, values.device)
    _check(lib().samd_conv2d_spaced_pack(values.data_ptr(), xfmt, wfmt, ctypes.byref(d), out.data_ptr(),
                                         _stream(values)))
    return out


def conv2d_spaced_from_packed(xp: torch.Tensor, xfmt: Fmt, wfmt: Fmt, shape,
                              out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Packed activations (the packed format) rewritten in the permanent-spacer layout."""
    _x_words(xp, shape, xfmt)
    out = _spaced_out(out, shape, xfmt, wfmt, xp.device)
    _check(lib().samd_conv2d_spaced_from_packed(xp.data_ptr(), xfmt, wfmt, ctypes.byref(Conv2dDesc.of(shape)),
                                                out.data_ptr(), _stream(xp)))
    return out


def conv2d_spaced(xs: torch.Tensor, xfmt: Fmt, wfmt: Fmt, shape, ws: torch.Tensor,
                  out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Convolution from activations in the permanent-spacer layout (no spread pass)."""
    _min(xs, torch.int32, conv2d_spaced_layout(shape, xfmt, wfmt).words, "xs")
    d = Conv2dDesc.of(shape)
    Ho, Wo = out_hw(shape)
    if out is None:
        out = torch.empty((d.N, d.M, Ho, Wo), dtype=torch.int32, device=xs.device)
    _out(out, d.N * d.M * Ho * Wo)
    _check(lib().samd_conv2d_spaced(xs.data_ptr(), xfmt, wfmt, ctypes.byref(d), out.data_ptr(), ws.data_ptr(),
                                    _ws_bytes(ws), _stream(xs)))
    return out


def relu_requant_spaced(acc: torch.Tensor, dev_max: torch.Tensor, bits: int, wfmt: Fmt, shape,
                        out: Optional[torch.Tensor] = None, dev_shift: Optional[torch.Tensor] = None) -> torch.Tensor:
    """ReLU + requantisation to unsigned `bits`, written as the next layer's (descriptor
    `shape`, weights `wfmt`) activations in the permanent-spacer layout."""
    d = Conv2dDesc.of(shape)
    _min(acc, torch.int32, d.N * d.C * d.H * d.W, "acc")
    xf = Fmt(bits, False)
    out = _spaced_out(out, shape, xf, wfmt, acc.device)
    _check(lib().samd_relu_requant_spaced(acc.data_ptr(), _opt(dev_max, "dev_max"), xf, wfmt, ctypes.byref(d),
                                          out.data_ptr(), _opt(dev_shift, "dev_shift"), _stream(acc)))
    return out


def conv2d_spaced_tune(xp: torch.Tensor, xfmt: Fmt, wp: torch.Tensor, wfmt: Fmt, shape, candidates: int = 16,
                       reps: int = 5, ws: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None) -> Conv2dPlan:
    """Tune the permanent-spacer layout's plan on packed inputs (blocks).  Tensors in the
    layout and workspaces of the shape must be written and prepared again afterwards."""
    _x_words(xp, shape, xfmt)
    _w_words(wp, shape, wfmt)
    d = Conv2dDesc.of(shape)
    Ho, Wo = out_hw(shape)
    if ws is None:
        n = _sz(0)
        _check(lib().samd_conv2d_spaced_tune_workspace(ctypes.byref(d), xfmt, wfmt, candidates, ctypes.byref(n)))
        ws = _workspace(int(n.value), xp.device)
    if out is None:
        out = torch.empty((d.N, d.M, Ho, Wo), dtype=torch.int32, device=xp.device)
    _out(out, d.N * d.M * Ho * Wo)
    plan = Conv2dPlan()
    _check(lib().samd_conv2d_spaced_tune(xp.data_ptr(), xfmt, wp.data_ptr(), wfmt, ctypes.byref(d), out.data_ptr(),
                                         ws.data_ptr(), _ws_bytes(ws), candidates, reps, ctypes.byref(plan),
                                         _stream(xp)))
    return plan
