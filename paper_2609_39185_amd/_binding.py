"""ctypes binding of libssmq.so (include/ssmq.h): argument marshalling only.

Tensors are torch device tensors; their data pointers and torch's current HIP
stream are handed to the C ABI unchanged. Every step of the computation runs in
the library's HIP kernels. If the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os

import torch  # imported first so the HIP runtime is the one torch already loaded

LIBRARY = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libssmq.so")

RULES = {"rtn": 0, "sr": 1, "weyl": 2, "philox": 3}
FORMATS = {"fp16": 0, "bf16": 1, "e4m3": 2, "fp32": 3, "int8": 4, "int4": 5}
CODE_BYTES = {"fp16": 2, "bf16": 2, "e4m3": 1, "fp32": 4, "int8": 1, "int4": 1}
# entries per element of the code tensor (INT4: two per byte, even entry in the low nibble)
ENTRIES_PER_CODE = {"fp16": 1, "bf16": 1, "e4m3": 1, "fp32": 1, "int8": 1, "int4": 2}
SCALED = ("e4m3", "int8", "int4")

_i32, _i64, _u32, _u64, _vp = (ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                               ctypes.c_uint64, ctypes.c_void_p)


class Dims(ctypes.Structure):
    _fields_ = [("batch", _i64), ("nheads", _i32), ("headdim", _i32), ("dstate", _i32),
                ("ngroups", _i32), ("a_per_state", _i32)]


class QParams(ctypes.Structure):
    _fields_ = [("rule", _i32), ("format", _i32), ("dither_block", _i32),
                ("scale_group", _i32), ("seed", _u32), ("layer", _u32), ("step", _u32),
                ("flags", _u32), ("entry_base", _u64)]


class StepOpts(ctypes.Structure):
    _fields_ = [("dt_bias", _vp), ("dt_softplus", _i32), ("reserved", _i32), ("z", _vp)]


class SsmqError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"ssmq status {status}: {message}")
        self.status = status


EXPORTS = ("ssmq_state_update", "ssmq_state_update_ex", "ssmq_conv1d_update", "ssmq_requantize",
           "ssmq_dither_fill", "ssmq_replay", "ssmq_status_string", "ssmq_last_error")

_lib = None


def library() -> ctypes.CDLL:
    """Load libssmq.so once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIBRARY):
        raise RuntimeError(f"{LIBRARY} is missing: build it with paper_2609_39185_amd.build.build()")
    L = ctypes.CDLL(LIBRARY)
    L.ssmq_state_update.argtypes = [ctypes.POINTER(Dims), ctypes.POINTER(QParams), _vp, _vp, _vp,
                                    _vp, _vp, _vp, _vp, _vp, _vp, _vp]
    L.ssmq_state_update.restype = _i32
    L.ssmq_state_update_ex.argtypes = [ctypes.POINTER(Dims), ctypes.POINTER(QParams),
                                       ctypes.POINTER(StepOpts), _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                       _vp, _vp, _vp]
    L.ssmq_state_update_ex.restype = _i32
    L.ssmq_conv1d_update.argtypes = [_i64, _i32, _i32, _vp, _vp, _vp, _vp, _i32, _vp, _vp]
    L.ssmq_conv1d_update.restype = _i32
    L.ssmq_requantize.argtypes = [ctypes.POINTER(QParams), _i64, _i64, _vp, _vp, _vp, _vp]
    L.ssmq_requantize.restype = _i32
    L.ssmq_dither_fill.argtypes = [_i32, _u32, _u32, _u32, _u64, _i64, _i32, _vp, _vp]
    L.ssmq_dither_fill.restype = _i32
    L.ssmq_replay.argtypes = [ctypes.POINTER(QParams), _i64, _i32, _i32, _vp, _vp, _vp, _vp, _vp,
                              _vp, _vp, _vp, _vp]
    L.ssmq_replay.restype = _i32
    L.ssmq_status_string.argtypes = [_i32]
    L.ssmq_status_string.restype = ctypes.c_char_p
    L.ssmq_last_error.argtypes = []
    L.ssmq_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(status: int) -> None:
    if status != 0:
        L = library()
        msg = L.ssmq_last_error().decode() or L.ssmq_status_string(status).decode()
        raise SsmqError(status, msg)


def _ptr(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch.Tensor")
    if not t.is_cuda:
        raise ValueError("tensors passed to libssmq must live in GPU memory")
    if not t.is_contiguous():
        raise ValueError("tensors passed to libssmq must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream, ref: torch.Tensor):
    if stream is None:
        stream = torch.cuda.current_stream(ref.device)
    return ctypes.c_void_p(stream.cuda_stream)


FLAG_FP32_STATE = 1


def qparams(rule: str, fmt: str, *, dither_block=16, scale_group=0, seed=0, layer=0, step=0,
            entry_base=0, flags=0) -> QParams:
    return QParams(RULES[rule], FORMATS[fmt], int(dither_block), int(scale_group),
                   int(seed) & 0xFFFFFFFF, int(layer) & 0xFFFFFFFF, int(step) & 0xFFFFFFFF,
                   int(flags), int(entry_base))


def state_update(state, scale, x, dt, A, B, C, D, y, *, rule: str, fmt: str, dither_block=16,
                 scale_group=0, seed=0, layer=0, step=0, entry_base=0, fp32_state=False,
                 dt_bias=None, dt_softplus=False, z=None, stream=None) -> None:
    """ssmq_state_update on [batch, nheads, headdim, dstate] state codes, in place
    (INT4: [batch, nheads, headdim, dstate / 2] bytes). fp32_state: a checkpoint
    write on an fp32 state [batch, nheads, headdim, dstate] (SSMQ_FLAG_FP32_STATE)."""
    batch, nheads, headdim, dstate = state.shape
    if fp32_state:
        if state.dtype != torch.float32:
            raise ValueError("a checkpoint write needs an fp32 state")
    else:
        dstate *= ENTRIES_PER_CODE[fmt]
        if state.element_size() != CODE_BYTES[fmt]:
            raise ValueError(f"state element size {state.element_size()} does not match {fmt}")
    dims = Dims(batch, nheads, headdim, dstate, B.shape[1], 1 if A.dim() == 2 else 0)
    q = qparams(rule, fmt, dither_block=dither_block, scale_group=scale_group, seed=seed,
                layer=layer, step=step, entry_base=entry_base,
                flags=FLAG_FP32_STATE if fp32_state else 0)
    if dt_bias is None and not dt_softplus and z is None:
        _check(library().ssmq_state_update(ctypes.byref(dims), ctypes.byref(q), _ptr(state),
                                           _ptr(scale), _ptr(x), _ptr(dt), _ptr(A), _ptr(B),
                                           _ptr(C), _ptr(D), _ptr(y), _stream(stream, state)))
    else:
        opts = StepOpts(_ptr(dt_bias), 1 if dt_softplus else 0, 0, _ptr(z))
        _check(library().ssmq_state_update_ex(ctypes.byref(dims), ctypes.byref(q),
                                              ctypes.byref(opts), _ptr(state), _ptr(scale),
                                              _ptr(x), _ptr(dt), _ptr(A), _ptr(B), _ptr(C),
                                              _ptr(D), _ptr(y), _stream(stream, state)))


def conv1d_update(conv_state, x, weight, bias, out, *, act=True, stream=None) -> None:
    """ssmq_conv1d_update: conv_state [batch, channels, width] shifted in place,
    out [batch, channels] written."""
    batch, channels, width = conv_state.shape
    _check(library().ssmq_conv1d_update(batch, channels, width, _ptr(conv_state), _ptr(x),
                                        _ptr(weight), _ptr(bias), 1 if act else 0, _ptr(out),
                                        _stream(stream, conv_state)))


def requantize(h, codes, scale, *, rule: str, fmt: str, head_size=0, dither_block=16,
               scale_group=0, seed=0, layer=0, step=0, entry_base=0, stream=None) -> None:
    """ssmq_requantize: fp32 h -> codes (and E4M3 / INT8 / INT4 group scales)."""
    if (codes.numel() * ENTRIES_PER_CODE[fmt] != h.numel()
            or codes.element_size() != CODE_BYTES[fmt]):
        raise ValueError("codes must match h in size and the format in element size")
    q = qparams(rule, fmt, dither_block=dither_block, scale_group=scale_group, seed=seed,
                layer=layer, step=step, entry_base=entry_base)
    _check(library().ssmq_requantize(ctypes.byref(q), h.numel(), int(head_size), _ptr(h),
                                     _ptr(codes), _ptr(scale), _stream(stream, h)))


def dither_fill(out, *, rule: str, seed=0, layer=0, step=0, entry_base=0, dither_block=16,
                stream=None) -> None:
    """ssmq_dither_fill into a uint32 (int32-typed) tensor."""
    if out.element_size() != 4:
        raise ValueError("thresholds are 32-bit words")
    _check(library().ssmq_dither_fill(RULES[rule], int(seed) & 0xFFFFFFFF, int(layer) & 0xFFFFFFFF,
                                      int(step) & 0xFFFFFFFF, int(entry_base), out.numel(),
                                      int(dither_block), _ptr(out), _stream(stream, out)))


def replay(h0, a, w, err, *, rule: str, fmt: str, ref=None, codes=None, scale=None, h_final=None,
           block_steps=None, dither_block=16, scale_group=0, seed=0, layer=0, step=0,
           entry_base=0, stream=None) -> None:
    """ssmq_replay: open-loop replay of decays a and writes w [T, n] from h0 [n]; err
    (and ref) [ceil(T / block_steps), n] float64 are written, and the final codes,
    scales and reference state when given."""
    n = h0.numel()
    steps = a.shape[0] if a.dim() == 2 else (0 if a.numel() == 0 else a.numel() // max(n, 1))
    if a.numel() != steps * n or w.numel() != steps * n:
        raise ValueError("a and w must be [steps, n]")
    bs = int(block_steps or max(steps, 1))
    if err.dtype != torch.float64 or err.numel() != ((steps + bs - 1) // bs) * n:
        raise ValueError("err must be float64 [ceil(steps / block_steps), n]")
    if ref is not None and (ref.dtype != torch.float64 or ref.numel() != err.numel()):
        raise ValueError("ref must be shaped as err")
    if codes is not None and (codes.numel() * ENTRIES_PER_CODE[fmt] != n
                              or codes.element_size() != CODE_BYTES[fmt]):
        raise ValueError("codes must hold n entries of the format")
    q = qparams(rule, fmt, dither_block=dither_block, scale_group=scale_group, seed=seed,
                layer=layer, step=step, entry_base=entry_base)
    _check(library().ssmq_replay(ctypes.byref(q), n, steps, bs, _ptr(h0), _ptr(a), _ptr(w),
                                 _ptr(err), _ptr(ref), _ptr(codes), _ptr(scale), _ptr(h_final),
                                 _stream(stream, h0)))
