"""CPU oracle for the quantized selective-state update (test infrastructure).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. It is a plain, slow statement of what the
GPU library computes (see ``ssmq_oracle.c`` for the definitions and the
floating-point order) and shares no code with it.

Formats: "fp16", "bf16", "e4m3" (OCP E4M3FN with an fp32 group scale), "fp32"
(unrounded), "int8" and "int4" (symmetric integers with an fp32 block scale; INT4
packs two entries per byte, the even entry in the low nibble). Rules: "rtn",
"sr" (hash), "weyl", "philox" (SR from Philox4x32-10).

Parity status: every function here is pinned by tests under ``tests/`` that use
what the paper and the mathematics fix (worked values, closed forms, exact
rational evaluation, library casts). The device ``exp`` and the quality of the
stochastic-rounding stream beyond its moments are not pinned.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build_oracle

FORMATS = {"fp16": 0, "bf16": 1, "e4m3": 2, "fp32": 3, "int8": 4, "int4": 5}
RULES = {"rtn": 0, "sr": 1, "weyl": 2, "philox": 3}
CODE_DTYPE = {"fp16": np.uint16, "bf16": np.uint16, "e4m3": np.uint8, "fp32": np.uint32,
              "int8": np.uint8, "int4": np.uint8}
SCALED = ("e4m3", "int8", "int4")
QMAX = {"e4m3": 448.0, "int8": 127.0, "int4": 7.0}


def entries_per_code_word(fmt: str) -> int:
    """Entries stored per element of the code array (2 for packed INT4)."""
    return 2 if fmt == "int4" else 1


def entry_codes(fmt: str, codes) -> np.ndarray:
    """One code per entry: INT4 bytes are split into their two nibbles (even entry
    in the low nibble); other formats are returned as they are."""
    c = np.asarray(codes)
    if fmt != "int4":
        return c
    b = c.astype(np.uint8).reshape(-1)
    out = np.empty(b.size * 2, np.uint8)
    out[0::2] = b & 0xF
    out[1::2] = b >> 4
    return out

_lib = None

_u32 = ctypes.c_uint32
_u64 = ctypes.c_uint64
_i64 = ctypes.c_int64
_int = ctypes.c_int
_vp = ctypes.c_void_p


def lib() -> ctypes.CDLL:
    """Load the oracle library, building it first only if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(build_oracle.LIBRARY):
        build_oracle.build()
    _lib = load_library(build_oracle.LIBRARY)
    return _lib


class using_library:
    """Context manager: route this module's functions through another build of the
    oracle (the mutation tests load copies with a planted mistake)."""

    def __init__(self, path: str):
        self.path = path

    def __enter__(self):
        global _lib
        self.saved = _lib
        _lib = load_library(self.path)
        return _lib

    def __exit__(self, *exc):
        global _lib
        _lib = self.saved
        return False


def load_library(path: str) -> ctypes.CDLL:
    """Open an oracle library at `path` and declare its functions' signatures."""
    L = ctypes.CDLL(path)
    L.orc_weyl_constants.argtypes = [ctypes.POINTER(_u32)]
    L.orc_weyl_constants.restype = None
    L.orc_fmix32.argtypes = [_u32]
    L.orc_fmix32.restype = _u32
    L.orc_philox4x32_10.argtypes = [_vp, _vp, _vp]
    L.orc_philox4x32_10.restype = None
    L.orc_grid.argtypes = [_int, _vp, _vp, _int]
    L.orc_grid.restype = _int
    L.orc_decode.argtypes = [_int, _u32]
    L.orc_decode.restype = ctypes.c_double
    L.orc_code_rank.argtypes = [_int, _u32]
    L.orc_code_rank.restype = _int
    L.orc_round.argtypes = [_int, _int, ctypes.c_float, _u32]
    L.orc_round.restype = _u32
    L.orc_round_array.argtypes = [_int, _int, _i64, _vp, _vp, _vp]
    L.orc_round_array.restype = None
    L.orc_threshold.argtypes = [_int, _u32, _u32, _u32, _u64, _u64]
    L.orc_threshold.restype = _u32
    L.orc_dither_fill.argtypes = [_int, _u32, _u32, _u32, _u64, _i64, _u64, _vp]
    L.orc_dither_fill.restype = None
    L.orc_requantize.argtypes = [_int, _int, _u32, _u32, _u32, _u64, _u64, _i64, _i64, _vp, _vp,
                                 _vp]
    L.orc_requantize.restype = _int
    L.orc_state_update.argtypes = [_int, _int, _u32, _u32, _u32, _u64, _u64, _i64, _i64, _i64,
                                   _i64, _i64, _i64, _int, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                   _vp, _vp]
    L.orc_state_update.restype = _int
    L.orc_state_update_fp32_grid.argtypes = [_int, _int, _u32, _u32, _u32, _u64, _u64, _i64, _i64,
                                             _i64, _i64, _i64, _i64, _int, _vp, _vp, _vp, _vp,
                                             _vp, _vp, _vp, _vp, _vp]
    L.orc_state_update_fp32_grid.restype = _int
    L.orc_state_update_ex.argtypes = [_int, _int, _u32, _u32, _u32, _u64, _u64, _i64, _i64, _i64,
                                      _i64, _i64, _i64, _int, _vp, _vp, _vp, _vp, _vp, _int, _vp,
                                      _vp, _vp, _vp, _vp, _vp, _vp]
    L.orc_state_update_ex.restype = _int
    L.orc_conv1d_update.argtypes = [_i64, _i64, _i64, _vp, _vp, _vp, _vp, _int, _vp]
    L.orc_conv1d_update.restype = _int
    L.orc_replay.argtypes = [_int, _int, _u32, _u32, _u32, _u64, _u64, _i64, _i64, _i64, _i64,
                             _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
    L.orc_replay.restype = _int
    return L


def _ptr(a):
    return None if a is None else a.ctypes.data_as(_vp)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def weyl_constants() -> dict:
    """The integer constants of the Weyl accumulator (A, B, L, S, Phi)."""
    out = (_u32 * 5)()
    lib().orc_weyl_constants(out)
    return dict(zip(("A", "B", "L", "S", "PHI"), [int(v) for v in out]))


def fmix32(h: int) -> int:
    return int(lib().orc_fmix32(h & 0xFFFFFFFF))


def philox4x32_10(ctr, key):
    """One block of Philox4x32-10: four 32-bit words for a counter and a key."""
    c = np.array(ctr, np.uint32)
    k = np.array(key, np.uint32)
    out = np.zeros(4, np.uint32)
    lib().orc_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return [int(v) for v in out]


def grid(fmt: str):
    """Sorted finite value set of a format and the code of each value."""
    f = FORMATS[fmt]
    n = lib().orc_grid(f, None, None, 0)
    vals = np.empty(n, np.float64)
    codes = np.empty(n, np.uint32)
    lib().orc_grid(f, _ptr(vals), _ptr(codes), n)
    return vals, codes


def decode(fmt: str, codes) -> np.ndarray:
    """Value of each code (no scale) as float64."""
    f = FORMATS[fmt]
    c = np.asarray(codes).astype(np.uint32).ravel()
    return np.array([lib().orc_decode(f, int(v)) for v in c], np.float64).reshape(np.shape(codes))


def code_rank(fmt: str, codes) -> np.ndarray:
    """Position of each code in value order (both zeros share one position)."""
    f = FORMATS[fmt]
    c = np.asarray(codes).astype(np.uint32).ravel()
    return np.array([lib().orc_code_rank(f, int(v)) for v in c], np.int64).reshape(np.shape(codes))


def round_values(fmt: str, rule: str, x, U24=None) -> np.ndarray:
    """Round fp32 values with given 24-bit thresholds; returns codes (uint32)."""
    x = _c(x, np.float32).ravel()
    U = None if U24 is None else _c(U24, np.uint32).ravel()
    out = np.empty(x.size, np.uint32)
    lib().orc_round_array(FORMATS[fmt], RULES[rule], x.size, _ptr(x), _ptr(U), _ptr(out))
    return out


def thresholds(rule: str, seed: int, layer: int, step: int, entry_base: int, n: int,
               block: int) -> np.ndarray:
    """The 24-bit threshold of entries entry_base .. entry_base + n - 1."""
    out = np.empty(n, np.uint32)
    lib().orc_dither_fill(RULES[rule], seed & 0xFFFFFFFF, layer & 0xFFFFFFFF, step & 0xFFFFFFFF,
                          entry_base, n, block, _ptr(out))
    return out


def requantize(fmt: str, rule: str, h, *, seed=0, layer=0, step=0, entry_base=0, block=16,
               group=0):
    """Codes (and E4M3 group scales) for fp32 values h."""
    h = _c(h, np.float32).ravel()
    per = entries_per_code_word(fmt)
    codes = np.zeros((h.size + per - 1) // per, CODE_DTYPE[fmt])
    scale = None
    if fmt in SCALED:
        if group <= 0:
            raise ValueError(f"{fmt} needs a positive group")
        scale = np.zeros(h.size // group, np.float32)
    rc = lib().orc_requantize(FORMATS[fmt], RULES[rule], seed & 0xFFFFFFFF, layer & 0xFFFFFFFF,
                              step & 0xFFFFFFFF, entry_base, block, h.size, group, _ptr(h),
                              _ptr(codes), _ptr(scale))
    if rc != 0:
        raise ValueError("oracle requantize rejected its arguments")
    return codes, scale


def state_update(fmt: str, rule: str, state, scale, x, dt, A, B, C, D, *, seed=0, layer=0,
                 step=0, entry_base=0, block=16, group=0, a_per_state=None, dt_bias=None,
                 dt_softplus=False, z=None):
    """One fused step. state has shape [batch, nheads, headdim, dstate] (codes).
    dt_bias / dt_softplus / z: the decode-step operations around the update
    (dt' = softplus(dt + dt_bias), y' = y * silu(z)).

    Returns (new_state, new_scale, y (float64), h_new (fp32 pre-rounding)).
    """
    state = np.array(state, dtype=CODE_DTYPE[fmt], copy=True, order="C")
    batch, nheads, headdim, dstate = state.shape
    dstate *= entries_per_code_word(fmt)
    B = _c(B, np.float32)
    ngroups = B.shape[1]
    A = _c(A, np.float32)
    if a_per_state is None:
        a_per_state = 1 if A.ndim == 2 else 0
    sc = None
    if fmt in SCALED:
        sc = np.array(scale, dtype=np.float32, copy=True).ravel()
    x = _c(x, np.float32)
    dt = _c(dt, np.float32)
    C = _c(C, np.float32)
    D = None if D is None else _c(D, np.float32)
    y = np.zeros((batch, nheads, headdim), np.float64)
    hnew = np.zeros((batch, nheads, headdim, dstate), np.float32)
    bias = None if dt_bias is None else _c(dt_bias, np.float32)
    zz = None if z is None else _c(z, np.float32)
    rc = lib().orc_state_update_ex(FORMATS[fmt], RULES[rule], seed & 0xFFFFFFFF,
                                   layer & 0xFFFFFFFF, step & 0xFFFFFFFF, entry_base, block, group,
                                   batch, nheads, headdim, dstate, ngroups, a_per_state,
                                   _ptr(state), _ptr(sc), _ptr(x), _ptr(dt), _ptr(bias),
                                   1 if dt_softplus else 0, _ptr(zz), _ptr(A), _ptr(B), _ptr(C),
                                   _ptr(D), _ptr(y), _ptr(hnew))
    if rc != 0:
        raise ValueError("oracle state_update rejected its arguments")
    return state, sc, y, hnew


def state_update_fp32_grid(fmt: str, rule: str, state, x, dt, A, B, C, D, *, seed=0, layer=0,
                           step=0, entry_base=0, block=16, group=0, a_per_state=None):
    """A checkpoint write on an fp32 state: one fp32 step, then every value rounded
    onto fmt's grid and stored as fp32. Returns (new fp32 state, group scales or
    None, y (float64))."""
    st = np.array(state, dtype=np.float32, copy=True, order="C")
    batch, nheads, headdim, dstate = st.shape
    B = _c(B, np.float32)
    A = _c(A, np.float32)
    if a_per_state is None:
        a_per_state = 1 if A.ndim == 2 else 0
    g = group if group else headdim * dstate
    sc = np.zeros(st.size // g, np.float32) if fmt in SCALED else None
    y = np.zeros((batch, nheads, headdim), np.float64)
    rc = lib().orc_state_update_fp32_grid(
        FORMATS[fmt], RULES[rule], seed & 0xFFFFFFFF, layer & 0xFFFFFFFF, step & 0xFFFFFFFF,
        entry_base, block, group, batch, nheads, headdim, dstate, B.shape[1], a_per_state,
        _ptr(st), _ptr(sc), _ptr(_c(x, np.float32)), _ptr(_c(dt, np.float32)), _ptr(A), _ptr(B),
        _ptr(_c(C, np.float32)), _ptr(None if D is None else _c(D, np.float32)), _ptr(y))
    if rc != 0:
        raise ValueError("oracle state_update_fp32_grid rejected its arguments")
    return st, sc, y


def conv1d_update(state, x, weight, bias=None, act=True):
    """Causal depthwise conv1d decode update: state [batch, channels, width] shifts
    and takes x [batch, channels]; returns (new state, out (float64))."""
    st = np.array(state, dtype=np.float32, copy=True, order="C")
    batch, channels, width = st.shape
    out = np.zeros((batch, channels), np.float64)
    rc = lib().orc_conv1d_update(batch, channels, width, _ptr(st), _ptr(_c(x, np.float32)),
                                 _ptr(_c(weight, np.float32)),
                                 _ptr(None if bias is None else _c(bias, np.float32)),
                                 1 if act else 0, _ptr(out))
    if rc != 0:
        raise ValueError("oracle conv1d_update rejected its arguments")
    return st, out


def dequantize(fmt: str, codes, scale=None, group=0) -> np.ndarray:
    """fp32 values of stored codes, one per entry (E4M3, INT8, INT4: times the group
    scale, one fp32 product). Shape: the codes' shape, INT4's last axis doubled."""
    codes = np.asarray(codes)
    if fmt == "fp32":
        return codes.astype(np.uint32).view(np.float32).astype(np.float32)
    shape = codes.shape
    if fmt == "int4":
        shape = shape[:-1] + (2 * shape[-1],) if len(shape) else (2,)
    v = decode(fmt, entry_codes(fmt, codes)).astype(np.float32).ravel()
    if fmt in SCALED:
        s = np.repeat(np.asarray(scale, np.float32).ravel(), group)
        v = (v * s).astype(np.float32)
    return v.reshape(shape)


def replay(fmt: str, rule: str, h0, a, w, *, seed=0, layer=0, step=0, entry_base=0, block=16,
           group=0, block_steps=None):
    """Open-loop replay of traces a, w [T, n] from the FP32 state h0 [n] (Appendix B
    "Open-loop replay"). Returns a dict: err and ref [n_blocks, n] (float64 sums of
    (hq_t - h_t)^2 and h_t^2 per block of block_steps steps), codes and scale of the
    final stored state, and h_final (the final FP32 reference state)."""
    h0 = _c(h0, np.float32).ravel()
    n = h0.size
    a = _c(a, np.float32).reshape(-1, n)
    w = _c(w, np.float32).reshape(-1, n)
    steps = a.shape[0]
    if w.shape[0] != steps:
        raise ValueError("a and w must hold the same number of steps")
    bs = block_steps or max(steps, 1)
    n_blocks = (steps + bs - 1) // bs
    err = np.zeros((n_blocks, n), np.float64)
    ref = np.zeros((n_blocks, n), np.float64)
    per = entries_per_code_word(fmt)
    codes = np.zeros((n + per - 1) // per, CODE_DTYPE[fmt])
    scale = np.zeros(n // group, np.float32) if fmt in SCALED and group else None
    h_final = np.zeros(n, np.float32)
    rc = lib().orc_replay(FORMATS[fmt], RULES[rule], seed & 0xFFFFFFFF, layer & 0xFFFFFFFF,
                          step & 0xFFFFFFFF, entry_base, block, n, group, steps, bs, _ptr(h0),
                          _ptr(a), _ptr(w), _ptr(err), _ptr(ref), _ptr(codes), _ptr(scale),
                          _ptr(h_final))
    if rc != 0:
        raise ValueError("oracle replay rejected its arguments")
    return {"err": err, "ref": ref, "codes": codes, "scale": scale, "h_final": h_final}
