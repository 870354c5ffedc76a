"""The C ABI library on the CPU: it loads, exports what include/ssmq.h declares,
and rejects bad arguments on the host before any HIP call (no GPU needed;
only calls that must fail validation, or are empty, are made here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ssmq.h")

EINVAL, EUNSUPPORTED, EALIGN = 1, 2, 3
FAKE = 0x10000  # a 16-byte aligned, never dereferenced address


@pytest.fixture(scope="module")
def lib():
    from paper_2609_39185_amd import _binding
    if not os.path.exists(_binding.LIBRARY):
        pytest.skip("libssmq.so has not been built")
    return _binding


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\S.*?\b(ssmq_\w+)\s*\(", text, flags=re.M)))


def test_exports_every_declared_function(lib):
    names = declared_functions()
    assert set(names) == set(lib.EXPORTS)
    L = lib.library()
    for name in names:
        assert hasattr(L, name), name


def test_conv1d_and_options_validation(lib):
    L = lib.library()
    c = L.ssmq_conv1d_update
    assert c(1, 0, 4, FAKE, FAKE, FAKE, None, 1, FAKE, None) == EINVAL       # no channels
    assert c(1, 8, 65, FAKE, FAKE, FAKE, None, 1, FAKE, None) == EINVAL      # width
    assert c(1, 8, 4, FAKE, FAKE, FAKE, None, 2, FAKE, None) == EINVAL       # act
    assert c(1, 8, 4, None, FAKE, FAKE, None, 1, FAKE, None) == EINVAL       # null state
    assert c(1, 8, 4, FAKE + 2, FAKE, FAKE, None, 1, FAKE, None) == EALIGN
    assert c(0, 8, 4, None, None, None, None, 1, None, None) == 0            # empty batch
    dims = lib.Dims(1, 4, 64, 128, 2, 0)
    q = lib.qparams("weyl", "bf16")
    for opts, want in ((lib.StepOpts(None, 2, 0, None), EINVAL), (lib.StepOpts(None, 1, 1, None), EINVAL),
                       (lib.StepOpts(FAKE + 2, 1, 0, None), EALIGN)):
        assert L.ssmq_state_update_ex(ctypes.byref(dims), ctypes.byref(q), ctypes.byref(opts),
                                      FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE,
                                      None) == want


def test_status_strings(lib):
    L = lib.library()
    assert L.ssmq_status_string(0) == b"ok"
    assert L.ssmq_status_string(99) == b"unknown status"


def _update(lib, dims, q, **ptrs):
    p = dict(state=FAKE, scale=None, x=FAKE, dt=FAKE, A=FAKE, B=FAKE, C=FAKE, D=None, y=FAKE)
    p.update(ptrs)
    L = lib.library()
    return L.ssmq_state_update(None if dims is None else ctypes.byref(dims),
                               None if q is None else ctypes.byref(q), p["state"], p["scale"],
                               p["x"], p["dt"], p["A"], p["B"], p["C"], p["D"], p["y"], None)


def test_state_update_validation(lib):
    D, Q = lib.Dims, lib.qparams
    good = D(1, 4, 64, 128, 2, 0)
    L = lib.library()
    assert _update(lib, None, Q("weyl", "bf16")) == EINVAL
    assert _update(lib, good, None) == EINVAL
    q = Q("weyl", "bf16"); q.rule = 7
    assert _update(lib, good, q) == EINVAL
    q = Q("weyl", "bf16"); q.format = 9
    assert _update(lib, good, q) == EINVAL
    q = Q("weyl", "bf16"); q.flags = 2
    assert _update(lib, good, q) == EINVAL                            # unknown flag
    q = Q("weyl", "fp32", flags=lib.FLAG_FP32_STATE)
    assert _update(lib, good, q) == EINVAL                            # fp32 onto fp32
    q = Q("weyl", "int8", flags=lib.FLAG_FP32_STATE)                   # whole-head groups
    assert _update(lib, good, q) == EUNSUPPORTED
    assert _update(lib, good, Q("philox", "int8")) == EINVAL           # INT8 needs its scale
    assert _update(lib, good, Q("weyl", "bf16", dither_block=24)) == EINVAL
    assert _update(lib, good, Q("weyl", "bf16", entry_base=8)) == EINVAL
    assert _update(lib, D(1, 4, 64, 128, 3, 0), Q("weyl", "bf16")) == EINVAL
    assert b"ngroups" in L.ssmq_last_error()
    assert _update(lib, D(-1, 4, 64, 128, 2, 0), Q("weyl", "bf16")) == EINVAL
    assert _update(lib, D(1, 4, 64, 128, 2, 2), Q("weyl", "bf16")) == EINVAL
    assert _update(lib, good, Q("weyl", "bf16"), x=None) == EINVAL
    assert _update(lib, good, Q("weyl", "e4m3")) == EINVAL            # no scale
    assert _update(lib, good, Q("weyl", "bf16"), state=FAKE + 8) == EALIGN
    assert _update(lib, good, Q("weyl", "bf16"), B=FAKE + 4) == EALIGN
    assert _update(lib, good, Q("weyl", "bf16"), x=FAKE + 2) == EALIGN
    assert _update(lib, D(1, 4, 64, 24, 2, 0), Q("weyl", "bf16")) == EUNSUPPORTED
    assert _update(lib, D(1, 4, 64, 1024, 2, 0), Q("weyl", "bf16")) == EUNSUPPORTED
    assert _update(lib, good, Q("weyl", "e4m3", scale_group=48), scale=FAKE) == EINVAL
    assert _update(lib, good, Q("weyl", "e4m3", scale_group=2048), scale=FAKE) == EUNSUPPORTED
    # an empty batch is a valid no-op that never reaches the device; its scalar
    # arguments are still checked, its pointers are not read and may be NULL
    assert _update(lib, D(0, 4, 64, 128, 2, 0), Q("weyl", "bf16")) == 0
    assert L.ssmq_last_error() == b""
    nulls = dict(state=None, x=None, dt=None, A=None, B=None, C=None, y=None)
    assert _update(lib, D(0, 4, 64, 128, 2, 0), Q("weyl", "e4m3"), **nulls) == 0
    assert _update(lib, D(0, 4, 64, 128, 3, 0), Q("weyl", "bf16"), **nulls) == EINVAL
    assert _update(lib, D(0, 4, 64, 128, 2, 0), Q("weyl", "e4m3", scale_group=48), **nulls) == EINVAL


def test_requantize_validation(lib):
    L = lib.library()
    Q = lib.qparams
    assert L.ssmq_requantize(None, 16, 0, FAKE, FAKE, None, None) == EINVAL
    assert L.ssmq_requantize(ctypes.byref(Q("sr", "bf16")), -1, 0, FAKE, FAKE, None, None) == EINVAL
    assert L.ssmq_requantize(ctypes.byref(Q("sr", "bf16")), 0, 0, None, None, None, None) == 0
    assert L.ssmq_requantize(ctypes.byref(Q("sr", "bf16")), 16, 0, FAKE + 4, FAKE, None, None) == EALIGN
    assert L.ssmq_requantize(ctypes.byref(Q("sr", "e4m3")), 32, 0, FAKE, FAKE, FAKE, None) == EINVAL
    assert L.ssmq_requantize(ctypes.byref(Q("sr", "e4m3", scale_group=16)), 40, 0, FAKE, FAKE,
                             FAKE, None) == EINVAL
    assert L.ssmq_requantize(ctypes.byref(Q("sr", "e4m3", scale_group=16)), 32, 0, FAKE, FAKE,
                             None, None) == EINVAL


def test_dither_fill_validation(lib):
    L = lib.library()
    assert L.ssmq_dither_fill(5, 0, 0, 0, 0, 16, 16, FAKE, None) == EINVAL
    assert L.ssmq_dither_fill(2, 0, 0, 0, 0, -1, 16, FAKE, None) == EINVAL
    assert L.ssmq_dither_fill(2, 0, 0, 0, 0, 16, 3, FAKE, None) == EINVAL
    assert L.ssmq_dither_fill(2, 0, 0, 0, 0, 16, 16, None, None) == EINVAL
    assert L.ssmq_dither_fill(2, 0, 0, 0, 0, 16, 16, FAKE + 2, None) == EALIGN
    assert L.ssmq_dither_fill(2, 0, 0, 0, 0, 0, 16, None, None) == 0


def test_replay_validation(lib):
    L = lib.library()
    Q = lib.qparams

    def rp(q, n=64, steps=8, bs=4, h0=FAKE, a=FAKE, w=FAKE, err=FAKE, ref=None, codes=None,
           scale=None, hf=None):
        return L.ssmq_replay(ctypes.byref(q) if q is not None else None, n, steps, bs, h0, a, w,
                             err, ref, codes, scale, hf, None)

    assert rp(None) == EINVAL
    assert rp(Q("weyl", "bf16"), n=-4) == EINVAL
    assert rp(Q("weyl", "bf16"), n=6) == EINVAL                    # not a multiple of 4
    assert rp(Q("weyl", "bf16"), steps=-1) == EINVAL
    assert rp(Q("weyl", "bf16"), bs=0) == EINVAL
    assert rp(Q("weyl", "bf16", flags=1)) == EINVAL                # no checkpoint flag here
    assert rp(Q("weyl", "bf16", entry_base=8)) == EINVAL           # a multiple of 16
    assert rp(Q("weyl", "int8", scale_group=0)) == EUNSUPPORTED    # no per-head groups
    assert rp(Q("weyl", "int8", scale_group=512)) == EUNSUPPORTED
    assert rp(Q("weyl", "e4m3", scale_group=24)) == EUNSUPPORTED
    assert rp(Q("weyl", "int4", scale_group=16), n=40) == EINVAL   # n not a multiple of the group
    assert rp(Q("weyl", "bf16"), a=None) == EINVAL
    assert rp(Q("weyl", "bf16"), err=None) == EINVAL
    assert rp(Q("weyl", "bf16"), h0=FAKE + 4) == EALIGN
    assert rp(Q("weyl", "bf16"), ref=FAKE + 8) == EALIGN
    # empty traces never reach the device
    assert rp(Q("weyl", "bf16"), n=0, h0=None, a=None, w=None, err=None) == 0
    assert L.ssmq_last_error() == b""


@pytest.mark.parametrize("lang,compiler,std", [("c", "gcc", "-std=c11"), ("c++", "g++", "-std=c++17")])
def test_header_is_self_contained(tmp_path, lang, compiler, std):
    """include/ssmq.h compiles on its own, as C and as C++, pedantic and warning-free."""
    import shutil
    import subprocess
    if shutil.which(compiler) is None:
        pytest.skip(f"{compiler} not available")
    src = tmp_path / "use.c"
    src.write_text('#include "ssmq.h"\nint main(void) { return ssmq_status_string(SSMQ_OK) == 0; }\n')
    r = subprocess.run([compiler, "-x", lang, std, "-Wall", "-Wextra", "-pedantic", "-Werror",
                        "-fsyntax-only", "-I", os.path.dirname(HEADER), str(src)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_last_error_is_per_thread(lib):
    """Threads that fail with different arguments each read their own message."""
    import threading

    L = lib.library()
    errors = []

    def worker(bad_n, rounds=2000):
        for _ in range(rounds):
            st = L.ssmq_dither_fill(2, 0, 0, 0, 0, bad_n, 16, FAKE, None)
            msg = L.ssmq_last_error()
            if st != EINVAL or msg != b"n < 0":
                errors.append((bad_n, st, msg))
                return

    def worker_block(rounds=2000):
        for _ in range(rounds):
            st = L.ssmq_dither_fill(2, 0, 0, 0, 0, 16, 3, FAKE, None)
            if st != EINVAL or b"dither_block" not in L.ssmq_last_error():
                errors.append(("block", st, L.ssmq_last_error()))
                return

    threads = [threading.Thread(target=worker, args=(-1,)), threading.Thread(target=worker_block),
               threading.Thread(target=worker, args=(-5,)), threading.Thread(target=worker_block)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert errors == []
