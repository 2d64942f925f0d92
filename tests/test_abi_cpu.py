"""CPU tests of libattn.so: exports, host-side validation, device description.

No compute call reaches a GPU here: every call below is rejected on the host
before any HIP work, or runs on a machine without a device.
"""
import ctypes
import math
import os
import re
import subprocess

import pytest
import torch

import paper_2609_29219_amd as pa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "attn.h")
HAS_GPU = torch.cuda.is_available()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(attn_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("attn_fwd", "attn_decode", "attn_set_stream", "attn_last_error",
                     "attn_get_plan"):
        assert required in names


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", pa.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (attn_\w+)", out))
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, f"declared but not exported: {missing}"
    for n in declared_functions():
        getattr(pa.lib, n)  # resolvable through ctypes
    assert set(pa.EXPORTED) == set(declared_functions())


ALIGNED = 1 << 20  # a fake, 16-byte-aligned address: never dereferenced


def fwd(q=ALIGNED, k=ALIGNED, v=ALIGNED, o=ALIGNED, B=1, H=1, Sq=4, Skv=4, d=64, scale=0.125,
        causal=0):
    return pa.lib.attn_fwd(q, k, v, o, B, H, Sq, Skv, d, scale, causal)


def dec(q=ALIGNED, k=ALIGNED, v=ALIGNED, o=ALIGNED, B=1, H=1, Skv=4, d=64, n=0):
    return pa.lib.attn_decode(q, k, v, o, B, H, Skv, d, n)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), pa.ATTN_EINVAL),
    (dict(o=None), pa.ATTN_EINVAL),
    (dict(k=ALIGNED + 2), pa.ATTN_EINVAL),
    (dict(B=0), pa.ATTN_EINVAL),
    (dict(H=-1), pa.ATTN_EINVAL),
    (dict(Sq=0), pa.ATTN_EINVAL),
    (dict(Skv=0), pa.ATTN_EINVAL),
    (dict(d=96), pa.ATTN_EUNSUPPORTED),
    (dict(d=256), pa.ATTN_EUNSUPPORTED),
    (dict(causal=1, Sq=5, Skv=4), pa.ATTN_EUNSUPPORTED),
    (dict(Skv=0x7FFFFFFF // 256 + 1, d=128), pa.ATTN_EUNSUPPORTED),  # one head's K: 2 GiB
    (dict(scale=float("nan")), pa.ATTN_EINVAL),
    (dict(scale=float("inf")), pa.ATTN_EINVAL),
])
def test_fwd_rejects_on_host(kw, code):
    assert fwd(**kw) == code
    assert pa.last_error() != ""


@pytest.mark.parametrize("kw,code", [
    (dict(v=None), pa.ATTN_EINVAL),
    (dict(q=ALIGNED + 8), pa.ATTN_EINVAL),
    (dict(Skv=0), pa.ATTN_EINVAL),
    (dict(B=0), pa.ATTN_EINVAL),
    (dict(d=32), pa.ATTN_EUNSUPPORTED),
])
def test_decode_rejects_on_host(kw, code):
    assert dec(**kw) == code
    assert pa.last_error() != ""


def dec_noalloc(q=ALIGNED, k=ALIGNED, v=ALIGNED, o=ALIGNED, lse=None, B=1, Hq=2, Hkv=1, Skv=4,
                d=64, n=0):
    return pa.lib.attn_decode_noalloc(q, k, v, o, lse, B, Hq, Hkv, Skv, d, n)


@pytest.mark.parametrize("kw,code", [
    (dict(k=None), pa.ATTN_EINVAL),
    (dict(o=ALIGNED + 4), pa.ATTN_EINVAL),
    (dict(lse=ALIGNED + 2), pa.ATTN_EINVAL),
    (dict(Hkv=3), pa.ATTN_EINVAL),
    (dict(Skv=0), pa.ATTN_EINVAL),
    (dict(d=96), pa.ATTN_EUNSUPPORTED),
])
def test_decode_noalloc_rejects_on_host(kw, code):
    assert dec_noalloc(**kw) == code
    assert pa.last_error() != ""


def gemm(a=ALIGNED, b=ALIGNED, c=ALIGNED, M=16, N=16, K=16, flags=0):
    return pa.lib.attn_gemm(a, b, c, M, N, K, flags)


@pytest.mark.parametrize("kw,code", [
    (dict(a=None), pa.ATTN_EINVAL),
    (dict(c=ALIGNED + 4), pa.ATTN_EINVAL),
    (dict(M=0), pa.ATTN_EINVAL),
    (dict(N=-8), pa.ATTN_EINVAL),
    (dict(flags=4), pa.ATTN_EINVAL),
    (dict(K=12), pa.ATTN_EUNSUPPORTED),
    (dict(N=20), pa.ATTN_EUNSUPPORTED),
    (dict(M=1 << 20, K=1 << 10), pa.ATTN_EUNSUPPORTED),  # A is 2 GiB
])
def test_gemm_rejects_on_host(kw, code):
    assert gemm(**kw) == code
    assert pa.last_error() != ""


@pytest.mark.skipif(HAS_GPU, reason="checks the no-device path")
def test_valid_call_without_device_is_a_hip_error_not_a_fallback():
    assert fwd() == pa.ATTN_EHIP
    # the largest key range a head may have passes the host checks
    assert fwd(Skv=0x7FFFFFFF // 256, d=128) == pa.ATTN_EHIP
    assert "device" in pa.last_error().lower() or "hip" in pa.last_error().lower()
    assert dec() == pa.ATTN_EHIP
    assert dec_noalloc() == pa.ATTN_EHIP
    assert gemm() == pa.ATTN_EHIP


def test_stream_round_trip():
    assert pa.lib.attn_set_stream(ctypes.c_void_p(0x1234)) == pa.ATTN_OK
    assert pa.lib.attn_get_stream() == 0x1234
    assert pa.lib.attn_set_stream(None) == pa.ATTN_OK
    assert not pa.lib.attn_get_stream()


def test_stream_and_last_error_are_per_thread():
    # two threads set different streams and fail with different errors at the
    # same time (ctypes releases the GIL in the calls); each sees its own
    import threading
    gate = threading.Barrier(2)
    seen = {}

    def worker(idx, stream, call):
        assert pa.lib.attn_set_stream(ctypes.c_void_p(stream)) == pa.ATTN_OK
        gate.wait()
        rc = call()
        gate.wait()
        seen[idx] = (rc, pa.lib.attn_get_stream(), pa.last_error())
        pa.lib.attn_set_stream(None)

    calls = [lambda: fwd(q=None), lambda: fwd(d=96)]
    ts = [threading.Thread(target=worker, args=(i, 0x1000 * (i + 1), calls[i])) for i in range(2)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert seen[0][0] == pa.ATTN_EINVAL and seen[0][1] == 0x1000 and "null" in seen[0][2]
    assert seen[1][0] == pa.ATTN_EUNSUPPORTED and seen[1][1] == 0x2000 and "96" in seen[1][2]
    assert not pa.lib.attn_get_stream()  # this thread's stream is untouched


@pytest.mark.skipif(HAS_GPU, reason="checks the no-device path")
def test_query_device_without_device_gives_spec_values():
    desc = pa.DeviceDesc()
    assert pa.lib.attn_query_device(ctypes.byref(desc)) == pa.ATTN_EHIP
    d = desc.as_dict()
    assert d["arch"] == "gfx950" and d["num_cus"] == 256 and d["num_xcds"] == 8
    assert d["lds_bytes_per_cu"] == 160 * 1024 and d["clock_ghz"] == pytest.approx(2.4)
    assert d["mfma_bf16_flops_per_clk_cu"] > 0 and d["hbm_bytes_per_s"] > 0


def test_null_descriptor_rejected():
    assert pa.lib.attn_query_device(None) == pa.ATTN_EINVAL
    assert pa.lib.attn_measure_device(None) == pa.ATTN_EINVAL


def test_workspace_growth_cannot_release_a_buffer_before_its_users_are_enqueued():
    # Host-only check of the library's workspace locking (no device): eight
    # threads share simulated streams and grow the workspace on most calls;
    # replaying each stream in order, no job may run after the release of the
    # buffer it was given.  The same replay with the entry lock dropped
    # before enqueueing (the order the library avoids) finds such jobs, so
    # the check can see the race it guards against.
    f = pa.lib.attn__workspace_selftest
    f.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
    f.restype = ctypes.c_int
    for _ in range(5):
        assert f(8, 200, 1) == 0
    assert any(f(8, 200, 0) > 0 for _ in range(20))
