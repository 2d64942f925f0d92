"""Tiled exact attention on MI355X (gfx950): Python binding of libattn.so.

This module only marshals arguments into the C ABI declared in
``include/attn.h``; every step of the computation runs in the HIP kernels of
``libattn.so``.  PyTorch is used for device memory and the current stream.
There is no fallback: if the library is missing, importing this package
raises ImportError, and the compute calls raise AttnError without a gfx950
device.

    o = attn_fwd(q, k, v, scale=None, causal=False)  # q [B,H,Sq,d], k/v [B,H,Skv,d] bf16
    o = attn_decode(q, k, v, n_splits=0)             # q [B,H,d], k/v [B,H,Skv,d] bf16
"""
from __future__ import annotations

import ctypes
import math
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libattn.so")

ATTN_OK = 0
ATTN_EINVAL = -1
ATTN_EUNSUPPORTED = -2
ATTN_EHIP = -3
ATTN_ENOMEM = -4
KIND_FWD = 0
KIND_DECODE = 1
ATTN_OUT_BF16 = 1
ATTN_GEMM_B_NK = 2

# Entry points declared in include/attn.h.
EXPORTED = ("attn_fwd", "attn_decode", "attn_fwd_ex", "attn_decode_ex",
            "attn_decode_workspace_bytes", "attn_set_stream", "attn_get_stream",
            "attn_last_error", "attn_query_device", "attn_measure_device", "attn_get_plan",
            "attn_get_plan_for", "attn_gemm", "attn_gemm_plan", "attn_decode_noalloc")
NOALLOC_SCRATCH_BYTES = 16 << 20  # ATTN_NOALLOC_SCRATCH_BYTES


class AttnError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"attn error {code}: {msg}")
        self.code = code


class DeviceDesc(ctypes.Structure):
    _fields_ = [
        ("arch", ctypes.c_char * 32),
        ("num_cus", ctypes.c_int),
        ("num_xcds", ctypes.c_int),
        ("simds_per_cu", ctypes.c_int),
        ("wave_size", ctypes.c_int),
        ("lds_bytes_per_cu", ctypes.c_int),
        ("vgprs_per_simd_lane", ctypes.c_int),
        ("max_waves_per_simd", ctypes.c_int),
        ("clock_ghz", ctypes.c_double),
        ("mfma_bf16_flops_per_clk_cu", ctypes.c_double),
        ("valu_lanes_per_clk_simd", ctypes.c_double),
        ("trans_cycles_per_op", ctypes.c_double),
        ("lds_bytes_per_clk_cu", ctypes.c_double),
        ("l2_bytes_per_clk_xcd", ctypes.c_double),
        ("hbm_bytes_per_s", ctypes.c_double),
        ("hbm_latency_us", ctypes.c_double),
        ("launch_us", ctypes.c_double),
        ("issue_cycles_per_score", ctypes.c_double),
        ("valu_mfma_overlap", ctypes.c_double),
        ("tile_sync_cycles", ctypes.c_double),
        ("tile_latency_cycles", ctypes.c_double),
    ]

    def as_dict(self) -> dict:
        d = {name: getattr(self, name) for name, _ in self._fields_}
        d["arch"] = self.arch.decode()
        return d


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python paper_2609_29219_amd/build.py` "
            "(or __graft_entry__.build())")
    # One HIP runtime per process: torch ships its own libamdhip64, and the
    # library must bind to that one (loaded first, it satisfies the library's
    # dependency), not load the system copy beside it.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    vp, ci, cf = ctypes.c_void_p, ctypes.c_int, ctypes.c_float
    lib.attn_fwd.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci, cf, ci]
    lib.attn_decode.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci]
    lib.attn_fwd_ex.argtypes = [vp, vp, vp, vp, vp, ci, ci, ci, ci, ci, ci, cf, ci, ci]
    lib.attn_decode_ex.argtypes = [vp, vp, vp, vp, vp, ci, ci, ci, ci, ci, ci, vp,
                                   ctypes.c_size_t]
    lib.attn_decode_noalloc.argtypes = [vp, vp, vp, vp, vp, ci, ci, ci, ci, ci, ci]
    lib.attn_decode_workspace_bytes.argtypes = [ci, ci, ci, ci, ci, ci]
    lib.attn_decode_workspace_bytes.restype = ctypes.c_longlong
    lib.attn_set_stream.argtypes = [vp]
    lib.attn_get_stream.argtypes = []
    lib.attn_get_stream.restype = vp
    lib.attn_last_error.argtypes = []
    lib.attn_last_error.restype = ctypes.c_char_p
    lib.attn_query_device.argtypes = [ctypes.POINTER(DeviceDesc)]
    lib.attn_measure_device.argtypes = [ctypes.POINTER(DeviceDesc)]
    lib.attn_get_plan.argtypes = [ci, ci, ci, ci, ci, ci, ci, ci, ctypes.c_char_p, ci]
    lib.attn_get_plan_for.argtypes = [ctypes.POINTER(DeviceDesc), ci, ci, ci, ci, ci, ci, ci,
                                      ci, ctypes.c_char_p, ci]
    lib.attn__fwd_candidates.argtypes = [ctypes.POINTER(DeviceDesc), ci, ci, ci, ci, ci, ci, ci,
                                         ctypes.c_char_p, ci]
    lib.attn_gemm.argtypes = [vp, vp, vp, ci, ci, ci, ci]
    lib.attn_gemm_plan.argtypes = [ctypes.POINTER(DeviceDesc), ci, ci, ci, ci, ctypes.c_char_p,
                                   ci]
    lib.attn__gemm_candidates.argtypes = [ctypes.POINTER(DeviceDesc), ci, ci, ci, ci, ci,
                                          ctypes.c_char_p, ci]
    for fn in (lib.attn_fwd, lib.attn_decode, lib.attn_fwd_ex, lib.attn_decode_ex,
               lib.attn_decode_noalloc,
               lib.attn_set_stream, lib.attn_query_device,
               lib.attn_measure_device, lib.attn_get_plan, lib.attn_get_plan_for,
               lib.attn__fwd_candidates, lib.attn_gemm, lib.attn_gemm_plan,
               lib.attn__gemm_candidates):
        fn.restype = ci
    return lib


lib = _load()


def last_error() -> str:
    return lib.attn_last_error().decode()


def _check(rc: int):
    if rc != ATTN_OK:
        raise AttnError(rc, last_error())


def _set_stream(t) -> None:
    import torch
    lib.attn_set_stream(ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream))


def _require(t, dtype, shape, name):
    import torch
    if not isinstance(t, torch.Tensor) or t.dtype != dtype or not t.is_cuda:
        raise TypeError(f"{name} must be a {dtype} tensor on a HIP device")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def attn_fwd(q, k, v, o=None, scale: float | None = None, causal: bool = False,
             out_dtype=None, return_lse: bool = False):
    """Prefill attention; returns o [B,Hq,Sq,d] (fp32, or out_dtype bf16),
    and with return_lse also the fp32 row log-sum-exp [B,Hq,Sq].  k and v
    may have fewer heads than q (grouped-query heads: Hkv divides Hq)."""
    import torch
    B, Hq, Sq, d = q.shape
    Hkv, Skv = k.shape[1], k.shape[2]
    _require(q, torch.bfloat16, (B, Hq, Sq, d), "q")
    _require(k, torch.bfloat16, (B, Hkv, Skv, d), "k")
    _require(v, torch.bfloat16, (B, Hkv, Skv, d), "v")
    if out_dtype is None:
        out_dtype = o.dtype if o is not None else torch.float32
    if out_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out_dtype must be torch.float32 or torch.bfloat16")
    if o is None:
        o = torch.empty((B, Hq, Sq, d), dtype=out_dtype, device=q.device)
    _require(o, out_dtype, (B, Hq, Sq, d), "o")
    lse = None
    if return_lse:
        lse = torch.empty((B, Hq, Sq), dtype=torch.float32, device=q.device)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    _set_stream(q)
    flags = ATTN_OUT_BF16 if out_dtype == torch.bfloat16 else 0
    _check(lib.attn_fwd_ex(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                           lse.data_ptr() if lse is not None else None, B, Hq, Hkv, Sq, Skv, d,
                           float(scale), int(bool(causal)), flags))
    return (o, lse) if return_lse else o


def attn_decode(q, k, v, o=None, n_splits: int = 0, workspace=None, return_lse: bool = False):
    """Split-KV single-query attention; returns o fp32 [B,Hq,d], and with
    return_lse also the row log-sum-exp [B,Hq].  k and v may have fewer heads
    than q (grouped-query heads).  workspace: None (the library's), or a
    device tensor of at least decode_workspace_bytes(...) bytes."""
    import torch
    B, Hq, d = q.shape
    Hkv, Skv = k.shape[1], k.shape[2]
    _require(q, torch.bfloat16, (B, Hq, d), "q")
    _require(k, torch.bfloat16, (B, Hkv, Skv, d), "k")
    _require(v, torch.bfloat16, (B, Hkv, Skv, d), "v")
    if o is None:
        o = torch.empty((B, Hq, d), dtype=torch.float32, device=q.device)
    _require(o, torch.float32, (B, Hq, d), "o")
    lse = None
    if return_lse:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=q.device)
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        if not isinstance(workspace, torch.Tensor) or not workspace.is_cuda or \
                not workspace.is_contiguous():
            raise TypeError("workspace must be a contiguous tensor on a HIP device")
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    _set_stream(q)
    _check(lib.attn_decode_ex(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                              lse.data_ptr() if lse is not None else None, B, Hq, Hkv, Skv, d,
                              int(n_splits), ws_ptr, ws_bytes))
    return (o, lse) if return_lse else o


def attn_decode_noalloc(q, k, v, o, n_splits: int = 0, lse=None):
    """attn_decode with its split partials in the library's static device
    scratch: allocates nothing, so o (fp32 [B,Hq,d]) and the optional lse
    (fp32 [B,Hq]) must be given.  Calls that can overlap on one device race
    on the scratch."""
    import torch
    B, Hq, d = q.shape
    Hkv, Skv = k.shape[1], k.shape[2]
    _require(q, torch.bfloat16, (B, Hq, d), "q")
    _require(k, torch.bfloat16, (B, Hkv, Skv, d), "k")
    _require(v, torch.bfloat16, (B, Hkv, Skv, d), "v")
    _require(o, torch.float32, (B, Hq, d), "o")
    if lse is not None:
        _require(lse, torch.float32, (B, Hq), "lse")
    _set_stream(q)
    _check(lib.attn_decode_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                   lse.data_ptr() if lse is not None else None, B, Hq, Hkv, Skv,
                                   d, int(n_splits)))
    return o


def decode_workspace_bytes(B: int, Hq: int, Hkv: int, Skv: int, d: int, n_splits: int = 0) -> int:
    """Bytes of workspace attn_decode needs with a caller-provided buffer."""
    n = lib.attn_decode_workspace_bytes(B, Hq, Hkv, Skv, d, int(n_splits))
    if n < 0:
        raise AttnError(int(n), last_error())
    return int(n)


def gemm(a, b, c=None, b_nk: bool = False, out_dtype=None):
    """C = A B on bf16 MFMA with fp32 accumulation.  a: bf16 [M,K]; b: bf16
    [K,N], or [N,K] with b_nk; returns c [M,N] fp32 (or out_dtype bf16)."""
    import torch
    M, K = a.shape
    N = b.shape[0] if b_nk else b.shape[1]
    _require(a, torch.bfloat16, (M, K), "a")
    _require(b, torch.bfloat16, (N, K) if b_nk else (K, N), "b")
    if out_dtype is None:
        out_dtype = c.dtype if c is not None else torch.float32
    if out_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out_dtype must be torch.float32 or torch.bfloat16")
    if c is None:
        c = torch.empty((M, N), dtype=out_dtype, device=a.device)
    _require(c, out_dtype, (M, N), "c")
    flags = (ATTN_OUT_BF16 if out_dtype == torch.bfloat16 else 0) | \
        (ATTN_GEMM_B_NK if b_nk else 0)
    _set_stream(a)
    _check(lib.attn_gemm(a.data_ptr(), b.data_ptr(), c.data_ptr(), M, N, K, flags))
    return c


def gemm_plan(M: int, N: int, K: int, b_nk: bool = False, desc: DeviceDesc | None = None) -> str:
    buf = ctypes.create_string_buffer(512)
    ptr = ctypes.byref(desc) if desc is not None else None
    rc = lib.attn_gemm_plan(ptr, M, N, K, ATTN_GEMM_B_NK if b_nk else 0, buf, 512)
    if rc < 0:
        raise AttnError(rc, last_error())
    return buf.value.decode()


def gemm_candidates(M: int, N: int, K: int, b_nk: bool = False, desc: DeviceDesc | None = None,
                    device_footprint: bool = False, analytic_only: bool = False) -> list[dict]:
    """Every feasible GEMM candidate with its modelled time (not ABI; for the
    block-size ablation).  analytic_only: without the measured per-variant
    costs."""
    buf = ctypes.create_string_buffer(1 << 16)
    ptr = ctypes.byref(desc) if desc is not None else None
    flags = int(bool(device_footprint)) | (2 if analytic_only else 0)
    rc = lib.attn__gemm_candidates(ptr, M, N, K, ATTN_GEMM_B_NK if b_nk else 0, flags, buf,
                                   1 << 16)
    if rc < 0:
        raise AttnError(rc, last_error())
    return [parse_plan(l) for l in buf.value.decode().splitlines() if l.strip()]


def query_device() -> dict:
    desc = DeviceDesc()
    lib.attn_query_device(ctypes.byref(desc))
    return desc.as_dict()


def measure_device() -> dict:
    """Run the device microbenchmarks (needs a gfx950 device)."""
    desc = DeviceDesc()
    _check(lib.attn_measure_device(ctypes.byref(desc)))
    return desc.as_dict()


def get_plan(kind: int, B: int, H: int, Sq: int, Skv: int, d: int, causal: bool = False,
             n_splits: int = 0, desc: DeviceDesc | None = None) -> str:
    buf = ctypes.create_string_buffer(512)
    if desc is None:
        rc = lib.attn_get_plan(kind, B, H, Sq, Skv, d, int(bool(causal)), n_splits, buf, 512)
    else:
        rc = lib.attn_get_plan_for(ctypes.byref(desc), kind, B, H, Sq, Skv, d, int(bool(causal)),
                                   n_splits, buf, 512)
    if rc < 0:
        raise AttnError(rc, last_error())
    return buf.value.decode()


def fwd_candidates(B: int, H: int, Sq: int, Skv: int, d: int, causal: bool = False,
                   desc: DeviceDesc | None = None, device_footprint: bool = False,
                   analytic_only: bool = False) -> list[dict]:
    """Every feasible prefill candidate with its modelled time (not ABI; for
    the block-size ablation).  desc None: this device's description and the
    compiled kernels' real register/occupancy footprint; with a desc, the
    footprint is estimated unless device_footprint is set.  analytic_only:
    without the measured per-variant tile costs."""
    buf = ctypes.create_string_buffer(1 << 18)
    ptr = ctypes.byref(desc) if desc is not None else None
    flags = int(bool(device_footprint)) | (2 if analytic_only else 0)
    rc = lib.attn__fwd_candidates(ptr, B, H, Sq, Skv, d, int(bool(causal)), flags, buf, 1 << 18)
    if rc < 0:
        raise AttnError(rc, last_error())
    return [parse_plan(l) for l in buf.value.decode().splitlines() if l.strip()]


def parse_plan(line: str) -> dict:
    out = {}
    for tok in line.split():
        key, _, val = tok.partition("=")
        try:
            out[key] = int(val)
        except ValueError:
            try:
                out[key] = float(val)
            except ValueError:
                out[key] = val
    return out
