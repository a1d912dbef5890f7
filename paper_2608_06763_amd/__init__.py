"""MI355X-native CubicQuant hot path: Python binding of ``libcq.so``.

The binding only marshals arguments: every step of the hot path runs in the
HIP kernels behind the C ABI declared in ``include/cq.h``.  PyTorch provides
device memory and the current stream.  Importing this package does not need a
GPU; calling a device entry point does, and a missing library raises.

Entry points (same names as the C ABI):
  cq_pack_groups, cq_decode_ref, cq_gemm_model_dtype, cq_quantize_act_a8,
  cq_gemm_a8, cq_gemm_a8_fused, cq_build_carriers, cq_gemm_a8_carriers,
  cq_gemm_routed_model_dtype, cq_gemm_routed_model_dtype_noalloc, cq_set_gemv_max_rows, cq_get_gemv_max_rows,
  cq_set_a8_fused_launch, cq_get_a8_fused_launch,
  cq_family_supported, cq_gemm_model_dtype_family, cq_gemm_a8_family,
  cq_select_set, cq_select_query, cq_probe_read (measurement aid, include/cq_measure.h)
The measured kernel-selection tuner that fills the selection table is in
``selection.py``.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcq.so")

CQ_BF16, CQ_FP16, CQ_FP32 = 0, 1, 2
STATUS = {0: "CQ_OK", 1: "CQ_ERR_ARG", 2: "CQ_ERR_SHAPE", 3: "CQ_ERR_ALIGN", 4: "CQ_ERR_META",
          5: "CQ_ERR_CODE", 6: "CQ_ERR_DTYPE", 7: "CQ_ERR_HIP", 8: "CQ_ERR_UNSUPPORTED"}

EXPORTS = ("cq_status_str", "cq_pack_groups", "cq_decode_ref", "cq_gemm_model_dtype", "cq_quantize_act_a8",
           "cq_gemm_a8", "cq_gemm_a8_fused", "cq_build_carriers", "cq_gemm_a8_carriers",
           "cq_gemm_routed_model_dtype", "cq_set_gemv_max_rows", "cq_get_gemv_max_rows",
           "cq_family_supported", "cq_gemm_model_dtype_family", "cq_gemm_a8_family", "cq_select_set",
           "cq_select_query", "cq_probe_read", "cq_gemm_routed_model_dtype_noalloc", "cq_set_a8_fused_launch",
           "cq_get_a8_fused_launch")

CQ_PATH_MODEL_DTYPE, CQ_PATH_A8 = 0, 1
FAMILIES = {"auto": 0, "gemv_stream": 1, "gemv_lut": 2, "gemv_narrow": 3, "gemv_generic": 4, "gemm_mfma": 5,
            "gemm_tiled": 6, "gemm_mfma_rounded": 7, "gemm_mfma_m32": 8, "gemm_mfma_m64": 9, "gemm_mfma_m128": 10,
            "gemm_mfma_m256": 11, "gemm_slab": 12,
            "gemm_slab_staged": 13, "gemv_rows": 14}
FAMILY_NAMES = {v: k for k, v in FAMILIES.items()}


class CQError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)}")


class cq_weight(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_int32), ("group", ctypes.c_int32), ("n", ctypes.c_int64),
                ("k", ctypes.c_int64), ("codes", ctypes.c_void_p), ("scale", ctypes.c_void_p),
                ("a", ctypes.c_void_p), ("b", ctypes.c_void_p)]


class cq_select_entry(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int32), ("family", ctypes.c_int32), ("bits", ctypes.c_int32),
                ("group", ctypes.c_int32), ("n", ctypes.c_int64), ("k", ctypes.c_int64), ("m_lo", ctypes.c_int64),
                ("m_hi", ctypes.c_int64), ("x_dtype", ctypes.c_int32), ("reserved", ctypes.c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libcq.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_06763_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    L.cq_status_str.restype = ctypes.c_char_p
    L.cq_status_str.argtypes = [ctypes.c_int]
    L.cq_pack_groups.restype = ctypes.c_int
    L.cq_pack_groups.argtypes = [i32, i32, i64, i64, vp, vp, vp, vp, vp, vp]
    L.cq_decode_ref.restype = ctypes.c_int
    L.cq_decode_ref.argtypes = [ctypes.POINTER(cq_weight), vp, vp, vp]
    L.cq_gemm_model_dtype.restype = ctypes.c_int
    L.cq_gemm_model_dtype.argtypes = [ctypes.POINTER(cq_weight), vp, ctypes.c_int, i64, vp, ctypes.c_int, vp]
    L.cq_quantize_act_a8.restype = ctypes.c_int
    L.cq_quantize_act_a8.argtypes = [vp, ctypes.c_int, i64, i64, vp, vp, vp]
    L.cq_gemm_a8.restype = ctypes.c_int
    L.cq_gemm_a8.argtypes = [ctypes.POINTER(cq_weight), vp, vp, i64, vp, ctypes.c_int, vp, vp]
    L.cq_gemm_a8_fused.restype = ctypes.c_int
    L.cq_gemm_a8_fused.argtypes = [ctypes.POINTER(cq_weight), vp, ctypes.c_int, i64, vp, vp, vp, ctypes.c_int, vp]
    L.cq_build_carriers.restype = ctypes.c_int
    L.cq_build_carriers.argtypes = [ctypes.POINTER(cq_weight), vp, vp]
    L.cq_gemm_a8_carriers.restype = ctypes.c_int
    L.cq_gemm_a8_carriers.argtypes = [ctypes.POINTER(cq_weight), vp, vp, vp, i64, vp, ctypes.c_int, vp]
    L.cq_gemm_routed_model_dtype.restype = ctypes.c_int
    L.cq_gemm_routed_model_dtype.argtypes = [ctypes.POINTER(cq_weight), i32, vp, ctypes.c_int, i64, vp, vp, i64, vp, vp,
                                             ctypes.c_int, vp]
    L.cq_gemm_routed_model_dtype_noalloc.restype = ctypes.c_int
    L.cq_gemm_routed_model_dtype_noalloc.argtypes = [ctypes.POINTER(cq_weight), i32, vp, ctypes.c_int, i64, vp, vp, i64,
                                                     vp, ctypes.c_int, vp]
    L.cq_set_gemv_max_rows.restype = ctypes.c_int
    L.cq_set_gemv_max_rows.argtypes = [i32, i64]
    L.cq_set_a8_fused_launch.restype = ctypes.c_int
    L.cq_set_a8_fused_launch.argtypes = [i32]
    L.cq_get_a8_fused_launch.restype = i32
    L.cq_get_a8_fused_launch.argtypes = []
    L.cq_get_gemv_max_rows.restype = i64
    L.cq_get_gemv_max_rows.argtypes = [i32]
    L.cq_family_supported.restype = i32
    L.cq_family_supported.argtypes = [i32, i32, ctypes.POINTER(cq_weight), i64]
    L.cq_gemm_model_dtype_family.restype = ctypes.c_int
    L.cq_gemm_model_dtype_family.argtypes = [ctypes.POINTER(cq_weight), vp, ctypes.c_int, i64, vp, ctypes.c_int, i32,
                                             vp]
    L.cq_gemm_a8_family.restype = ctypes.c_int
    L.cq_gemm_a8_family.argtypes = [ctypes.POINTER(cq_weight), vp, vp, i64, vp, ctypes.c_int, i32, vp]
    L.cq_select_set.restype = ctypes.c_int
    L.cq_select_set.argtypes = [ctypes.POINTER(cq_select_entry), i64]
    L.cq_select_query.restype = ctypes.c_int
    L.cq_select_query.argtypes = [i32, ctypes.POINTER(cq_weight), ctypes.c_int, i64, ctypes.POINTER(i32)]
    L.cq_probe_read.restype = ctypes.c_int
    L.cq_probe_read.argtypes = [vp, i64, vp, vp]
    _lib = L
    return L


def _check(status: int, where: str):
    if status != 0:
        raise CQError(status, where)


def _np_ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# ---------------------------------------------------------------- host packer


def cq_pack_groups(codes, scale, a_bits, b_bits, bits: int, group: int) -> np.ndarray:
    """Validate and pack host arrays; returns uint8 [N, K*B/8]."""
    codes = np.ascontiguousarray(codes, dtype=np.int8)
    n, k = codes.shape
    scale = np.ascontiguousarray(scale, dtype=np.float32)
    a_bits = np.ascontiguousarray(a_bits, dtype=np.uint16)
    b_bits = np.ascontiguousarray(b_bits, dtype=np.uint16)
    out = np.zeros((n, (k * bits + 7) // 8), np.uint8)
    bad = ctypes.c_int64(-1)
    st = lib().cq_pack_groups(bits, group, n, k, _np_ptr(codes), _np_ptr(scale), _np_ptr(a_bits),
                              _np_ptr(b_bits), _np_ptr(out), ctypes.byref(bad))
    if st != 0:
        err = CQError(st, "cq_pack_groups")
        err.bad_index = bad.value
        raise err
    return out


# ---------------------------------------------------------------- device weights


def _torch():
    import torch
    return torch


def _stream_ptr(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class CQWeight:
    """Device copy of one packed matrix plus its C descriptor."""

    def __init__(self, packed, scale, a_bits, b_bits, bits: int, group: int, n: int, k: int,
                 device="cuda"):
        torch = _torch()

        def dev(arr, dtype):
            if isinstance(arr, torch.Tensor):
                return arr.to(device=device).contiguous().view(dtype)
            return torch.from_numpy(np.ascontiguousarray(arr)).to(device).view(dtype)

        self.codes = dev(packed, torch.uint8)
        self.scale = dev(scale, torch.float32)
        self.a = dev(np.asarray(a_bits, np.uint16).view(np.int16) if not isinstance(a_bits, torch.Tensor)
                     else a_bits, torch.int16)
        self.b = dev(np.asarray(b_bits, np.uint16).view(np.int16) if not isinstance(b_bits, torch.Tensor)
                     else b_bits, torch.int16)
        self.bits, self.group, self.n, self.k = int(bits), int(group), int(n), int(k)
        self.desc = cq_weight(self.bits, self.group, self.n, self.k, self.codes.data_ptr(),
                              self.scale.data_ptr(), self.a.data_ptr(), self.b.data_ptr())

    @classmethod
    def from_codes(cls, codes, scale, a_bits, b_bits, bits: int, group: int, device="cuda"):
        packed = cq_pack_groups(codes, scale, a_bits, b_bits, bits, group)
        n, k = np.asarray(codes).shape
        return cls(packed, scale, a_bits, b_bits, bits, group, n, k, device)

    def clone(self) -> "CQWeight":
        """Same bytes at new device addresses."""
        return CQWeight(self.codes.clone(), self.scale.clone(), self.a.clone(), self.b.clone(),
                        self.bits, self.group, self.n, self.k, self.codes.device)

    @property
    def nbytes(self) -> int:
        return (self.codes.numel() + self.scale.numel() * 4 + self.a.numel() * 2 + self.b.numel() * 2)


def _dt(t) -> int:
    torch = _torch()
    if t == torch.bfloat16:
        return CQ_BF16
    if t == torch.float16:
        return CQ_FP16
    if t == torch.float32:
        return CQ_FP32
    raise ValueError(f"unsupported dtype {t}")


def cq_decode_ref(w: CQWeight, want_codes=True, want_values=True, stream=None):
    torch = _torch()
    codes = torch.empty((w.n, w.k), dtype=torch.int8, device=w.codes.device) if want_codes else None
    vals = torch.empty((w.n, w.k), dtype=torch.float32, device=w.codes.device) if want_values else None
    st = lib().cq_decode_ref(ctypes.byref(w.desc), codes.data_ptr() if codes is not None else None,
                             vals.data_ptr() if vals is not None else None, _stream_ptr(stream))
    _check(st, "cq_decode_ref")
    return codes, vals


def cq_gemm_model_dtype(w: CQWeight, x, y_dtype=None, out=None, stream=None):
    """y = x W_hat^T; x is a [M, K] bf16/fp16 device tensor."""
    torch = _torch()
    assert x.dim() == 2 and x.shape[1] == w.k and x.is_contiguous()
    y_dtype = y_dtype or x.dtype
    if out is None:
        out = torch.empty((x.shape[0], w.n), dtype=y_dtype, device=x.device)
    st = lib().cq_gemm_model_dtype(ctypes.byref(w.desc), x.data_ptr(), _dt(x.dtype), x.shape[0],
                                   out.data_ptr(), _dt(out.dtype), _stream_ptr(stream))
    _check(st, "cq_gemm_model_dtype")
    return out


def cq_quantize_act_a8(x, x8=None, dx=None, stream=None):
    torch = _torch()
    assert x.dim() == 2 and x.is_contiguous()
    m, k = x.shape
    if x8 is None:
        x8 = torch.empty((m, k), dtype=torch.int8, device=x.device)
    if dx is None:
        dx = torch.empty((m,), dtype=torch.float32, device=x.device)
    st = lib().cq_quantize_act_a8(x.data_ptr(), _dt(x.dtype), m, k, x8.data_ptr(), dx.data_ptr(),
                                  _stream_ptr(stream))
    _check(st, "cq_quantize_act_a8")
    return x8, dx


def cq_gemm_a8(w: CQWeight, x8, dx, y_dtype=None, want_partials=False, out=None, stream=None):
    torch = _torch()
    assert x8.dim() == 2 and x8.shape[1] == w.k and x8.is_contiguous()
    m = x8.shape[0]
    y_dtype = y_dtype or torch.bfloat16
    if out is None:
        out = torch.empty((m, w.n), dtype=y_dtype, device=x8.device)
    parts = torch.empty((m, w.n, w.k // w.group), dtype=torch.int32, device=x8.device) if want_partials else None
    st = lib().cq_gemm_a8(ctypes.byref(w.desc), x8.data_ptr(), dx.data_ptr(), m, out.data_ptr(), _dt(out.dtype),
                          parts.data_ptr() if parts is not None else None, _stream_ptr(stream))
    _check(st, "cq_gemm_a8")
    return (out, parts) if want_partials else out


def cq_gemm_a8_fused(w: CQWeight, x, y_dtype=None, out=None, x8=None, dx=None, stream=None):
    """Dynamic-A8 product straight from model-dtype activations; returns (y, x8, dx)."""
    torch = _torch()
    assert x.dim() == 2 and x.shape[1] == w.k and x.is_contiguous()
    m = x.shape[0]
    y_dtype = y_dtype or x.dtype
    if out is None:
        out = torch.empty((m, w.n), dtype=y_dtype, device=x.device)
    if x8 is None:
        x8 = torch.empty((m, w.k), dtype=torch.int8, device=x.device)
    if dx is None:
        dx = torch.empty((m,), dtype=torch.float32, device=x.device)
    st = lib().cq_gemm_a8_fused(ctypes.byref(w.desc), x.data_ptr(), _dt(x.dtype), m, x8.data_ptr(), dx.data_ptr(),
                                out.data_ptr(), _dt(out.dtype), _stream_ptr(stream))
    _check(st, "cq_gemm_a8_fused")
    return out, x8, dx


def cq_build_carriers(w: CQWeight, out=None, stream=None):
    """Load-time carrier table int8 [N, K/G, 2^(B-1)] (None for W1)."""
    torch = _torch()
    if w.bits == 1:
        return None
    if out is None:
        out = torch.empty((w.n, w.k // w.group, 1 << (w.bits - 1)), dtype=torch.int8, device=w.codes.device)
    _check(lib().cq_build_carriers(ctypes.byref(w.desc), out.data_ptr(), _stream_ptr(stream)), "cq_build_carriers")
    return out


def cq_gemm_a8_carriers(w: CQWeight, carriers, x8, dx, y_dtype=None, out=None, stream=None):
    torch = _torch()
    assert x8.dim() == 2 and x8.shape[1] == w.k and x8.is_contiguous()
    m = x8.shape[0]
    y_dtype = y_dtype or torch.bfloat16
    if out is None:
        out = torch.empty((m, w.n), dtype=y_dtype, device=x8.device)
    st = lib().cq_gemm_a8_carriers(ctypes.byref(w.desc), carriers.data_ptr() if carriers is not None else None,
                                   x8.data_ptr(), dx.data_ptr(), m, out.data_ptr(), _dt(out.dtype), _stream_ptr(stream))
    _check(st, "cq_gemm_a8_carriers")
    return out


def cq_gemm_routed_model_dtype(bank: CQWeight, n_experts: int, x, route_token, route_expert, y_dtype=None, out=None,
                               workspace=None, stream=None):
    """Route-major routed product; ``bank`` stacks n_experts experts along its rows."""
    torch = _torch()
    assert x.dim() == 2 and x.shape[1] == bank.k and x.is_contiguous()
    assert bank.n % n_experts == 0
    n = bank.n // n_experts
    routes = route_token.numel()
    assert route_expert.numel() == routes and route_token.dtype == torch.int32 and route_expert.dtype == torch.int32
    y_dtype = y_dtype or x.dtype
    if out is None:
        out = torch.empty((routes, n), dtype=y_dtype, device=x.device)
    if workspace is None:
        workspace = torch.empty((n_experts + 1 + routes,), dtype=torch.int32, device=x.device)
    desc = cq_weight(bank.bits, bank.group, n, bank.k, bank.codes.data_ptr(), bank.scale.data_ptr(), bank.a.data_ptr(),
                     bank.b.data_ptr())
    st = lib().cq_gemm_routed_model_dtype(ctypes.byref(desc), n_experts, x.data_ptr(), _dt(x.dtype), x.shape[0],
                                          route_token.data_ptr(), route_expert.data_ptr(), routes, workspace.data_ptr(),
                                          out.data_ptr(), _dt(out.dtype), _stream_ptr(stream))
    _check(st, "cq_gemm_routed_model_dtype")
    return out


def cq_gemm_routed_model_dtype_noalloc(bank: CQWeight, n_experts: int, x, route_token, route_expert, y_dtype=None,
                                       out=None, stream=None):
    """The routed product without a workspace: the library's per-device scratch
    holds the expert grouping (n_experts + 1 + routes <= 2^20)."""
    torch = _torch()
    assert x.dim() == 2 and x.shape[1] == bank.k and x.is_contiguous()
    assert bank.n % n_experts == 0
    n = bank.n // n_experts
    routes = route_token.numel()
    assert route_expert.numel() == routes and route_token.dtype == torch.int32 and route_expert.dtype == torch.int32
    y_dtype = y_dtype or x.dtype
    if out is None:
        out = torch.empty((routes, n), dtype=y_dtype, device=x.device)
    desc = cq_weight(bank.bits, bank.group, n, bank.k, bank.codes.data_ptr(), bank.scale.data_ptr(), bank.a.data_ptr(),
                     bank.b.data_ptr())
    st = lib().cq_gemm_routed_model_dtype_noalloc(ctypes.byref(desc), n_experts, x.data_ptr(), _dt(x.dtype),
                                                  x.shape[0], route_token.data_ptr(), route_expert.data_ptr(), routes,
                                                  out.data_ptr(), _dt(out.dtype), _stream_ptr(stream))
    _check(st, "cq_gemm_routed_model_dtype_noalloc")
    return out


def cq_set_gemv_max_rows(path: int, max_rows: int):
    _check(lib().cq_set_gemv_max_rows(path, max_rows), "cq_set_gemv_max_rows")


def cq_get_gemv_max_rows(path: int) -> int:
    return int(lib().cq_get_gemv_max_rows(path))


def cq_set_a8_fused_launch(single: int):
    _check(lib().cq_set_a8_fused_launch(int(single)), "cq_set_a8_fused_launch")


def cq_get_a8_fused_launch() -> int:
    return int(lib().cq_get_a8_fused_launch())


# ---------------------------------------------------------------- kernel families and the selection table


def _family(f) -> int:
    return FAMILIES[f] if isinstance(f, str) else int(f)


def _desc(w):
    return w.desc if isinstance(w, CQWeight) else w


def cq_family_supported(path: int, family, w, m: int) -> bool:
    """Whether a family can take this call; w is a CQWeight or a cq_weight descriptor."""
    return bool(lib().cq_family_supported(path, _family(family), ctypes.byref(_desc(w)), m))


def cq_gemm_model_dtype_family(w: CQWeight, x, family, y_dtype=None, out=None, stream=None):
    """cq_gemm_model_dtype on one kernel family."""
    torch = _torch()
    assert x.dim() == 2 and x.shape[1] == w.k and x.is_contiguous()
    y_dtype = y_dtype or x.dtype
    if out is None:
        out = torch.empty((x.shape[0], w.n), dtype=y_dtype, device=x.device)
    st = lib().cq_gemm_model_dtype_family(ctypes.byref(w.desc), x.data_ptr(), _dt(x.dtype), x.shape[0],
                                          out.data_ptr(), _dt(out.dtype), _family(family), _stream_ptr(stream))
    _check(st, "cq_gemm_model_dtype_family")
    return out


def cq_gemm_a8_family(w: CQWeight, x8, dx, family, y_dtype=None, out=None, stream=None):
    """cq_gemm_a8 on one kernel family (no partials dump)."""
    torch = _torch()
    assert x8.dim() == 2 and x8.shape[1] == w.k and x8.is_contiguous()
    m = x8.shape[0]
    y_dtype = y_dtype or torch.bfloat16
    if out is None:
        out = torch.empty((m, w.n), dtype=y_dtype, device=x8.device)
    st = lib().cq_gemm_a8_family(ctypes.byref(w.desc), x8.data_ptr(), dx.data_ptr(), m, out.data_ptr(),
                                 _dt(out.dtype), _family(family), _stream_ptr(stream))
    _check(st, "cq_gemm_a8_family")
    return out


def cq_select_set(entries):
    """Install the selection table: a list of dicts with keys path, family, bits,
    group, n, k, m_lo, m_hi and optionally x_dtype (-1 = any)."""
    arr = (cq_select_entry * max(1, len(entries)))()
    for i, e in enumerate(entries):
        arr[i] = cq_select_entry(int(e["path"]), _family(e["family"]), int(e["bits"]), int(e["group"]), int(e["n"]),
                                 int(e["k"]), int(e["m_lo"]), int(e["m_hi"]), int(e.get("x_dtype", -1)), 0)
    _check(lib().cq_select_set(arr, len(entries)), "cq_select_set")


def cq_select_query(path: int, w, m: int, x_dtype: int = CQ_BF16) -> str:
    """Name of the family the dispatcher would run for this call."""
    out = ctypes.c_int32(-1)
    _check(lib().cq_select_query(path, ctypes.byref(_desc(w)), x_dtype, m, ctypes.byref(out)), "cq_select_query")
    return FAMILY_NAMES[out.value]


def cq_probe_read(buf, sink, stream=None):
    """Read the whole device tensor ``buf`` once (HBM read ceiling probe);
    ``sink`` is a one-element int32 device tensor."""
    _check(lib().cq_probe_read(buf.data_ptr(), buf.numel() * buf.element_size(), sink.data_ptr(), _stream_ptr(stream)),
           "cq_probe_read")
