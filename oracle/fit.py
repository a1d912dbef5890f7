"""Continuous groupwise reference fitter (Sec. 4.1), float64.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Each [1, G] group is fitted independently by minimising the original-domain
squared error of eq. offline-objective over the codes, the scale and an
admissible shape (a, b):
  * s is both the endpoint and the clipping threshold, values beyond s
    saturate at the signed endpoint, and each value goes to its nearest level;
  * a deterministic set of monotone (a, b) candidates is traversed, always
    starting with the uniform-integer point (1, 0) (eq. int-special-case);
  * scale and clipping are refined jointly for every candidate;
  * the objective is re-evaluated after mapping s to FP32 and (a, b) to FP16,
    so the stored representation is what is scored;
  * NRMSE_C = sqrt(sum (w - w_hat)^2 / sum w^2) (eq. nrmse).

The paper leaves the candidate grid, the clipping candidates and the iteration
counts open.  This oracle fixes them (the same constants are the defaults of
the product-side fitter, which is tested against this one):
  * coarse grid a in {0.10, 0.20, ..., 1.50} x b in {-1.20, -1.10, ..., 0.40},
    each value rounded to FP16 first, kept when m(a, b) >= 1e-3;
  * two 3x3 local refinements around the incumbent, steps 0.05 then 0.02,
    admissible candidates only;
  * clip initialisations s = alpha max|w|, alpha in {1.00, 0.90, 0.80, 0.70};
  * three assignment / least-squares-scale rounds, then a final assignment
    that is scored; the lowest SSE wins and ties keep the earlier candidate;
  * W2 has no interior level, so only (1, 0) is used; W1 takes k = sign(w)
    (w = 0 gives +1) and s = fl32(mean |w|), the exact least-squares scale;
  * an all-zero group stores s = 0, (a, b) = (1, 0) and zero codes (+1 for W1).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

from .format import f16_bits_to_f64, f64_to_f16_bits, max_code, shape_margin

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fit_eval.c")
_LIB = os.path.join(_HERE, "_fit_eval.so")

CLIPS = (1.00, 0.90, 0.80, 0.70)
ITERS = 3
MARGIN_MIN = 1e-3


def build_c(force: bool = False) -> str:
    """Compile the candidate scorer with gcc (plain C, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build_c())
        p = ctypes.c_void_p
        lib.cq_oracle_eval_candidates.argtypes = [p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, p, p, p,
                                                  ctypes.c_int, ctypes.c_int, p, ctypes.c_int, ctypes.c_int,
                                                  p, p, p]
        lib.cq_oracle_assign_serialized.argtypes = [p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, p, p, p, p, p]
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def coarse_candidates() -> tuple[np.ndarray, np.ndarray]:
    """(1, 0) followed by the admissible FP16-rounded coarse grid, fixed order."""
    a_vals = np.round(np.arange(1, 16) * 0.1, 10)
    b_vals = np.round(-1.2 + np.arange(0, 17) * 0.1, 10)
    ca, cb = [1.0], [0.0]
    for a in a_vals:
        for b in b_vals:
            a16 = float(f16_bits_to_f64(f64_to_f16_bits(a)))
            b16 = float(f16_bits_to_f64(f64_to_f16_bits(b)))
            if (a16, b16) == (1.0, 0.0):
                continue
            if shape_margin(a16, b16) >= MARGIN_MIN:
                ca.append(a16)
                cb.append(b16)
    return np.array(ca), np.array(cb)


@dataclass
class FitResult:
    codes: np.ndarray      # int8 [N, K]
    scale: np.ndarray      # float32 [N, K/G]
    a_bits: np.ndarray     # uint16 [N, K/G]
    b_bits: np.ndarray     # uint16 [N, K/G]
    sse: np.ndarray        # float64 [N, K/G], serialized representation

    def nrmse(self, w) -> float:
        w = np.asarray(w, dtype=np.float64)
        return float(np.sqrt(self.sse.sum() / np.sum(w * w)))


def _refine(wg, bits, g, inc_a, inc_b, inc_sse, inc_s, step, clips, iters):
    """One 3x3 local refinement around each group's incumbent."""
    lib = _load()
    ng = wg.shape[0]
    offs = [(da, db) for da in (-1, 0, 1) for db in (-1, 0, 1) if (da, db) != (0, 0)]
    ca = np.empty((ng, len(offs)))
    cb = np.empty((ng, len(offs)))
    for i, (da, db) in enumerate(offs):
        ca[:, i] = f16_bits_to_f64(f64_to_f16_bits(inc_a + da * step))
        cb[:, i] = f16_bits_to_f64(f64_to_f16_bits(inc_b + db * step))
    valid = (shape_margin(ca, cb) >= MARGIN_MIN).astype(np.uint8)
    idx = np.empty(ng, np.int32)
    sse = np.empty(ng)
    s = np.empty(ng)
    clips_a = np.asarray(clips, dtype=np.float64)
    ca = np.ascontiguousarray(ca)
    cb = np.ascontiguousarray(cb)
    lib.cq_oracle_eval_candidates(_ptr(wg), ng, g, bits, _ptr(ca), _ptr(cb), _ptr(valid), len(offs), 0,
                                  _ptr(clips_a), len(clips_a), iters, _ptr(idx), _ptr(sse), _ptr(s))
    better = (idx >= 0) & (sse < inc_sse)
    rows = np.nonzero(better)[0]
    inc_a = inc_a.copy()
    inc_b = inc_b.copy()
    inc_sse = inc_sse.copy()
    inc_s = inc_s.copy()
    inc_a[rows] = ca[rows, idx[rows]]
    inc_b[rows] = cb[rows, idx[rows]]
    inc_sse[rows] = sse[rows]
    inc_s[rows] = s[rows]
    return inc_a, inc_b, inc_sse, inc_s


def fit(w, bits: int, group: int, candidates=None, refine_steps=(0.05, 0.02),
        clips=CLIPS, iters=ITERS) -> FitResult:
    """Fit every [1, G] group of the float32 matrix w [N, K]."""
    w = np.ascontiguousarray(np.asarray(w, dtype=np.float32))
    n, k = w.shape
    if k % group:
        raise ValueError("K must be a multiple of G")
    ng = n * (k // group)
    wg = w.reshape(ng, group)
    u = np.abs(wg.astype(np.float64))
    zero = np.all(u == 0, axis=1)

    a_bits = np.full(ng, f64_to_f16_bits(1.0), np.uint16)
    b_bits = np.full(ng, f64_to_f16_bits(0.0), np.uint16)

    if bits == 1:
        codes = np.where(wg >= 0, 1, -1).astype(np.int8)
        s = np.mean(u, axis=1).astype(np.float32)
        s[zero] = 0
        sse = np.sum((u - s.astype(np.float64)[:, None]) ** 2, axis=1)
        return FitResult(codes.reshape(n, k), s.reshape(n, -1), a_bits.reshape(n, -1),
                         b_bits.reshape(n, -1), sse.reshape(n, -1))

    lib = _load()
    if bits == 2:
        ca, cb = np.array([1.0]), np.array([0.0])
        steps = ()
    elif candidates is None:
        ca, cb = coarse_candidates()
        steps = refine_steps
    else:
        ca, cb = (np.asarray(c, dtype=np.float64) for c in candidates)
        steps = refine_steps
    valid = np.ones(len(ca), np.uint8)
    idx = np.empty(ng, np.int32)
    sse = np.empty(ng)
    s = np.empty(ng)
    clips_a = np.asarray(clips, dtype=np.float64)
    rc = lib.cq_oracle_eval_candidates(_ptr(wg), ng, group, bits, _ptr(np.ascontiguousarray(ca)),
                                       _ptr(np.ascontiguousarray(cb)), _ptr(valid), len(ca), 1,
                                       _ptr(clips_a), len(clips_a), iters, _ptr(idx), _ptr(sse), _ptr(s))
    if rc:
        raise RuntimeError("oracle candidate scorer rejected its arguments")
    inc_a, inc_b = ca[idx], cb[idx]
    for step in steps:
        inc_a, inc_b, sse, s = _refine(wg, bits, group, inc_a, inc_b, sse, s, step, clips, iters)

    # serialize: s -> FP32, (a, b) already FP16; reassign under stored values
    s32 = s.astype(np.float32)
    s32[zero] = 0
    inc_a = np.where(zero, 1.0, inc_a)
    inc_b = np.where(zero, 0.0, inc_b)
    codes = np.empty((ng, group), np.int8)
    sse_ser = np.empty(ng)
    lib.cq_oracle_assign_serialized(_ptr(wg), ng, group, bits, _ptr(s32), _ptr(np.ascontiguousarray(inc_a)),
                                    _ptr(np.ascontiguousarray(inc_b)), _ptr(codes), _ptr(sse_ser))
    a_bits = f64_to_f16_bits(inc_a)
    b_bits = f64_to_f16_bits(inc_b)
    assert np.all(np.abs(codes.astype(np.int64)) <= max_code(bits))
    return FitResult(codes.reshape(n, k), s32.reshape(n, -1), a_bits.reshape(n, -1),
                     b_bits.reshape(n, -1), sse_ser.reshape(n, -1))
