"""Groupwise reference fitters, float64: the continuous fitter (Sec. 4.1) and
the carrier-aware joint fitter (Sec. 4.3, ``fit_joint``).

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
counts open.  This oracle fixes them:
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
        lib.cq_oracle_eval_candidates_joint.argtypes = lib.cq_oracle_eval_candidates.argtypes
        lib.cq_oracle_assign_serialized_joint.argtypes = [p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, p, p, p, p, p,
                                                          p, p]
        lib.cq_oracle_carriers.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_double, p]
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


def _refine(wg, bits, g, inc_a, inc_b, inc_sse, inc_s, step, clips, iters, joint=False):
    """One 3x3 local refinement around each group's incumbent."""
    lib = _load()
    scorer = lib.cq_oracle_eval_candidates_joint if joint else lib.cq_oracle_eval_candidates
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
    scorer(_ptr(wg), ng, g, bits, _ptr(ca), _ptr(cb), _ptr(valid), len(offs), 0,
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


# ---------------------------------------------------------------- carrier-aware joint fit (Sec. 4.3)


@dataclass
class JointFitResult:
    codes: np.ndarray      # int8 [N, K]
    scale: np.ndarray      # float32 [N, K/G]
    a_bits: np.ndarray     # uint16 [N, K/G]
    b_bits: np.ndarray     # uint16 [N, K/G]
    loss_c: np.ndarray     # float64 [N, K/G], L_C of the serialized representation
    loss_a8: np.ndarray    # float64 [N, K/G], L_A8 of the serialized representation

    def nrmse_joint(self, w) -> float:
        """eq. carrier-aware-nrmse: sqrt((L_C + L_A8) / (2 sum w^2))."""
        w = np.asarray(w, dtype=np.float64)
        return float(np.sqrt((self.loss_c.sum() + self.loss_a8.sum()) / (2.0 * np.sum(w * w))))

    def nrmse_a8(self, w) -> float:
        """The A8-only diagnostic sqrt(L_A8 / sum w^2)."""
        w = np.asarray(w, dtype=np.float64)
        return float(np.sqrt(self.loss_a8.sum() / np.sum(w * w)))


def carriers_c(bits: int, a: float, b: float) -> np.ndarray:
    """The C scorer's integer-exact carriers r(0..M) for one FP16 shape pair."""
    out = np.empty(max_code(bits) + 1, np.int32)
    if _load().cq_oracle_carriers(bits, float(a), float(b), _ptr(out)):
        raise ValueError("bits must be 2..8")
    return out


def joint_loss(w, codes, bits: int, group: int, scale, a_bits, b_bits):
    """(L_C, L_A8) per group of a given representation (eq. continuous-and-carrier-loss),
    from the oracle's exact carrier table."""
    from .a8 import carrier_table
    from .format import decode
    w = np.asarray(w, dtype=np.float64)
    n, k = w.shape
    wc = decode(codes, bits, group, scale, a_bits, b_bits)
    m = 1 if bits == 1 else max_code(bits)
    ng = k // group
    wa = np.empty_like(wc)
    cache = {}
    for r in range(n):
        for g in range(ng):
            key = (int(a_bits[r, g]), int(b_bits[r, g]))
            if key not in cache:
                cache[key] = carrier_table(bits, *key)
            tab = cache[key]
            kk = codes[r, g * group:(g + 1) * group].astype(np.int64)
            mag = np.abs(kk) if bits > 1 else np.ones_like(kk)
            car = np.array([tab[i] for i in mag], np.float64)
            wa[r, g * group:(g + 1) * group] = np.sign(kk) * float(scale[r, g]) * car / 127.0
    lc = ((w - wc) ** 2).reshape(n, ng, group).sum(axis=2)
    la = ((w - wa) ** 2).reshape(n, ng, group).sum(axis=2)
    return lc, la


def fit_joint(w, bits: int, group: int, candidates=None, refine_steps=(0.05, 0.02),
              clips=CLIPS, iters=ITERS) -> JointFitResult:
    """Carrier-aware joint fit of every [1, G] group (Sec. 4.3): the same
    candidate traversal as ``fit``, scoring L_C + L_A8 (eq.
    carrier-aware-objective) with the joint assignment and closed-form scale,
    then the final joint assignment under the stored FP32 scale, FP16 shapes
    and their exact carriers.  W1 levels already lie on the carrier grid
    (L_C = L_A8), so W1 keeps the continuous fit."""
    from .a8 import carrier_table
    w = np.ascontiguousarray(np.asarray(w, dtype=np.float32))
    n, k = w.shape
    if k % group:
        raise ValueError("K must be a multiple of G")
    if bits == 1:
        r = fit(w, bits, group)
        return JointFitResult(r.codes, r.scale, r.a_bits, r.b_bits, r.sse, r.sse.copy())
    ng = n * (k // group)
    wg = w.reshape(ng, group)
    zero = np.all(wg == 0, axis=1)
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
    loss = np.empty(ng)
    s = np.empty(ng)
    clips_a = np.asarray(clips, dtype=np.float64)
    rc = lib.cq_oracle_eval_candidates_joint(_ptr(wg), ng, group, bits, _ptr(np.ascontiguousarray(ca)),
                                             _ptr(np.ascontiguousarray(cb)), _ptr(valid), len(ca), 1,
                                             _ptr(clips_a), len(clips_a), iters, _ptr(idx), _ptr(loss), _ptr(s))
    if rc:
        raise RuntimeError("oracle candidate scorer rejected its arguments")
    inc_a, inc_b = ca[idx], cb[idx]
    for step in steps:
        inc_a, inc_b, loss, s = _refine(wg, bits, group, inc_a, inc_b, loss, s, step, clips, iters, joint=True)

    s32 = s.astype(np.float32)
    s32[zero] = 0
    inc_a = np.where(zero, 1.0, inc_a)
    inc_b = np.where(zero, 0.0, inc_b)
    a_bits = f64_to_f16_bits(inc_a)
    b_bits = f64_to_f16_bits(inc_b)
    m = max_code(bits)
    car = np.empty((ng, m + 1), np.int32)
    cache = {}
    for gi in range(ng):
        key = (int(a_bits[gi]), int(b_bits[gi]))
        if key not in cache:
            cache[key] = carrier_table(bits, *key)
        car[gi] = cache[key]
    codes = np.empty((ng, group), np.int8)
    lc = np.empty(ng)
    la = np.empty(ng)
    lib.cq_oracle_assign_serialized_joint(_ptr(wg), ng, group, bits, _ptr(s32), _ptr(np.ascontiguousarray(inc_a)),
                                          _ptr(np.ascontiguousarray(inc_b)), _ptr(car), _ptr(codes), _ptr(lc),
                                          _ptr(la))
    assert np.all(np.abs(codes.astype(np.int64)) <= m)
    return JointFitResult(codes.reshape(n, k), s32.reshape(n, -1), a_bits.reshape(n, -1), b_bits.reshape(n, -1),
                          lc.reshape(n, -1), la.reshape(n, -1))
