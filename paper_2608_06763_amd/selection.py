"""Measured shape- and device-dependent kernel selection (Sec. 5.6).

For one operator signature (path, B, G, N, K, activation dtype) the tuner
  1. filters the kernel families with ``cq_family_supported`` for every
     representative row count,
  2. runs each admissible family once and keeps it only if its output agrees
     with the built-in choice's output (the families compute the same product
     up to FP32 rounding order; a candidate that does not is reported, never
     selected),
  3. times the valid ones with HIP events on the launch stream over rotated
     copies of the weight, so that every timed call streams its weight from
     HBM, in three rounds over all valid families (alternating order) and
     keeps each family's median round,
  4. maps every row count to its fastest family: each representative row
     count owns the rows up to the geometric midpoint towards the next one,
     and neighbouring regimes with the same family merge.
The result is a deterministic function of the signature and the measured
device; ``install`` hands it to the library (``cq_select_set``), and
``save``/``load`` keep it as JSON keyed by the device it was measured on.
Selection changes neither codes nor metadata.
"""
from __future__ import annotations

import json
import math

import numpy as np

from . import (CQ_BF16, CQ_FP16, CQ_PATH_A8, CQ_PATH_MODEL_DTYPE, FAMILIES, CQWeight, cq_family_supported,
               cq_gemm_a8, cq_gemm_a8_family, cq_gemm_model_dtype, cq_gemm_model_dtype_family, cq_quantize_act_a8,
               cq_select_set)

MODEL_DTYPE_FAMILIES = ("gemv_stream", "gemv_rows", "gemv_lut", "gemv_narrow", "gemv_generic", "gemm_slab", "gemm_slab_staged",
                        "gemm_mfma",
                        "gemm_mfma_m32", "gemm_mfma_m64", "gemm_mfma_m128", "gemm_mfma_m256", "gemm_tiled")
# Families timed only when a caller asks for them: the single-rounded operand
# family trades accuracy for speed (its error can exceed the 2e-3 budget).
OPT_IN_FAMILIES = ("gemm_mfma_rounded",)
A8_FAMILIES = ("gemv_stream", "gemv_narrow", "gemv_generic", "gemm_mfma", "gemm_mfma_m32", "gemm_mfma_m64",
               "gemm_mfma_m128", "gemm_mfma_m256", "gemm_tiled")
M_MAX = (1 << 40) - 1
# relative agreement with the built-in choice (max |dy| / max |y|, FP32 output)
AGREE = 2e-3
# weight bytes in play while timing: twice the 256 MB Infinity Cache
ROTATE_BYTES = 512 << 20


def device_signature() -> dict:
    import torch
    p = torch.cuda.get_device_properties(torch.cuda.current_device())
    return {"name": p.name, "arch": getattr(p, "gcnArchName", ""), "compute_units": p.multi_processor_count,
            "hip": torch.version.hip}


def _batch(torch, fn, calls: int) -> float:
    """Mean time per call of one batch of ``calls`` back-to-back calls, microseconds."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(calls):
        fn(i)
    e1.record()
    e1.synchronize()
    return e0.elapsed_time(e1) * 1e3 / calls


def regimes(ms, choice):
    """[(m_lo, m_hi, family)] from the winner at each representative row count."""
    ms = sorted(ms)
    bounds = [int(math.floor(math.sqrt(a * b))) for a, b in zip(ms[:-1], ms[1:])]
    out = []
    for i, m in enumerate(ms):
        lo = 1 if i == 0 else bounds[i - 1] + 1
        hi = M_MAX if i == len(ms) - 1 else bounds[i]
        if out and out[-1][2] == choice[m]:
            out[-1] = (out[-1][0], hi, choice[m])
        else:
            out.append((lo, hi, choice[m]))
    return out


def tune(w: CQWeight, path: int, ms, x_dtype=None, activations=None, target_ms: float = 2.0, max_calls: int = 50,
         log=None, opt_in=()) -> dict:
    """Measure every admissible family of ``path`` on ``w`` at the row counts ``ms``.

    activations(m) -> bf16/fp16 [m, K] device tensor; by default N(0, 1) rows.
    opt_in: families of OPT_IN_FAMILIES to time as well (still subject to the
    agreement check).
    Returns {"signature", "device", "timings": {m: {family: us}}, "rejected",
    "choice": {m: family}, "entries": [...]} with entries ready for install().
    """
    import torch
    x_dtype = x_dtype or torch.bfloat16
    gen = torch.Generator(device="cuda")
    gen.manual_seed(0)
    if activations is None:
        activations = lambda m: torch.randn((m, w.k), generator=gen, device="cuda", dtype=torch.float32).to(x_dtype)
    copies = [w] + [w.clone() for _ in range(max(0, min(15, math.ceil(ROTATE_BYTES / w.nbytes) - 1)))]
    names = MODEL_DTYPE_FAMILIES if path == CQ_PATH_MODEL_DTYPE else A8_FAMILIES
    names = names + tuple(f for f in opt_in if f in OPT_IN_FAMILIES and path == CQ_PATH_MODEL_DTYPE)
    timings, rejected, choice = {}, {}, {}
    for m in ms:
        x = activations(m)
        y = torch.empty((m, w.n), dtype=torch.float32, device="cuda")
        if path == CQ_PATH_MODEL_DTYPE:
            ref = cq_gemm_model_dtype(w, x, y_dtype=torch.float32)
            run = lambda f, c, out: cq_gemm_model_dtype_family(c, x, f, out=out)
        else:
            x8, dx = cq_quantize_act_a8(x)
            ref = cq_gemm_a8(w, x8, dx, y_dtype=torch.float32)
            run = lambda f, c, out: cq_gemm_a8_family(c, x8, dx, f, out=out)
        scale = float(ref.abs().max()) or 1.0
        timings[m] = {}
        calls = {}
        for f in names:
            if not cq_family_supported(path, f, w, m):
                continue
            run(f, w, y)
            err = float((y - ref).abs().max()) / scale
            if not err <= AGREE:
                rejected.setdefault(m, {})[f] = err
                continue
            run(f, copies[0], y)
            torch.cuda.synchronize()
            t0 = min(_batch(torch, lambda i: run(f, copies[i % len(copies)], y), 2) for _ in range(3))
            calls[f] = int(min(max_calls, max(len(copies), target_ms * 1e3 / max(t0, 1e-3))))
        # three rounds over all candidates, the order reversed every other round,
        # so that no family is timed only right after the host work between row
        # counts (clock ramp); the median batch per family is kept
        samples = {f: [] for f in calls}
        for r in range(3):
            for f in (list(calls) if r % 2 == 0 else list(calls)[::-1]):
                samples[f].append(_batch(torch, lambda i: run(f, copies[i % len(copies)], y), calls[f]))
        timings[m] = {f: float(np.median(v)) for f, v in samples.items()}
        choice[m] = min(timings[m], key=lambda f: timings[m][f])
        if log:
            log(f"[select] path {path} m={m}: " + ", ".join(f"{f} {t:.1f} us" for f, t in timings[m].items())
                + f" -> {choice[m]}")
    xd = -1 if path == CQ_PATH_A8 else (CQ_BF16 if x_dtype == torch.bfloat16 else CQ_FP16)
    entries = [{"path": path, "family": f, "bits": w.bits, "group": w.group, "n": w.n, "k": w.k, "m_lo": lo,
                "m_hi": hi, "x_dtype": xd} for lo, hi, f in regimes(ms, choice)]
    return {"signature": {"path": path, "bits": w.bits, "group": w.group, "n": w.n, "k": w.k, "x_dtype": xd},
            "device": device_signature(), "timings": timings, "rejected": rejected, "choice": choice,
            "entries": entries}


def install(tables):
    """Install the entries of one or more tune() results (replaces the table)."""
    if isinstance(tables, dict):
        tables = [tables]
    cq_select_set([e for t in tables for e in t["entries"]])


def clear():
    cq_select_set([])


def save(path: str, tables):
    if isinstance(tables, dict):
        tables = [tables]
    with open(path, "w") as f:
        json.dump({"device": device_signature(), "tables": tables}, f, indent=1, default=str)


def load(path: str, allow_other_device: bool = False) -> list:
    """Read a saved table; refuses one measured on another device unless asked."""
    with open(path) as f:
        doc = json.load(f)
    if not allow_other_device and doc["device"] != device_signature():
        raise ValueError(f"{path} was measured on {doc['device']}, this is {device_signature()}")
    for t in doc["tables"]:
        for e in t["entries"]:
            if e["family"] not in FAMILIES:
                raise ValueError(f"unknown family {e['family']}")
    return doc["tables"]
