"""GPU parity at the full workload sizes, on sampled outputs.

The library runs each configuration at its real shape, in the launch
configuration the benchmark times (same entry points, same dispatch); the
oracle recomputes a seeded sample of output rows (weight rows decoded in
float64, A8 carriers from exact rationals) and the sampled outputs must meet
the same bars as the small parity tests: eps_comp <= 2e-3 for bf16 outputs,
1e-5 for FP32 outputs of the FP32-product paths, and bit-exact INT32 group
partials where they are dumped.

Weights.  The checked rows carry the configuration's own law, quantized by
the oracle fit: exactly the sampled weight rows are drawn (row-seeded
generators) and fitted, and spliced at their indices into a seeded packed
stand-in that fills the rest of the full-size matrix.  Rows of y depend only
on their own weight row, so the unchecked rows only set the shape, the
launch configuration and the memory traffic.
"""
import functools

import numpy as np
import pytest

from oracle import a8 as A8
from oracle import ref as R
from tests._cases import say
from workloads import (LLAMA8B_LAYERS, PREFILL70B_SHAPES, bf16_bits_to_f32, crossover_act, crossover_weight, gemv_4k,
                       llama8b_act, llama8b_weight, prefill70b_act, prefill70b_weight, sweep_act, sweep_weight,
                       synthetic_representation)

pytestmark = pytest.mark.gpu

TOL = 2e-3


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2608_06763_amd as cq
    cq.lib()
    return torch


def _cq():
    import paper_2608_06763_amd as cq
    return cq


def _dev_x(torch, bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def _sample(seed, count, total):
    return np.sort(np.random.default_rng(seed).choice(total, size=min(count, total), replace=False))


# the configurations' weight laws, as functions of the sampled rows
LAWS = {
    "llama8b": lambda layer, k, n: (lambda rows: llama8b_weight(layer, k, n, rows)),
    "sweep": lambda k, n: (lambda rows: sweep_weight(k, n, rows)),
    "crossover": lambda k, n: (lambda rows: crossover_weight(k, n, rows)),
    "prefill70b": lambda k, n, off: (lambda rows: prefill70b_weight(k, n, off, rows)),
}


@functools.lru_cache(maxsize=None)
def _fitted_rows(law_key, rows_key, bits, group):
    """Oracle fit of the sampled rows of a configuration's weights (cached)."""
    from oracle import fit as FIT
    law, args = law_key[0], law_key[1:]
    w = LAWS[law](*args)(np.asarray(rows_key))
    return FIT.fit(w, bits, group)


def _spliced_np(seed, n, k, bits, group, law_key, rows):
    """Seeded stand-in [N, K] with the oracle-fitted rows of the law at `rows`."""
    codes, s, a, b = synthetic_representation(seed, n, k, bits, group)
    fr = _fitted_rows(law_key, tuple(int(r) for r in rows), bits, group)
    codes[rows], s[rows], a[rows], b[rows] = fr.codes, fr.scale, fr.a_bits, fr.b_bits
    return codes, s, a, b


@functools.lru_cache(maxsize=2)
def _spliced(seed, n, k, bits, group, law_key, rows_key):
    """The spliced matrix, packed by the library and uploaded once per module run."""
    codes, s, a, b = _spliced_np(seed, n, k, bits, group, law_key, np.asarray(rows_key))
    return codes, s, a, b, _cq().CQWeight.from_codes(codes, s, a, b, bits, group)


def _ref_rows(xv, codes, s, a, b, bits, group, rows):
    """Oracle model-dtype outputs y[:, rows] (float64)."""
    return R.gemm_model_dtype(xv, codes[rows], bits, group, s[rows], a[rows], b[rows])


def _ref_a8_rows(x8, dx, codes, s, a, b, bits, group, rows):
    y, p = A8.gemm_a8(x8, dx, codes[rows], bits, group, s[rows], a[rows], b[rows])
    return y, p


def _check_rounded_bound(got, y_ref, xs, codes, s, a, b, bits, group, rows):
    """|y - y_ref| <= 2^-8 sum_j |x_j| |w_j| (one BF16 rounding per weight) plus
    the FP32 accumulation, elementwise."""
    from oracle import format as F
    wabs = np.abs(F.decode(codes[rows], bits, group, s[rows], a[rows], b[rows]))
    bound = 2.0 ** -8 * (np.abs(xs) @ wabs.T) * (1 + 2e-3) + 1e-6 * np.max(np.abs(y_ref))
    assert np.all(np.abs(np.asarray(got, np.float64) - y_ref) <= bound)


def _eps(got, ref, dtype):
    return R.eps_comp(np.asarray(got, np.float64), ref, dtype)


def _check_both_paths(torch, w, xb, codes, s, a, b, bits, group, rows, tag, xrows=None):
    """Run both entry points at full size; compare sampled columns (and
    sampled activation rows when xrows is given) with the oracle.  Where the
    single-rounded matrix-core family can take the shape, it is held to the
    same bar (its error is printed)."""
    cq = _cq()
    xs = bf16_bits_to_f32(xb if xrows is None else xb[xrows]).astype(np.float64)
    x = _dev_x(torch, xb)
    say(tag, "model-dtype")
    y = cq.cq_gemm_model_dtype(w, x).float().cpu().numpy()
    y_ref = _ref_rows(xs, codes, s, a, b, bits, group, rows)
    got = y[:, rows] if xrows is None else y[xrows][:, rows]
    assert _eps(got, y_ref, "bf16") <= TOL
    m = xb.shape[0]
    if m > 16 and cq.cq_family_supported(cq.CQ_PATH_MODEL_DTYPE, "gemm_mfma_rounded", w, m):
        # the single-rounded operand family: every weight rounded once to BF16
        # (relative error <= 2^-8), products exact, FP32 accumulation; its
        # FP32 output must lie within that rounding's own bound elementwise
        say(tag, "model-dtype rounded operand")
        yr = cq.cq_gemm_model_dtype_family(w, x, "gemm_mfma_rounded", y_dtype=torch.float32).cpu().numpy()
        yr = yr[:, rows] if xrows is None else yr[xrows][:, rows]
        say(tag, f"rounded operand eps_comp {_eps(yr, y_ref, 'fp32'):.3e}")
        _check_rounded_bound(yr, y_ref, xs, codes, s, a, b, bits, group, rows)
    say(tag, "a8")
    x8, dx = cq.cq_quantize_act_a8(x)
    x8_ref, d_ref = A8.quantize_act(xs)
    x8_got = x8.cpu().numpy() if xrows is None else x8.cpu().numpy()[xrows]
    d_got = dx.cpu().numpy() if xrows is None else dx.cpu().numpy()[xrows]
    assert np.array_equal(x8_got, x8_ref)
    assert np.array_equal(d_got, d_ref.astype(np.float32))
    ya = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch.float32).cpu().numpy()
    ya_ref, _ = _ref_a8_rows(x8_ref, d_ref, codes, s, a, b, bits, group, rows)
    gota = ya[:, rows] if xrows is None else ya[xrows][:, rows]
    assert _eps(gota, ya_ref, "fp32") <= 1e-5


def test_fullsize_single_gemv_fitted(torch_dev):
    # W4 G128, M = 1, K = N = 4096, weights fitted by the oracle; every output
    x_bits, w = gemv_4k()
    from oracle import fit as FIT
    say("fullsize gemv_4k fit")
    r = FIT.fit(w, 4, 128)
    cq = _cq()
    wt = cq.CQWeight.from_codes(r.codes, r.scale, r.a_bits, r.b_bits, 4, 128)
    _check_both_paths(torch_dev, wt, x_bits, r.codes, r.scale, r.a_bits, r.b_bits, 4, 128,
                      np.arange(4096), "gemv_4k")


@pytest.mark.parametrize("m", [1, 4, 16])
@pytest.mark.parametrize("layer", range(4))
def test_fullsize_llama8b_decode_layers(torch_dev, layer, m):
    # the benchmark's layer shapes and launches; 96 sampled output rows carry
    # the layer's Laplace-with-outlier-channels weights, fitted by the oracle
    name, k, n = LLAMA8B_LAYERS[layer]
    rows = _sample(7 + layer, 96, n)
    say(f"llama8b {name} fit of the sampled rows")
    codes, s, a, b, w = _spliced(2000 + layer, n, k, 4, 128, ("llama8b", layer, k, n), tuple(rows.tolist()))
    xb = llama8b_act(m, k, layer)
    _check_both_paths(torch_dev, w, xb, codes, s, a, b, 4, 128, rows, f"llama8b {name} m={m}")


@pytest.mark.parametrize("m", [1, 2, 8, 32, 128, 512, 2048, 8192])
def test_fullsize_crossover_shape(torch_dev, m):
    # K = 8192, N = 28672, W4 G128 at every row count of the crossover sweep;
    # 48 sampled weight rows (Student-t weights fitted by the oracle) x (all or
    # 24 sampled) activation rows
    k, n = 8192, 28672
    rows = _sample(11, 48, n)
    say(f"crossover fit of the sampled rows")
    codes, s, a, b, w = _spliced(4001, n, k, 4, 128, ("crossover", k, n), tuple(rows.tolist()))
    xb = crossover_act(m, k)
    xrows = None if m <= 32 else _sample(12, 24, m)
    _check_both_paths(torch_dev, w, xb, codes, s, a, b, 4, 128, rows, f"crossover m={m}", xrows)


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 6, 8])
@pytest.mark.parametrize("group", [32, 64, 128, 256])
def test_fullsize_width_group_sweep(torch_dev, bits, group):
    # M = 1, K = N = 8192 for every B x G of the sweep; 32 sampled rows of
    # N(0, 0.015^2) weights fitted by the oracle at this B and G
    k = n = 8192
    rows = _sample(13, 32, n)
    say(f"sweep B={bits} G={group} fit of the sampled rows")
    codes, s, a, b, w = _spliced(5000 + 10 * bits + group // 32, n, k, bits, group, ("sweep", k, n),
                                 tuple(rows.tolist()))
    xb = sweep_act(k)
    _check_both_paths(torch_dev, w, xb, codes, s, a, b, bits, group, rows, f"sweep B={bits} G={group}")


@pytest.mark.parametrize("m", [2048, 8192])
@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("shape", range(3))
def test_fullsize_prefill70b(torch_dev, shape, bits, m):
    # 70B-class prefill GEMMs, W3 and W4 G128; 16 x 24 sampled outputs, the
    # 16 weight rows Laplace times their row multiplier, fitted by the oracle
    k, n = PREFILL70B_SHAPES[shape]
    rows = _sample(17, 16, n)
    say(f"prefill70b {k}x{n} B={bits} fit of the sampled rows")
    codes, s, a, b, w = _spliced(6000 + 10 * shape + bits, n, k, bits, 128, ("prefill70b", k, n, shape),
                                 tuple(rows.tolist()))
    xb = prefill70b_act(m, k)
    xrows = _sample(18, 24, m)
    _check_both_paths(torch_dev, w, xb, codes, s, a, b, bits, 128, rows, f"prefill70b {k}x{n} m={m} B={bits}",
                      xrows)


def test_fullsize_fitted_slice_partials(torch_dev):
    # oracle-fitted Laplace-with-outliers weights at a full decode-layer width
    # (K = 14336), 64 rows: INT32 group partials of both matrix-core families
    # compared bit for bit
    from workloads import llama8b_weight
    w_full = llama8b_weight(3, 14336, 64)
    say("fitted slice K=14336 fit")
    from oracle import fit as FIT
    r = FIT.fit(w_full, 4, 128)
    cq = _cq()
    wt = cq.CQWeight.from_codes(r.codes, r.scale, r.a_bits, r.b_bits, 4, 128)
    for m in (1, 16, 300):
        xb = llama8b_act(m, 14336, 9)
        xv = bf16_bits_to_f32(xb).astype(np.float64)
        x8_ref, d_ref = A8.quantize_act(xv)
        _, p_ref = A8.gemm_a8(x8_ref, d_ref, r.codes, 4, 128, r.scale, r.a_bits, r.b_bits)
        say("fitted slice partials m=", m)
        x8 = torch_dev.from_numpy(x8_ref).cuda()
        dx = torch_dev.from_numpy(d_ref).cuda()
        _, parts = cq.cq_gemm_a8(wt, x8, dx, y_dtype=torch_dev.float32, want_partials=True)
        assert np.array_equal(parts.cpu().numpy(), p_ref)


@pytest.mark.parametrize("layer", range(4))
def test_fullsize_fused_a8_decode_layers(torch_dev, layer):
    # the benchmark's single-row fused A8 call on each decode layer: carriers
    # and d_x bit-exact, 96 sampled output rows against the A8 oracle
    name, k, n = LLAMA8B_LAYERS[layer]
    rows = _sample(31 + layer, 96, n)
    say("fused a8", name, "fit of the sampled rows")
    codes, s, a, b, w = _spliced(2000 + layer, n, k, 4, 128, ("llama8b", layer, k, n), tuple(rows.tolist()))
    cq = _cq()
    xb = llama8b_act(1, k, layer)
    xv = bf16_bits_to_f32(xb).astype(np.float64)
    say("fused a8", name)
    cq.cq_set_a8_fused_launch(1)  # the single launch (the default runs the two calls)
    try:
        y, x8, dx = cq.cq_gemm_a8_fused(w, _dev_x(torch_dev, xb), y_dtype=torch_dev.float32)
    finally:
        cq.cq_set_a8_fused_launch(0)
    x8_ref, d_ref = A8.quantize_act(xv)
    assert np.array_equal(x8.cpu().numpy(), x8_ref)
    assert np.array_equal(dx.cpu().numpy(), d_ref.astype(np.float32))
    y_ref, _ = _ref_a8_rows(x8_ref, d_ref, codes, s, a, b, 4, 128, rows)
    assert _eps(y.cpu().numpy()[:, rows], y_ref, "fp32") <= 1e-5


@pytest.mark.parametrize("layer", range(2))
@pytest.mark.parametrize("tokens", [1, 16, 64])
def test_fullsize_routed_mixtral_experts(torch_dev, layer, tokens):
    # the routed sweep's configuration: a bank of 8 copies of one synthetic
    # expert (as the benchmark builds it), top-2 skewed routes; every route's
    # output on 48 sampled columns against the oracle
    from workloads import MOE_EXPERTS, MOE_LAYERS, MOE_TOPK, route_map
    name, k, n = MOE_LAYERS[layer]
    codes, s, a, b = synthetic_representation(7000 + layer, n, k, 4, 128)
    cq = _cq()
    w1 = cq.CQWeight.from_codes(codes, s, a, b, 4, 128)
    rep = lambda t: t.repeat(MOE_EXPERTS, 1) if t.dim() == 2 else t.repeat(MOE_EXPERTS)
    bank = cq.CQWeight(rep(w1.codes), rep(w1.scale), rep(w1.a), rep(w1.b), 4, 128, n * MOE_EXPERTS, k)
    tok, exp = route_map(7100 + tokens, tokens, MOE_EXPERTS, MOE_TOPK)
    xb = llama8b_act(tokens, k, 5)
    xv = bf16_bits_to_f32(xb).astype(np.float64)
    cols = _sample(41 + tokens, 48, n)
    say("routed fullsize", name, tokens)
    y = cq.cq_gemm_routed_model_dtype(bank, MOE_EXPERTS, _dev_x(torch_dev, xb), torch_dev.from_numpy(tok).cuda(),
                                      torch_dev.from_numpy(exp).cuda(), y_dtype=torch_dev.float32)
    y_ref = _ref_rows(xv[tok], codes, s, a, b, 4, 128, cols)
    assert _eps(y.cpu().numpy()[:, cols], y_ref, "fp32") <= 2e-4
    y16 = cq.cq_gemm_routed_model_dtype(bank, MOE_EXPERTS, _dev_x(torch_dev, xb), torch_dev.from_numpy(tok).cuda(),
                                        torch_dev.from_numpy(exp).cuda())
    assert _eps(y16.float().cpu().numpy()[:, cols], y_ref, "bf16") <= TOL
