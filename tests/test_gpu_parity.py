"""GPU parity: every entry point of the C ABI against the CPU oracle.

Integer stages (unpacked codes, INT8 activation carriers, their scales, INT32
group partials) must match bit for bit.  Floating-point outputs must satisfy
eps_comp <= 2e-3 (bf16/fp16 outputs; the final output rounding is excused
once, see oracle/ref.py) and tighter bounds for FP32 outputs of paths that
multiply in FP32.
"""
import numpy as np
import pytest

from oracle import a8 as A8
from oracle import format as F
from oracle import ref as R
from tests._cases import act, carrier_probe, fitted, ref_a8, ref_model_dtype, say

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


def _weight(r, bits, group):
    return _cq().CQWeight.from_codes(r.codes, r.scale, r.a_bits, r.b_bits, bits, group)


def _x(torch, bits_np, dtype):
    t = torch.from_numpy(bits_np.view(np.int16)).cuda()
    return t.view(torch.bfloat16 if dtype == "bf16" else torch.float16)


def _np(t):
    import torch
    if t.dtype in (torch.bfloat16, torch.float16):
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy()


WIDTHS = list(range(1, 9))
GROUPS = [32, 64, 128, 256]


# ---------------------------------------------------------------- decode


@pytest.mark.parametrize("bits", WIDTHS)
@pytest.mark.parametrize("group", GROUPS)
def test_decode_ref(torch_dev, bits, group):
    r = fitted(1, 40, 512, bits, group)
    say("decode_ref", bits, group)
    w = _weight(r, bits, group)
    codes, vals = _cq().cq_decode_ref(w)
    torch_dev.cuda.synchronize()
    assert np.array_equal(codes.cpu().numpy(), r.codes)
    want = F.decode(r.codes, bits, group, r.scale, r.a_bits, r.b_bits)
    got = vals.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got - want) <= 2e-6 * np.abs(want) + 1e-30)


@pytest.mark.parametrize("bits,raw", [(4, 0x88), (3, None), (2, 0xAA), (8, 0x80)])
def test_decode_reserved_pattern(torch_dev, bits, raw):
    # a stream made only of the reserved pattern (bypassing the packer)
    k = 128
    n = 2
    if bits == 3:
        row = bytes([0x24, 0x49, 0x92]) * (k * 3 // 24)
    else:
        row = bytes([raw]) * (k * bits // 8)
    packed = np.frombuffer(row * n, np.uint8).reshape(n, -1).copy()
    s = np.ones((n, 1), np.float32)
    a = np.full((n, 1), F.f64_to_f16_bits(0.7), np.uint16)
    b = np.full((n, 1), F.f64_to_f16_bits(-0.1), np.uint16)
    assert np.all(F.unpack(packed, bits, k) == 0)
    say("decode_reserved", bits)
    w = _cq().CQWeight(packed, s, a, b, bits, 128, n, k)
    codes, vals = _cq().cq_decode_ref(w)
    assert np.all(codes.cpu().numpy() == 0) and np.all(vals.cpu().numpy() == 0)
    x = torch_dev.ones((1, k), dtype=torch_dev.bfloat16, device="cuda")
    y = _cq().cq_gemm_model_dtype(w, x, y_dtype=torch_dev.float32)
    assert np.all(y.cpu().numpy() == 0)


# ---------------------------------------------------------------- model dtype


@pytest.mark.parametrize("bits", WIDTHS)
@pytest.mark.parametrize("group", GROUPS)
@pytest.mark.parametrize("m", [1, 5, 16])
def test_gemv_model_dtype(torch_dev, bits, group, m):
    r = fitted(2, 72, 768, bits, group)
    xb, xv = act(3 + m, m, 768)
    y_ref = ref_model_dtype(xv, r, bits, group)
    say("gemv_a16", bits, group, m)
    w = _weight(r, bits, group)
    x = _x(torch_dev, xb, "bf16")
    y16 = _cq().cq_gemm_model_dtype(w, x)
    y32 = _cq().cq_gemm_model_dtype(w, x, y_dtype=torch_dev.float32)
    assert R.eps_comp(_np(y16), y_ref, "bf16") <= TOL
    # FP32 output of the FP32-multiply GEMV: rounding-order differences only
    assert R.eps_comp(_np(y32), y_ref, "fp32") <= 1e-5


@pytest.mark.parametrize("bits", [1, 2])
@pytest.mark.parametrize("group", [32, 128, 512])
@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_gemv_w1_w2_direct(torch_dev, bits, group, dtype):
    # W1/W2 single rows take the table-free decode (level pairs in the
    # activation dtype, two-term dot products): both single-row forms, BF16
    # and FP16 activations, 2560 codes (a ragged second column block), 301
    # rows (a lone last row), FP32 and activation-dtype outputs
    n, k = 301, 2560
    r = fitted(640 + bits, n, k, bits, group)
    xb, xv = act(641 + bits, 1, k, dtype)
    y_ref = ref_model_dtype(xv, r, bits, group)
    cq = _cq()
    w = _weight(r, bits, group)
    x = _x(torch_dev, xb, dtype)
    for fam in ("gemv_stream", "gemv_rows"):
        say("gemv w1/w2 direct", bits, group, dtype, fam)
        y32 = cq.cq_gemm_model_dtype_family(w, x, fam, y_dtype=torch_dev.float32)
        assert R.eps_comp(_np(y32), y_ref, "fp32") <= 1e-5, fam
        yd = cq.cq_gemm_model_dtype_family(w, x, fam)
        assert R.eps_comp(_np(yd), y_ref, dtype) <= TOL, fam


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
@pytest.mark.parametrize("m", [1, 16])
def test_gemv_model_dtype_fp16(torch_dev, bits, m):
    r = fitted(4, 40, 512, bits, 128)
    xb, xv = act(5, m, 512, "fp16")
    y_ref = ref_model_dtype(xv, r, bits, 128)
    say("gemv_a16_fp16", bits, m)
    w = _weight(r, bits, 128)
    y = _cq().cq_gemm_model_dtype(w, _x(torch_dev, xb, "fp16"))
    assert y.dtype == torch_dev.float16
    assert R.eps_comp(_np(y), y_ref, "fp16") <= TOL


@pytest.mark.parametrize("bits", WIDTHS)
@pytest.mark.parametrize("group", [32, 128])
@pytest.mark.parametrize("m", [1, 37, 130])
def test_gemm_model_dtype_tiled(torch_dev, bits, group, m):
    cq = _cq()
    r = fitted(6, 136, 768, bits, group)
    xb, xv = act(7 + m, m, 768)
    y_ref = ref_model_dtype(xv, r, bits, group)
    say("gemm_a16", bits, group, m)
    w = _weight(r, bits, group)
    x = _x(torch_dev, xb, "bf16")
    cq.cq_set_gemv_max_rows(0, 0)
    try:
        y = cq.cq_gemm_model_dtype(w, x)
        y32 = cq.cq_gemm_model_dtype(w, x, y_dtype=torch_dev.float32)
    finally:
        cq.cq_set_gemv_max_rows(0, -1)
    assert R.eps_comp(_np(y), y_ref, "bf16") <= TOL
    # bf16 output is the RNE of the fp32 output of the same kernel
    assert np.array_equal(_np(y), _np(y32.to(torch_dev.bfloat16)))


@pytest.mark.parametrize("m", [1, 64])
def test_gemm_model_dtype_fp16_tiled(torch_dev, m):
    cq = _cq()
    r = fitted(8, 72, 512, 4, 128)
    xb, xv = act(9, m, 512, "fp16")
    y_ref = ref_model_dtype(xv, r, 4, 128)
    say("gemm_a16_fp16", m)
    w = _weight(r, 4, 128)
    cq.cq_set_gemv_max_rows(0, 0)
    try:
        y = cq.cq_gemm_model_dtype(w, _x(torch_dev, xb, "fp16"))
    finally:
        cq.cq_set_gemv_max_rows(0, -1)
    assert R.eps_comp(_np(y), y_ref, "fp16") <= TOL


def test_model_dtype_deterministic(torch_dev):
    r = fitted(10, 64, 1024, 4, 128)
    xb, _ = act(11, 3, 1024)
    say("determinism_a16")
    w = _weight(r, 4, 128)
    x = _x(torch_dev, xb, "bf16")
    y1 = _cq().cq_gemm_model_dtype(w, x, y_dtype=torch_dev.float32)
    y2 = _cq().cq_gemm_model_dtype(w, x, y_dtype=torch_dev.float32)
    assert torch_dev.equal(y1, y2)


# ---------------------------------------------------------------- Dynamic A8


@pytest.mark.parametrize("m,k", [(1, 32), (7, 4096), (64, 768), (1, 4096), (1, 14336), (3, 18432), (2, 65568), (1, 139264), (600, 2080)])
@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_quantize_act_a8_bitexact(torch_dev, m, k, dtype):
    xb, xv = act(12 + m, m, k, dtype)
    if m >= 7:
        xv = xv.copy()
        xb = xb.copy()
        xb[1] = 0            # an all-zero row
        xv[1] = 0
    x8_ref, d_ref = A8.quantize_act(xv)
    say("quant_a8", m, k, dtype)
    x8, dx = _cq().cq_quantize_act_a8(_x(torch_dev, xb, dtype))
    assert np.array_equal(x8.cpu().numpy(), x8_ref)
    assert np.array_equal(dx.cpu().numpy().view(np.uint32), d_ref.view(np.uint32))


def test_quantize_act_a8_halfway_cases(torch_dev):
    vals = np.array([[127.0, 2.5, -2.5, 0.5, -0.5, 1.5, 126.5, -127.0] * 4])
    from workloads import to_bf16_bits
    xb = to_bf16_bits(vals)
    x8_ref, _ = A8.quantize_act(vals)
    say("quant_a8_halfway")
    x8, dx = _cq().cq_quantize_act_a8(_x(torch_dev, xb, "bf16"))
    assert dx.item() == 1.0
    assert np.array_equal(x8.cpu().numpy(), x8_ref)


@pytest.mark.parametrize("bits", WIDTHS)
@pytest.mark.parametrize("group", GROUPS)
@pytest.mark.parametrize("m,family", [(1, "gemv"), (16, "gemv"), (3, "gemm"), (70, "gemm")])
def test_gemm_a8_partials_bitexact(torch_dev, bits, group, m, family):
    cq = _cq()
    r = fitted(13, 72, 768, bits, group)
    xb, xv = act(14 + m, m, 768)
    x8_ref, d_ref, y_ref, p_ref = ref_a8(xv, r, bits, group)
    say("gemm_a8", bits, group, m, family)
    w = _weight(r, bits, group)
    x8 = torch_dev.from_numpy(x8_ref).cuda()
    dx = torch_dev.from_numpy(d_ref).cuda()
    if family == "gemm":
        cq.cq_set_gemv_max_rows(1, 0)
    try:
        y, parts = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32, want_partials=True)
        y16 = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.bfloat16)
    finally:
        cq.cq_set_gemv_max_rows(1, -1)
    assert np.array_equal(parts.cpu().numpy(), p_ref)
    assert R.eps_comp(_np(y), y_ref, "fp32") <= 1e-5
    assert R.eps_comp(_np(y16), y_ref, "bf16") <= TOL


def test_a8_carrier_tie_rounds_to_even(torch_dev):
    # W8, a = 2^-7, b = 127/128, code 64: 127 q = 32.5 exactly -> carrier 32
    n, k, g = 16, 128, 128
    codes = np.zeros((n, k), np.int8)
    codes[:, 0] = 64
    codes[:, 1] = -64
    s = np.ones((n, 1), np.float32)
    a = np.full((n, 1), F.f64_to_f16_bits(2.0 ** -7), np.uint16)
    b = np.full((n, 1), F.f64_to_f16_bits(127 / 128), np.uint16)
    x8 = np.zeros((1, k), np.int8)
    x8[0, 0] = 1
    x8[0, 1] = 3
    dx = np.ones(1, np.float32)
    cq = _cq()
    say("a8_tie")
    w = cq.CQWeight.from_codes(codes, s, a, b, 8, g)
    for thr in (-1, 0):
        cq.cq_set_gemv_max_rows(1, thr)
        try:
            _, parts = cq.cq_gemm_a8(w, torch_dev.from_numpy(x8).cuda(), torch_dev.from_numpy(dx).cuda(),
                                     y_dtype=torch_dev.float32, want_partials=True)
        finally:
            cq.cq_set_gemv_max_rows(1, -1)
        assert np.all(parts.cpu().numpy() == 32 * 1 - 32 * 3)


def test_a8_operator_end_to_end(torch_dev):
    # quantizer + GEMM through the device, against the oracle's A8 semantics
    r = fitted(15, 96, 1024, 4, 128)
    xb, xv = act(16, 9, 1024)
    _, _, y_ref, _ = ref_a8(xv, r, 4, 128)
    say("a8_operator")
    w = _weight(r, 4, 128)
    x8, dx = _cq().cq_quantize_act_a8(_x(torch_dev, xb, "bf16"))
    y = _cq().cq_gemm_a8(w, x8, dx)
    assert R.eps_comp(_np(y), y_ref, "bf16") <= TOL


def test_a8_deterministic(torch_dev):
    r = fitted(17, 64, 1024, 5, 64)
    xb, _ = act(18, 33, 1024)
    say("determinism_a8")
    w = _weight(r, 5, 64)
    x8, dx = _cq().cq_quantize_act_a8(_x(torch_dev, xb, "bf16"))
    y1 = _cq().cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32)
    y2 = _cq().cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32)
    assert torch_dev.equal(y1, y2)


# ---------------------------------------------------------------- edge shapes


@pytest.mark.parametrize("n,k,g,m", [(1, 128, 128, 1), (1, 128, 128, 16), (3, 512, 512, 2), (257, 256, 32, 17)])
def test_edge_shapes(torch_dev, n, k, g, m):
    r = fitted(19, n, k, 4, g)
    xb, xv = act(20, m, k)
    y_ref = ref_model_dtype(xv, r, 4, g)
    _, _, ya_ref, p_ref = ref_a8(xv, r, 4, g)
    say("edge", n, k, g, m)
    w = _weight(r, 4, g)
    x = _x(torch_dev, xb, "bf16")
    y = _cq().cq_gemm_model_dtype(w, x)
    assert R.eps_comp(_np(y), y_ref, "bf16") <= TOL
    x8, dx = _cq().cq_quantize_act_a8(x)
    ya, parts = _cq().cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32, want_partials=True)
    assert np.array_equal(parts.cpu().numpy(), p_ref)
    assert R.eps_comp(_np(ya), ya_ref, "fp32") <= 1e-5


# ---------------------------------------------------------------- single-row A8 streaming family


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5, 6, 7, 8])
@pytest.mark.parametrize("group", GROUPS)
@pytest.mark.parametrize("k", [768, 4096 + 2048 + 512])
def test_gemv_a8_stream(torch_dev, bits, group, k):
    # m == 1 without a partials dump takes the streaming kernel (W1..W4 carrier
    # tables in registers, W5..W8 one carrier per weight)
    if k % group:
        pytest.skip("K must be a multiple of G")
    r = fitted(23, 67, k, bits, group)
    xb, xv = act(24, 1, k)
    x8_ref, d_ref, y_ref, _ = ref_a8(xv, r, bits, group)
    say("gemv_a8_stream", bits, group, k)
    w = _weight(r, bits, group)
    x8 = torch_dev.from_numpy(x8_ref).cuda()
    dx = torch_dev.from_numpy(d_ref).cuda()
    y = _cq().cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32)
    y16 = _cq().cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.bfloat16)
    assert R.eps_comp(_np(y), y_ref, "fp32") <= 1e-5
    assert R.eps_comp(_np(y16), y_ref, "bf16") <= TOL


@pytest.mark.parametrize("bits", [3, 4, 5, 6, 7, 8])
@pytest.mark.parametrize("family", ["stream", "gemv", "gemm"])
def test_a8_near_tie_carriers_exact(torch_dev, bits, family):
    # rows whose shapes put a carrier within 3e-4 of a half-integer; with unit
    # scales and d_x = 127 the FP32 output is the exact integer sum of P_g
    codes, s, a, b, x8, dx, p = carrier_probe(bits, 128)
    say("a8_near_tie", bits, family, len(a))
    cq = _cq()
    w = cq.CQWeight.from_codes(codes, s, a, b, bits, 128)
    x8_t = torch_dev.from_numpy(x8).cuda()
    dx_t = torch_dev.from_numpy(dx).cuda()
    if family == "gemm":
        cq.cq_set_gemv_max_rows(1, 0)
    try:
        if family == "stream":
            y = cq.cq_gemm_a8(w, x8_t, dx_t, y_dtype=torch_dev.float32)
        else:
            y, parts = cq.cq_gemm_a8(w, x8_t, dx_t, y_dtype=torch_dev.float32, want_partials=True)
            assert np.array_equal(parts.cpu().numpy(), p)
    finally:
        cq.cq_set_gemv_max_rows(1, -1)
    assert np.array_equal(_np(y).astype(np.float64), p.sum(axis=-1).astype(np.float64))


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("m", [2, 5, 16, 17, 32])
def test_a8_narrow_near_tie_carriers_exact(torch_dev, bits, m):
    # the narrow-row A8 kernel (W3 and W4) on the near-tie rows: the probe's
    # activation row repeated m times, every output row the exact integer sum
    # of the oracle's P_g (unit scales, d_x = 127), bit for bit
    codes, s, a, b, x8, dx, p = carrier_probe(bits, 128)
    say("a8_narrow_near_tie", bits, m, len(a))
    cq = _cq()
    w = cq.CQWeight.from_codes(codes, s, a, b, bits, 128)
    x8_t = torch_dev.from_numpy(np.repeat(x8, m, axis=0)).cuda()
    dx_t = torch_dev.from_numpy(np.repeat(dx, m)).cuda()
    assert cq.cq_family_supported(cq.CQ_PATH_A8, "gemv_narrow", w, m)
    y = _np(cq.cq_gemm_a8_family(w, x8_t, dx_t, "gemv_narrow", y_dtype=torch_dev.float32))
    want = p.sum(axis=-1).astype(np.float64).reshape(1, -1)
    assert np.array_equal(y, np.repeat(want, m, axis=0))


@pytest.mark.parametrize("group", [64, 128, 256, 512])
@pytest.mark.parametrize("m", [2, 7, 16, 19, 32])
def test_gemv_a8_narrow_w3(torch_dev, group, m):
    # W3 narrow-row A8 against the A8 oracle: 300 weight rows (a ragged last
    # strip), K = 2048 + one group (at least 128 codes: W3 rows are whole
    # 16-byte units), fitted weights
    bits, n = 3, 300
    k = 2048 + max(group, 128)
    r = fitted(620 + group, n, k, bits, group)
    xb, xv = act(621 + m, m, k)
    x8_ref, d_ref, y_ref, _ = ref_a8(xv, r, bits, group)
    cq = _cq()
    w = _weight(r, bits, group)
    x8 = torch_dev.from_numpy(x8_ref).cuda()
    dx = torch_dev.from_numpy(d_ref).cuda()
    say("gemv_a8_narrow w3", group, m)
    assert cq.cq_select_query(cq.CQ_PATH_A8, w, m) == "gemv_narrow"
    y = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32)
    assert R.eps_comp(_np(y), y_ref, "fp32") <= 1e-5
    assert R.eps_comp(_np(cq.cq_gemm_a8(w, x8, dx)), y_ref, "bf16") <= TOL


@pytest.mark.parametrize("group", [64, 128, 256, 512])
@pytest.mark.parametrize("m", [17, 24, 32])
def test_gemv_a8_narrow_two_blocks_w4(torch_dev, group, m):
    # W4 narrow-row A8 above 16 rows (two 16-row blocks of x per decoded
    # operand) against the A8 oracle and the 32-row tiled GEMM; 300 weight
    # rows (a ragged last strip), K = 2048 + one group
    bits, n = 4, 300
    k = 2048 + group
    r = fitted(630 + group, n, k, bits, group)
    xb, xv = act(631 + m, m, k)
    x8_ref, d_ref, y_ref, _ = ref_a8(xv, r, bits, group)
    cq = _cq()
    w = _weight(r, bits, group)
    x8 = torch_dev.from_numpy(x8_ref).cuda()
    dx = torch_dev.from_numpy(d_ref).cuda()
    say("gemv_a8_narrow two blocks", group, m)
    assert cq.cq_select_query(cq.CQ_PATH_A8, w, m) == "gemv_narrow"
    y = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32)
    assert R.eps_comp(_np(y), y_ref, "fp32") <= 1e-5
    yt = cq.cq_gemm_a8_family(w, x8, dx, "gemm_mfma_m32", y_dtype=torch_dev.float32)
    assert R.eps_comp(_np(yt), y_ref, "fp32") <= 1e-5


# ---------------------------------------------------------------- many-row matrix-core GEMMs


@pytest.mark.parametrize("bits,group", [(4, 64), (4, 128), (4, 512), (3, 128)])
@pytest.mark.parametrize("m,n", [(300, 600), (129, 257)])
def test_gemm_multi_tile(torch_dev, bits, group, m, n):
    # several row and column tiles with ragged edges; A8 partials bit-exact
    k = 1024
    r = fitted(31, n, k, bits, group)
    xb, xv = act(32, m, k)
    x8_ref, d_ref, ya_ref, p_ref = ref_a8(xv, r, bits, group)
    y_ref = ref_model_dtype(xv, r, bits, group)
    say("gemm_multi_tile", bits, group, m, n)
    cq = _cq()
    w = _weight(r, bits, group)
    x8 = torch_dev.from_numpy(x8_ref).cuda()
    dx = torch_dev.from_numpy(d_ref).cuda()
    ya, parts = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32, want_partials=True)
    assert np.array_equal(parts.cpu().numpy(), p_ref)
    assert R.eps_comp(_np(ya), ya_ref, "fp32") <= 1e-5
    ya16 = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.bfloat16)
    assert R.eps_comp(_np(ya16), ya_ref, "bf16") <= TOL
    ya32 = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32)
    assert torch_dev.equal(ya32, ya)
    y = cq.cq_gemm_model_dtype(w, _x(torch_dev, xb, "bf16"))
    assert R.eps_comp(_np(y), y_ref, "bf16") <= TOL


# ---------------------------------------------------------------- narrow rows (2 <= m <= 16), matrix cores


@pytest.mark.parametrize("group", [64, 128, 256, 512])
@pytest.mark.parametrize("m", [2, 7, 16])
def test_narrow_rows_both_paths(torch_dev, group, m):
    # 75 weight rows (ragged 16-row strip), K = 2560: group counts not a
    # multiple of the four waves that share a strip
    k = 2560 if 2560 % group == 0 else 2048
    r = fitted(41, 75, k, 4, group)
    xb, xv = act(42 + m, m, k)
    x8_ref, d_ref, ya_ref, _ = ref_a8(xv, r, 4, group)
    y_ref = ref_model_dtype(xv, r, 4, group)
    say("narrow", group, m, k)
    cq = _cq()
    w = _weight(r, 4, group)
    x8 = torch_dev.from_numpy(x8_ref).cuda()
    dx = torch_dev.from_numpy(d_ref).cuda()
    ya = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32)
    assert R.eps_comp(_np(ya), ya_ref, "fp32") <= 1e-5
    for dtype in ("bf16", "fp16"):
        xb2, xv2 = act(42 + m, m, k, dtype)
        y2_ref = ref_model_dtype(xv2, r, 4, group)
        y = cq.cq_gemm_model_dtype(w, _x(torch_dev, xb2, dtype), y_dtype=torch_dev.float32)
        assert R.eps_comp(_np(y), y2_ref, "fp32") <= 2e-4
        y16 = cq.cq_gemm_model_dtype(w, _x(torch_dev, xb2, dtype))
        assert R.eps_comp(_np(y16), y2_ref, dtype) <= TOL


# ---------------------------------------------------------------- fused single-row A8


@pytest.fixture
def single_launch():
    # cq_gemm_a8_fused as one launch for a single row (the default is two)
    cq = _cq()
    cq.cq_set_a8_fused_launch(1)
    yield
    cq.cq_set_a8_fused_launch(0)


def test_gemm_a8_fused_default_is_two_calls(torch_dev):
    # by default the fused call runs the quantizer and the product: its outputs
    # equal the two calls' bit for bit
    cq = _cq()
    assert cq.cq_get_a8_fused_launch() == 0
    bits, group, k = 4, 128, 4096
    r = fitted(50, 37, k, bits, group)
    w = _weight(r, bits, group)
    xb, xv = act(49, 1, k)
    x = _x(torch_dev, xb, "bf16")
    y, x8, dx = cq.cq_gemm_a8_fused(w, x, y_dtype=torch_dev.float32)
    x8b, dxb = cq.cq_quantize_act_a8(x)
    assert torch_dev.equal(x8, x8b) and torch_dev.equal(dx, dxb)
    assert torch_dev.equal(y, cq.cq_gemm_a8(w, x8b, dxb, y_dtype=torch_dev.float32))


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
@pytest.mark.parametrize("group", [32, 128, 512])
@pytest.mark.parametrize("k", [512, 2048, 4096, 4096 + 2048 + 512, 14336, 16384])
def test_gemm_a8_fused_single_row(torch_dev, single_launch, bits, group, k):
    # m == 1: one launch that quantizes its own activations (one to eight
    # column blocks, the last one ragged for K = 6656); carriers and d_x are
    # compared bit for bit, y against the A8 oracle
    if k % group:
        pytest.skip("K must be a multiple of G")
    r = fitted(51, 37, k, bits, group)
    cq = _cq()
    w = _weight(r, bits, group)
    for dtype in ("bf16", "fp16"):
        xb, xv = act(52, 1, k, dtype)
        x8_ref, d_ref, y_ref, _ = ref_a8(xv, r, bits, group)
        say("gemm_a8_fused", bits, group, k, dtype)
        x = _x(torch_dev, xb, dtype)
        y, x8, dx = cq.cq_gemm_a8_fused(w, x, y_dtype=torch_dev.float32)
        assert np.array_equal(x8.cpu().numpy(), x8_ref)
        assert np.array_equal(dx.cpu().numpy(), d_ref.astype(np.float32))
        assert R.eps_comp(_np(y), y_ref, "fp32") <= 1e-5
        y16, _, _ = cq.cq_gemm_a8_fused(w, x)
        assert R.eps_comp(_np(y16), y_ref, dtype) <= TOL
        # the two-call path on the same row: same carriers, y equal to rounding
        y2 = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32)
        assert R.eps_comp(_np(y), _np(y2).astype(np.float64), "fp32") <= 1e-6


@pytest.mark.parametrize("case", ["rows3", "w6", "k18432", "zero_row", "gemv_rows_0"])
def test_gemm_a8_fused_fallbacks(torch_dev, single_launch, case):
    # with the single launch enabled, shapes it does not take run the two
    # calls; an all-zero row gives d_x = eps / 127, zero carriers and a zero
    # output
    cq = _cq()
    bits, group, k, m, n = 4, 128, 2048, 1, 21
    if case == "rows3":
        m = 3
    elif case == "w6":
        bits = 6
    elif case == "k18432":
        k = 18432
    r = fitted(61, n, k, bits, group)
    xb, xv = act(62, m, k)
    if case == "zero_row":
        xb = np.zeros_like(xb)
        xv = np.zeros_like(xv)
    x8_ref, d_ref, y_ref, _ = ref_a8(xv, r, bits, group)
    say("gemm_a8_fused fallback", case)
    w = _weight(r, bits, group)
    if case == "gemv_rows_0":
        cq.cq_set_gemv_max_rows(1, 0)
    try:
        y, x8, dx = cq.cq_gemm_a8_fused(w, _x(torch_dev, xb, "bf16"), y_dtype=torch_dev.float32)
    finally:
        cq.cq_set_gemv_max_rows(1, -1)
    assert np.array_equal(x8.cpu().numpy(), x8_ref)
    assert np.array_equal(dx.cpu().numpy(), d_ref.astype(np.float32))
    if case == "zero_row":
        assert np.all(y.cpu().numpy() == 0)
        assert dx.cpu().numpy()[0] == np.float32(np.float32(1e-10) / np.float32(127))
    else:
        assert R.eps_comp(_np(y), y_ref, "fp32") <= 1e-5


def _all_values(dtype):
    """Every finite non-negative value of the activation dtype (float64)."""
    if dtype == "bf16":
        return (np.arange(0, 0x7F80, dtype=np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float64)


def _encode(vals, dtype):
    from workloads import to_bf16_bits, to_f16_bits
    return to_bf16_bits(vals) if dtype == "bf16" else to_f16_bits(vals)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_gemm_a8_fused_carriers_near_rounding_boundaries(torch_dev, single_launch, dtype):
    # the single-row call forms carriers from x * (1/d) and divides only near
    # a rounding boundary; for 24 random row scales, every representable
    # activation whose quotient lies within 2^-15 of a half-integer (plus a
    # random sample of the others), both signs, must give the oracle's
    # IEEE-division carriers; at xbar = 127 (d = 1) every half-integer is an
    # exact tie, and there the whole value range is checked
    from workloads import synthetic_representation
    allv = _all_values(dtype)
    rng = np.random.default_rng(81)
    k = 4096
    codes, s, a, b = synthetic_representation(72, 5, k, 4, 128)
    w = _cq().CQWeight.from_codes(codes, s, a, b, 4, 128)
    cands = allv[(allv >= 0.01) & (allv <= 1000.0)]
    rows = []
    for amax in rng.choice(cands, 24, replace=False):
        d = np.float64(np.float32(np.float32(amax) / np.float32(127.0)))
        v = allv[allv <= amax]
        f = np.abs(np.abs(v / d - np.round(v / d)) - 0.5)
        pick = np.concatenate([v[f < 2.0 ** -15], rng.choice(v, 800)])
        rows.append((amax, pick))
    top = allv[allv <= 127.0]
    for i in range(0, len(top), 2000):
        rows.append((127.0, top[i:i + 2000]))
    hits = 0
    batch = []
    for amax, pick in rows:
        row = np.zeros((1, k))
        vals = np.concatenate([pick, -pick])[:k - 1]
        row[0, 0] = amax
        row[0, 1:1 + len(vals)] = vals
        x8_ref, d_ref = A8.quantize_act(row)
        q = row / np.float64(d_ref[0])
        hits += int(np.sum(np.abs(np.abs(q - np.round(q)) - 0.5) < 2.0 ** -15))
        say("fused boundary", dtype, amax, len(vals))
        xt = _x(torch_dev, _encode(row, dtype), dtype)
        _, x8, dx = _cq().cq_gemm_a8_fused(w, xt, y_dtype=torch_dev.float32)
        assert np.array_equal(dx.cpu().numpy(), d_ref.astype(np.float32))
        assert np.array_equal(x8.cpu().numpy(), x8_ref), (dtype, amax)
        # the standalone quantizer takes the same reciprocal path
        x8q, dxq = _cq().cq_quantize_act_a8(xt)
        assert np.array_equal(dxq.cpu().numpy(), d_ref.astype(np.float32))
        assert np.array_equal(x8q.cpu().numpy(), x8_ref), (dtype, amax)
        batch.append(row[0])
    assert hits >= 48
    # many rows at once (the 256-thread configuration), rows repeated to 600
    rows_np = np.stack(batch)
    rows_np = np.concatenate([rows_np] * (600 // len(rows_np) + 1))[:600]
    x8_ref, d_ref = A8.quantize_act(rows_np)
    say("quantizer boundary batch", dtype, rows_np.shape)
    x8q, dxq = _cq().cq_quantize_act_a8(_x(torch_dev, _encode(rows_np, dtype), dtype))
    assert np.array_equal(dxq.cpu().numpy(), d_ref.astype(np.float32))
    assert np.array_equal(x8q.cpu().numpy(), x8_ref)


# ---------------------------------------------------------------- routed (mixture-of-experts) product


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("group", [32, 128])
@pytest.mark.parametrize("experts,tokens", [(1, 5), (3, 40), (8, 1), (8, 4), (8, 16)])
def test_routed_model_dtype(torch_dev, bits, group, experts, tokens):
    # route-major outputs for a skewed top-2 route map (top-1 with one expert);
    # 37 rows per expert (ragged strip, odd: route rows start at odd offsets),
    # experts with more than 16 routes run several chunks; at most one route
    # per two experts (8 experts, 1 token) takes the streaming mode; the
    # grouped mode runs the staged slab (G B <= 512) or the narrow kernel
    # (W5 G128); every route against the oracle
    from oracle import routed as RT
    from workloads import route_map, synthetic_representation
    n, k = 37, 1024
    codes, s, a, b = synthetic_representation(90 + bits, experts * n, k, bits, group)
    cq = _cq()
    bank = cq.CQWeight.from_codes(codes, s, a, b, bits, group)
    tok, exp = route_map(91 + tokens, tokens, experts, 1 if experts == 1 else 2)
    tt = torch_dev.from_numpy(tok).cuda()
    te = torch_dev.from_numpy(exp).cuda()
    for dtype in ("bf16", "fp16"):
        xb, xv = act(92, tokens, k, dtype)
        y_ref = RT.routed_model_dtype(xv, tok, exp, codes, bits, group, s, a, b, experts)
        say("routed", bits, group, experts, tokens, dtype)
        x = _x(torch_dev, xb, dtype)
        y = cq.cq_gemm_routed_model_dtype(bank, experts, x, tt, te, y_dtype=torch_dev.float32)
        assert R.eps_comp(_np(y), y_ref, "fp32") <= 2e-4
        y16 = cq.cq_gemm_routed_model_dtype(bank, experts, x, tt, te)
        assert R.eps_comp(_np(y16), y_ref, dtype) <= TOL
        y2 = cq.cq_gemm_routed_model_dtype(bank, experts, x, tt, te, y_dtype=torch_dev.float32)
        assert torch_dev.equal(y, y2)


@pytest.mark.parametrize("experts", [4, 16])
def test_routed_invalid_routes_untouched(torch_dev, experts):
    # routes naming a missing token or expert are dropped; their rows keep
    # the caller's contents, the others match the oracle (7 routes: grouped
    # mode with 4 experts, streaming mode with 16)
    from oracle import routed as RT
    from workloads import synthetic_representation
    bits, group, n, k, tokens = 4, 128, 20, 512, 6
    codes, s, a, b = synthetic_representation(95, experts * n, k, bits, group)
    cq = _cq()
    bank = cq.CQWeight.from_codes(codes, s, a, b, bits, group)
    tok = np.array([0, 5, 6, -1, 2, 3, 1], np.int32)
    exp = np.array([1, 3, 0, 2, 4, -3, 0], np.int32)
    xb, xv = act(96, tokens, k)
    y_ref = RT.routed_model_dtype(xv, tok, exp, codes, bits, group, s, a, b, experts)
    say("routed invalid")
    y = torch_dev.full((len(tok), n), 7.0, dtype=torch_dev.float32, device="cuda")
    cq.cq_gemm_routed_model_dtype(bank, experts, _x(torch_dev, xb, "bf16"), torch_dev.from_numpy(tok).cuda(),
                                  torch_dev.from_numpy(exp).cuda(), out=y)
    got = _np(y)
    valid = np.isfinite(y_ref[:, 0])
    assert list(valid) == [True, True, False, False, experts > 4, False, True]
    assert np.all(got[~valid] == 7.0)
    assert R.eps_comp(got[valid], y_ref[valid], "fp32") <= 2e-4


# ---------------------------------------------------------------- load-time carrier tables


@pytest.mark.parametrize("bits", [2, 3, 4, 5, 6, 7, 8])
def test_build_carriers_exact(torch_dev, bits):
    # every (row, group) entry against the oracle's exact table, on fitted
    # weights and on shapes searched to sit next to a carrier tie
    from tests._cases import near_tie_shapes
    r = fitted(101, 24, 1024, bits, 128)
    a_bits, b_bits = r.a_bits.copy(), r.b_bits.copy()
    if bits >= 3:
        ties = near_tie_shapes(bits, count=16)
        for i, (a, b) in enumerate(ties):
            a_bits.flat[i] = a
            b_bits.flat[i] = b
    cq = _cq()
    w = cq.CQWeight.from_codes(r.codes, r.scale, a_bits, b_bits, bits, 128)
    say("build_carriers", bits)
    tab = cq.cq_build_carriers(w).cpu().numpy()
    assert tab.shape == (24, 8, 1 << (bits - 1))
    cache = {}
    for row in range(24):
        for g in range(8):
            key = (int(a_bits[row, g]), int(b_bits[row, g]))
            if key not in cache:
                cache[key] = A8.carrier_table(bits, *key)
            assert list(tab[row, g].astype(np.int64)) == cache[key], (row, g)


@pytest.mark.parametrize("bits", WIDTHS)
@pytest.mark.parametrize("group", [32, 128, 256])
@pytest.mark.parametrize("m", [1, 5, 16, 70, 300])
def test_gemm_a8_carriers_equals_gemm_a8(torch_dev, bits, group, m):
    # the table-fed product is the same computation: bit-equal to cq_gemm_a8
    # on every family, and within the A8 bar of the oracle
    r = fitted(102, 67, 1024, bits, group)
    xb, xv = act(103 + m, m, 1024)
    x8_ref, d_ref, y_ref, _ = ref_a8(xv, r, bits, group)
    cq = _cq()
    w = _weight(r, bits, group)
    x8 = torch_dev.from_numpy(x8_ref).cuda()
    dx = torch_dev.from_numpy(d_ref).cuda()
    say("gemm_a8_carriers", bits, group, m)
    tab = cq.cq_build_carriers(w)
    y = cq.cq_gemm_a8_carriers(w, tab, x8, dx, y_dtype=torch_dev.float32)
    y0 = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32)
    assert torch_dev.equal(y, y0)
    assert R.eps_comp(_np(y), y_ref, "fp32") <= 1e-5
    y16 = cq.cq_gemm_a8_carriers(w, tab, x8, dx)
    assert R.eps_comp(_np(y16), y_ref, "bf16") <= TOL


# ---------------------------------------------------------------- kernel families and the selection table

MD_FAMILIES = ("gemv_stream", "gemv_rows", "gemv_lut", "gemv_narrow", "gemv_generic", "gemm_slab", "gemm_slab_staged", "gemm_mfma",
               "gemm_mfma_m32",
               "gemm_mfma_m64", "gemm_mfma_m128", "gemm_mfma_m256", "gemm_tiled", "gemm_mfma_rounded")
A8_FAMILIES = ("gemv_stream", "gemv_narrow", "gemv_generic", "gemm_mfma", "gemm_mfma_m32", "gemm_mfma_m64",
               "gemm_mfma_m128", "gemm_mfma_m256", "gemm_tiled")


@pytest.mark.parametrize("bits,group", [(4, 128), (3, 64), (6, 32), (2, 256)])
@pytest.mark.parametrize("m", [1, 3, 8, 24])
def test_every_family_matches_oracle(torch_dev, bits, group, m):
    # every admissible family of both paths computes the oracle's product; the
    # matrix-core model-dtype families carry the level as a BF16 hi + lo pair
    # (16 significant bits), hence 2e-4 on their FP32 output; the rounded
    # family rounds every weight once to BF16 (relative error <= 2^-8) and is
    # held to that rounding's own elementwise bound
    n, k = 131, 1024
    r = fitted(140 + bits, n, k, bits, group)
    xb, xv = act(141, m, k)
    y16_ref = ref_model_dtype(xv, r, bits, group)
    x8_ref, d_ref, y8_ref, _ = ref_a8(xv, r, bits, group)
    cq = _cq()
    w = _weight(r, bits, group)
    x = _x(torch_dev, xb, "bf16")
    x8 = torch_dev.from_numpy(x8_ref).cuda()
    dx = torch_dev.from_numpy(d_ref).cuda()
    ran = 0
    for f in MD_FAMILIES:
        if not cq.cq_family_supported(cq.CQ_PATH_MODEL_DTYPE, f, w, m):
            with pytest.raises(cq.CQError):
                cq.cq_gemm_model_dtype_family(w, x, f)
            continue
        say("family model dtype", f, bits, group, m)
        y = cq.cq_gemm_model_dtype_family(w, x, f, y_dtype=torch_dev.float32)
        if f == "gemm_mfma_rounded":
            wabs = np.abs(F.decode(r.codes, bits, group, r.scale, r.a_bits, r.b_bits))
            bound = 2.0 ** -8 * (np.abs(xv) @ wabs.T) * (1 + 2e-3) + 1e-6 * np.max(np.abs(y16_ref))
            assert np.all(np.abs(_np(y).astype(np.float64) - y16_ref) <= bound), f
            ran += 1
            continue
        assert R.eps_comp(_np(y), y16_ref, "fp32") <= 2e-4, f
        assert R.eps_comp(_np(cq.cq_gemm_model_dtype_family(w, x, f)), y16_ref, "bf16") <= TOL, f
        ran += 1
    for f in A8_FAMILIES:
        if not cq.cq_family_supported(cq.CQ_PATH_A8, f, w, m):
            continue
        say("family a8", f, bits, group, m)
        y = cq.cq_gemm_a8_family(w, x8, dx, f, y_dtype=torch_dev.float32)
        assert R.eps_comp(_np(y), y8_ref, "fp32") <= 1e-5, f
        ran += 1
    assert ran >= 2


# ---------------------------------------------------------------- x-tile heights of the matrix-core GEMM

@pytest.mark.parametrize("m", [5, 17, 40, 64, 100, 129, 300])
def test_gemm_tile_heights_bit_equal(torch_dev, m):
    # every x-tile height runs the same FP32 accumulation chain per output:
    # the fixed-height families are bit-equal to each other and to the oracle
    # within the dense-path bar
    cq = _cq()
    n, k, bits, group = 300, 1024, 4, 128
    r = fitted(340, n, k, bits, group)
    w = _weight(r, bits, group)
    xb, xv = act(341 + m, m, k)
    x = _x(torch_dev, xb, "bf16")
    y_ref = ref_model_dtype(xv, r, bits, group)
    outs = []
    for f in ("gemm_mfma_m32", "gemm_mfma_m64", "gemm_mfma_m128", "gemm_mfma_m256", "gemm_mfma"):
        say("tile height", f, m)
        outs.append(cq.cq_gemm_model_dtype_family(w, x, f, y_dtype=torch_dev.float32))
    for o in outs[1:]:
        assert torch_dev.equal(o, outs[0])
    assert R.eps_comp(_np(outs[0]), y_ref, "fp32") <= 2e-4


# ---------------------------------------------------------------- few-row GEMM with lane-decoded operands


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("group,k", [(32, 640), (64, 640), (128, 640), (256, 1280), (512, 2560)])
@pytest.mark.parametrize("m", [1, 7, 17, 32])
def test_gemm_slab(torch_dev, bits, group, k, m):
    # five groups per row (a last sweep with one group of four), 83 weight rows
    # (a ragged 16-row block), one and two x-row blocks; FP32 and BF16 outputs
    n = 83
    r = fitted(360 + bits, n, k, bits, group)
    w = _weight(r, bits, group)
    xb, xv = act(361 + m, m, k)
    y_ref = ref_model_dtype(xv, r, bits, group)
    cq = _cq()
    x = _x(torch_dev, xb, "bf16")
    say("gemm_slab", bits, group, k, m)
    y = cq.cq_gemm_model_dtype_family(w, x, "gemm_slab", y_dtype=torch_dev.float32)
    assert R.eps_comp(_np(y), y_ref, "fp32") <= 2e-4
    y16 = cq.cq_gemm_model_dtype_family(w, x, "gemm_slab")
    assert R.eps_comp(_np(y16), y_ref, "bf16") <= TOL


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("group,k", [(32, 1024), (64, 1024), (128, 2048)])
@pytest.mark.parametrize("m", [1, 7, 12, 16, 21, 32])
def test_gemm_slab_staged(torch_dev, bits, group, k, m):
    # codes and metadata staged through LDS: 83 weight rows (ragged block),
    # four or more sweeps; W5 stages groups of up to 64 codes
    n = 83
    cq = _cq()
    r = fitted(380 + bits, n, k, bits, group)
    w = _weight(r, bits, group)
    if not cq.cq_family_supported(cq.CQ_PATH_MODEL_DTYPE, "gemm_slab_staged", w, m):
        assert bits == 5 and group == 128
        return
    xb, xv = act(381 + m, m, k)
    y_ref = ref_model_dtype(xv, r, bits, group)
    x = _x(torch_dev, xb, "bf16")
    say("gemm_slab_staged", bits, group, k, m)
    y = cq.cq_gemm_model_dtype_family(w, x, "gemm_slab_staged", y_dtype=torch_dev.float32)
    assert R.eps_comp(_np(y), y_ref, "fp32") <= 2e-4
    y16 = cq.cq_gemm_model_dtype_family(w, x, "gemm_slab_staged")
    assert R.eps_comp(_np(y16), y_ref, "bf16") <= TOL


@pytest.mark.parametrize("bits,group,k,m", [(4, 32, 4096, 5), (4, 128, 8192, 16), (3, 64, 8192, 2),
                                             (4, 128, 8192, 24), (3, 64, 8192, 32), (5, 64, 4096, 19)])
def test_gemm_slab_staged_many_sweeps(torch_dev, bits, group, k, m):
    # 8200 weight rows (513 row blocks, few waves per block): every wave walks
    # several sweeps and crosses metadata batches; sampled output columns
    # against the oracle, both families against each other
    from workloads import synthetic_representation
    n = 8200
    cq = _cq()
    codes, sc, a, b = synthetic_representation(390 + bits, n, k, bits, group)
    w = cq.CQWeight.from_codes(codes, sc, a, b, bits, group)
    xb, xv = act(391 + m, m, k)
    x = _x(torch_dev, xb, "bf16")
    say("gemm_slab_staged many sweeps", bits, group, k, m)
    y = _np(cq.cq_gemm_model_dtype_family(w, x, "gemm_slab_staged", y_dtype=torch_dev.float32))
    y1 = _np(cq.cq_gemm_model_dtype_family(w, x, "gemm_slab", y_dtype=torch_dev.float32))
    rows = np.sort(np.random.default_rng(392).choice(n, size=48, replace=False))
    rows = np.concatenate([rows, [0, 15, 16, n - 8, n - 1]])
    y_ref = R.gemm_model_dtype(xv, codes[rows], bits, group, sc[rows], a[rows], b[rows])
    assert R.eps_comp(y[:, rows], y_ref, "fp32") <= 2e-4
    assert R.eps_comp(y1[:, rows], y_ref, "fp32") <= 2e-4
    assert np.max(np.abs(y - y1)) <= 1e-4 * np.max(np.abs(y1))


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5, 6, 7, 8])
@pytest.mark.parametrize("group", [32, 128, 512])
def test_gemv_rows(torch_dev, bits, group):
    # resident-activation single-row GEMV: 4608 codes per row are 2.25 column
    # blocks (three waves, the last one partly past the row), 1601 rows are
    # 801 row pairs (the last one single), walked in batches of four tiles by
    # each workgroup; every row against the oracle, and against the streaming
    # family (the same products summed in another order)
    from workloads import synthetic_representation
    n, k = 1601, 4608
    cq = _cq()
    codes, sc, a, b = synthetic_representation(600 + bits, n, k, bits, group)
    w = cq.CQWeight.from_codes(codes, sc, a, b, bits, group)
    xb, xv = act(601 + bits, 1, k)
    x = _x(torch_dev, xb, "bf16")
    say("gemv_rows", bits, group)
    y = _np(cq.cq_gemm_model_dtype_family(w, x, "gemv_rows", y_dtype=torch_dev.float32))
    y_ref = R.gemm_model_dtype(xv, codes, bits, group, sc, a, b)
    assert R.eps_comp(y, y_ref, "fp32") <= 2e-4
    assert R.eps_comp(_np(cq.cq_gemm_model_dtype_family(w, x, "gemv_rows")), y_ref, "bf16") <= TOL
    ys = _np(cq.cq_gemm_model_dtype_family(w, x, "gemv_stream", y_dtype=torch_dev.float32))
    assert np.max(np.abs(y - ys)) <= 1e-5 * np.max(np.abs(ys))


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_gemv_rows_many_tiles(torch_dev, dtype):
    # 20001 rows over 7168 codes (3.5 column blocks): each workgroup walks
    # about twelve row tiles, three batches, the last partly filled; sampled
    # rows against the oracle, every row against the streaming family
    from workloads import synthetic_representation
    n, k, bits, group = 20001, 7168, 4, 128
    cq = _cq()
    codes, sc, a, b = synthetic_representation(610, n, k, bits, group)
    w = cq.CQWeight.from_codes(codes, sc, a, b, bits, group)
    xb, xv = act(611, 1, k, dtype)
    x = _x(torch_dev, xb, dtype)
    say("gemv_rows many tiles", dtype)
    assert cq.cq_select_query(cq.CQ_PATH_MODEL_DTYPE, w, 1) == "gemv_rows"
    y = _np(cq.cq_gemm_model_dtype(w, x, y_dtype=torch_dev.float32))
    rows = np.sort(np.random.default_rng(612).choice(n, size=64, replace=False))
    rows = np.concatenate([rows, [0, 1, 2, 3, n - 2, n - 1]])
    y_ref = R.gemm_model_dtype(xv, codes[rows], bits, group, sc[rows], a[rows], b[rows])
    assert R.eps_comp(y[:, rows], y_ref, "fp32") <= 2e-4
    ys = _np(cq.cq_gemm_model_dtype_family(w, x, "gemv_stream", y_dtype=torch_dev.float32))
    assert np.max(np.abs(y - ys)) <= 1e-5 * np.max(np.abs(ys))
    y16 = _np(cq.cq_gemm_model_dtype(w, x))
    assert R.eps_comp(y16[:, rows], y_ref, dtype) <= TOL


@pytest.mark.parametrize("n,k,m", [(40, 8192, 5), (300, 4096, 32), (16, 1024, 1), (1024, 4096, 16), (72, 8192, 23)])
def test_gemm_slab_split_k_and_fp16(torch_dev, n, k, m):
    # few weight rows over long K: up to 16 waves per workgroup split K and
    # meet in LDS; FP16 activations carry the weight as an FP16 hi + lo pair
    bits, group = 4, 128
    r = fitted(370, n, k, bits, group)
    w = _weight(r, bits, group)
    cq = _cq()
    for dtype in ("bf16", "fp16"):
        xb, xv = act(371 + m, m, k, dtype)
        y_ref = ref_model_dtype(xv, r, bits, group)
        say("gemm_slab split-k", n, k, m, dtype)
        y = cq.cq_gemm_model_dtype_family(w, _x(torch_dev, xb, dtype), "gemm_slab", y_dtype=torch_dev.float32)
        assert R.eps_comp(_np(y), y_ref, "fp32") <= 2e-4
        y16 = cq.cq_gemm_model_dtype_family(w, _x(torch_dev, xb, dtype), "gemm_slab")
        assert R.eps_comp(_np(y16), y_ref, dtype) <= TOL
        y2 = cq.cq_gemm_model_dtype_family(w, _x(torch_dev, xb, dtype), "gemm_slab", y_dtype=torch_dev.float32)
        assert torch_dev.equal(y, y2)
        # the staged variant (two x-row blocks per wave above 16 rows)
        ys = cq.cq_gemm_model_dtype_family(w, _x(torch_dev, xb, dtype), "gemm_slab_staged", y_dtype=torch_dev.float32)
        assert R.eps_comp(_np(ys), y_ref, "fp32") <= 2e-4


@pytest.mark.parametrize("bits,group", [(4, 128), (3, 64), (4, 512), (3, 256)])
@pytest.mark.parametrize("m", [3, 17, 40, 64, 100, 129, 300])
def test_gemm_a8_tile_heights_bit_equal(torch_dev, bits, group, m):
    # A8: every x-tile height rescales the exact INT32 group partials; heights
    # whose workgroups run one K range (128 and 256 rows) add the rescaled
    # groups in group order and are bit-equal, the 32- and 64-row tiles split
    # K over two or four groups of waves whose FP32 sums meet at the end; all
    # meet the A8 oracle within 1e-5, and the load-time carrier tables change
    # nothing for the same height
    cq = _cq()
    n, k = 300, 2048
    r = fitted(350 + bits, n, k, bits, group)
    w = _weight(r, bits, group)
    xb, xv = act(351 + m, m, k)
    x8_ref, d_ref, y8_ref, _ = ref_a8(xv, r, bits, group)
    x8 = torch_dev.from_numpy(x8_ref).cuda()
    dx = torch_dev.from_numpy(d_ref).cuda()
    outs = {}
    for f in ("gemm_mfma_m32", "gemm_mfma_m64", "gemm_mfma_m128", "gemm_mfma_m256", "gemm_mfma"):
        say("a8 tile height", f, bits, group, m)
        outs[f] = cq.cq_gemm_a8_family(w, x8, dx, f, y_dtype=torch_dev.float32)
        assert R.eps_comp(_np(outs[f]), y8_ref, "fp32") <= 1e-5, f
        assert torch_dev.equal(cq.cq_gemm_a8_family(w, x8, dx, f, y_dtype=torch_dev.float32), outs[f])
    assert torch_dev.equal(outs["gemm_mfma_m128"], outs["gemm_mfma_m256"])
    tab = cq.cq_build_carriers(w)
    # the table call runs the built-in rules' kernel (above 16 rows: the
    # narrow-row kernel up to 32, the tiled GEMM beyond) and equals cq_gemm_a8
    auto = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32)
    assert torch_dev.equal(cq.cq_gemm_a8_carriers(w, tab, x8, dx, y_dtype=torch_dev.float32), auto) or m <= 16
    if m > 32:
        assert torch_dev.equal(auto, outs["gemm_mfma"])


def test_selection_table_drives_dispatch(torch_dev):
    # with a table installed the ordinary calls run the named family: their
    # outputs equal the forced-family call bit for bit; clearing restores the
    # built-in rules
    cq = _cq()
    n, k, bits, group = 300, 2048, 4, 128
    r = fitted(150, n, k, bits, group)
    w = _weight(r, bits, group)
    md, a8 = cq.CQ_PATH_MODEL_DTYPE, cq.CQ_PATH_A8
    table = [{"path": md, "family": "gemv_generic", "bits": bits, "group": group, "n": n, "k": k, "m_lo": 1,
              "m_hi": 4, "x_dtype": cq.CQ_BF16},
             {"path": md, "family": "gemm_tiled", "bits": bits, "group": group, "n": n, "k": k, "m_lo": 5,
              "m_hi": 100},
             {"path": a8, "family": "gemm_tiled", "bits": bits, "group": group, "n": n, "k": k, "m_lo": 1,
              "m_hi": 100}]
    try:
        for m in (1, 3, 40):
            xb, _ = act(151 + m, m, k)
            x = _x(torch_dev, xb, "bf16")
            x8, dx = cq.cq_quantize_act_a8(x)
            say("selection table", m)
            cq.cq_select_set([])
            base_md = cq.cq_select_query(md, w, m)
            y_default = cq.cq_gemm_model_dtype(w, x, y_dtype=torch_dev.float32)
            assert torch_dev.equal(y_default, cq.cq_gemm_model_dtype_family(w, x, base_md, y_dtype=torch_dev.float32))
            cq.cq_select_set(table)
            f_md = cq.cq_select_query(md, w, m)
            assert f_md == ("gemv_generic" if m <= 4 else "gemm_tiled")
            y = cq.cq_gemm_model_dtype(w, x, y_dtype=torch_dev.float32)
            assert torch_dev.equal(y, cq.cq_gemm_model_dtype_family(w, x, f_md, y_dtype=torch_dev.float32))
            assert cq.cq_select_query(a8, w, m) == "gemm_tiled"
            y8 = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32)
            assert torch_dev.equal(y8, cq.cq_gemm_a8_family(w, x8, dx, "gemm_tiled", y_dtype=torch_dev.float32))
            # the partials dump keeps the built-in rules and the same product
            y8p, parts = cq.cq_gemm_a8(w, x8, dx, y_dtype=torch_dev.float32, want_partials=True)
            assert torch_dev.allclose(y8p, y8, rtol=1e-5, atol=1e-6)
            # fp16 activations do not match the bf16-only entry for m <= 4
            assert cq.cq_select_query(md, w, m, cq.CQ_FP16) == ("gemm_tiled" if m > 4 else base_md)
    finally:
        cq.cq_select_set([])
    assert cq.cq_select_query(md, w, 1) == "gemv_stream"


def test_tuner_selects_valid_families(torch_dev):
    # the measured selection on a small shape: every timed family agreed with
    # the built-in choice, the winner at each row count is the fastest one, the
    # regimes cover every row count, and installing the table makes the
    # dispatcher follow it
    cq = _cq()
    from paper_2608_06763_amd import selection as S
    n, k, bits, group = 512, 2048, 4, 128
    r = fitted(160, n, k, bits, group)
    w = _weight(r, bits, group)
    ms = [1, 3, 24]
    try:
        tables = []
        for path in (cq.CQ_PATH_MODEL_DTYPE, cq.CQ_PATH_A8):
            say("tuner", path)
            t = S.tune(w, path, ms, target_ms=0.5, max_calls=8)
            assert not t["rejected"]
            for m in ms:
                assert t["choice"][m] == min(t["timings"][m], key=t["timings"][m].get)
                assert len(t["timings"][m]) >= 2
            e = t["entries"]
            assert e[0]["m_lo"] == 1 and e[-1]["m_hi"] == S.M_MAX
            assert all(a["m_hi"] + 1 == b["m_lo"] for a, b in zip(e[:-1], e[1:]))
            tables.append(t)
        S.install(tables)
        for t in tables:
            path = t["signature"]["path"]
            for m in ms:
                assert cq.cq_select_query(path, w, m) == t["choice"][m]
    finally:
        S.clear()


def test_probe_read_reads_without_writing(torch_dev):
    # the HBM read probe of the benchmark: completes on odd sizes and leaves
    # its sink untouched for real data
    cq = _cq()
    sink = torch_dev.zeros((4,), dtype=torch_dev.int32, device="cuda")
    for n in (4, 1000, 1 << 20):
        buf = torch_dev.ones((n,), dtype=torch_dev.float32, device="cuda")
        say("probe_read", n)
        cq.cq_probe_read(buf, sink)
    torch_dev.cuda.synchronize()
    assert int(sink.abs().sum()) == 0
