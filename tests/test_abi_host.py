"""Host-side checks of the C ABI (no GPU needed).

The library must load and export every function ``include/*.h`` declares;
``cq_pack_groups`` must equal the oracle's packer byte for byte and reject
every invalid input the format forbids; device entry points must reject bad
arguments on the host before touching a device.
"""
import ctypes
import time
import os
import re

import numpy as np
import pytest

import paper_2608_06763_amd as cq
from oracle import fit as FIT
from oracle import format as F
from workloads import small_weight

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
HEADERS = sorted(os.path.join(INCLUDE, f) for f in os.listdir(INCLUDE) if f.endswith(".h"))


def declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(cq_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 8
    L = cq.lib()
    for name in names:
        assert hasattr(L, name), name
    assert set(names) == set(cq.EXPORTS)


def test_status_strings():
    L = cq.lib()
    for s in range(9):
        assert L.cq_status_str(s).decode().startswith(cq.STATUS[s])


@pytest.mark.parametrize("bits", range(1, 9))
@pytest.mark.parametrize("group", [8, 16, 32, 64, 128, 256])
def test_pack_matches_oracle(bits, group):
    if (group * bits) % 8:
        pytest.skip("G*B not byte aligned")
    rng = np.random.default_rng(bits * 1000 + group)
    n, k = 5, group * 3
    codes = rng.choice(F.valid_codes(bits), size=(n, k)).astype(np.int8)
    s = rng.uniform(0.1, 1.0, (n, k // group)).astype(np.float32)
    a = np.full((n, k // group), F.f64_to_f16_bits(0.8), np.uint16)
    b = np.full((n, k // group), F.f64_to_f16_bits(-0.2), np.uint16)
    assert np.array_equal(cq.cq_pack_groups(codes, s, a, b, bits, group), F.pack(codes, bits))


def test_pack_fitted_weights_matches_oracle():
    w = small_weight(5, 16, 512, "laplace")
    for bits in (2, 3, 4, 5, 8):
        r = FIT.fit(w, bits, 128)
        got = cq.cq_pack_groups(r.codes, r.scale, r.a_bits, r.b_bits, bits, 128)
        assert np.array_equal(got, F.pack(r.codes, bits))


def _meta(n, ng, a=1.0, b=0.0, s=1.0):
    return (np.full((n, ng), s, np.float32), np.full((n, ng), F.f64_to_f16_bits(a), np.uint16),
            np.full((n, ng), F.f64_to_f16_bits(b), np.uint16))


def _pack_err(codes, s, a, b, bits, group):
    with pytest.raises(cq.CQError) as ei:
        cq.cq_pack_groups(codes, s, a, b, bits, group)
    return ei.value


def test_pack_rejects_out_of_range_codes():
    codes = np.zeros((2, 64), np.int8)
    codes[1, 5] = -8  # reserved pattern at W4
    e = _pack_err(codes, *_meta(2, 2), 4, 32)
    assert e.status == 5 and e.bad_index == 64 + 5
    codes[1, 5] = 8
    assert _pack_err(codes, *_meta(2, 2), 4, 32).status == 5
    w1 = np.ones((1, 32), np.int8)
    w1[0, 3] = 0  # W1 has no zero code
    e = _pack_err(w1, *_meta(1, 1), 1, 32)
    assert e.status == 5 and e.bad_index == 3


def test_pack_rejects_bad_metadata():
    codes = np.ones((1, 64), np.int8)
    s, a, b = _meta(1, 2, a=2.0, b=0.0)  # q'(1) = -1: not monotone
    e = _pack_err(codes, s, a, b, 4, 32)
    assert e.status == 4 and e.bad_index == 0
    s, a, b = _meta(1, 2, a=0.0, b=0.0)  # q = t^3: closure, not strict
    assert _pack_err(codes, s, a, b, 3, 32).status == 4
    s, a, b = _meta(1, 2)
    s[0, 1] = np.nan
    e = _pack_err(codes, s, a, b, 4, 32)
    assert e.status == 4 and e.bad_index == 1
    s, a, b = _meta(1, 2)
    s[0, 0] = -1.0
    assert _pack_err(codes, s, a, b, 4, 32).status == 4
    s, a, b = _meta(1, 2)
    s[0, 0] = 0.0  # zero scale with nonzero codes
    assert _pack_err(codes, s, a, b, 4, 32).status == 4
    s, a, b = _meta(1, 2)
    a[0, 0] = 0x7C00  # +inf fp16
    assert _pack_err(codes, s, a, b, 4, 32).status == 4
    # non-monotone shapes are irrelevant at W2 (no interior level)
    s, a, b = _meta(1, 2, a=2.0, b=0.0)
    cq.cq_pack_groups(codes, s, a, b, 2, 32)


def test_pack_zero_group_with_zero_scale_is_valid():
    codes = np.zeros((1, 64), np.int8)
    s, a, b = _meta(1, 2, s=0.0)
    assert np.all(cq.cq_pack_groups(codes, s, a, b, 4, 32) == 0)


def test_pack_rejects_bad_shapes():
    codes = np.zeros((1, 60), np.int8)
    assert _pack_err(codes, *_meta(1, 2), 4, 32).status == 2     # K % G
    codes = np.zeros((1, 12), np.int8)
    assert _pack_err(codes, *_meta(1, 3), 3, 4).status == 2      # G*B % 8
    L = cq.lib()
    z = np.zeros(4, np.uint8)
    p = z.ctypes.data_as(ctypes.c_void_p)
    assert L.cq_pack_groups(9, 32, 1, 32, p, p, p, p, p, None) == 1
    assert L.cq_pack_groups(4, 32, 1, 32, None, p, p, p, p, None) == 1


def _desc(bits=4, group=128, n=64, k=256, ptr=4096):
    return cq.cq_weight(bits, group, n, k, ptr, ptr, ptr, ptr)


def test_device_calls_validate_on_host():
    # every case below must be rejected before any device work is issued
    L = cq.lib()
    P = ctypes.c_void_p
    ok = 4096
    bad_align = 4100
    w = _desc()
    cases = [
        (_desc(bits=0), 1), (_desc(bits=9), 1), (_desc(group=48), 1), (_desc(group=1024), 1),
        (_desc(group=16), 1), (_desc(k=320), 2), (_desc(bits=3, group=32, k=96), 2),
        (_desc(n=0), 1), (_desc(ptr=bad_align), 3),
    ]
    for d, want in cases:
        assert L.cq_gemm_model_dtype(ctypes.byref(d), P(ok), 0, 1, P(ok), 0, None) == want
        assert L.cq_gemm_a8(ctypes.byref(d), P(ok), P(ok), 1, P(ok), 0, None, None) == want
        assert L.cq_decode_ref(ctypes.byref(d), P(ok), None, None) == want
        assert L.cq_gemm_a8_fused(ctypes.byref(d), P(ok), 0, 1, P(ok), P(ok), P(ok), 0, None) == want
    assert L.cq_gemm_model_dtype(None, P(ok), 0, 1, P(ok), 0, None) == 1
    assert L.cq_gemm_model_dtype(ctypes.byref(w), P(ok), 0, 0, P(ok), 0, None) == 1        # m = 0
    assert L.cq_gemm_model_dtype(ctypes.byref(w), P(ok), 2, 1, P(ok), 2, None) == 6        # fp32 x
    assert L.cq_gemm_model_dtype(ctypes.byref(w), P(ok), 0, 1, P(ok), 1, None) == 6        # bf16 -> fp16
    assert L.cq_gemm_model_dtype(ctypes.byref(w), P(bad_align), 0, 1, P(ok), 0, None) == 3
    assert L.cq_gemm_a8(ctypes.byref(w), P(ok), P(ok), 1, P(ok), 7, None, None) == 6
    assert L.cq_gemm_a8(ctypes.byref(w), P(ok), P(ok), 1, P(ok), 0, P(bad_align), None) == 3
    assert L.cq_decode_ref(ctypes.byref(w), None, None, None) == 1
    fused = L.cq_gemm_a8_fused
    assert fused(ctypes.byref(w), None, 0, 1, P(ok), P(ok), P(ok), 0, None) == 1            # no x
    assert fused(ctypes.byref(w), P(ok), 0, 1, None, P(ok), P(ok), 0, None) == 1            # no x8
    assert fused(ctypes.byref(w), P(ok), 0, 0, P(ok), P(ok), P(ok), 0, None) == 1           # m = 0
    assert fused(ctypes.byref(w), P(ok), 2, 1, P(ok), P(ok), P(ok), 0, None) == 6           # fp32 x
    assert fused(ctypes.byref(w), P(ok), 0, 1, P(ok), P(ok), P(ok), 7, None) == 6           # bad y dtype
    assert fused(ctypes.byref(w), P(ok), 0, 1, P(ok), P(bad_align), P(ok), 0, None) == 3
    assert L.cq_quantize_act_a8(P(ok), 0, 1, 48, P(ok), P(ok), None) == 2                 # k % 32
    assert L.cq_quantize_act_a8(P(ok), 2, 1, 64, P(ok), P(ok), None) == 6
    assert L.cq_quantize_act_a8(P(ok), 0, 0, 64, P(ok), P(ok), None) == 1
    assert L.cq_quantize_act_a8(P(ok), 0, 1, 64, P(bad_align), P(ok), None) == 3


def test_gemv_threshold_override():
    assert cq.cq_get_gemv_max_rows(0) >= 1
    cq.cq_set_gemv_max_rows(0, 0)
    assert cq.cq_get_gemv_max_rows(0) == 0
    cq.cq_set_gemv_max_rows(0, -1)
    assert cq.cq_get_gemv_max_rows(0) >= 1
    with pytest.raises(cq.CQError):
        cq.cq_set_gemv_max_rows(2, 1)


def test_routed_argument_errors_need_no_gpu():
    # every argument check of the routed entry returns before any device work
    L = cq.lib()
    P = ctypes.c_void_p
    ok, bad_align = 4096, 4100
    w = _desc()
    f = L.cq_gemm_routed_model_dtype
    assert f(ctypes.byref(_desc(bits=0)), 2, P(ok), 0, 4, P(ok), P(ok), 8, P(ok), P(ok), 0, None) == 1
    assert f(ctypes.byref(w), 0, P(ok), 0, 4, P(ok), P(ok), 8, P(ok), P(ok), 0, None) == 1      # no experts
    assert f(ctypes.byref(w), 2, P(ok), 0, 0, P(ok), P(ok), 8, P(ok), P(ok), 0, None) == 1      # no tokens
    assert f(ctypes.byref(w), 2, P(ok), 0, 4, None, P(ok), 8, P(ok), P(ok), 0, None) == 1       # no route map
    assert f(ctypes.byref(w), 2, P(ok), 0, 4, P(ok), P(ok), 8, None, P(ok), 0, None) == 1       # no workspace
    assert f(ctypes.byref(w), 2, P(ok), 2, 4, P(ok), P(ok), 8, P(ok), P(ok), 2, None) == 6      # fp32 x
    assert f(ctypes.byref(w), 2, P(ok), 0, 4, P(ok), P(ok), 8, P(ok), P(ok), 1, None) == 6      # bf16 -> fp16
    assert f(ctypes.byref(w), 2, P(bad_align), 0, 4, P(ok), P(ok), 8, P(ok), P(ok), 0, None) == 3
    assert f(ctypes.byref(w), 2, P(ok), 0, 4, P(ok + 2), P(ok), 8, P(ok), P(ok), 0, None) == 3  # int32 alignment
    assert f(ctypes.byref(_desc(bits=6)), 2, P(ok), 0, 4, P(ok), P(ok), 8, P(ok), P(ok), 0, None) == 8
    assert f(ctypes.byref(w), 2, P(ok), 0, 4, P(ok), P(ok), 0, P(ok), P(ok), 0, None) == 0      # no routes


def test_carrier_table_argument_errors_need_no_gpu():
    L = cq.lib()
    P = ctypes.c_void_p
    ok, bad_align = 4096, 4100
    w = _desc()
    assert L.cq_build_carriers(ctypes.byref(_desc(bits=0)), P(ok), None) == 1
    assert L.cq_build_carriers(ctypes.byref(w), None, None) == 1
    assert L.cq_build_carriers(ctypes.byref(w), P(bad_align), None) == 3
    assert L.cq_build_carriers(ctypes.byref(_desc(bits=1)), None, None) == 0        # W1: no table
    f = L.cq_gemm_a8_carriers
    assert f(ctypes.byref(w), None, P(ok), P(ok), 1, P(ok), 0, None) == 1            # W4 needs a table
    assert f(ctypes.byref(w), P(ok), None, P(ok), 1, P(ok), 0, None) == 1
    assert f(ctypes.byref(w), P(ok), P(ok), P(ok), 0, P(ok), 0, None) == 1           # m = 0
    assert f(ctypes.byref(w), P(ok), P(ok), P(ok), 1, P(ok), 7, None) == 6
    assert f(ctypes.byref(w), P(bad_align), P(ok), P(ok), 1, P(ok), 0, None) == 3
    assert f(ctypes.byref(_desc(group=48)), P(ok), P(ok), P(ok), 1, P(ok), 0, None) == 1


# ---------------------------------------------------------------- kernel selection (host logic only)


def _fake(bits, group, n, k):
    # descriptor with aligned placeholder addresses: the selection calls read
    # only its fields
    return cq.cq_weight(bits, group, n, k, 256, 512, 768, 1024)


@pytest.fixture
def clean_table():
    cq.cq_select_set([])
    yield
    cq.cq_select_set([])
    cq.cq_set_gemv_max_rows(0, -1)
    cq.cq_set_gemv_max_rows(1, -1)


@pytest.mark.parametrize("bits,group,m,md,a8", [
    (4, 128, 1, "gemv_stream", "gemv_stream"),
    (4, 128, 3, "gemm_slab", "gemv_narrow"),
    (4, 256, 3, "gemm_slab", "gemv_narrow"),
    (4, 128, 8, "gemm_slab", "gemv_narrow"),
    (4, 32, 8, "gemm_slab_staged", "gemv_generic"),
    (3, 128, 1, "gemv_stream", "gemv_stream"),
    (3, 128, 8, "gemm_slab", "gemv_narrow"),
    (6, 128, 1, "gemv_stream", "gemv_stream"),
    (6, 128, 8, "gemv_generic", "gemv_generic"),
    (4, 128, 17, "gemm_slab", "gemv_narrow"),
    (4, 128, 32, "gemm_slab_staged", "gemv_narrow"),
    (4, 128, 33, "gemm_mfma", "gemm_mfma"),
    (4, 128, 4, "gemm_slab", "gemv_narrow"),
    (3, 64, 300, "gemm_mfma", "gemm_mfma"),
    (3, 32, 300, "gemm_mfma", "gemm_tiled"),
    (6, 128, 300, "gemm_tiled", "gemm_tiled"),
])
def test_builtin_rules(clean_table, bits, group, m, md, a8):
    d = _fake(bits, group, 4096, 4096)
    assert cq.cq_select_query(cq.CQ_PATH_MODEL_DTYPE, d, m) == md
    assert cq.cq_select_query(cq.CQ_PATH_A8, d, m) == a8
    assert cq.cq_family_supported(cq.CQ_PATH_MODEL_DTYPE, md, d, m)
    assert cq.cq_family_supported(cq.CQ_PATH_A8, a8, d, m)


@pytest.mark.parametrize("n,k,m,want", [
    (28672, 8192, 4, "gemm_slab_staged"), (28672, 4096, 16, "gemm_slab_staged"), (4096, 14336, 2, "gemm_slab_staged"),
    (6144, 4096, 4, "gemm_slab"), (4096, 4096, 8, "gemm_slab"), (28672, 8192, 1, "gemv_rows"),
    (4096, 14336, 1, "gemv_rows"), (6144, 4096, 1, "gemv_stream"),
    (28672, 8192, 24, "gemm_slab_staged"), (4096, 4096, 17, "gemm_slab"), (6144, 4096, 21, "gemm_slab_staged"), (6144, 4096, 17, "gemm_slab_staged"), (6144, 4096, 24, "gemm_slab_staged"), (4096, 4096, 24, "gemm_slab"),
    (4096, 4096, 32, "gemm_slab_staged"),
    (4096, 14336, 17, "gemm_slab_staged"),
    (28672, 8192, 33, "gemm_mfma")])
def test_builtin_slab_variant(clean_table, n, k, m, want):
    # the staged variant when every wave of the K split gets two sweeps
    assert cq.cq_select_query(cq.CQ_PATH_MODEL_DTYPE, _fake(4, 128, n, k), m) == want


def test_a8_fused_launch_knob():
    assert cq.cq_get_a8_fused_launch() == 0
    cq.cq_set_a8_fused_launch(1)
    assert cq.cq_get_a8_fused_launch() == 1
    cq.cq_set_a8_fused_launch(0)
    assert cq.cq_get_a8_fused_launch() == 0
    assert cq.lib().cq_set_a8_fused_launch(2) == 1 and cq.cq_get_a8_fused_launch() == 0


def test_builtin_rules_follow_gemv_threshold(clean_table):
    d = _fake(4, 128, 4096, 4096)
    cq.cq_set_gemv_max_rows(0, 0)
    assert cq.cq_select_query(cq.CQ_PATH_MODEL_DTYPE, d, 1) == "gemm_mfma"
    assert cq.cq_select_query(cq.CQ_PATH_MODEL_DTYPE, _fake(4, 128, 28672, 4096), 24) == "gemm_slab_staged"
    assert cq.cq_select_query(cq.CQ_PATH_A8, d, 1) == "gemv_stream"


def test_family_predicates():
    d = _fake(4, 128, 4096, 4096)
    md, a8 = cq.CQ_PATH_MODEL_DTYPE, cq.CQ_PATH_A8
    assert not cq.cq_family_supported(md, "gemv_stream", d, 2)
    assert not cq.cq_family_supported(md, "gemv_lut", d, 5)
    assert not cq.cq_family_supported(md, "gemv_narrow", d, 1)
    assert not cq.cq_family_supported(md, "gemv_generic", d, 17)
    assert cq.cq_family_supported(md, "gemm_tiled", d, 1)
    assert cq.cq_family_supported(md, "gemm_mfma", d, 1)
    assert cq.cq_family_supported(md, "gemm_mfma_rounded", d, 1)
    assert not cq.cq_family_supported(a8, "gemm_mfma_rounded", d, 300)
    assert cq.cq_family_supported(md, "gemm_slab", d, 1) and cq.cq_family_supported(md, "gemm_slab", d, 32)
    assert not cq.cq_family_supported(md, "gemm_slab", d, 33)
    assert not cq.cq_family_supported(a8, "gemm_slab", d, 8)
    assert cq.cq_family_supported(md, "gemm_slab_staged", d, 16)
    assert cq.cq_family_supported(md, "gemm_slab_staged", d, 32)
    assert not cq.cq_family_supported(md, "gemm_slab_staged", d, 33)
    assert not cq.cq_family_supported(md, "gemm_slab_staged", _fake(4, 256, 4096, 4096), 2)
    assert not cq.cq_family_supported(md, "gemm_slab_staged", _fake(4, 128, 4096, 640), 2)
    assert not cq.cq_family_supported(a8, "gemm_slab_staged", d, 8)
    assert cq.cq_family_supported(md, "gemv_rows", d, 1)
    assert not cq.cq_family_supported(md, "gemv_rows", d, 2)
    assert not cq.cq_family_supported(a8, "gemv_rows", d, 1)
    assert cq.cq_family_supported(md, "gemv_rows", _fake(4, 128, 4096, 14336), 1)
    assert not cq.cq_family_supported(md, "gemv_rows", _fake(4, 128, 4096, 18432), 1)  # nine column blocks
    assert not cq.cq_family_supported(md, "gemv_rows", _fake(5, 128, 4096, 16384), 1)  # tables above 64 KB
    assert cq.cq_family_supported(md, "gemv_rows", _fake(6, 128, 4096, 16384), 1)
    assert not cq.cq_family_supported(a8, "gemv_lut", d, 2)
    assert not cq.cq_family_supported(a8, "auto", d, 2)
    assert not cq.cq_family_supported(7, "gemm_tiled", d, 2)
    # 32-bit buffer offsets: the streaming and matrix-core families stop below 2 GiB
    big = _fake(8, 128, 1 << 18, 8192)
    assert not cq.cq_family_supported(md, "gemv_stream", big, 1)
    assert not cq.cq_family_supported(md, "gemm_mfma", big, 64)
    assert cq.cq_family_supported(md, "gemv_generic", big, 1)
    assert cq.cq_family_supported(md, "gemm_tiled", big, 64)


def _entry(**kw):
    e = {"path": 0, "family": "gemv_generic", "bits": 4, "group": 128, "n": 4096, "k": 4096, "m_lo": 1,
         "m_hi": 16, "x_dtype": -1}
    e.update(kw)
    return e


def test_table_overrides_and_falls_back(clean_table):
    d = _fake(4, 128, 4096, 4096)
    other = _fake(4, 128, 4096, 8192)
    cq.cq_select_set([_entry(m_lo=1, m_hi=4, family="gemv_generic"),
                      _entry(m_lo=5, m_hi=1000, family="gemm_tiled"),
                      _entry(path=1, m_lo=1, m_hi=1, family="gemm_mfma"),
                      # narrow cannot take one row: the built-in rules decide there
                      _entry(path=1, m_lo=2, m_hi=8, family="gemv_generic"),
                      _entry(path=1, m_lo=9, m_hi=16, family="gemv_narrow", group=32)])
    md, a8 = cq.CQ_PATH_MODEL_DTYPE, cq.CQ_PATH_A8
    assert cq.cq_select_query(md, d, 1) == "gemv_generic"
    assert cq.cq_select_query(md, d, 4) == "gemv_generic"
    assert cq.cq_select_query(md, d, 5) == "gemm_tiled"
    assert cq.cq_select_query(md, d, 1000) == "gemm_tiled"
    assert cq.cq_select_query(md, d, 1001) == "gemm_mfma"
    assert cq.cq_select_query(md, other, 1) == "gemv_stream"
    assert cq.cq_select_query(a8, d, 1) == "gemm_mfma"
    assert cq.cq_select_query(a8, d, 8) == "gemv_generic"
    assert cq.cq_select_query(a8, d, 12) == "gemv_narrow"
    # an entry whose family cannot take the call is skipped
    cq.cq_select_set([_entry(m_lo=1, m_hi=16, family="gemv_narrow")])
    assert cq.cq_select_query(md, d, 1) == "gemv_stream"
    assert cq.cq_select_query(md, d, 2) == "gemv_narrow"
    cq.cq_select_set([])
    assert cq.cq_select_query(md, d, 4) == "gemm_slab"


def test_table_matches_activation_dtype(clean_table):
    d = _fake(4, 128, 4096, 4096)
    cq.cq_select_set([_entry(x_dtype=cq.CQ_FP16, family="gemv_generic")])
    assert cq.cq_select_query(0, d, 1, cq.CQ_FP16) == "gemv_generic"
    assert cq.cq_select_query(0, d, 1, cq.CQ_BF16) == "gemv_stream"


@pytest.mark.parametrize("bad", [
    dict(path=2), dict(family="auto"), dict(family=15), dict(path=1, family="gemv_lut"),
    dict(path=1, family="gemm_mfma_rounded"), dict(path=1, family="gemm_slab"),
    dict(path=1, family="gemm_slab_staged"), dict(bits=0),
    dict(bits=9), dict(group=48), dict(group=1024), dict(n=0), dict(k=0), dict(m_lo=0), dict(m_lo=5, m_hi=4),
    dict(x_dtype=2), dict(path=1, x_dtype=0)])
def test_table_rejects_malformed_entries(clean_table, bad):
    d = _fake(4, 128, 4096, 4096)
    cq.cq_select_set([_entry(family="gemv_generic")])
    with pytest.raises(cq.CQError) as e:
        cq.cq_select_set([_entry(m_lo=20, m_hi=30, family="gemm_tiled"), _entry(**bad)])
    assert e.value.status == 1
    # the previous table stays
    assert cq.cq_select_query(0, d, 1) == "gemv_generic"


def test_table_rejects_overlaps_and_reserved(clean_table):
    with pytest.raises(cq.CQError):
        cq.cq_select_set([_entry(m_lo=1, m_hi=8), _entry(m_lo=8, m_hi=9, family="gemm_tiled")])
    with pytest.raises(cq.CQError):
        cq.cq_select_set([_entry(x_dtype=-1), _entry(x_dtype=cq.CQ_BF16)])
    # different dtypes, shapes or paths do not overlap
    cq.cq_select_set([_entry(x_dtype=cq.CQ_FP16), _entry(x_dtype=cq.CQ_BF16), _entry(k=8192), _entry(path=1)])
    L = cq.lib()
    arr = (cq.cq_select_entry * 1)()
    arr[0] = cq.cq_select_entry(0, 4, 4, 128, 4096, 4096, 1, 2, -1, 1)
    assert L.cq_select_set(arr, 1) == 1
    assert L.cq_select_set(None, 1) == 1
    assert L.cq_select_set(arr, -1) == 1
    assert L.cq_select_set(arr, 65537) == 1


def test_table_large_and_shuffled(clean_table):
    # 4096 shapes x 4 row ranges given in shuffled order: installed in one
    # sort, each call finds its own shape's entry
    rng = np.random.default_rng(7)
    fams = ["gemv_generic", "gemm_tiled", "gemm_mfma", "gemv_narrow"]
    ranges = [(1, 4), (5, 16), (17, 256), (257, 1 << 40)]
    entries = [_entry(n=64 * (i + 1), m_lo=lo, m_hi=hi, family=fams[(i + j) % 4])
               for i in range(4096) for j, (lo, hi) in enumerate(ranges)]
    order = rng.permutation(len(entries))
    t0 = time.perf_counter()
    cq.cq_select_set([entries[i] for i in order])
    assert time.perf_counter() - t0 < 5.0
    for i in (0, 1, 777, 4095):
        d = _fake(4, 128, 64 * (i + 1), 4096)
        for j, (lo, hi) in enumerate(ranges):
            want = fams[(i + j) % 4]
            got = cq.cq_select_query(cq.CQ_PATH_MODEL_DTYPE, d, lo)
            if cq.cq_family_supported(cq.CQ_PATH_MODEL_DTYPE, want, d, lo):
                assert got == want, (i, j)
    # one overlapping pair anywhere in a large table is found
    bad = [entries[i] for i in order] + [_entry(n=64 * 3000, m_lo=16, m_hi=16, family="gemm_tiled")]
    with pytest.raises(cq.CQError):
        cq.cq_select_set(bad)


def test_table_dtype_classes_in_sorted_order(clean_table):
    # bf16-only and fp16-only entries never meet; a wildcard meets both
    cq.cq_select_set([_entry(x_dtype=cq.CQ_BF16, m_lo=1, m_hi=4), _entry(x_dtype=-1, m_lo=5, m_hi=8),
                      _entry(x_dtype=cq.CQ_FP16, m_lo=1, m_hi=4)])
    cq.cq_select_set([_entry(x_dtype=cq.CQ_BF16, m_lo=1, m_hi=4), _entry(x_dtype=cq.CQ_FP16, m_lo=3, m_hi=6)])
    for pair in ([_entry(x_dtype=-1, m_lo=1, m_hi=4), _entry(x_dtype=cq.CQ_FP16, m_lo=4, m_hi=6)],
                 [_entry(x_dtype=cq.CQ_BF16, m_lo=6, m_hi=9), _entry(x_dtype=cq.CQ_FP16, m_lo=1, m_hi=2),
                  _entry(x_dtype=-1, m_lo=3, m_hi=6)]):
        with pytest.raises(cq.CQError):
            cq.cq_select_set(pair)


def test_forced_family_errors_need_no_gpu():
    d = _fake(4, 128, 4096, 4096)
    L = cq.lib()
    buf = 4096
    # unsupported family for the shape: rejected before any launch
    assert L.cq_gemm_model_dtype_family(ctypes.byref(d), buf, 0, 2, buf, 0, cq.FAMILIES["gemv_stream"], None) == 8
    assert L.cq_gemm_a8_family(ctypes.byref(d), buf, buf, 2, buf, 0, cq.FAMILIES["gemv_lut"], None) == 8
    assert L.cq_gemm_a8_family(ctypes.byref(d), buf, buf, 1, buf, 0, 99, None) == 8
    # argument checks come first
    assert L.cq_gemm_model_dtype_family(ctypes.byref(d), None, 0, 2, buf, 0, 6, None) == 1
    assert L.cq_gemm_model_dtype_family(ctypes.byref(d), buf, 2, 2, buf, 2, 6, None) == 6
    assert L.cq_gemm_a8_family(ctypes.byref(d), buf + 4, buf, 2, buf, 0, 6, None) == 3
    out = ctypes.c_int32(-1)
    assert L.cq_select_query(3, ctypes.byref(d), 0, 1, ctypes.byref(out)) == 1
    assert L.cq_select_query(0, ctypes.byref(d), 2, 1, ctypes.byref(out)) == 6
    assert L.cq_select_query(0, ctypes.byref(d), 0, 0, ctypes.byref(out)) == 1
    assert L.cq_family_supported(0, 1, None, 1) == 0


def test_probe_read_argument_errors_need_no_gpu():
    L = cq.lib()
    assert L.cq_probe_read(None, 16, 4096, None) == 1
    assert L.cq_probe_read(4096, 16, None, None) == 1
    assert L.cq_probe_read(4096, 17, 4096, None) == 1
    assert L.cq_probe_read(4096, -16, 4096, None) == 1
    assert L.cq_probe_read(4104, 16, 4096, None) == 3
    assert L.cq_probe_read(4096, 16, 4098, None) == 3
