"""The no-allocation routed call against the ordinary routed call (GPU).

Both run the same kernels; the no-allocation entry point takes the expert
grouping's scratch from the library's per-device array instead of a caller
workspace.  Two calls in a row, the second smaller (the array keeps the first
call's contents), must each equal the ordinary call bit for bit and the
oracle within the routed product's bars; a request beyond the scratch limit
is refused before any launch.
"""
import ctypes

import numpy as np
import pytest

from oracle import ref as R
from oracle import routed as RT
from tests._cases import act, fitted, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2608_06763_amd as cq
    cq.lib()
    return torch


def _bank(cq, experts, n, k, bits, group):
    fits = [fitted(600 + e, n, k, bits, group) for e in range(experts)]
    cat = lambda f: np.concatenate([getattr(r, f) for r in fits], axis=0)
    codes, s, a, b = cat("codes"), cat("scale"), cat("a_bits"), cat("b_bits")
    return cq.CQWeight.from_codes(codes, s, a, b, bits, group), (codes, s, a, b)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_noalloc_routed_matches_workspace_call(torch_dev, dtype):
    import paper_2608_06763_amd as cq
    torch = torch_dev
    experts, n, k, bits, group = 6, 48, 512, 4, 128
    bank, (codes, s, a, b) = _bank(cq, experts, n, k, bits, group)
    rng = np.random.default_rng(7)
    # first a larger route map, then a smaller one: both group (routes > experts)
    for tokens, routes in ((30, 57), (9, 14)):
        tok = rng.integers(0, tokens, routes).astype(np.int32)
        exp = rng.integers(0, experts, routes).astype(np.int32)
        tok[3] = tokens + 5  # a dropped route: its row stays unwritten
        xb, xv = act(610 + tokens, tokens, k, dtype)
        x = torch.from_numpy(xb.view(np.int16)).cuda().view(torch.bfloat16 if dtype == "bf16" else torch.float16)
        tt, te = torch.from_numpy(tok).cuda(), torch.from_numpy(exp).cuda()
        say("noalloc routed", dtype, tokens, routes)
        y_ws = torch.full((routes, n), float("nan"), dtype=torch.float32, device="cuda")
        y_na = torch.full((routes, n), float("nan"), dtype=torch.float32, device="cuda")
        cq.cq_gemm_routed_model_dtype(bank, experts, x, tt, te, out=y_ws)
        cq.cq_gemm_routed_model_dtype_noalloc(bank, experts, x, tt, te, out=y_na)
        torch.cuda.synchronize()
        assert torch.equal(torch.nan_to_num(y_ws, nan=-7.0), torch.nan_to_num(y_na, nan=-7.0))
        assert bool(torch.isnan(y_na[3]).all())
        y_ref = RT.routed_model_dtype(xv, tok, exp, codes, bits, group, s, a, b, experts)
        ok = ~np.isnan(y_ref[:, 0])
        assert R.eps_comp(y_na.cpu().numpy()[ok], y_ref[ok], "fp32") <= 2e-4
        y16 = cq.cq_gemm_routed_model_dtype_noalloc(bank, experts, x, tt, te)
        assert R.eps_comp(y16.float().cpu().numpy()[ok], y_ref[ok], dtype) <= 2e-3


def test_noalloc_routed_refuses_beyond_scratch(torch_dev):
    import paper_2608_06763_amd as cq
    torch = torch_dev
    bank, _ = _bank(cq, 2, 48, 512, 4, 128)
    n = 48
    x = torch.zeros((4, 512), dtype=torch.bfloat16, device="cuda")
    big = (1 << 20)  # n_experts + 1 + routes > 2^20
    tt = torch.zeros((big,), dtype=torch.int32, device="cuda")
    y = torch.empty((big, n), dtype=torch.bfloat16, device="cuda")
    desc = cq.cq_weight(4, 128, n, 512, bank.codes.data_ptr(), bank.scale.data_ptr(), bank.a.data_ptr(),
                        bank.b.data_ptr())
    st = cq.lib().cq_gemm_routed_model_dtype_noalloc(ctypes.byref(desc), 2, x.data_ptr(), cq.CQ_BF16, 4,
                                                     tt.data_ptr(), tt.data_ptr(), big, y.data_ptr(), cq.CQ_BF16, None)
    assert st == 2  # CQ_ERR_SHAPE, nothing launched
