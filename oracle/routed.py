"""Routed (mixture-of-experts) product, plain definition.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Sec. 5.5 (workload regimes and routed execution): a routed operator applies,
for every active route r = (token t_r, matrix e_r) of a route map supplied
by the serving system, the packed matrix e_r to activation row t_r, with one
output row per route (route-major).  Grouping routes by matrix, compacting
them or reducing them are kernel organisations; they change neither the
reconstruction nor the result of a route.  Routing weights and expert choice
are the serving system's and are not applied here.

The oracle evaluates every route with the model-dtype product of Sec. 5.3
(``ref.gemm_model_dtype``) on the expert's rows of the bank, in float64.
Routes whose token or expert lies outside the inputs have no output row here
(NaN), matching the library, which leaves those rows unwritten.
"""
from __future__ import annotations

import numpy as np

from .ref import gemm_model_dtype


def routed_model_dtype(x, route_token, route_expert, codes, bits: int, group: int, scale, a_bits, b_bits,
                       n_experts: int) -> np.ndarray:
    """y[r] = x[t_r] W_{e_r}^T in float64; the bank holds n_experts matrices of
    equal shape stacked along the rows (expert e owns rows e n .. e n + n - 1)."""
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    tokens = x.shape[0]
    n = codes.shape[0] // n_experts
    route_token = np.asarray(route_token, dtype=np.int64)
    route_expert = np.asarray(route_expert, dtype=np.int64)
    y = np.full((len(route_token), n), np.nan)
    for r, (t, e) in enumerate(zip(route_token, route_expert)):
        if not (0 <= t < tokens and 0 <= e < n_experts):
            continue
        rows = slice(e * n, (e + 1) * n)
        y[r] = gemm_model_dtype(x[t:t + 1], codes[rows], bits, group, scale[rows], a_bits[rows], b_bits[rows])[0]
    return y
