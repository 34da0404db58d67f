"""The allocation-free entry point wam_cosine_similarity_noalloc (partial sums in the
library's static device scratch) against wam_cosine_similarity with a caller workspace:
the same kernels and summation order, so the results agree bit for bit, on two calls in
a row, the second over a smaller input (the scratch keeps the first call's partials)."""
import numpy as np
import pytest

import oracle
from gpu_helpers import host, log

pytestmark = pytest.mark.gpu


def test_cosine_noalloc_matches_the_workspace_entry_point():
    import torch
    import paper_2602_15922_amd as w
    g = torch.Generator(device="cuda").manual_seed(21)
    ws = torch.empty(w.wam_cosine_workspace_bytes(), dtype=torch.uint8, device="cuda")
    for n in (3_000_017, 1_537):
        log(f"cosine noalloc n={n}")
        a = torch.randn(n, generator=g, device="cuda")
        b = 0.6 * a + 0.8 * torch.randn(n, generator=g, device="cuda")
        ref = torch.full((1,), float("nan"), device="cuda")
        got = torch.full((1,), float("nan"), device="cuda")
        w.wam_cosine_similarity(a, b, ref, ws)
        w.wam_cosine_similarity_noalloc(a, b, got)
        torch.cuda.synchronize()
        assert torch.equal(got, ref), (float(got), float(ref))
        exact = oracle.cosine_similarity(host(a), host(b))
        assert abs(float(got) - exact) <= 1e-6
    # a zero vector gives 0 (the documented convention), also from the static scratch
    z = torch.zeros(777, device="cuda")
    got = torch.full((1,), float("nan"), device="cuda")
    w.wam_cosine_similarity_noalloc(z, z, got)
    torch.cuda.synchronize()
    assert float(got) == 0.0
    assert np.isfinite(float(got))
