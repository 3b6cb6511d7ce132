"""The allocation-free gating entry point (cgconv_gate_value_noalloc): through
the C ABI, two calls in a row on one GPU (the second with a smaller input)
give exactly what the plan-based cgconv_gate_value gives on the same inputs,
and both match the oracle; oversize inputs are refused on the host."""

import numpy as np
import pytest

from tests.conftest import rel_l2

pytestmark = pytest.mark.gpu


def _setup():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    torch.cuda.set_device(0)
    import paper_2509_24093_amd as P
    return torch, P


def test_noalloc_gate_matches_plan_entry_point_twice():
    torch, P = _setup()
    from oracle.gate import gate_value
    stream = torch.cuda.current_stream().cuda_stream
    # second call smaller in every size; the array keeps the first call's contents
    for n, (B, N, L, C, seed) in enumerate([(2, 512, 4, 12, 71), (1, 64, 2, 5, 72)]):
        print(f"[gpu] noalloc gate call {n}: B={B} N={N} L={L} C={C}", flush=True)
        K = (L + 1) ** 2
        rng = np.random.default_rng(seed)
        u = rng.normal(size=(B, N, K, C)).astype(np.float32)
        v = rng.normal(size=(B, N, K, C)).astype(np.float32)
        ud, vd = torch.from_numpy(u).cuda(), torch.from_numpy(v).cuda()
        f_na = torch.full_like(ud, float("nan"))
        P.cgconv_gate_value_noalloc(B, N, L, C, ud.data_ptr(), vd.data_ptr(), f_na.data_ptr(), stream)
        plan = P.Plan(B, N, L, C)
        try:
            f_pl = torch.full_like(ud, float("nan"))
            P.cgconv_gate_value(plan._h, ud.data_ptr(), vd.data_ptr(), f_pl.data_ptr(), stream)
            torch.cuda.synchronize()
        finally:
            plan.close()
        a, b = f_na.cpu().numpy(), f_pl.cpu().numpy()
        assert np.isfinite(a).all()
        assert np.array_equal(a, b)
        assert rel_l2(a, gate_value(u.astype(np.float64), v.astype(np.float64), L)) <= 1e-4


def test_noalloc_gate_rejects_oversize_and_bad_arguments():
    torch, P = _setup()
    lib = P.library()
    buf = torch.zeros(1024, device="cuda")
    p = buf.data_ptr()
    # 8 * (65536/64 + 1) * 9 * 64 * 8 bytes = 37.8 MB > 16 MiB: refused before any launch
    assert lib.cgconv_gate_value_noalloc(8, 65536, 8, 64, p, p + 1024, p + 2048, None) == P.CGCONV_ERR_UNSUPPORTED
    assert "exceeds" in P.cgconv_last_error()
    assert lib.cgconv_gate_value_noalloc(1, 64, 9, 4, p, p + 1024, p + 2048, None) == P.CGCONV_ERR_UNSUPPORTED
    assert lib.cgconv_gate_value_noalloc(0, 64, 2, 4, p, p + 1024, p + 2048, None) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_gate_value_noalloc(1, 64, 2, 4, p + 4, p + 1024, p + 2048, None) == P.CGCONV_ERR_ALIGNMENT
    assert lib.cgconv_gate_value_noalloc(1, 64, 2, 4, p, p + 1024, p, None) == P.CGCONV_ERR_INVALID_ARG
