"""The C-ABI library on the CPU (no GPU compute): it loads, exports every
symbol include/cgconv.h declares, its host-built CG table matches the
oracle's, its host reference of the frequency-domain contraction (the same
coefficient table the generated GPU code carries) matches the oracle's dense
contraction, and argument errors come back as statuses with messages."""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2509_24093_amd as P
from oracle.cg import dense_R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cgconv.h")

pytestmark = pytest.mark.skipif(not os.path.exists(P.LIB_PATH), reason="libcgconv.so not built")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cgconv_\w+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = _declared_functions()
    assert {"cgconv_plan_create", "cgconv_forward", "cgconv_forward_bf16", "cgconv_plan_destroy",
            "cgconv_plan_info", "cgconv_cg_table", "cgconv_contract_host", "cgconv_last_error"} <= set(names)
    lib = ctypes.CDLL(P.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


@pytest.mark.parametrize("L", [0, 1, 2, 3, 4, 5, 6, 7, 8])
def test_library_table_matches_oracle(L):
    idx, coef = P.cgconv_cg_table(L)
    R = dense_R(L)
    Rl = np.zeros_like(R)
    for (l1, m1, l2, m2, J, M), c in zip(idx, coef):
        Rl[J * J + J + M, l1 * l1 + l1 + m1, l2 * l2 + l2 + m2] += c
    assert len(coef) == int((np.abs(R) > 1e-12).sum())
    assert np.abs(Rl - R).max() < 1e-12


@pytest.mark.parametrize("L", [0, 1, 2, 3, 4, 5, 6, 7, 8])
def test_contraction_table_matches_oracle(L):
    rng = np.random.default_rng(100 + L)
    K = (L + 1) ** 2
    R = dense_R(L)
    for _ in range(3):
        q = rng.normal(size=K) + 1j * rng.normal(size=K)
        k = rng.normal(size=K) + 1j * rng.normal(size=K)
        u = P.cgconv_contract_host(L, q, k)
        ref = np.einsum("oab,a,b->o", R, q, k)
        assert np.abs(u - ref).max() < 1e-13 * max(1.0, np.abs(ref).max())


def test_plan_create_rejects_bad_arguments():
    lib = P.library()
    for args, word in [((0, 64, 2, 4), "invalid sizes"), ((1, 64, 2, 0), "invalid sizes"),
                       ((1, 1, 2, 4), "invalid sizes"), ((1, 63, 2, 4), "unsupported N"),
                       ((1, 65536 * 2, 2, 4), "unsupported N"), ((1, 64, 9, 4), "unsupported L_max"),
                       ((1, 64, -1, 4), "invalid L_max")]:
        assert not lib.cgconv_plan_create(*args)
        assert word in P.cgconv_last_error()


def test_forward_and_info_reject_null_plan():
    lib = P.library()
    assert lib.cgconv_forward(None, 16, 16, 32, None) == P.CGCONV_ERR_INVALID_ARG
    assert "NULL" in P.cgconv_last_error()
    assert lib.cgconv_forward_bf16(None, 16, 16, 32, None) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_plan_info(None, None, None, None) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_plan_contraction_info(None, None, None) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_plan_export_table(None, None, None, 0) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_gate_value(None, 16, 16, 32, None) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_gate_value_backward(None, 16, 16, 32, 48, 64, None) == P.CGCONV_ERR_INVALID_ARG
    assert "NULL" in P.cgconv_last_error()
    lib.cgconv_plan_destroy(None)  # no-op


def test_table_and_contract_reject_bad_arguments():
    lib = P.library()
    assert lib.cgconv_cg_table(9, None, None, 0) == P.CGCONV_ERR_UNSUPPORTED
    assert lib.cgconv_cg_table(2, None, None, 5) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_contract_host(2, None, None, None) == P.CGCONV_ERR_INVALID_ARG
    # cap smaller than the table: only cap entries are written, full count returned
    n = lib.cgconv_cg_table(2, None, None, 0)
    idx = (ctypes.c_int32 * 12)(*([-7] * 12))
    coef = (ctypes.c_double * 3)(9.0, 9.0, 9.0)
    assert lib.cgconv_cg_table(2, idx, coef, 2) == n
    assert coef[2] == 9.0 and coef[0] != 9.0


def test_package_has_no_cpu_fallback(monkeypatch):
    """Without the library every entry point raises (no silent CPU path)."""
    monkeypatch.setattr(P, "_lib", None)
    monkeypatch.setattr(P, "LIB_PATH", P.LIB_PATH + ".missing")
    with pytest.raises(RuntimeError, match="missing"):
        P.Plan(1, 64, 2, 4)
    with pytest.raises(RuntimeError, match="missing"):
        P.cgconv_cg_table(2)


def test_timing_entry_points_reject_null_plan():
    lib = P.library()
    assert lib.cgconv_plan_enable_timing(None, 4) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_plan_stage_times(None, None, 0, None, None) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_plan_stage_name(None, 0) == b""


@pytest.mark.parametrize("L", range(0, 9))
def test_paths_match_oracle_order(L):
    """The weight order of the mixing entry point is the oracle's path list."""
    from oracle.cg import paths
    got = [tuple(int(x) for x in row) for row in P.cgconv_paths(L)]
    assert got == paths(L)


def test_mixed_entry_points_reject_bad_arguments():
    lib = P.library()
    assert lib.cgconv_forward_mixed(None, 16, 16, 16, 32, None) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_paths(9, None, 0) == P.CGCONV_ERR_UNSUPPORTED
    assert lib.cgconv_paths(2, None, 3) == P.CGCONV_ERR_INVALID_ARG
    buf = (ctypes.c_int32 * 6)(*([-7] * 6))
    n = lib.cgconv_paths(2, buf, 2)
    assert n == 15 and buf[5] != -7


def test_gate_entry_point_rejects_null_plan():
    lib = P.library()
    assert lib.cgconv_gate_value(None, 16, 32, 48, None) == P.CGCONV_ERR_INVALID_ARG


def test_backward_entry_point_rejects_null_plan():
    lib = P.library()
    assert lib.cgconv_backward(None, 16, 32, 48, 64, 80, None) == P.CGCONV_ERR_INVALID_ARG


def test_graph_entry_points_reject_bad_arguments():
    lib = P.library()
    assert lib.cgconv_forward_graph(None, 16, 32, 48, 64, None) == P.CGCONV_ERR_INVALID_ARG
    assert lib.cgconv_backward_graph(None, 16, 32, 48, 64, 80, 96, None) == P.CGCONV_ERR_INVALID_ARG


def _dense_from_entries(idx, coef, L):
    K = (L + 1) ** 2
    R = np.zeros((K, K, K))
    for (l1, m1, l2, m2, J, M), c in zip(idx, coef):
        R[J * J + J + M, l1 * l1 + l1 + m1, l2 * l2 + l2 + m2] += c
    return R


@pytest.mark.gpu
@pytest.mark.parametrize("L", [0, 1, 2, 3, 4, 5, 6, 7, 8])
def test_plan_export_table_matches_oracle(L):
    """The tensor a plan's kernels evaluate, exported through the C ABI,
    equals the oracle's dense R (entries, count, order), for a token plan
    (recovered from its contraction terms) and a graph plan."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("plan creation needs a GPU")
    torch.cuda.set_device(0)
    print(f"[gpu] export table L={L}", flush=True)
    R = dense_R(L)
    n_ref = int((np.abs(R) > 1e-12).sum())
    for plan in (P.Plan(1, 64, L, 2), P.GraphPlan(1, 16, L, 2)):
        try:
            n_paths, nnz, ws = plan.info()
            idx, coef = plan.export_table()
            assert nnz == len(coef) == n_ref
            assert np.abs(_dense_from_entries(idx, coef, L) - R).max() < 1e-12
            keys = [tuple(r) for r in idx[:, [4, 5, 0, 1, 2, 3]]]
            assert keys == sorted(keys)
            assert n_paths == len(P.cgconv_paths(L))
            nc, npr = plan.contraction_info()
            assert nc > 0 and 0 < npr <= nc
            # a short buffer: the full count comes back, nothing past cap is written
            lib = P.library()
            ib = (ctypes.c_int32 * 12)(*([-7] * 12))
            cb = (ctypes.c_double * 3)(9.0, 9.0, 9.0)
            assert lib.cgconv_plan_export_table(plan._h, ib, cb, 1 if n_ref > 1 else 0) == n_ref
            assert cb[1] == 9.0 and ib[6] == -7
        finally:
            plan.close()
