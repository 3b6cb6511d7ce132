"""GPU parity of the CG convolution with per-path channel mixing
(cgconv_forward_mixed, MFMA mixing stage) against the mixing oracle on the
same seeded inputs and weights.

Bar: relative L2 error <= 1e-4 (fp32).  Whole outputs for the small
workloads and for shapes that cover the single-pass and two-pass pipelines,
every L_max the stage supports, odd, small and full channel counts and point
counts that leave a ragged last block; at the point-cloud size the mixed
output with weights that depend only on the output degree is compared with
that channel map applied to the plain forward, plus random weights against
the oracle at a reduced token count with the same L_max and C.
"""

import numpy as np
import pytest

import workloads as W
from oracle.cg import paths
from oracle.mix import cgconv_mixed_direct, cgconv_mixed_fft
from tests.conftest import rel_l2

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _weights(L, C, seed):
    rng = np.random.default_rng(seed)
    return (rng.normal(size=(len(paths(L)), C, C)) / np.sqrt(C)).astype(np.float32)


def gpu_mixed(q, k, L, Wm, tag=""):
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, K, C = q.shape
    print(f"[gpu] {tag} cgconv_forward_mixed B={B} N={N} L={L} C={C}", flush=True)
    plan = P.Plan(B, N, L, C)
    out = plan.forward_mixed(torch.from_numpy(np.ascontiguousarray(q, dtype=np.float32)).cuda(),
                             torch.from_numpy(np.ascontiguousarray(k, dtype=np.float32)).cuda(),
                             torch.from_numpy(Wm).cuda())
    torch.cuda.synchronize()
    res = out.cpu().numpy()
    plan.close()
    return res


def _rand(B, N, L, C, seed):
    rng = np.random.default_rng(seed)
    K = (L + 1) ** 2
    return (rng.normal(size=(B, N, K, C)).astype(np.float32), rng.normal(size=(B, N, K, C)).astype(np.float32))


@pytest.mark.parametrize("name", ["tiny", "nbody", "molecule"])
def test_mixed_small_workloads(name):
    cfg = W.WORKLOADS[name]
    q, k = W.make(name)
    L, C = cfg["L"], cfg["C"]
    Wm = _weights(L, C, 500 + cfg["seed"])
    got = gpu_mixed(q, k, L, Wm, name)
    ref = cgconv_mixed_direct(q, k, L, Wm) if name == "tiny" else cgconv_mixed_fft(q, k, L, Wm)
    err = rel_l2(got, ref)
    print(f"[parity] mixed {name}: rel_l2 {err:.3e}", flush=True)
    assert err < TOL


# (B, N, L, C): N <= 256 single pass; 512..32768 the shapes of fused plans
# (mixing runs the unfused passes there with N2 = 64: radix-512 outer passes
# at 32768); 65536 the plain two-pass split.
SHAPES = [(1, 64, 0, 1), (2, 128, 1, 3), (3, 256, 2, 5), (1, 512, 6, 32), (2, 1024, 4, 16),
          (1, 2048, 5, 7), (1, 32768, 2, 2), (1, 65536, 1, 3), (5, 16, 3, 32), (1, 2, 6, 9)]


@pytest.mark.parametrize("B,N,L,C", SHAPES)
def test_mixed_shapes(B, N, L, C):
    q, k = _rand(B, N, L, C, 600 + N + L)
    Wm = _weights(L, C, 700 + L)
    got = gpu_mixed(q, k, L, Wm, "shape")
    ref = cgconv_mixed_fft(q, k, L, Wm)
    err = rel_l2(got, ref)
    print(f"[parity] mixed B={B} N={N} L={L} C={C}: rel_l2 {err:.3e}", flush=True)
    assert err < TOL


def test_identity_weights_equal_plain_forward():
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, L, C = 2, 1024, 6, 32
    q, k = _rand(B, N, L, C, 11)
    Wm = np.ascontiguousarray(np.broadcast_to(np.eye(C, dtype=np.float32), (len(paths(L)), C, C)))
    plan = P.Plan(B, N, L, C)
    qt, kt = torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda()
    mixed = plan.forward_mixed(qt, kt, torch.from_numpy(Wm).cuda())
    plain = plan(qt, kt)
    torch.cuda.synchronize()
    err = rel_l2(mixed.cpu().numpy().astype(np.float64), plain.cpu().numpy().astype(np.float64))
    plan.close()
    print(f"[parity] identity weights vs plain forward: rel_l2 {err:.3e}", flush=True)
    assert err < 1e-5


def test_pointcloud_size_output_degree_maps():
    """W_p = A_J (J = output degree of p): mixed output of degree J = A_J
    applied over channels to the plain output, at the point-cloud size."""
    torch = _torch()
    import paper_2509_24093_amd as P
    cfg = W.WORKLOADS["pointcloud"]
    B, N, L, C = cfg["B"], cfg["N"], cfg["L"], cfg["C"]
    rng = np.random.default_rng(71)
    A = [(rng.normal(size=(C, C)) / np.sqrt(C)).astype(np.float32) for _ in range(L + 1)]
    Wm = np.stack([A[J] for (_, _, J) in paths(L)]).astype(np.float32)
    g = torch.Generator(device="cuda")
    g.manual_seed(72)
    K = (L + 1) ** 2
    qt = torch.randn(B, N, K, C, device="cuda", generator=g)
    kt = torch.randn(B, N, K, C, device="cuda", generator=g)
    print(f"[gpu] pointcloud-size mixed B={B} N={N} L={L} C={C}", flush=True)
    plan = P.Plan(B, N, L, C)
    mixed = plan.forward_mixed(qt, kt, torch.from_numpy(Wm).cuda())
    plain = plan(qt, kt)
    torch.cuda.synchronize()
    num = den = 0.0
    for J in range(L + 1):
        sl = slice(J * J, (J + 1) ** 2)
        want = torch.einsum("dc,bnmc->bnmd", torch.from_numpy(A[J]).cuda().double(), plain[:, :, sl, :].double())
        num += float(((mixed[:, :, sl, :].double() - want) ** 2).sum())
        den += float((want ** 2).sum())
    plan.close()
    err = (num / den) ** 0.5
    print(f"[parity] pointcloud-size degree maps: rel_l2 {err:.3e}", flush=True)
    assert err < TOL


def test_pointcloud_L_C_random_weights_reduced_tokens():
    """Random weights at L_max = 6, C = 32 (the point-cloud stage) on a
    reduced token count the oracle finishes quickly."""
    B, N, L, C = 2, 4096, 6, 32
    q, k = _rand(B, N, L, C, 81)
    Wm = _weights(L, C, 82)
    got = gpu_mixed(q, k, L, Wm, "L6C32")
    ref = cgconv_mixed_fft(q, k, L, Wm)
    err = rel_l2(got, ref)
    print(f"[parity] mixed B={B} N={N} L={L} C={C}: rel_l2 {err:.3e}", flush=True)
    assert err < TOL


def test_mixed_unsupported_and_bad_arguments():
    torch = _torch()
    import paper_2509_24093_amd as P
    for (L, C) in [(7, 4), (2, 33)]:
        plan = P.Plan(1, 64, L, C)
        K = (L + 1) ** 2
        q = torch.zeros(1, 64, K, C, device="cuda")
        w = torch.zeros(len(paths(L)), C, C, device="cuda")
        with pytest.raises(P.CgconvError) as e:
            plan.forward_mixed(q, q, w)
        assert e.value.status == P.CGCONV_ERR_UNSUPPORTED
        plan.close()
    plan = P.Plan(1, 64, 2, 4)
    q = torch.zeros(1, 64, 9, 4, device="cuda")
    with pytest.raises(ValueError):
        plan.forward_mixed(q, q, torch.zeros(3, 4, 4, device="cuda"))
    lib = P.library()
    out = torch.empty_like(q)
    assert lib.cgconv_forward_mixed(plan._h, q.data_ptr(), q.data_ptr(), None, out.data_ptr(), None) \
        == P.CGCONV_ERR_INVALID_ARG
    plan.close()


def test_mixed_stage_timing_names():
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, L, C = 1, 2048, 3, 8
    plan = P.Plan(B, N, L, C)
    q = torch.randn(B, N, 16, C, device="cuda")
    w = torch.randn(len(paths(L)), C, C, device="cuda")
    plan.enable_timing(2)
    plan.forward_mixed(q, q, w)
    plan(q, q)  # a plain call after a timed mixed one is not timed
    st, n = plan.stage_times()
    plan.close()
    assert n == 1 and list(st) == ["fft_fwd_1", "fft_fwd_2", "cg_mix", "fft_inv_1", "fft_inv_2"]
