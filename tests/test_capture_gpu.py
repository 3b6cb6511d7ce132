"""HIP graph capture of the library's entry points (torch.cuda.graph).

After plan creation every entry point only enqueues kernels on the caller's
stream: no allocation, memset, copy or host synchronisation.  So a call
captured into a graph replays correctly.  Each test captures one call with
preallocated outputs, then replays the graph three times; between replays
the program does its own eager work (new inputs written in place, an eager
call of the same entry point, synchronisations).  Every replay is compared
bit for bit with the eager call on the same inputs (the kernels are
deterministic), and the first replay is also checked against the oracle.
"""

import numpy as np
import pytest

from oracle.conv import cgconv_fft
from tests.conftest import rel_l2

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _replay_matches_eager(tag, inputs, outs, call, seed):
    """Capture call() (which reads `inputs` and writes `outs`, and takes the
    stream to enqueue on), then replay with fresh inputs three times."""
    torch = _torch()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up outside the capture
        call(side.cuda_stream)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    print(f"[gpu] capture {tag}", flush=True)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    gen = torch.Generator(device="cuda").manual_seed(seed)
    replays = []
    for rep in range(3):
        for t in inputs:
            t.copy_(torch.randn(t.shape, generator=gen, device="cuda").to(t.dtype))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [o.clone() for o in outs]
        for o in outs:
            o.fill_(float("nan"))
        call(torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        for a, b in zip(got, outs):
            assert torch.equal(a, b), f"{tag}: replay {rep} differs from the eager call"
        replays.append(([t.clone() for t in inputs], got))
        print(f"[gpu] capture {tag}: replay {rep} equals the eager call", flush=True)
    del g
    return replays


def test_forward_fused_and_unfused_capture():
    torch = _torch()
    import paper_2509_24093_amd as P
    for B, N, L, C in ((2, 1024, 3, 5), (1, 256, 2, 3)):
        plan = P.Plan(B, N, L, C)
        q, k, out = (torch.zeros(plan.shape, device="cuda") for _ in range(3))
        reps = _replay_matches_eager(f"forward N={N}", [q, k], [out],
                                     lambda s: P.cgconv_forward(plan._h, q.data_ptr(), k.data_ptr(), out.data_ptr(), s),
                                     7000 + N)
        (qi, ki), (got,) = reps[0]
        err = rel_l2(got.cpu().numpy(), cgconv_fft(qi.cpu().numpy(), ki.cpu().numpy(), L))
        print(f"[parity] captured forward N={N}: rel_l2 {err:.3e}", flush=True)
        assert err <= 1e-4
        plan.close()


def test_forward_bf16_capture():
    torch = _torch()
    import paper_2509_24093_amd as P
    plan = P.Plan(2, 2048, 4, 3)
    q, k, out = (torch.zeros(plan.shape, device="cuda", dtype=torch.bfloat16) for _ in range(3))
    _replay_matches_eager("forward bf16", [q, k], [out],
                          lambda s: P.cgconv_forward_bf16(plan._h, q.data_ptr(), k.data_ptr(), out.data_ptr(), s), 7100)
    plan.close()


def test_backward_capture():
    torch = _torch()
    import paper_2509_24093_amd as P
    plan = P.Plan(2, 512, 3, 4)
    q, k, g, gq, gk = (torch.zeros(plan.shape, device="cuda") for _ in range(5))
    _replay_matches_eager("backward", [q, k, g], [gq, gk],
                          lambda s: P.cgconv_backward(plan._h, q.data_ptr(), k.data_ptr(), g.data_ptr(),
                                                      gq.data_ptr(), gk.data_ptr(), s), 7200)
    plan.close()


def test_mixed_forward_capture():
    torch = _torch()
    import paper_2509_24093_amd as P
    B, N, L, C = 1, 1024, 3, 8
    plan = P.Plan(B, N, L, C)
    n_paths = len(P.cgconv_paths(L))
    q, k, out = (torch.zeros(plan.shape, device="cuda") for _ in range(3))
    w = torch.zeros(n_paths, C, C, device="cuda")
    _replay_matches_eager("mixed forward", [q, k, w], [out],
                          lambda s: P.cgconv_forward_mixed(plan._h, q.data_ptr(), k.data_ptr(), w.data_ptr(),
                                                           out.data_ptr(), s), 7300)
    plan.close()


def test_gate_forward_and_backward_capture():
    torch = _torch()
    import paper_2509_24093_amd as P
    plan = P.Plan(2, 300, 4, 3, boundary="linear")
    u, v, f, gf, gu, gv = (torch.zeros(plan.shape, device="cuda") for _ in range(6))
    _replay_matches_eager("gate_value", [u, v], [f],
                          lambda s: P.cgconv_gate_value(plan._h, u.data_ptr(), v.data_ptr(), f.data_ptr(), s), 7400)
    _replay_matches_eager("gate_value_backward", [u, v, gf], [gu, gv],
                          lambda s: P.cgconv_gate_value_backward(plan._h, u.data_ptr(), v.data_ptr(), gf.data_ptr(),
                                                                 gu.data_ptr(), gv.data_ptr(), s), 7500)
    plan.close()


def test_graph_fourier_forward_capture():
    torch = _torch()
    import paper_2509_24093_amd as P
    B, n, L, C = 1, 200, 3, 3
    plan = P.GraphPlan(B, n, L, C)
    U = torch.from_numpy(np.linalg.qr(np.random.default_rng(7600).normal(size=(n, n)))[0]
                         .astype(np.float32)[None]).cuda()
    q, k, out = (torch.zeros(plan.shape, device="cuda") for _ in range(3))
    _replay_matches_eager("graph forward", [q, k], [out],
                          lambda s: P.cgconv_forward_graph(plan._h, U.data_ptr(), q.data_ptr(), k.data_ptr(),
                                                           out.data_ptr(), s), 7700)
    plan.close()

