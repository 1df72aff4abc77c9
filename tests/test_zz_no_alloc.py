"""yoso_backward_noalloc (the fixed per-GPU scratch, no workspace) against
yoso_backward, both through the C ABI: two calls in a row, the second smaller, so
that the second call runs on scratch the first call left behind."""
import numpy as np
import pytest

from workloads import Workload, make_inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2111_09714_amd as Y  # noqa: E402


def _case(bh, n, m, tau, dtype, seed):
    w = Workload("noalloc", 1, bh, n, 64, tau, m, dtype, "gauss", seed)
    inp = make_inputs(w)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda().to(tdt)
    q, k, v, dy = (dev(inp[s]) for s in ("q", "k", "v", "dy"))
    R = torch.from_numpy(inp["R"]).cuda()
    qc, kc = Y.hash_qk(q, k, R, m, tau)
    return qc, kc, q, k, v, dy


def _both(qc, kc, q, k, v, dy, m, tau):
    ref = Y.backward(qc, kc, q, k, v, dy, m, tau)
    got = tuple(torch.empty_like(t) for t in ref)
    Y.yoso_backward_noalloc(qc, kc, q, k, v, dy, m, tau, *got)
    torch.cuda.synchronize()
    return ref, got


def test_noalloc_matches_backward_on_two_calls():
    assert torch.cuda.is_available()
    limit = Y.yoso_backward_noalloc_limit()
    big = (1, 4096, 32, 8, "f32", 11)     # about 56 MB of scratch
    small = (2, 700, 16, 9, "bf16", 12)   # smaller, other dtype and tau
    for bh, n, m, tau, dtype, seed in (big, small):
        need = Y.yoso_workspace_bytes(Y.OP_BACKWARD, bh, n, n, 64, m, tau, Y.BF16 if dtype == "bf16" else Y.F32)
        assert 0 < need <= limit
        print(f"[noalloc] bh={bh} n={n} m={m} tau={tau} {dtype}: scratch {need} of {limit} bytes", flush=True)
        ref, got = _both(*_case(bh, n, m, tau, dtype, seed), m, tau)
        for name, a, b in zip(("dq", "dk", "dv"), got, ref):
            # the same kernels in the same order on the same inputs: bit for bit
            assert torch.equal(a, b), name


def test_noalloc_refuses_oversized_shapes():
    qc, kc, q, k, v, dy = _case(8, 4096, 32, 8, "f32", 13)  # about 0.2 GB of scratch
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    with pytest.raises(Y.YosoError) as e:
        Y.yoso_backward_noalloc(qc, kc, q, k, v, dy, 32, 8, dq, dk, dv)
    assert e.value.status == 6
