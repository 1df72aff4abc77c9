"""The whole step (hash Q, hash K, forward, backward) captured into one HIP graph
(torch.cuda.graph: stream capture) and replayed: every replay must reproduce the
eager step bit for bit (every kernel is deterministic), with eager work that
reuses the same workspaces and device synchronisations between the replays.
The library enqueues kernels only (no memset nodes, no allocation), so capture
records nothing but its kernels."""
import sys

import numpy as np
import pytest

from workloads import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2111_09714_amd as Y  # noqa: E402


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


# (one head of 700 rows: the tables and the dense backward; all 384 heads of 512 rows:
# the dense forward, the one-wave sort and the dense backward; the bench workload:
# the tables, the pair passes, the table form and the reductions)
@pytest.mark.parametrize("wname,n", [("single_head_n512", 700), ("bert_base_n512", None), ("lra_n4096", None)])
def test_step_graph_replays_match_eager(wname, n):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    w = WORKLOADS[wname]
    heads = None if n is None else [0]
    inp = make_inputs(w, heads=heads, n=n)
    q, k, v, dy = (torch.from_numpy(inp[s]).cuda().contiguous() for s in ("q", "k", "v", "dy"))
    R = torch.from_numpy(inp["R"]).cuda()
    bh, nn = q.shape[0], q.shape[1]
    qc = torch.empty((bh, nn, w.m), dtype=torch.int16, device="cuda")
    kc = torch.empty_like(qc)
    y, dq, dk, dv = (torch.empty_like(q) for _ in range(4))
    ws_f = Y.workspace(Y.OP_FORWARD, q, w.m, w.tau)
    ws_b = Y.workspace(Y.OP_BACKWARD, q, w.m, w.tau)

    def step(stream=None):
        Y.yoso_hash(q, R, w.m, w.tau, qc, stream)
        Y.yoso_hash(k, R, w.m, w.tau, kc, stream)
        Y.yoso_forward(qc, kc, v, w.m, w.tau, y, ws_f, stream)
        Y.yoso_backward(qc, kc, q, k, v, dy, w.m, w.tau, dq, dk, dv, ws_b, stream)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (qc, kc, y, dq, dk, dv)]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    other = torch.from_numpy(np.random.default_rng(3).standard_normal(tuple(v.shape)).astype(np.float32)).cuda()
    for rep in range(4):
        for t in (qc, kc, y, dq, dk, dv):
            t.zero_()
        g.replay()
        torch.cuda.synchronize()
        same = all(torch.equal(a, b) for a, b in zip((qc, kc, y, dq, dk, dv), ref))
        log(f"[graph {wname}] replay {rep}: bitwise equal to the eager step: {same}")
        assert same, rep
        # eager work between replays, through the same workspaces (other values of V)
        y2 = torch.empty_like(y)
        Y.yoso_forward(qc, kc, other, w.m, w.tau, y2, ws_f)
        d2 = [torch.empty_like(q) for _ in range(3)]
        Y.yoso_backward(qc, kc, q, k, other, dy, w.m, w.tau, *d2, ws_b)
        torch.cuda.synchronize()
