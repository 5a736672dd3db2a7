"""The scoring step captured as a HIP graph (torch.cuda.CUDAGraph) and
replayed: every replay, with eager work and synchronizations between the
replays, gives the eager step's outputs bit for bit, and a replay after the
pool changed in place gives the eager outputs for the new pool.  Covers the
one-pass kernel with the one-workgroup selection (Tiny) and the two walks
with the multi-workgroup selection and its grid barrier (Medium), each
followed by a second-level re-rank of the selected rows (model A: here the
V ensemble, over the same columns)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import gen  # noqa: E402
from paper_2411_10764_amd import ml2  # noqa: E402


def _note(msg):
    print(f"[graph] {msg}", flush=True)


class Step:
    """ml2_score, ml2_filter_topk and ml2_rerank into buffers of its own."""

    def __init__(self, v, p, n, k, dev):
        self.v, self.p, self.k = v, p, k
        self.keep = max(1, k // 2)
        self.a_scores = torch.empty(k, dtype=torch.float32, device=dev)
        self.a_idx = torch.empty(self.keep, dtype=torch.int32, device=dev)
        self.a_top = torch.empty(self.keep, dtype=torch.float32, device=dev)
        self.a_num = torch.empty(1, dtype=torch.int32, device=dev)
        self.a_wsb = ml2.ml2_rerank_workspace_bytes(v, k)
        self.a_ws = torch.empty(self.a_wsb, dtype=torch.uint8, device=dev)
        self.valid = torch.empty(n, dtype=torch.uint8, device=dev)
        self.score = torch.empty(n, dtype=torch.float32, device=dev)
        self.idx = torch.empty(k, dtype=torch.int32, device=dev)
        self.top = torch.empty(k, dtype=torch.float32, device=dev)
        self.num = torch.empty(1, dtype=torch.int32, device=dev)
        self.wsb = ml2.ml2_topk_workspace_bytes(n, k)
        self.ws = torch.empty(self.wsb, dtype=torch.uint8, device=dev)

    def __call__(self, X):
        ml2.ml2_score(self.v, self.p, X, self.valid, None, self.score)
        ml2.ml2_filter_topk(self.valid, self.score, self.k, self.idx, self.top, self.num,
                            self.ws, self.wsb, X.shape[0])
        ml2.ml2_rerank(self.v, X, self.idx, self.keep, self.a_scores, self.a_idx, self.a_top,
                       self.a_num, self.a_ws, self.a_wsb, m=self.k)

    def clear(self):
        self.valid.fill_(7)
        self.score.fill_(float("nan"))
        self.idx.fill_(-5)
        self.top.fill_(float("nan"))
        self.num.fill_(-5)
        for t in (self.a_scores, self.a_top):
            t.fill_(float("nan"))
        self.a_idx.fill_(-5)
        self.a_num.fill_(-5)

    def outputs(self):
        return (self.valid.cpu().numpy(), self.score.cpu().numpy().view(np.uint32),
                self.idx.cpu().numpy(), self.top.cpu().numpy().view(np.uint32),
                self.num.cpu().numpy(), self.a_scores.cpu().numpy().view(np.uint32),
                self.a_idx.cpu().numpy(), self.a_top.cpu().numpy().view(np.uint32),
                self.a_num.cpu().numpy())


def _same(a, b):
    return all(np.array_equal(x, y) for x, y in zip(a, b))


@pytest.mark.parametrize("name", ["tiny", "medium"])
def test_graph_replays_match_eager(name):
    w = gen.WORKLOADS[name]
    dev = torch.device("cuda:0")
    X = torch.from_numpy(w.features()).to(dev)
    v = ml2.ml2_load_ensemble(w.validity())
    p = ml2.ml2_load_ensemble(w.perf())
    _note(f"{name}: n={w.n} F={w.F} k={w.k} one pass={ml2.ml2_score_single_pass(v, p, X)}")
    eager = Step(v, p, w.n, w.k, dev)
    eager(X)
    torch.cuda.synchronize()
    want = eager.outputs()

    run = Step(v, p, w.n, w.k, dev)
    run(X)  # first use outside the capture (per-kernel attributes, clock rate)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(X)
    torch.cuda.synchronize()
    other = torch.empty_like(X)
    for r in range(4):
        run.clear()
        other.copy_(X).mul_(0.5)  # eager work between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert _same(run.outputs(), want), f"{name}: replay {r} differs from the eager step"
        _note(f"{name}: replay {r} ok")

    # the graph reads the pool where it is: a new pool in the same buffer
    X.mul_(-1.25)
    eager(X)
    torch.cuda.synchronize()
    want2 = eager.outputs()
    assert not _same(want2, want)
    for r in range(2):
        run.clear()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert _same(run.outputs(), want2), f"{name}: replay {r} on the new pool differs"
    del g
    v.free()
    p.free()
