"""Concurrent use of one set of loaded ensembles: host threads, each with a
stream of its own, run the scoring step at the same time (ctypes releases
the interpreter lock during library calls, so the host calls overlap too,
and the walks and selections of the streams overlap on the GPU).  Every
run gives the outputs of a run alone, bit for bit; an argument error on
one thread leaves the other threads' runs and error strings untouched."""
import threading

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import gen  # noqa: E402
from paper_2411_10764_amd import ml2  # noqa: E402

DEV = torch.device("cuda:0")


def _outputs(pipe):
    return [t.cpu().numpy().copy().view(np.uint8)
            for t in (pipe.valid, pipe.margin, pipe.score, pipe.idx, pipe.top, pipe.num)]


@pytest.mark.parametrize("name,threads,reps", [("medium", 4, 3), ("large", 2, 2)])
def test_threads_and_streams_match_a_lone_run(name, threads, reps):
    w = gen.WORKLOADS[name]
    X = torch.from_numpy(w.features()).to(DEV)
    v, p = ml2.ml2_load_ensemble(w.validity()), ml2.ml2_load_ensemble(w.perf())
    alone = ml2.Pipeline(v, p, w.n, w.k, device=DEV, with_margin=True)
    alone.run(X)
    torch.cuda.synchronize()
    want = _outputs(alone)
    print(f"[concurrency] {name}: {threads} threads x {reps} runs", flush=True)

    errors = []

    def worker(t):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                pipe = ml2.Pipeline(v, p, w.n, w.k, device=DEV, with_margin=True)
                for r in range(reps):
                    pipe.run(X)
                    s.synchronize()
                    got = _outputs(pipe)
                    for a, b in zip(want, got):
                        if not np.array_equal(a, b):
                            errors.append(f"thread {t} run {r} differs")
                            return
                    # an argument error here must not disturb the others
                    bad = ml2.lib().ml2_filter_topk(None, None, -1, 1, None, None, None, None,
                                                    0, None)
                    if bad != ml2.ML2_ERR_INVALID_ARG:
                        errors.append(f"thread {t}: bad call returned {bad}")
                        return
        except Exception as e:  # noqa: BLE001 - reported below
            errors.append(f"thread {t}: {e!r}")

    ts = [threading.Thread(target=worker, args=(t,)) for t in range(threads)]
    for t in ts:
        t.start()
    for t in ts:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in ts), "a worker did not finish"
    assert not errors, errors
    v.free()
    p.free()
