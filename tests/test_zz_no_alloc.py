"""dtr_sim_run_static (working memory in the library's static device array,
for callers that cannot allocate) against dtr_sim_run on the same handles:
two calls in a row, the second on a smaller batch, bit-exact."""
import numpy as np
import pytest

from paper_2006_09616_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2006_09616_amd import dtr as D
    D.lib()
    return D


def _batches():
    rn = W.make_config("resnet50blk")
    small = [W.random_program(s, n_ops=20 + s % 40, n_const=s % 3, backward=s % 2 == 0) for s in range(12)]
    rows = [(i, h, max(1, W.natural_peak(t) * f // 4), 3 + i)
            for i, t in enumerate(small) for h in (W.H_DTR, W.H_EQ, W.H_LRU, W.H_RAND) for f in (1, 2, 3)]
    return [(rn.traces, rn.specs), (small, W.make_specs(rows))]


def test_static_scratch_matches_workspace_run(gpu):
    batches = _batches()
    assert len(batches[1][1]) < len(batches[0][1])
    refs = [gpu.run(traces, specs) for traces, specs in batches]
    sims = [gpu.Simulator(traces, specs, device="cuda:0", flags=gpu.OPT_STATIC_SCRATCH)
            for traces, specs in batches]
    try:
        with pytest.raises(gpu.DtrError) as e:
            sims[0].run()                          # its workspace has no working memory
        assert e.value.code == gpu.DTR_ESTATE
        got = []
        for sim in sims:                           # two static calls in a row, the second smaller
            sim.run_static()
            got.append(sim.results())
        ws = [gpu.Simulator(traces, specs, device="cuda:0").bytes for traces, specs in batches]
        assert all(s.bytes < w for s, w in zip(sims, ws))
    finally:
        for sim in sims:
            sim.close()
    for g, r in zip(got, refs):
        assert g.tobytes() == r.tobytes()


def test_static_scratch_on_a_workspace_handle(gpu):
    """A handle created with its own working memory may also run statically;
    two static runs in a row on it give the same results as dtr_sim_run."""
    traces, specs = _batches()[1]
    sim = gpu.Simulator(traces, specs, device="cuda:0")
    try:
        sim.run()
        ref = sim.results()
        sim.run_static()
        a = sim.results()
        sim.run_static()
        b = sim.results()
    finally:
        sim.close()
    assert a.tobytes() == ref.tobytes() == b.tobytes()
