"""routepack_aggregate_demand_noalloc (the aggregation for callers that
cannot allocate: its band partials live in a fixed device array) against
routepack_aggregate_demand, bit for bit, on two calls in a row, the second
with a smaller input: the mid window (4096 x 24 x 256), then the tiny one
(64 x 4 x 16); then a shape whose default band grid (171 bands of 6144
columns) exceeds the array, so the call takes 170 taller bands."""
import numpy as np
import pytest

import synth

gpu = pytest.mark.gpu


def _log(msg):
    print(f"[no-alloc] {msg}", flush=True)


@gpu
def test_noalloc_aggregation_equals_the_allocating_one():
    import torch
    import paper_2608_12146_amd as rp
    for name in ("mid", "tiny"):
        w = synth.make_window(name)
        prob = rp.Problem.from_dict(synth.window_problem(w))
        d = torch.as_tensor(w.demand, device="cuda")
        _log(f"{name}: {tuple(d.shape)}")
        want = rp.aggregate_demand(prob, d)
        out = torch.full((w.n_layers, w.n_experts), -1, dtype=torch.int64, device="cuda")
        got = rp.aggregate_demand_noalloc(prob, d, out=out)
        torch.cuda.synchronize()
        assert got.data_ptr() == out.data_ptr()
        assert torch.equal(got, want)
        assert np.array_equal(got.cpu().numpy(), w.demand.sum(axis=0, dtype=np.int64))


@gpu
def test_noalloc_aggregation_with_fewer_bands():
    import torch
    import paper_2608_12146_amd as rp
    N, L, E = 16384, 24, 256
    _log(f"random counts {N} x {L} x {E}")
    g = torch.Generator(device="cuda")
    g.manual_seed(12146)
    d = torch.randint(0, 1 << 20, (N, L, E), dtype=torch.int32, device="cuda", generator=g)
    prob = rp.Problem(N, L, E, 8, 16, 8, 1, [0] * 8, 65536, [4096], [1])
    want = rp.aggregate_demand(prob, d)
    got = rp.aggregate_demand_noalloc(prob, d)
    assert torch.equal(got, want)
    assert torch.equal(want, d.sum(dim=0, dtype=torch.int64))
    del d
    torch.cuda.empty_cache()
