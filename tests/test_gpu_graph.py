"""poseidon_sync_iteration captured into a HIP graph (stream capture on the
caller's stream) and replayed: every replay must update the tensors exactly
as the eager iteration does, with eager work and synchronisations between the
replays."""
import pytest
import torch

from _helpers import dev, log
from paper_1706_03292_amd import api
from paper_1706_03292_amd import inputs as I

pytestmark = pytest.mark.gpu


def _to_dev(host, d):
    return [{k: (v.to(d) if isinstance(v, torch.Tensor) else v) for k, v in h.items()} for h in host]


# 1: two launches on the caller's stream (latency-bound); 2: one stream, an SF
# and a PS launch; 4: the spread rebuild beside the PS applies, forked onto a
# pool stream and joined back; 5: the grouped rebuild beside the lean applies.
@pytest.mark.parametrize("cfg", [1, 2, 4, 5])
def test_sync_iteration_replays_as_a_hip_graph(cfg):
    d = dev()
    wl = I.workload(cfg)
    host = I.make_tensors(wl)
    eager, graphed, warm = _to_dev(host, d), _to_dev(host, d), _to_dev(host, d)
    cs = torch.cuda.current_stream(d)
    pool_e, pool_g = api.StreamPool(2), api.StreamPool(2)
    it_e = api.SyncIteration(pool_e, eager, wl.B, wl.P, wl.lr, wl.momentum)
    it_g = api.SyncIteration(pool_g, graphed, wl.B, wl.P, wl.lr, wl.momentum)
    # one eager iteration on a third copy first, as before any capture
    api.SyncIteration(pool_g, warm, wl.B, wl.P, wl.lr, wl.momentum)(cs)
    torch.cuda.synchronize()
    del warm
    s = torch.cuda.Stream(d)
    g = torch.cuda.CUDAGraph()
    log(f"graph capture, workload {cfg}")
    with torch.cuda.graph(g, stream=s):
        schemes = it_g(s)
    torch.cuda.synchronize()
    busy = torch.randn(2048, 2048, device=d)
    for r in range(3):
        log(f"graph replay {r}, workload {cfg}")
        want = it_e(cs)
        g.replay()
        torch.mm(busy, busy)                    # eager work between the replays
        torch.cuda.synchronize()
        assert schemes == want
        for x, y in zip(eager, graphed):
            assert torch.equal(x["W"], y["W"]), (r, x["spec"].name)
            if "buf" in x:
                assert torch.equal(x["buf"], y["buf"]), (r, x["spec"].name)
    del g
    pool_e.close()
    pool_g.close()
