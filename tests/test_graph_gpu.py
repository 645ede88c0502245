"""The library's calls inside a captured HIP graph: a whole chunked prefill
step (appends, attention, split merges) is captured once and replayed, with
eager work and synchronisation between replays; every replay must equal the
eager run bit for bit."""
import pytest
import torch

from helpers import say
from paper_2606_22968_amd import synth
from paper_2606_22968_amd.prefill import ChunkedPrefill

pytestmark = pytest.mark.gpu


def _all_lse(r):
    return torch.cat([r.lse(c).flatten() for c in range(len(r.lengths))])


@pytest.mark.parametrize("splits,remote", [(0, None), (3, None), (0, (0, 1664)), (2, (512, 1664))])
def test_graph_replay_equals_eager(gpu, splits, remote):
    # remote: the two-store call, with positions [begin, end) read from a
    # second store (every chunk boundary inside the range is a multiple of 64).
    lengths = [704, 1024, 333, 1500]
    say(f"[case] graph capture, splits={splits} remote={remote}")
    q, k, v = (t.cuda() for t in synth.make_qkv(81, sum(lengths), 32, 8, 128))
    r = ChunkedPrefill(32, 8, 128, lengths, num_splits=splits, remote=remote)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        r.run(q, k, v, 0.088)  # plans are made (and cached) before capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    o_ref, lse_ref = r.o.clone(), _all_lse(r).clone()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        r.run(q, k, v, 0.088)
    torch.cuda.synchronize()
    for rep in range(4):
        r.o.fill_(float("nan"))
        r._lse_flat.fill_(float("nan"))
        r.store.k_pool.fill_(float("nan"))
        r.store.v_pool.fill_(float("nan"))
        if r.remote_store is not None:
            r.remote_store.k_pool.fill_(float("nan"))
            r.remote_store.v_pool.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(r.o.view(torch.int16), o_ref.view(torch.int16)), f"replay {rep}: O differs"
        assert torch.equal(_all_lse(r).view(torch.int32), lse_ref.view(torch.int32)), f"replay {rep}: LSE differs"
