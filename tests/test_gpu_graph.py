"""A whole training step (every layer's forward and backward plus the loss)
captured into a HIP graph gives, on every replay, bit-identical results to
eager execution: the library allocates nothing, uses no memset and is
deterministic. Replays are interleaved with eager work and synchronisations."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _snapshot(net):
    out = [net.loss.cpu().numpy().copy()]
    for e in net.L:
        out += [e["t_out"].cpu().numpy().copy(), e["gW"].cpu().numpy().copy(),
                e["g_out"].cpu().numpy().copy()]
    return out


@pytest.mark.parametrize("name,batch", [("mlp3", 16), ("conv20", 2)])
def test_graph_replay_matches_eager(name, batch):
    import torch
    import bench
    from paper_2607_14672_amd import dstd, workloads
    assert torch.cuda.is_available()
    dstd._load()
    dev = torch.device("cuda:0")
    net = bench.Net(workloads.with_batch(workloads.get(name), batch), dev)
    net.step()
    torch.cuda.synchronize()
    ref = _snapshot(net)
    graph = net.capture()
    for rep in range(3):
        for e in net.L:  # clobber outputs so a replay that does nothing fails
            e["t_out"].fill_(-1.0)
            e["gW"].fill_(-1.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = _snapshot(net)
        for a, b in zip(ref, got):
            assert np.array_equal(a, b, equal_nan=True), f"replay {rep} differs"
        net.step()  # eager work between replays
        torch.cuda.synchronize()
        for a, b in zip(ref, _snapshot(net)):
            assert np.array_equal(a, b, equal_nan=True)
