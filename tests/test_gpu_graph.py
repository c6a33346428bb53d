"""Graph capture of the split paths on a stream whose scratch is already
large enough (the capture contract in the header): the captured softmax and
top-k calls allocate nothing, their counter arrays were cleared by a fill
kernel (no memset node), and every replay gives the eager results bit for
bit, with eager work and synchronisation between the replays."""
import pytest
import torch

import oracle
import paper_1805_02867_amd as osm
from paper_1805_02867_amd import synth
from parity import assert_topk_equal, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X; none is visible")
    return torch.device("cuda:0")


def test_captured_split_calls_replay_like_eager(dev):
    N, V, K = 10, 1_000_000, 5
    assert osm.topk_plan(N, V, K)[0] == osm.KERNEL_SPLIT
    assert osm.plan(N, V, mode="online")[0] == osm.KERNEL_SPLIT
    x = synth.logits(N, V, sigma=3.0, seed=91, device=dev)
    s = torch.cuda.Stream()
    vals = torch.empty((N, K), device=dev)
    idx = torch.empty((N, K), dtype=torch.int32, device=dev)
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):  # warm-up: the stream's scratch and counters
        osm.softmax_topk(x, K, vals, idx)
        osm.softmax_fwd(x, y, mode="online")
    s.synchronize()
    ref_vals, ref_idx, ref_y = vals.clone(), idx.clone(), y.clone()
    print("captured split calls: capture", flush=True)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        osm.softmax_topk(x, K, vals, idx)
        osm.softmax_fwd(x, y, mode="online")
    torch.cuda.synchronize()
    scratch = torch.empty_like(x)
    for rep in range(3):
        print(f"captured split calls: replay {rep}", flush=True)
        vals.fill_(-1.0)
        idx.fill_(-1)
        y.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(vals, ref_vals) and torch.equal(idx, ref_idx), f"replay {rep} top-k"
        assert torch.equal(y, ref_y), f"replay {rep} softmax"
        # eager work between replays, on the same stream and on torch's
        with torch.cuda.stream(s):
            osm.softmax_topk(x, K, vals, idx)
        scratch.copy_(x).mul_(0.5)
        torch.cuda.synchronize()
        assert torch.equal(idx, ref_idx), f"eager after replay {rep}"
    v64, z64 = oracle.topk(to_host(x), K, "f32")
    assert_topk_equal(to_host(ref_vals), to_host(ref_idx), v64, z64, "captured split 10x1e6 K=5")
