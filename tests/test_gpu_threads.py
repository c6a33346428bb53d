"""Calls from several host threads on one stream (the boundary's re-entrancy).

Split softmax, split top-k and the fused projection + top-k all keep their
partials in the stream's one scratch buffer.  Three host threads enqueue them
on the same stream at once, with shapes that grow from call to call so that
the buffer is replaced (its old copy freed in stream order) while other
threads' calls are being enqueued.  No thread synchronises until all have
finished; then every result is checked against the oracle.  A call whose
kernels interleaved with another's on the shared buffer, or ran on a freed
one, would read the other call's partials.
"""
import threading

import numpy as np
import pytest
import torch

import oracle
import paper_1805_02867_amd as osm
from paper_1805_02867_amd import synth
from parity import assert_softmax_close, assert_topk_equal, host_dtype, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X; none is visible")
    return torch.device("cuda:0")


# (N, V, S): N * S pairs of 8 bytes, from 128 KB to 2 MB (the buffer starts
# at 256 KB and doubles)
SOFTMAX_CASES = [(32, 4096, 512), (64, 4096, 1024), (64, 8192, 2048), (128, 8192, 2048)]
# (N, V, K, S): N * S partials of 8K + 8 bytes, 0.3 to 9 MB, plus N counters
TOPK_CASES = [(16, 8192, 16, 256), (32, 8192, 16, 512), (64, 16384, 16, 1024),
              (64, 16384, 64, 1024)]
# (N, H, V, K): exact inputs (every logit exact in binary32)
PROJ_CASES = [(64, 64, 4096, 8), (200, 64, 8192, 16), (300, 128, 16384, 16)]


def _exact_proj_inputs(N, H, V, seed, dev):
    g = torch.Generator().manual_seed(seed)
    h = (torch.randint(-4, 5, (N, H), generator=g).float() * 0.125).to(torch.bfloat16)
    w = (torch.randint(-4, 5, (V, H), generator=g).float() * 0.0625).to(torch.bfloat16)
    return h.to(dev), w.to(dev)


def test_three_threads_one_stream(dev):
    stream = torch.cuda.Stream(device=dev)
    sp = stream.cuda_stream
    rounds = 3
    jobs = {"softmax": [], "topk": [], "proj": []}
    for rnd in range(rounds):
        for i, (N, V, S) in enumerate(SOFTMAX_CASES):
            x = synth.logits(N, V, sigma=3.0, seed=100 * rnd + i, device=dev)
            jobs["softmax"].append((x, torch.empty_like(x), S))
        for i, (N, V, K, S) in enumerate(TOPK_CASES):
            x = synth.logits(N, V, sigma=2.0, seed=200 * rnd + i, device=dev)
            vals = torch.empty((N, K), dtype=torch.float32, device=dev)
            idx = torch.empty((N, K), dtype=torch.int32, device=dev)
            jobs["topk"].append((x, vals, idx, K, S))
        for i, (N, H, V, K) in enumerate(PROJ_CASES):
            h, w = _exact_proj_inputs(N, H, V, 300 * rnd + i, dev)
            vals = torch.empty((N, K), dtype=torch.float32, device=dev)
            idx = torch.empty((N, K), dtype=torch.int32, device=dev)
            jobs["proj"].append((h, w, vals, idx, K))
    torch.cuda.synchronize()
    osm.stream_release(sp)

    per_round = {k: len(v) // rounds for k, v in jobs.items()}
    start = threading.Barrier(3)
    round_done = threading.Barrier(3)
    errors = []

    def worker(kind):
        try:
            for rnd in range(rounds):
                start.wait()
                n = per_round[kind]
                for job in jobs[kind][rnd * n:(rnd + 1) * n]:
                    if kind == "softmax":
                        x, y, S = job
                        osm.softmax_fwd(x, y, mode="online", kernel=osm.KERNEL_SPLIT, param=S,
                                        stream=sp)
                    elif kind == "topk":
                        x, vals, idx, K, S = job
                        osm.softmax_topk(x, K, vals, idx, kernel=osm.KERNEL_SPLIT, param=S,
                                         stream=sp)
                    else:
                        h, w, vals, idx, K = job
                        osm.proj_softmax_topk(h, w, K, vals, idx, stream=sp)
                round_done.wait()
                if kind == "softmax":
                    # every stream buffer dropped between rounds (in stream
                    # order), so the next round grows it again from nothing
                    osm.stream_release(sp)
        except Exception as e:  # reported by the main thread
            errors.append((kind, repr(e)))
            start.abort()
            round_done.abort()

    threads = [threading.Thread(target=worker, args=(k,)) for k in jobs]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    torch.cuda.synchronize()
    assert not errors, errors

    for x, y, S in jobs["softmax"]:
        what = f"split softmax {tuple(x.shape)} S={S}"
        assert_softmax_close(to_host(y), oracle.softmax(to_host(x), host_dtype(x)), what)
    for x, vals, idx, K, S in jobs["topk"]:
        v64, z64 = oracle.topk(to_host(x), K, host_dtype(x))
        assert_topk_equal(to_host(vals), to_host(idx), v64, z64,
                          f"split top-{K} {tuple(x.shape)} S={S}")
    for h, w, vals, idx, K in jobs["proj"]:
        lg = oracle.proj(to_host(h), to_host(w), "bf16", "bf16")
        v64, z64 = oracle.topk(lg, K, "f64")
        assert np.array_equal(to_host(idx), z64), f"proj top-{K} {tuple(h.shape)}"
        assert_softmax_close(to_host(vals), v64, f"proj top-{K} values")
    osm.stream_release(sp)
