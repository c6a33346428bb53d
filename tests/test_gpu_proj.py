"""GPU parity of the projection (proj_fwd) and of the projection fused with
the online softmax and top-k (proj_softmax_topk) against the binary64 oracle.

* Exact inputs: small integers times powers of two in bfloat16 make every
  product and every partial sum exact in binary32, whatever the order of the
  sums, so the GPU logits must equal the oracle's bit for bit, and the fused
  top-k must return the oracle's indices (with many exact ties, settled by
  the lower index) and its softmax values within the binary32 rule.
* Random inputs: the GPU sums H exact products in binary32, so each logit is
  within 2 H 2^-24 sum_k |h_k w_k| of the exact value (a bound for any order
  of round-to-nearest additions, doubled for margin); values and indices are
  checked against the oracle with that bound.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1805_02867_amd as osm
from parity import assert_softmax_close, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X; none is visible")
    return torch.device("cuda:0")


def exact_inputs(N, H, V, seed, dev):
    g = torch.Generator().manual_seed(seed)
    h = (torch.randint(-4, 5, (N, H), generator=g).float() * 0.125).to(torch.bfloat16)
    w = (torch.randint(-4, 5, (V, H), generator=g).float() * 0.0625).to(torch.bfloat16)
    return h.to(dev), w.to(dev)


def random_inputs(N, H, V, seed, dev, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    h = (torch.randn(N, H, generator=g) * scale).to(torch.bfloat16)
    w = (torch.randn(V, H, generator=g) * (1.0 / np.sqrt(H))).to(torch.bfloat16)
    return h.to(dev), w.to(dev)


def host_bf16(t):
    return to_host(t)


def oracle_logits(h, w):
    return oracle.proj(host_bf16(h), host_bf16(w), "bf16", "bf16")


def accumulation_bound(h, w):
    """2 H 2^-24 sum_k |h_k w_k| for every (n, v)."""
    ha = np.abs(oracle.bf16_to_f64(host_bf16(h)))
    wa = np.abs(oracle.bf16_to_f64(host_bf16(w)))
    H = ha.shape[1]
    return 2.0 * H * 2.0 ** -24 * (ha @ wa.T)


SHAPES = [(1, 8, 1), (5, 64, 7), (127, 72, 128), (128, 64, 129), (129, 136, 1000),
          (300, 1032, 4099), (64, 1024, 257)]


@pytest.mark.parametrize("N,H,V", SHAPES)
def test_proj_fwd_exact(dev, N, H, V):
    h, w = exact_inputs(N, H, V, seed=N + H + V, dev=dev)
    out = osm.proj(h, w)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(out).astype(np.float64), oracle_logits(h, w))


@pytest.mark.parametrize("N,H,V", [(33, 256, 500), (200, 1024, 3000)])
def test_proj_fwd_random_within_accumulation_bound(dev, N, H, V):
    h, w = random_inputs(N, H, V, seed=7, dev=dev)
    out = to_host(osm.proj(h, w)).astype(np.float64)
    err = np.abs(out - oracle_logits(h, w))
    assert (err <= accumulation_bound(h, w) + 1e-30).all(), float(err.max())


@pytest.mark.parametrize("N,H,V", SHAPES)
@pytest.mark.parametrize("K", [1, 5, 8, 16])
def test_proj_topk_exact(dev, N, H, V, K):
    if K > V:
        return
    h, w = exact_inputs(N, H, V, seed=3 * N + H + V + K, dev=dev)
    vals, idx = osm.proj_softmax_topk(h, w, K)
    torch.cuda.synchronize()
    v64, z64 = oracle.topk(oracle_logits(h, w), K, "f64")
    zi = to_host(idx)
    if not np.array_equal(zi, z64):
        r = np.argwhere(zi != z64)[0][0]
        raise AssertionError(f"N={N} H={H} V={V} K={K} row {r}: gpu {zi[r].tolist()} "
                             f"oracle {z64[r].tolist()}")
    assert_softmax_close(to_host(vals), v64, f"proj top-{K} values")


@pytest.mark.parametrize("N,H,V,K", [(64, 512, 3000, 5), (257, 1024, 8000, 10),
                                     (16, 256, 32000, 16), (1100, 256, 5000, 12)])
def test_proj_topk_random(dev, N, H, V, K):
    """Indices: where the oracle's K-th and (K+1)-th logits are further apart
    than twice the bound, the GPU must return exactly the oracle's indices;
    elsewhere its indices must be a valid top-k within the bound.  Values:
    the oracle's softmax at the GPU's indices, within 1e-5 plus the effect of
    the logit bound."""
    h, w = random_inputs(N, H, V, seed=N + K, dev=dev, scale=2.0)
    vals, idx = osm.proj_softmax_topk(h, w, K)
    torch.cuda.synchronize()
    check_topk_within_bound(oracle_logits(h, w), accumulation_bound(h, w).max(axis=1),
                            to_host(idx), to_host(vals), K)


def check_topk_within_bound(lg, bound, zi, vals, K):
    """The GPU's top-K of logit rows lg (binary64 oracle logits), given each
    row's accumulation bound: exact indices where the oracle's order is
    separated by more than twice the bound, else a valid top-K within it;
    values within 1e-5 plus the bound's effect."""
    zi = zi.astype(np.int64)
    order = np.argsort(-lg, axis=1, kind="stable")
    srt = np.take_along_axis(lg, order, 1)
    for r in range(lg.shape[0]):
        sel = lg[r, zi[r]]
        assert len(set(zi[r].tolist())) == K
        assert (np.diff(sel) <= 2 * bound[r]).all(), f"row {r} not sorted"
        if srt[r, K - 1] - srt[r, K] > 2 * bound[r] and \
                (np.diff(srt[r, :K]) < -2 * bound[r]).all():
            assert zi[r].tolist() == order[r, :K].tolist(), f"row {r}"
        else:
            assert sel.min() >= srt[r, K - 1] - 2 * bound[r], f"row {r}"
    y64 = oracle.softmax(lg, "f64")
    want = np.take_along_axis(y64, zi, 1)
    rel = np.abs(vals - want) / want
    allowed = 1e-5 + 4 * bound[:, None]
    assert (rel <= allowed).all(), float((rel / allowed).max())


@pytest.mark.slow
@pytest.mark.parametrize("N,H,V,nrows", [(4000, 1024, 32000, 48), (4000, 4096, 128256, 12)])
def test_proj_topk_full_size_sampled_rows(dev, N, H, V, nrows):
    """The fused call at full size, in the launch configuration the benchmark
    times (K = 5): sampled rows (the first and last of the batch and of a
    256-row strip, and random ones) against the oracle's binary64 logits."""
    K = 5
    g = torch.Generator(device=dev).manual_seed(N + H)
    h = (torch.randn(N, H, device=dev, generator=g) * 2.0).to(torch.bfloat16)
    w = (torch.randn(V, H, device=dev, generator=g) * (1.0 / np.sqrt(H))).to(torch.bfloat16)
    vals, idx = osm.proj_softmax_topk(h, w, K)
    torch.cuda.synchronize()
    rng = np.random.default_rng(N + H + V)
    rows = np.unique(np.concatenate([[0, 255, 256, N - 1],
                                     rng.choice(N, nrows - 4, replace=False)]))
    print(f"proj full size N={N} H={H} V={V} rows={rows.tolist()}", flush=True)
    hs = h[torch.as_tensor(rows, device=dev)]
    check_topk_within_bound(oracle_logits(hs, w), accumulation_bound(hs, w).max(axis=1),
                            to_host(idx)[rows], to_host(vals)[rows], K)


def test_proj_topk_deterministic(dev):
    h, w = random_inputs(100, 512, 5000, seed=1, dev=dev)
    a = osm.proj_softmax_topk(h, w, 8)
    b = osm.proj_softmax_topk(h, w, 8)
    torch.cuda.synchronize()
    assert torch.equal(a[1], b[1]) and torch.equal(a[0].view(torch.int32), b[0].view(torch.int32))


@pytest.mark.parametrize("K", [1, 2, 5, 16])
def test_proj_topk_all_equal_logits(dev, K):
    """w = 0: every logit is exactly 0, so the top-k is the K lowest indices
    (ties in increasing index order) and each value is exactly 1 / V."""
    N, H, V = 70, 64, 3000
    h, _ = random_inputs(N, H, V, seed=K, dev=dev)
    w = torch.zeros(V, H, dtype=torch.bfloat16, device=dev)
    vals, idx = osm.proj_softmax_topk(h, w, K)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(idx), np.tile(np.arange(K, dtype=np.int32), (N, 1)))
    assert_softmax_close(to_host(vals), np.full((N, K), 1.0 / V), "all-equal logits")


@pytest.mark.parametrize("N", [64, 65, 128, 129, 257, 1024, 1025])
@pytest.mark.parametrize("K", [5, 9, 16])
def test_proj_topk_tile_shapes(dev, N, K):
    """Batch sizes on each side of the fused kernel's tile and layout choices
    (256 x 64, 256 x 128 in one or two wavefronts along the vocabulary, and
    256 x 256 tiles), with a ragged last vocabulary tile and a K that is not a
    multiple of the 64-element step."""
    H, V = 136, 3001
    h, w = exact_inputs(N, H, V, seed=N * 31 + K, dev=dev)
    vals, idx = osm.proj_softmax_topk(h, w, K)
    torch.cuda.synchronize()
    v64, z64 = oracle.topk(oracle_logits(h, w), K, "f64")
    assert np.array_equal(to_host(idx), z64)
    assert_softmax_close(to_host(vals), v64, f"tile shapes N={N} K={K}")
