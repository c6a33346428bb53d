"""softmax_topk_ex_noalloc (the entry point that allocates nothing) against
softmax_topk_ex, the entry point whose kernels it shares, and the oracle.

Each case makes two calls in a row through the C ABI, the second on a smaller
input, so that the second call runs on the fixed scratch array as the first
left it (partials and row counters of a larger batch).  Indices must be
identical and values bit-identical to softmax_topk_ex with the same kernel
choice (same kernels, same reduction order), and both must meet the oracle's
bar (indices bit-exact, values within the binary32 rule).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1805_02867_amd as osm
from paper_1805_02867_amd import synth
from parity import assert_topk_equal, host_dtype, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X; none is visible")
    return torch.device("cuda:0")


def _check_pair(x, K, kernel, param, what):
    ref_v, ref_i = osm.softmax_topk(x, K, kernel=kernel, param=param)
    v, i = osm.softmax_topk_noalloc(x, K, kernel=kernel, param=param)
    torch.cuda.synchronize()
    v, i, ref_v, ref_i = to_host(v), to_host(i), to_host(ref_v), to_host(ref_i)
    assert np.array_equal(i, ref_i), what
    assert np.array_equal(v.view(np.uint32), ref_v.view(np.uint32)), what
    v64, z64 = oracle.topk(to_host(x), K, host_dtype(x))
    assert_topk_equal(v, i, v64, z64, what)


# (first shape, second smaller shape, K, kernel, param); the first two use the
# plan (split for these small batches of long rows)
CASES = [
    ((12, 1000000), (5, 300000), 5, osm.KERNEL_AUTO, 0),
    ((40, 100000), (3, 50001), 16, osm.KERNEL_AUTO, 0),
    ((16, 65536), (9, 20000), 64, osm.KERNEL_SPLIT, 96),
    ((64, 32000), (7, 1000), 10, osm.KERNEL_SPLIT, 7),
    ((700, 4000), (300, 999), 5, osm.KERNEL_ROWS, 64),
    ((8, 50000), (2, 8192), 50, osm.KERNEL_ROWS, 256),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_noalloc_matches_existing_entry_point(dev, dtype, case):
    first, second, K, kernel, param = CASES[case]
    for n, (N, V) in enumerate((first, second)):
        what = f"noalloc {dtype} call {n + 1} N={N} V={V} K={K} kernel {kernel} param {param}"
        print(what, flush=True)
        x = synth.logits(N, V, sigma=2.0, seed=N * 31 + V + n, dtype=dtype, device=dev)
        _check_pair(x, K, kernel, param, what)


def test_noalloc_rejects_what_the_array_cannot_hold(dev):
    """A forced split whose partials exceed the fixed array: OSM_ESCRATCH,
    nothing enqueued (the outputs keep their contents)."""
    N, V, K, S = 64, 65536, 64, 256  # 64 * 256 * (8 * 64 + 8) bytes = 8.5 MB
    assert N * S * (8 * K + 8) > osm.NOALLOC_SCRATCH_BYTES
    x = synth.logits(N, V, sigma=2.0, seed=1, device=dev)
    vals = torch.full((N, K), 7.0, device=dev)
    idx = torch.full((N, K), -5, dtype=torch.int32, device=dev)
    with pytest.raises(osm.OsmError) as e:
        osm.softmax_topk_noalloc(x, K, vals, idx, kernel=osm.KERNEL_SPLIT, param=S)
    assert e.value.status == osm.ESCRATCH
    torch.cuda.synchronize()
    assert (vals == 7.0).all() and (idx == -5).all()
    # the same call on the allocating entry point works
    _check_pair(x[:4].contiguous(), K, osm.KERNEL_SPLIT, S, "allocating split after ESCRATCH")
