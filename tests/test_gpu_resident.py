"""GPU parity of the row-resident softmax (OSM_RESIDENT) against the binary64
oracle: every workgroup shape, binary32 and bfloat16, row lengths from one
element up to the longest row the mode holds (with every 16-byte phase of
the row start), x and y off each other's 16-byte phase, special values,
determinism, and the workload shapes at full size."""
import numpy as np
import pytest
import torch

import oracle
import paper_1805_02867_amd as osm
from paper_1805_02867_amd import synth
from parity import assert_softmax_close, host_dtype, to_host

pytestmark = pytest.mark.gpu

E = {"f32": 4, "bf16": 8}
TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X; none is visible")
    return torch.device("cuda:0")


def run_case(x, block=None, y=None, what=""):
    if block is None:
        y = osm.softmax_fwd(x, y, mode="resident")
    else:
        y = osm.softmax_fwd(x, y, mode="resident", kernel=osm.KERNEL_ROWS, param=block)
    torch.cuda.synchronize()
    assert_softmax_close(to_host(y), oracle.softmax(to_host(x), host_dtype(x)), what)
    return y


def holds(V, dtype, block):
    """Whether a workgroup of `block` threads can hold a row of V (16 vectors
    per lane at most)."""
    return V // E[dtype] <= block * 16


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("block", [None, 256, 512, 1024])
def test_lengths(dev, dtype, block):
    for V in (1, 2, 3, 7, 8, 9, 63, 64, 65, 1000, 1001, 4095, 4097, 16383, 16385, 32000, 50001):
        if block is not None and not holds(V, dtype, block):
            continue
        N = 37 if V <= 4097 else 7
        print(f"resident dtype={dtype} block={block} V={V}", flush=True)
        x = synth.logits(N, V, sigma=3.0, seed=V, dtype=dtype, device=dev)
        run_case(x, block, what=f"resident {dtype} block {block} V={V}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_longest_rows(dev, dtype):
    """Rows of exactly OSM_RESIDENT_MAX_VEC vectors plus a partial vector at
    either end, and at every 16-byte phase of the row start."""
    e = E[dtype]
    top = osm.RESIDENT_MAX_VEC * e
    for V in (top, top + e - 1):
        for off in range(e):
            buf = synth.logits(1, 3 * V + off, sigma=2.0, seed=off, dtype=dtype, device=dev)
            x = buf[0, off:off + 3 * V].view(3, V)
            run_case(x, what=f"longest {dtype} V={V} offset {off}")
    x = synth.logits(2, top + e, sigma=2.0, seed=1, dtype=dtype, device=dev)
    with pytest.raises(osm.OsmError) as err:
        osm.softmax_fwd(x, mode="resident")
    assert err.value.status == osm.EUNSUPPORTED


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_unaligned_x_and_y(dev, dtype):
    """x rows at every 16-byte phase, y congruent and not congruent with x."""
    e = E[dtype]
    for V in (999, 4097, 30001):
        N = 9
        for xoff in (0, 1, e - 1):
            xb = synth.logits(1, N * V + xoff, sigma=2.0, seed=xoff + V, dtype=dtype, device=dev)
            x = xb[0, xoff:].view(N, V)
            for yoff in (0, 1):
                yb = torch.empty(N * V + yoff, dtype=TDT[dtype], device=dev)
                y = yb[yoff:].view(N, V)
                run_case(x, y=y, what=f"unaligned {dtype} V={V} x+{xoff} y+{yoff}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_special_values(dev, dtype):
    ninf, pinf, nan = float("-inf"), float("inf"), float("nan")
    V = 3000
    rows = [
        [0.0] * V,
        [1000.0] * (V - 1) + [1001.0],
        [-1000.0] * V,
        [ninf] * (V - 2) + [0.0, 1.0],
        [ninf] * V,
        [0.0] * (V - 1) + [pinf],
        [nan] + [0.0] * (V - 1),
        list(np.linspace(-80, 80, V)),
    ]
    x = torch.tensor(rows, dtype=TDT[dtype], device=dev)
    for block in (None, 256, 1024):
        run_case(x, block, what=f"special {dtype} block {block}")
    y = osm.softmax_fwd(torch.tensor([[5.0]], dtype=TDT[dtype], device=dev), mode="resident")
    assert y.item() == 1.0


def test_deterministic_and_stream(dev):
    x = synth.logits(300, 32000, sigma=2.0, seed=9, device=dev)
    a = osm.softmax_fwd(x, mode="resident")
    b = osm.softmax_fwd(x, mode="resident")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        c = osm.softmax_fwd(x, mode="resident", stream=s)
    s.synchronize()
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    assert torch.equal(a.view(torch.int32), c.view(torch.int32))


@pytest.mark.slow
def test_workload_4000x32000_f32(dev):
    w = synth.WORKLOADS["softmax_4000x32000_f32_shift"]
    x = synth.logits(w["N"], w["V"], sigma=w["sigma"], seed=0, device=dev,
                     shift_frac=w["shift_frac"])
    assert osm.plan(w["N"], w["V"], mode="resident") == (osm.KERNEL_ROWS, 512)
    run_case(x, what="4000x32000 resident")


@pytest.mark.slow
def test_workload_4000x50000_f32(dev):
    w = synth.WORKLOADS["topk_4000x50000_f32_ties"]
    x = synth.logits(w["N"], w["V"], sigma=w["sigma"], seed=0, device=dev,
                     tie_frac=w["tie_frac"])
    run_case(x, what="4000x50000 resident")


@pytest.mark.slow
def test_workload_32768x128256_bf16_sampled(dev):
    """Full-size bfloat16 batch; the oracle checks a seeded sample of 4096 rows
    plus the first and last."""
    w = synth.WORKLOADS["softmax_topk_32768x128256_bf16"]
    x = synth.logits(w["N"], w["V"], sigma=w["sigma"], seed=0, dtype="bf16", device=dev)
    y = osm.softmax_fwd(x, mode="resident")
    torch.cuda.synchronize()
    g = torch.Generator().manual_seed(124)
    rows = torch.cat([torch.tensor([0, w["N"] - 1]),
                      torch.randperm(w["N"], generator=g)[:4096]]).tolist()
    for i in range(0, len(rows), 128):
        rr = torch.tensor(rows[i:i + 128], device=dev)
        xh = to_host(x.index_select(0, rr))
        yh = to_host(y.index_select(0, rr))
        assert_softmax_close(yh, oracle.softmax(xh, "bf16"), "bf16 32768x128256 resident sample")
