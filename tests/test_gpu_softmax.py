"""GPU parity of softmax_fwd / softmax_fwd_ex against the binary64 oracle.

Every kernel family and lane-group size, every mode, binary32 and bfloat16,
over row lengths that cover single elements, partial 16-byte vectors, one and
several wavefronts, ragged tails and misaligned rows; split-V with forced
chunk counts (including 1 and more chunks than needed); special values; and
the paper's workload shapes at full size.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1805_02867_amd as osm
from paper_1805_02867_amd import synth
from parity import assert_softmax_close, host_dtype, to_host

pytestmark = pytest.mark.gpu

MODES = ("naive", "safe", "online")
TEAMS = (4, 8, 16, 32, 64, 128, 256, 512, 1024)
VS = (1, 2, 3, 5, 8, 10, 31, 63, 64, 65, 127, 250, 1000, 1001, 4097, 8191, 32000, 50001)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X; none is visible")
    return torch.device("cuda:0")


def run_case(x, mode, kernel=osm.KERNEL_AUTO, param=0, y=None, what=""):
    y = osm.softmax_fwd(x, y, mode=mode, kernel=kernel, param=param)
    torch.cuda.synchronize()
    xh = to_host(x)
    y64 = oracle.softmax(xh, host_dtype(x))
    assert_softmax_close(to_host(y), y64, what)
    return y


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("team", TEAMS)
def test_rows_kernel_all_modes_and_lengths(dev, team, dtype):
    for V in VS:
        N = 67 if V <= 8191 else 9
        x = synth.logits(N, V, sigma=3.0, seed=V, dtype=dtype, device=dev)
        for mode in MODES:
            print(f"rows team={team} dtype={dtype} V={V} mode={mode}", flush=True)
            run_case(x, mode, osm.KERNEL_ROWS, team, what=f"team {team} {dtype} V={V} {mode}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("S", [1, 2, 3, 5, 64, 257])
def test_split_kernel_forced_chunks(dev, S, dtype):
    for V in (1, 7, 4097, 100003, 1000000):
        N = 3 if V >= 100000 else 5
        x = synth.logits(N, V, sigma=3.0, seed=V + S, dtype=dtype, device=dev)
        for mode in MODES:
            print(f"split S={S} dtype={dtype} V={V} mode={mode}", flush=True)
            run_case(x, mode, osm.KERNEL_SPLIT, S, what=f"split S={S} {dtype} V={V} {mode}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_unaligned_output_uses_scalar_path(dev, dtype):
    """y offset by one element from x's 16-byte phase: every element goes
    through the scalar path."""
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    for V, kernel, param in ((1000, osm.KERNEL_ROWS, 64), (4097, osm.KERNEL_ROWS, 256),
                             (3000, osm.KERNEL_ROWS, 8), (50000, osm.KERNEL_SPLIT, 7)):
        N = 11
        x = synth.logits(N, V, sigma=2.0, seed=3, dtype=dtype, device=dev)
        buf = torch.empty(N * V + 1, dtype=tdt, device=dev)
        y = buf[1:].view(N, V)
        for mode in MODES:
            run_case(x, mode, kernel, param, y=y, what=f"unaligned {dtype} V={V} {mode}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_special_values(dev, dtype):
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    ninf, pinf, nan = float("-inf"), float("inf"), float("nan")
    V = 300
    rows = [
        [0.0] * V,                                   # all equal -> 1/V
        [1000.0] * (V - 1) + [1001.0],               # large values
        [-1000.0] * V,                               # very negative, all equal
        [ninf] * (V - 2) + [0.0, 1.0],               # -inf elements next to finite ones
        [ninf] * V,                                  # only -inf -> NaN row
        [0.0] * (V - 1) + [pinf],                    # +inf -> NaN row
        [nan] + [0.0] * (V - 1),                     # NaN -> NaN row
        list(np.linspace(-80, 80, V)),               # wide range, deep underflow
    ]
    x = torch.tensor(rows, dtype=tdt, device=dev)
    for team in (4, 64, 256, 1024):
        for mode in ("safe", "online"):
            run_case(x, mode, osm.KERNEL_ROWS, team, what=f"special {dtype} team {team} {mode}")
    for S in (1, 3):
        for mode in ("safe", "online"):
            run_case(x, mode, osm.KERNEL_SPLIT, S, what=f"special {dtype} split {S} {mode}")
    y = osm.softmax_fwd(torch.tensor([[5.0]], dtype=tdt, device=dev))
    assert y.item() == 1.0


def test_naive_overflows_where_the_paper_says(dev):
    """Alg. 1 overflows on rows shifted by +1000; safe and online stay exact."""
    x = synth.logits(64, 2000, sigma=2.0, seed=5, device=dev, shift_frac=0.25)
    shifted, _ = synth.special_rows(64, seed=5, shift_frac=0.25)
    plain = [r for r in range(64) if r not in set(shifted)]
    yn = to_host(osm.softmax_fwd(x, mode="naive"))
    assert not np.isfinite(yn[shifted]).any()
    y64 = oracle.softmax(to_host(x))
    assert_softmax_close(yn[plain], y64[plain], "naive on unshifted rows")
    for mode in ("safe", "online"):
        assert_softmax_close(to_host(osm.softmax_fwd(x, mode=mode)), y64, mode)


def test_deterministic(dev):
    x = synth.logits(300, 32000, sigma=2.0, seed=9, device=dev)
    for kernel, param in ((osm.KERNEL_ROWS, 512), (osm.KERNEL_ROWS, 64), (osm.KERNEL_SPLIT, 9)):
        a = osm.softmax_fwd(x, kernel=kernel, param=param)
        b = osm.softmax_fwd(x, kernel=kernel, param=param)
        torch.cuda.synchronize()
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_nonzero_stream(dev):
    x = synth.logits(100, 5000, sigma=2.0, seed=11, device=dev)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        y = osm.softmax_fwd(x, stream=s)
        ys = osm.softmax_fwd(x, kernel=osm.KERNEL_SPLIT, param=4, stream=s)
    s.synchronize()
    y64 = oracle.softmax(to_host(x))
    assert_softmax_close(to_host(y), y64, "side stream")
    assert_softmax_close(to_host(ys), y64, "side stream split")


# ------------------------------------------------------ full workload shapes
@pytest.mark.slow
def test_workload_4000x32000_f32_all_modes(dev):
    w = synth.WORKLOADS["softmax_4000x32000_f32_shift"]
    x = synth.logits(w["N"], w["V"], sigma=w["sigma"], seed=0, device=dev,
                     shift_frac=w["shift_frac"])
    shifted, _ = synth.special_rows(w["N"], seed=0, shift_frac=w["shift_frac"])
    xh = to_host(x)
    y64 = oracle.softmax(xh)
    plain = np.setdiff1d(np.arange(w["N"]), shifted)
    for mode in MODES:
        print(f"4000x32000 {mode} plan={osm.plan(w['N'], w['V'], mode=mode)}", flush=True)
        y = to_host(osm.softmax_fwd(x, mode=mode))
        if mode == "naive":
            assert not np.isfinite(y[shifted]).any()
            assert_softmax_close(y[plain], y64[plain], "naive 4000x32000 unshifted rows")
        else:
            assert_softmax_close(y, y64, f"{mode} 4000x32000")
        del y


@pytest.mark.slow
def test_workload_10x1e6_f32(dev):
    w = synth.WORKLOADS["softmax_10x1e6_f32"]
    x = synth.logits(w["N"], w["V"], sigma=w["sigma"], seed=0, device=dev)
    assert osm.plan(w["N"], w["V"])[0] == osm.KERNEL_SPLIT
    y64 = oracle.softmax(to_host(x))
    for mode in MODES:
        assert_softmax_close(to_host(osm.softmax_fwd(x, mode=mode)), y64, f"{mode} 10x1e6")


@pytest.mark.slow
def test_workload_32768x128256_bf16_sampled(dev):
    """Full-size bfloat16 batch in the benchmark's launch configuration;
    the oracle checks a seeded sample of 4096 rows plus the first and last."""
    w = synth.WORKLOADS["softmax_topk_32768x128256_bf16"]
    x = synth.logits(w["N"], w["V"], sigma=w["sigma"], seed=0, dtype="bf16", device=dev)
    y = osm.softmax_fwd(x, mode="online")
    torch.cuda.synchronize()
    g = torch.Generator().manual_seed(123)
    rows = torch.cat([torch.tensor([0, w["N"] - 1]),
                      torch.randperm(w["N"], generator=g)[:4096]]).tolist()
    for i in range(0, len(rows), 128):
        rr = torch.tensor(rows[i:i + 128], device=dev)
        xh = to_host(x.index_select(0, rr))
        yh = to_host(y.index_select(0, rr))
        assert_softmax_close(yh, oracle.softmax(xh, "bf16"), "bf16 32768x128256 sample")


def test_ref_stream_copy_is_exact(dev):
    """The reference copy kernel (a measurement aid) copies every byte, ragged
    tail included; the read kernel runs on the same buffer."""
    x = torch.randint(-2**31, 2**31 - 1, (1_000_003 * 4,), dtype=torch.int32, device=dev)
    y = torch.empty_like(x)
    osm.ref_stream("copy", x, y)
    sink = torch.zeros(1024, dtype=torch.float32, device=dev)
    osm.ref_stream("read", x, sink)
    torch.cuda.synchronize()
    assert torch.equal(x, y)


def _subnormal_rows(V: int, tdt):
    """Rows whose outputs sweep through the binary32 and bfloat16 subnormal
    range: the row maximum is 0 and the rest descend from -80 to -110 (e^-87.3
    is 2^-126, e^-92.2 the smallest bfloat16 subnormal 2^-133, e^-103.3 the
    smallest binary32 subnormal 2^-149)."""
    base = np.linspace(-80.0, -110.0, V - 1)
    rows = [np.concatenate([[0.0], base]), np.concatenate([base[::-1], [0.0]]),
            np.concatenate([base[: V // 2], [0.0], base[V // 2:]])]
    return torch.tensor(np.array(rows), dtype=tdt)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_subnormal_outputs(dev, dtype):
    """Outputs below 2^-126 are rounded, not flushed: bfloat16 within 1 ulp of
    the oracle's rounding (no exception for subnormals), binary32 within the
    normal range's relative bound plus one subnormal unit, 1e-5 y64 + 2^-149,
    where the oracle is subnormal."""
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    for V in (301, 4001):
        x = _subnormal_rows(V, tdt).to(dev)
        xh = to_host(x)
        y64 = oracle.softmax(xh, host_dtype(x))
        assert (y64 < 2.0 ** -126).sum() > 30 and (y64 > 2.0 ** -149).sum() > 30
        cases = [(m, osm.KERNEL_ROWS, t) for m in MODES for t in (8, 64, 256, 1024)]
        cases += [(m, osm.KERNEL_SPLIT, s) for m in MODES for s in (1, 3)]
        cases += [("resident", osm.KERNEL_AUTO, 0)]
        for mode, kernel, param in cases:
            what = f"subnormal {dtype} V={V} {mode} kernel {kernel} param {param}"
            print(what, flush=True)
            y = osm.softmax_fwd(x, mode=mode, kernel=kernel, param=param)
            torch.cuda.synchronize()
            yh = to_host(y)
            assert_softmax_close(yh, y64, what)
            if dtype == "f32":
                tiny = y64 < 2.0 ** -126
                err = np.abs(yh.astype(np.float64) - y64)[tiny]
                bound = 1e-5 * y64[tiny] + 2.0 ** -149
                assert (err <= bound).all(), (what, (err / bound).max())
                assert (yh[tiny] > 0).sum() >= (y64[tiny] >= 2.0 ** -148).sum()
