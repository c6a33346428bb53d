"""GPU parity of the fused softmax + top-k against the binary64 oracle:
indices bit-exact (ties to the lower index), values within the binary32 rule."""
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


SHAPES = (64, 128, 256)  # lanes per row: one, two or four wavefronts


def check(x, K, what, lanes=None):
    if lanes is None:
        vals, idx = osm.softmax_topk(x, K)
    else:
        vals, idx = osm.softmax_topk(x, K, kernel=osm.KERNEL_ROWS, param=lanes)
    torch.cuda.synchronize()
    v64, z64 = oracle.topk(to_host(x), K, host_dtype(x))
    assert_topk_equal(to_host(vals), to_host(idx), v64, z64, what)


@pytest.mark.parametrize("lanes", SHAPES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_lengths_and_k(dev, dtype, lanes):
    for V in (1, 2, 3, 5, 8, 9, 63, 64, 65, 255, 256, 257, 1000, 1001, 4097, 32000, 50001):
        for K in sorted({1, 2, 5, 10, 50, 64, V}):
            if K > V or K > osm.TOPK_KMAX:
                continue
            N = 23 if V < 10000 else 7
            print(f"topk dtype={dtype} lanes={lanes} V={V} K={K}", flush=True)
            x = synth.logits(N, V, sigma=2.0, seed=V * 7 + K, dtype=dtype, device=dev)
            check(x, K, f"{dtype} lanes={lanes} V={V} K={K}", lanes)


@pytest.mark.parametrize("lanes", SHAPES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_heavy_ties(dev, dtype, lanes):
    """Values on a coarse grid: long runs of equal values straddle slot K."""
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    g = torch.Generator(device=dev).manual_seed(4)
    for V in (100, 3000, 40000):
        x = torch.randint(-3, 4, (13, V), generator=g, device=dev).to(tdt) * 0.5
        for K in (1, 5, 17, 64):
            check(x, K, f"ties {dtype} V={V} K={K}", lanes)
    # every element equal
    x = torch.full((5, 5000), 1.25, dtype=tdt, device=dev)
    check(x, 64, "all equal", lanes)
    check(x, 3, "all equal", lanes)


@pytest.mark.parametrize("lanes", SHAPES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_special_values(dev, dtype, lanes):
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    ninf = float("-inf")
    V = 700
    base = torch.linspace(-5, 5, V)
    rows = torch.stack([
        base,
        base.flip(0),
        torch.where(torch.arange(V) % 3 == 0, torch.tensor(ninf), base),  # -inf elements
        torch.cat([torch.full((V - 3,), ninf), torch.tensor([1.0, 2.0, 3.0])]),  # few finite
        torch.zeros(V) * torch.where(torch.arange(V) % 2 == 0, 1.0, -1.0),  # +-0.0 ties
        base + 1000.0,
    ]).to(tdt).to(dev)
    for K in (1, 3, 5, 10):
        check(rows, K, f"special {dtype} K={K}", lanes)
    # K larger than the finite elements: -inf elements fill in, lowest index first
    check(rows[3:4], 8, f"-inf fill {dtype}", lanes)


@pytest.mark.parametrize("lanes", SHAPES)
def test_unaligned_rows(dev, lanes):
    """x starting off the 16-byte phase (a view into a larger buffer)."""
    buf = synth.logits(1, 37 * 999 + 3, sigma=2.0, seed=8, device=dev)
    x = buf[0, 3:].view(37, 999)
    check(x, 5, "unaligned x", lanes)
    bbuf = synth.logits(1, 21 * 4097 + 5, sigma=2.0, seed=9, dtype="bf16", device=dev)
    check(bbuf[0, 5:].view(21, 4097), 7, "unaligned bf16 x", lanes)


def test_batch_not_multiple_of_rows_per_workgroup(dev):
    """One wavefront per row packs four rows per workgroup: ragged last block."""
    for N in (1, 2, 3, 5, 1027):
        x = synth.logits(N, 3001, sigma=2.0, seed=N, device=dev)
        check(x, 5, f"N={N}", 64)


def test_deterministic(dev):
    x = synth.logits(500, 32000, sigma=2.0, seed=10, device=dev)
    for lanes in SHAPES:
        a = osm.softmax_topk(x, 10, kernel=osm.KERNEL_ROWS, param=lanes)
        b = osm.softmax_topk(x, 10, kernel=osm.KERNEL_ROWS, param=lanes)
        torch.cuda.synchronize()
        assert torch.equal(a[1], b[1])
        assert torch.equal(a[0].view(torch.int32), b[0].view(torch.int32))


def test_small_workload_16x1000(dev):
    w = synth.WORKLOADS["softmax_topk_16x1000_f32"]
    x = synth.logits(w["N"], w["V"], sigma=w["sigma"], seed=0, device=dev)
    # short rows: one wavefront per row, whatever the batch size
    assert osm.topk_plan(w["N"], w["V"], w["K"]) == (osm.KERNEL_ROWS, 64)
    check(x, w["K"], "16x1000 K=5")


@pytest.mark.slow
def test_workload_4000x32000_k5(dev):
    w = synth.WORKLOADS["softmax_4000x32000_f32_shift"]
    x = synth.logits(w["N"], w["V"], sigma=w["sigma"], seed=0, device=dev,
                     shift_frac=w["shift_frac"])
    check(x, 5, "4000x32000 K=5")


@pytest.mark.slow
@pytest.mark.parametrize("K", [5, 10])
def test_workload_4000x50000_ties(dev, K):
    w = synth.WORKLOADS["topk_4000x50000_f32_ties"]
    x = synth.logits(w["N"], w["V"], sigma=w["sigma"], seed=0, device=dev,
                     tie_frac=w["tie_frac"])
    _, tied = synth.special_rows(w["N"], seed=0, tie_frac=w["tie_frac"])
    xh = to_host(x)
    # the tie rows really hold their maximum four times
    for r in tied[:5]:
        assert (xh[r] == xh[r].max()).sum() == 4
    vals, idx = osm.softmax_topk(x, K)
    torch.cuda.synchronize()
    v64, z64 = oracle.topk(xh, K)
    assert_topk_equal(to_host(vals), to_host(idx), v64, z64, f"4000x50000 K={K}")
    zt = to_host(idx)[tied]
    for r, z in zip(tied, zt):
        assert list(z[:4]) == sorted(z[:4]), "tied maxima must come in increasing index order"


@pytest.mark.slow
def test_workload_32768x128256_bf16_k50_sampled(dev):
    w = synth.WORKLOADS["softmax_topk_32768x128256_bf16"]
    x = synth.logits(w["N"], w["V"], sigma=w["sigma"], seed=0, dtype="bf16", device=dev)
    vals, idx = osm.softmax_topk(x, w["K"])
    torch.cuda.synchronize()
    g = torch.Generator().manual_seed(321)
    rows = torch.cat([torch.tensor([0, w["N"] - 1]),
                      torch.randperm(w["N"], generator=g)[:4096]])
    rr = rows.to(dev)
    xh = to_host(x.index_select(0, rr))
    v64, z64 = oracle.topk(xh, w["K"], "bf16")
    assert_topk_equal(to_host(vals.index_select(0, rr)), to_host(idx.index_select(0, rr)),
                      v64, z64, "bf16 32768x128256 K=50 sample")


def test_split_row_counters_reset(dev):
    """Split top-k merges each row in the workgroup that completes it, counted
    in a per-stream array that every call must leave cleared: back-to-back
    calls with other batch sizes, chunk counts and K on one stream, then on a
    second stream, each checked against the oracle."""
    cases = [(10, 100003, 5, 7), (3, 50001, 9, 13), (10, 100003, 5, 7), (37, 20011, 64, 3),
             (1, 200000, 1, 40), (10, 100003, 16, 2)]
    xs = {c: synth.logits(c[0], c[1], sigma=2.0, seed=sum(c), device=dev) for c in cases}
    s2 = torch.cuda.Stream()
    for stream in (None, s2):
        for c in cases:
            N, V, K, S = c
            print(f"split counters stream={'2nd' if stream else 'current'} N={N} V={V} K={K} S={S}",
                  flush=True)
            x = xs[c]
            if stream is None:
                vals, idx = osm.softmax_topk(x, K, kernel=osm.KERNEL_SPLIT, param=S)
            else:
                with torch.cuda.stream(stream):
                    vals, idx = osm.softmax_topk(x, K, kernel=osm.KERNEL_SPLIT, param=S,
                                                 stream=stream)
                stream.synchronize()
            torch.cuda.synchronize()
            v64, z64 = oracle.topk(to_host(x), K, "f32")
            assert_topk_equal(to_host(vals), to_host(idx), v64, z64, f"split counters {c}")


def test_split_calls_on_two_streams_at_once(dev):
    """Split top-k and split softmax enqueued alternately on two streams with
    no synchronisation between the calls: each stream has its own scratch and
    row counters, so every result must match the oracle."""
    cases = [(10, 100003, 5, 7), (3, 50001, 9, 13), (6, 30011, 64, 5)]
    xs = [synth.logits(N, V, sigma=2.0, seed=300 + i, device=dev)
          for i, (N, V, K, S) in enumerate(cases)]
    torch.cuda.synchronize()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    for rep in range(3):
        for i, (N, V, K, S) in enumerate(cases):
            s = sa if (rep + i) % 2 == 0 else sb
            print(f"two streams rep={rep} case={cases[i]}", flush=True)
            with torch.cuda.stream(s):
                vals, idx = osm.softmax_topk(xs[i], K, kernel=osm.KERNEL_SPLIT, param=S, stream=s)
                y = osm.softmax_fwd(xs[i], kernel=osm.KERNEL_SPLIT, param=S, stream=s)
            outs.append((i, vals, idx, y))
    sa.synchronize()
    sb.synchronize()
    torch.cuda.synchronize()
    ref = {}
    for i, vals, idx, y in outs:
        N, V, K, S = cases[i]
        if i not in ref:
            xh = to_host(xs[i])
            ref[i] = (oracle.topk(xh, K, "f32"), oracle.softmax(xh))
        (v64, z64), y64 = ref[i]
        assert_topk_equal(to_host(vals), to_host(idx), v64, z64, f"two streams {cases[i]}")
        assert_softmax_close(to_host(y), y64, f"two streams softmax {cases[i]}")


def test_split_merge_many_partials(dev):
    """The merge seeds its list with the largest of the partials' first keys
    for up to 256 partials per row and streams the rest: rows with more
    partials than that, K on both sides of the round-selection limit (16),
    chunks shorter than K (partials holding empty slots), and tied values."""
    cases = [(2, 300000, 5, 600), (2, 300000, 64, 300), (3, 20000, 17, 400), (1, 500000, 1, 1000),
             (5, 40000, 16, 257), (2, 65536, 64, 2048)]
    g = torch.Generator(device=dev).manual_seed(21)
    for N, V, K, S in cases:
        print(f"split merge N={N} V={V} K={K} S={S}", flush=True)
        x = synth.logits(N, V, sigma=2.0, seed=N * V + K, device=dev)
        vals, idx = osm.softmax_topk(x, K, kernel=osm.KERNEL_SPLIT, param=S)
        torch.cuda.synchronize()
        v64, z64 = oracle.topk(to_host(x), K, "f32")
        assert_topk_equal(to_host(vals), to_host(idx), v64, z64, f"split merge {N}x{V} K={K} S={S}")
        t = torch.randint(-2, 3, (N, V), generator=g, device=dev).float()
        vals, idx = osm.softmax_topk(t, K, kernel=osm.KERNEL_SPLIT, param=S)
        torch.cuda.synchronize()
        v64, z64 = oracle.topk(to_host(t), K, "f32")
        assert_topk_equal(to_host(vals), to_host(idx), v64, z64, f"split merge ties {N}x{V} K={K} S={S}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_subnormal_values(dev, dtype):
    """Top-k values below 2^-126 are rounded, not flushed: the row maximum is 0
    and the next largest elements sit at -88 ... -100, so the K-th value is a
    binary32 subnormal; each value within 1e-5 of the oracle's plus one
    subnormal unit (2^-149)."""
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    V = 5000
    rows = []
    for r in range(6):
        row = np.full(V, -200.0)
        row[(r * 997) % V] = 0.0
        pos = (np.arange(12) * 389 + r * 17) % V
        pos = pos[pos != (r * 997) % V]
        row[pos] = -88.0 - np.arange(len(pos))
        rows.append(row)
    x = torch.tensor(np.array(rows), dtype=tdt, device=dev)
    K = 10
    cases = [(osm.KERNEL_ROWS, p) for p in SHAPES] + [(osm.KERNEL_SPLIT, 3)]
    for kernel, param in cases:
        vals, idx = osm.softmax_topk(x, K, kernel=kernel, param=param)
        torch.cuda.synchronize()
        v64, z64 = oracle.topk(to_host(x), K, host_dtype(x))
        what = f"subnormal top-k {dtype} kernel {kernel} param {param}"
        assert_topk_equal(to_host(vals), to_host(idx), v64, z64, what)
        assert (v64 < 2.0 ** -126).sum() > 20
        err = np.abs(to_host(vals).astype(np.float64) - v64)
        tiny = v64 < 2.0 ** -126
        assert (err[tiny] <= 1e-5 * v64[tiny] + 2.0 ** -149).all(), what


def test_split_plan_stays_within_two_workgroups_per_cu(dev):
    """The top-k plan splits a small batch of long rows into chunks (a
    workgroup each) whose count keeps the grid within two workgroups per CU,
    with at least two chunks a row and at most 512 / K (the merge's one
    register batch); and the planned call agrees with the oracle."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    for N, V, K in ((10, 1_000_000, 5), (10, 4_000_000, 5), (20, 1_000_000, 10), (200, 200_000, 5),
                    (300, 100_000, 5), (4, 1_000_000, 10), (64, 128_256, 50)):
        kernel, S = osm.topk_plan(N, V, K)
        print(f"plan N={N} V={V} K={K}: ({kernel}, {S})", flush=True)
        assert kernel == osm.KERNEL_SPLIT, (N, V, K, kernel, S)
        assert 2 <= S <= max(2, 2 * cus // N), (N, V, K, S, cus)
        assert S <= V // 4096 and S * K <= 512, (N, V, K, S)
        if 2 * cus // N >= 2:
            assert N * S <= 2 * cus, (N, S, cus)
    # one planned call, checked against the oracle
    x = synth.logits(10, 1_000_000, sigma=3.0, seed=77, device=dev)
    vals, idx = osm.softmax_topk(x, 5)
    torch.cuda.synchronize()
    v64, z64 = oracle.topk(to_host(x), 5, "f32")
    assert_topk_equal(to_host(vals), to_host(idx), v64, z64, "planned split 10x1e6 K=5")
