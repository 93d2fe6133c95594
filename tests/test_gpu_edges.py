"""Edge cases of the device path through the C ABI: non-finite inputs, a
target on a held node, the largest history the kernels take at the full
FLUX cache shape, and stream ordering of push and prediction."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_23429_amd as cheb
from synth import CONFIGS, make_history, split_segments, by_name
from tests.gpu_util import TOL, check_parity, decode, oracle_combine, say, to_host_bits

pytestmark = pytest.mark.gpu


def _classes(v):
    return np.where(np.isnan(v), 0, np.where(np.isposinf(v), 1, np.where(np.isneginf(v), 2, 3)))


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
def test_nonfinite_inputs_propagate_like_ieee(dtype):
    """NaN and +-Inf planted in the history: the output is NaN / +-Inf
    exactly where the fp64 oracle's is, finite elements keep the bound."""
    td = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[dtype]
    n, numel = 5, 100_003
    g = torch.Generator(device="cuda")
    g.manual_seed(19)
    srcs = [torch.randn(numel, generator=g, device="cuda").to(td) for _ in range(n)]
    rng = np.random.default_rng(19)
    for k in range(n):
        for val in (float("nan"), float("inf"), float("-inf")):
            idx = torch.from_numpy(rng.integers(0, numel, 300)).to("cuda")
            srcs[k].index_fill_(0, idx, val)
    w = oracle.weights_row([900, 820, 740, 660, 580], 560)
    out = torch.empty(numel, dtype=td, device="cuda")
    cheb.combine(srcs, w, out)
    torch.cuda.synchronize()
    hosts = [to_host_bits(s) for s in srcs]
    exp, mag = oracle_combine(hosts, w, dtype)
    got = decode(to_host_bits(out), dtype)
    fin = np.isfinite(exp)
    assert (~fin).sum() > 1000
    assert np.array_equal(_classes(got[~fin]), _classes(exp[~fin]))
    e = oracle.parity_error(got[fin], exp[fin], mag[fin])[0]
    assert e <= TOL[dtype]


def test_target_on_a_held_node_is_a_bit_copy():
    cfg = by_name("flux_dev_1024").shrunk(400_000)
    entries = make_history(cfg, "cuda")
    cache = cheb.ChebCache(cfg.n_hist, torch.bfloat16, cfg.seg_numel)
    for x, e in zip(cfg.nodes, entries):
        cache.push(x, split_segments(e, cfg))
    for j, x in enumerate(cfg.nodes):
        out, w = cache.extrapolate_at(x)
        torch.cuda.synchronize()
        assert w.tolist() == [1.0 if k == j else 0.0 for k in range(cfg.n_hist)]
        assert torch.equal(out.view(torch.int16), entries[j].view(torch.int16))
    cache.close()


def test_eight_entry_history_full_flux_shape():
    """K + 1 = 8 (the largest history the kernels take) on the full FLUX
    cache: eight full steps, sampled against the oracle."""
    cfg = by_name("flux_dev_1024")
    nodes = [1.0 - s / 50.0 for s in (2, 5, 8, 10, 14, 17, 20, 25)]
    say(f"eight-entry history: {cfg.numel} elements x 8")
    entries = make_history(cfg, "cuda", nodes=nodes)
    cache = cheb.ChebCache(8, torch.bfloat16, cfg.seg_numel)
    for x, e in zip(nodes, entries):
        cache.push(x, split_segments(e, cfg))
    targets = [0.48, 0.44, 0.40]
    outs, w = cache.extrapolate_at_multi(targets)
    torch.cuda.synchronize()
    idx = np.unique(np.random.default_rng(8).integers(0, cfg.numel, 1 << 18))
    it = torch.from_numpy(idx).to("cuda")
    hosts = [to_host_bits(e.index_select(0, it)) for e in entries]
    for m, t in enumerate(targets):
        check_parity(to_host_bits(outs[m].index_select(0, it)), hosts,
                     oracle.weights_row(nodes, t), "bf16", f"8 entries t={t}")
    cache.close()
    del entries, outs
    torch.cuda.empty_cache()


def test_push_then_predict_ordered_on_one_stream():
    """Pushes and predictions issued back to back on one non-default stream,
    with no host synchronisation between them, see each other's writes."""
    cfg = by_name("dit_xl2_256").shrunk(300_000)
    s = torch.cuda.Stream()
    entries = make_history(cfg, "cuda", nodes=[900.0, 820.0, 740.0, 660.0, 580.0, 500.0, 420.0])
    torch.cuda.synchronize()
    cache = cheb.ChebCache(5, torch.bfloat16, cfg.seg_numel)
    outs = []
    with torch.cuda.stream(s):
        for i, (x, e) in enumerate(zip([900.0, 820.0, 740.0, 660.0, 580.0, 500.0, 420.0], entries)):
            cache.push(x, split_segments(e, cfg), stream=s)
            if i >= 4:
                outs.append((cache.history().tolist(), cache.extrapolate_at(400.0, stream=s)[0]))
    s.synchronize()
    hosts = [to_host_bits(e) for e in entries]
    for hist, out in outs:
        first = [900.0, 820.0, 740.0, 660.0, 580.0, 500.0, 420.0].index(hist[0])
        check_parity(to_host_bits(out), hosts[first:first + 5], oracle.weights_row(hist, 400.0),
                     "bf16", f"history from {hist[0]}")
    cache.close()


def _max_numel(dtype):
    """Largest element count one launch takes: 2^31 - 1 whole 16-byte
    vectors plus a ragged tail of one element less than a vector."""
    per_vec = 4 if dtype == "f32" else 8
    return ((1 << 31) - 1) * per_vec + per_vec - 1


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
def test_largest_launch(dtype):
    """The largest problem the host accepts in one launch (32 GiB per
    buffer; the kernel's 32-bit vector indices reach 2^31 - 1): two sources,
    then two outputs from one pass, sampled against the oracle at both ends,
    around the last tile and at random."""
    numel = _max_numel(dtype)
    nbytes = numel * (4 if dtype == "f32" else 2)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()                        # blocks cached by earlier tests
    free, _ = torch.cuda.mem_get_info()
    if free < 4 * nbytes + (8 << 30):
        pytest.skip(f"needs {4 * nbytes + (8 << 30)} free bytes, {free} free")
    say(f"largest launch {dtype}: {numel} elements, {nbytes} bytes per buffer")
    td = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[dtype]
    g = torch.Generator(device="cuda")
    g.manual_seed(31)
    srcs = [torch.empty(numel, dtype=td, device="cuda").uniform_(-1.0, 1.0, generator=g)
            for _ in range(2)]
    outs = [torch.empty(numel, dtype=td, device="cuda") for _ in range(2)]
    nodes, targets = [0.0, 1.0], [1.25, 2.0]
    w = cheb.precompute_weights(nodes, targets)
    cheb.combine(srcs, w[0], outs[0])
    torch.cuda.synchronize()
    rng = np.random.default_rng(31)
    idx = np.unique(np.concatenate([
        np.arange(4096), np.arange(numel - 16384, numel),
        np.arange((numel // 2) - 2048, (numel // 2) + 2048),
        rng.integers(0, numel, 1 << 20)]))
    it = torch.from_numpy(idx).to("cuda")
    hosts = [to_host_bits(s.index_select(0, it)) for s in srcs]
    check_parity(to_host_bits(outs[0].index_select(0, it)), hosts,
                 oracle.weights_row(nodes, targets[0]), dtype, f"largest single {dtype}")
    outs[0].zero_()
    cheb.combine_multi(srcs, w, outs)
    torch.cuda.synchronize()
    for m, t in enumerate(targets):
        check_parity(to_host_bits(outs[m].index_select(0, it)), hosts,
                     oracle.weights_row(nodes, t), dtype, f"largest multi {dtype} t={t}")
    del srcs, outs
    torch.cuda.empty_cache()
