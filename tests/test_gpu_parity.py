"""GPU parity of libcheb against the fp64 CPU oracle, through the C ABI.

Inputs are seeded and drawn once on the device; the oracle gets exact host
copies of the same stored values.  Floating-point results must satisfy the
floored relative bound (1e-2 for bfloat16 storage, 1e-5 for float32 storage);
bit patterns are compared exactly where the result is fixed bit for bit.
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle
import paper_2608_23429_amd as cheb
from synth import CONFIGS, make_history, split_segments, by_name
from tests.gpu_util import TOL, check_parity, decode, say, to_host_bits

pytestmark = pytest.mark.gpu

DT = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}
SHAPES = [
    {"block": 1024, "unroll": 1, "nontemporal": 1, "blocks_per_cu": 0},
    {"block": 256, "unroll": 4, "nontemporal": 1, "blocks_per_cu": 0},
    {"block": 256, "unroll": 1, "nontemporal": 0, "blocks_per_cu": 0},
    {"block": 256, "unroll": 2, "nontemporal": 1, "blocks_per_cu": 0},
    {"block": 512, "unroll": 2, "nontemporal": 0, "blocks_per_cu": 2},
    {"block": 512, "unroll": 1, "nontemporal": 1, "blocks_per_cu": 0},
    {"block": 256, "unroll": 4, "nontemporal": 0, "blocks_per_cu": 2},
    {"block": 1024, "unroll": 1, "nontemporal": 1, "blocks_per_cu": 8},
    {"block": 64, "unroll": 1, "nontemporal": 1, "blocks_per_cu": 0, "waves_per_cu": 0},
    {"block": 64, "unroll": 1, "nontemporal": 0, "blocks_per_cu": 0, "waves_per_cu": 4},
    {"block": 64, "unroll": 1, "nontemporal": 1, "blocks_per_cu": 4, "waves_per_cu": -1},
    {"block": 64, "unroll": 1, "nontemporal": 1, "blocks_per_cu": 0, "waves_per_cu": 32},
    {"block": 256, "unroll": 1, "nontemporal": 1, "blocks_per_cu": 0, "waves_per_cu": 12},
    {"block": 1024, "unroll": 1, "nontemporal": 1, "blocks_per_cu": 0, "waves_per_cu": 8},
]


@pytest.fixture(autouse=True)
def _default_shape():
    old = cheb.cheb_get_launch_config()
    yield
    cheb.cheb_set_launch_config(**old)
    torch.cuda.synchronize()


def _rand(n, numel, dtype, seed, scale=1.0):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return [(torch.randn(numel, generator=g, device="cuda") * scale).to(DT[dtype])
            for _ in range(n)]


# --------------------------------------------------------------------------
# Stateless combination: every history size, ragged sizes, every launch shape
# --------------------------------------------------------------------------

NUMELS = [1, 7, 8, 9, 255, 1000, 65536 + 13, 3 * 4 * 256 * 8 + 5, 1 << 20]


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("n", range(1, 9))
def test_combine_all_sizes(dtype, n):
    rng = np.random.default_rng(1000 + n)
    for numel in NUMELS:
        say(f"combine dtype={dtype} n={n} numel={numel}")
        srcs = _rand(n, numel, dtype, seed=numel * 31 + n)
        # extrapolation-like weights: from equispaced nodes, target ahead
        w = oracle.weights_row(np.arange(n, dtype=float), n - 1 + rng.uniform(0.1, 2.0))
        out = torch.empty(numel, dtype=DT[dtype], device="cuda")
        cheb.combine(srcs, w, out)
        torch.cuda.synchronize()
        check_parity(to_host_bits(out), [to_host_bits(s) for s in srcs], w, dtype,
                     f"n={n} numel={numel}")


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "b{block}_u{unroll}_nt{nontemporal}_g{blocks_per_cu}_w{waves}".format(
                             waves=s.get("waves_per_cu", 0), **s))
@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
def test_combine_launch_shapes(shape, dtype):
    cheb.cheb_set_launch_config(**shape)
    n = 6
    for numel in [5, 4096 * 8 + 3, 2_000_003]:
        say(f"shape={shape} dtype={dtype} numel={numel}")
        srcs = _rand(n, numel, dtype, seed=numel)
        w = oracle.weights_row([2, 5, 10, 14, 20, 25], 27)
        out = torch.empty(numel, dtype=DT[dtype], device="cuda")
        cheb.combine(srcs, w, out)
        torch.cuda.synchronize()
        check_parity(to_host_bits(out), [to_host_bits(s) for s in srcs], w, dtype, str(shape))


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
def test_launch_shapes_give_identical_bits(dtype):
    """Each element's sum runs in the same order whatever the launch shape,
    so every shape and occupancy cap of the tuning interface gives the same
    bits, for one output and for several (ragged size, interleaved-layout
    chunk formula not involved)."""
    n, numel = 6, 3 * 65536 + 4099
    srcs = _rand(n, numel, dtype, seed=77)
    w = oracle.weights([2, 5, 10, 14, 20, 25], [26, 27, 28])
    ref_one, ref_many = None, None
    for shape in SHAPES + [{"block": 64, "unroll": 1, "nontemporal": 1, "blocks_per_cu": 0,
                            "waves_per_cu": wv} for wv in (-1, 1, 6, 9, 16, 24)]:
        cheb.cheb_set_launch_config(**shape)
        one = torch.empty(numel, dtype=DT[dtype], device="cuda")
        cheb.combine(srcs, w[0], one)
        many = [torch.empty(numel, dtype=DT[dtype], device="cuda") for _ in range(3)]
        cheb.combine_multi(srcs, w, many)
        torch.cuda.synchronize()
        if ref_one is None:
            ref_one, ref_many = one, many
            check_parity(to_host_bits(one), [to_host_bits(s) for s in srcs], w[0], dtype, str(shape))
            continue
        assert torch.equal(one.view(torch.uint8), ref_one.view(torch.uint8)), shape
        for a, b in zip(many, ref_many):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), shape
        assert torch.equal(many[0].view(torch.uint8), one.view(torch.uint8)), shape


def test_combine_empty_and_nonzero_stream():
    out = torch.empty(0, dtype=torch.bfloat16, device="cuda")
    cheb.combine([out, out], [0.5, 0.5], out)
    s = torch.cuda.Stream()
    srcs = _rand(3, 300_001, "bf16", seed=5)
    out = torch.empty(300_001, dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        cheb.combine(srcs, [0.25, -1.0, 1.75], out, stream=s)
    s.synchronize()
    check_parity(to_host_bits(out), [to_host_bits(x) for x in srcs], [0.25, -1.0, 1.75], "bf16")


# --------------------------------------------------------------------------
# Bit-exact special cases
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
def test_unit_weights_copy_bitwise(dtype):
    """w = e_j: every output is entry j's stored value (K = 0 is the n = 1 case)."""
    numel = 123_457
    for n in (1, 4, 6, 8):
        srcs = _rand(n, numel, dtype, seed=77 + n)
        for j in range(n):
            w = np.zeros(n)
            w[j] = 1.0
            out = torch.empty(numel, dtype=DT[dtype], device="cuda")
            cheb.combine(srcs, w, out)
            torch.cuda.synchronize()
            got = decode(to_host_bits(out), dtype)
            ref = decode(to_host_bits(srcs[j]), dtype)
            assert np.array_equal(got, ref), (n, j)


def test_bf16_midpoint_weights_round_to_nearest_even():
    """w = (1/2, 1/2) on bfloat16 inputs in [1, 2): the fp32 sum is
    exact, so the output must be the correctly rounded bfloat16 of the exact
    mean, which the oracle's rounding routine gives bit for bit."""
    numel = 1 << 18
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    a = ((torch.rand(numel, generator=g, device="cuda") + 1.0)).to(torch.bfloat16)
    b = ((torch.rand(numel, generator=g, device="cuda") + 1.0)).to(torch.bfloat16)
    out = torch.empty(numel, dtype=torch.bfloat16, device="cuda")
    cheb.combine([a, b], [0.5, 0.5], out)
    torch.cuda.synchronize()
    ha, hb = to_host_bits(a), to_host_bits(b)
    exact = 0.5 * oracle.bf16_to_f64(ha) + 0.5 * oracle.bf16_to_f64(hb)
    expect = oracle.round_bf16(exact)
    got = to_host_bits(out)
    assert np.array_equal(got, expect)
    # ties really occur in this input, so the even rule is exercised
    # (inputs are multiples of 2^-7, so a tie is an odd multiple of 2^-8)
    ties = np.mod(exact * 256.0, 2.0) == 1.0
    assert ties.any()


def test_f16_midpoint_weights_round_to_nearest_even():
    """w = (1/2, 1/2) on float16 inputs in [1, 2): the fp32 sum is exact, so
    the output must be the correctly rounded float16 of the exact mean (the
    oracle's binary16 rounding), ties included."""
    numel = 1 << 18
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    a = (torch.rand(numel, generator=g, device="cuda") + 1.0).to(torch.float16)
    b = (torch.rand(numel, generator=g, device="cuda") + 1.0).to(torch.float16)
    out = torch.empty(numel, dtype=torch.float16, device="cuda")
    cheb.combine([a, b], [0.5, 0.5], out)
    torch.cuda.synchronize()
    exact = 0.5 * oracle.f16_to_f64(to_host_bits(a)) + 0.5 * oracle.f16_to_f64(to_host_bits(b))
    assert np.array_equal(to_host_bits(out), oracle.round_f16(exact))
    ties = np.mod(exact * 2048.0, 2.0) == 1.0    # inputs are multiples of 2^-10
    assert ties.any()


def test_f16_overflow_and_subnormal_outputs():
    """float16 results past the largest finite value become +-Inf, and tiny
    results land on the subnormals, exactly as the oracle's rounding of the
    fp32 sum (weights (1, 1) keep every sum exact in fp32)."""
    numel = 1 << 16
    g = torch.Generator(device="cuda")
    g.manual_seed(6)
    big = ((torch.rand(numel, generator=g, device="cuda") * 2 - 1) * 60000.0).to(torch.float16)
    tiny = ((torch.rand(numel, generator=g, device="cuda") * 2 - 1) * 6e-5).to(torch.float16)
    for x in (big, tiny):
        out = torch.empty_like(x)
        cheb.combine([x, x], [1.0, 1.0], out)
        torch.cuda.synchronize()
        exact = 2.0 * oracle.f16_to_f64(to_host_bits(x))
        assert np.array_equal(to_host_bits(out), oracle.round_f16(exact))
    assert np.isinf(oracle.f16_to_f64(oracle.round_f16(2.0 * oracle.f16_to_f64(to_host_bits(big))))).any()


# --------------------------------------------------------------------------
# History ring on the device
# --------------------------------------------------------------------------

RAGGED = [13, 1, 8, 1_000_003, 0, 4096 * 3 + 7]


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
def test_ring_push_eviction_and_padding(dtype):
    n = 4
    cache = cheb.ChebCache(n, DT[dtype], RAGGED)
    pushed = []
    ts = [999.0, 979.0, 959.0, 939.0, 919.0, 899.0, 879.0]
    for i, t in enumerate(ts):
        say(f"ring dtype={dtype} push {i}")
        segs = []
        for s, m in enumerate(RAGGED):
            g = torch.Generator(device="cuda")
            g.manual_seed(100 * i + s)
            segs.append(torch.randn(m, generator=g, device="cuda").to(DT[dtype]))
        cache.push(t, segs)
        pushed.append((t, segs))
        torch.cuda.synchronize()
        held = pushed[-n:]
        assert cache.history().tolist() == [p[0] for p in held]
        for age, (_, psegs) in enumerate(held):
            flat = to_host_bits(cache.entry(age))
            for s, (off, m) in enumerate(zip(cache.seg_offset, cache.seg_numel)):
                assert np.array_equal(flat[off:off + m], to_host_bits(psegs[s])), (i, age, s)
                end = off + m
                vec = 4 if dtype == "f32" else 8
                pad_end = -(-m // vec) * vec + off
                assert np.all(flat[end:pad_end] == 0), "padding not zeroed"
    # Prediction over the held entries, per segment, against the oracle.
    out, w = cache.extrapolate_at(859.0)
    torch.cuda.synchronize()
    w_or = oracle.weights_row(cache.history(), 859.0)
    assert np.max(np.abs(w - w_or)) <= 1e-12 * np.abs(w_or).sum() ** 2
    got = to_host_bits(out)
    hosts = [to_host_bits(cache.entry(a)) for a in range(n)]
    for s, (off, m) in enumerate(zip(cache.seg_offset, cache.seg_numel)):
        check_parity(got[off:off + m], [h[off:off + m] for h in hosts], w_or, dtype, f"seg{s}")
    cache.close()


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
def test_fused_push_matches_copy_push(dtype):
    seg = [4096 * 8, 1000, 24]
    a = cheb.ChebCache(3, DT[dtype], seg)
    b = cheb.ChebCache(3, DT[dtype], seg)
    pushed = []
    for i, t in enumerate([0.96, 0.9, 0.8, 0.72]):
        segs = [(_rand(1, m, dtype, seed=10 * i + k)[0]) for k, m in enumerate(seg)]
        pushed.append(segs)
        a.push(t, segs)
        slot = b.begin_push()
        for view, src in zip(b.segment_views(slot), segs):
            view.copy_(src)
        b.commit(t)
    torch.cuda.synchronize()
    assert a.history().tolist() == b.history().tolist() == [0.9, 0.8, 0.72]
    oa, _ = a.extrapolate_at(0.6)
    ob, _ = b.extrapolate_at(0.6)
    torch.cuda.synchronize()
    w = oracle.weights_row([0.9, 0.8, 0.72], 0.6)
    for s_idx, va in enumerate(a.segment_views(oa)):
        check_parity(to_host_bits(va), [to_host_bits(p[s_idx]) for p in pushed[1:]], w, dtype,
                     f"copy push segment {s_idx}")
    for va, vb in zip(a.segment_views(oa), b.segment_views(ob)):
        assert torch.equal(va.view(torch.int32 if dtype == "f32" else torch.int16),
                           vb.view(torch.int32 if dtype == "f32" else torch.int16))
    a.close()
    b.close()


# --------------------------------------------------------------------------
# The five workloads
# --------------------------------------------------------------------------

def _run_workload(cfg, nodes, targets, time_scale=None, label=""):
    """Seeded history on the device -> push through the ring -> one
    prediction per target; returns (cache, entries, outputs, weights)."""
    entries = make_history(cfg, "cuda", nodes=nodes, time_scale=time_scale)
    cache = cheb.ChebCache(cfg.n_hist, DT[cfg.dtype], cfg.seg_numel)
    for x, e in zip(nodes, entries):
        cache.push(x, split_segments(e, cfg))
    outs, ws = [], []
    for t in targets:
        out, w = cache.extrapolate_at(t)
        outs.append(out)
        ws.append(w)
    torch.cuda.synchronize()
    return cache, entries, outs, ws


# The paper's PixArt-Sigma and DiT-XL/2 also run with float16 activations:
# the same workloads with float16 storage.
F16_WORKLOADS = [replace(by_name("pixart_sigma_1024"), name="pixart_sigma_1024_f16", dtype="f16"),
                 replace(by_name("dit_xl2_256"), name="dit_xl2_256_f16", dtype="f16")]


@pytest.mark.parametrize("cfg", CONFIGS + F16_WORKLOADS, ids=lambda c: c.name)
def test_workload_small_all_elements(cfg):
    """Each workload's schedule and generator on a cache cut down so the
    oracle checks every element (ragged segment mix kept)."""
    small = cfg.shrunk(600_000)
    readings = [(small.nodes, small.targets, None)]
    if small.alt_nodes is not None:
        readings.append((small.alt_nodes, small.alt_targets,
                         20.0 if cfg.name.startswith("pixart") else None))
    for nodes, targets, ts in readings:
        say(f"workload {cfg.name} (small, {small.numel} elems) nodes={nodes}")
        cache, entries, outs, ws = _run_workload(small, nodes, targets, ts)
        hosts = [to_host_bits(e) for e in entries]
        for t, out, w in zip(targets, outs, ws):
            w_or = oracle.weights_row(nodes, t)
            check_parity(to_host_bits(out), hosts, w_or, small.dtype, f"{cfg.name} t={t}")
        cache.close()
        del entries, outs
    torch.cuda.empty_cache()


def _sample_indices(numel, seg_offsets, seg_numel, count, seed):
    rng = np.random.default_rng(seed)
    idx = [rng.integers(0, numel, size=count)]
    idx.append(np.arange(min(4096, numel)))
    idx.append(np.arange(max(0, numel - 4096), numel))
    for off, m in zip(seg_offsets, seg_numel):       # both ends of every segment
        idx.append(np.arange(off, off + min(16, m)))
        idx.append(np.arange(max(off, off + m - 16), off + m))
    return np.unique(np.concatenate(idx))


@pytest.mark.parametrize("cfg", CONFIGS + F16_WORKLOADS, ids=lambda c: c.name)
def test_workload_full_size_sampled(cfg):
    """Full cache shape, default launch shape (the one the benchmark times):
    the oracle recomputes a sample of outputs (random elements, both ends of
    the cache and of every segment) from the same stored inputs."""
    cheb.cheb_set_launch_config(**cheb.DEFAULT_LAUNCH_CONFIG)
    say(f"workload {cfg.name} full size: {cfg.numel} elements x {cfg.n_hist}")
    cache, entries, outs, ws = _run_workload(cfg, cfg.nodes, cfg.targets)
    idx = _sample_indices(cfg.numel, cache.seg_offset, cache.seg_numel, 1 << 20, cfg.seed)
    idx_t = torch.from_numpy(idx).to("cuda")
    hosts = [to_host_bits(e.index_select(0, idx_t)) for e in entries]
    for t, out in zip(cfg.targets, outs):
        w_or = oracle.weights_row(cfg.nodes, t)
        got = to_host_bits(out.index_select(0, idx_t))
        e, nw = check_parity(got, hosts, w_or, cfg.dtype, f"{cfg.name} t={t}")
        say(f"  t={t}: floored error {e:.3e}, normwise {nw:.3e}, {idx.size} samples")
    cache.close()
    del entries, outs, cache
    torch.cuda.empty_cache()


@pytest.mark.parametrize("cfg", [c for c in CONFIGS if c.name != "tiny"], ids=lambda c: c.name)
def test_workload_full_size_every_element(cfg):
    """Full cache shape, interleaved history and the default launch shape
    (what the benchmark times), the workload's farthest target: every
    element against the oracle, in chunks of 2^26 elements, with the
    history read back from the ring."""
    cheb.cheb_set_launch_config(**cheb.DEFAULT_LAUNCH_CONFIG)
    say(f"workload {cfg.name} full size, every element: {cfg.numel} x {cfg.n_hist}")
    entries = make_history(cfg, "cuda")
    cache = cheb.ChebCache(cfg.n_hist, DT[cfg.dtype], cfg.seg_numel, layout="interleaved")
    for x, e in zip(cfg.nodes, entries):
        cache.push(x, split_segments(e, cfg))
    del entries
    t = cfg.targets[-1]
    out, _ = cache.extrapolate_at(t)
    stored = [cache.entry(k)[:cfg.numel] for k in range(cfg.n_hist)]
    torch.cuda.synchronize()
    w_or = oracle.weights_row(cfg.nodes, t)
    chunk = 1 << 26
    worst = 0.0
    for start in range(0, cfg.numel, chunk):
        stop = min(cfg.numel, start + chunk)
        hosts = [to_host_bits(h[start:stop]) for h in stored]
        e, _ = check_parity(to_host_bits(out[start:stop]), hosts, w_or, cfg.dtype,
                            f"{cfg.name} t={t} elements {start}..{stop}")
        worst = max(worst, e)
    say(f"  t={t}: floored error {worst:.3e} over all {cfg.numel} elements")
    cache.close()
    del stored, out, cache
    torch.cuda.empty_cache()


def test_tiny_recovers_quadratic():
    """Tiny workload: F_k = A + B tau + C tau^2 + 1e-3 noise, stored in fp32.
    The prediction at the next timesteps equals the quadratic at the target
    up to the combined noise (|w| sums to at most 2.14 here) and fp32
    storage rounding."""
    cfg = by_name("tiny")
    cache, entries, outs, ws = _run_workload(cfg, cfg.nodes, cfg.targets)
    g = torch.Generator(device="cuda")
    g.manual_seed(cfg.seed)
    coeffs = [torch.randn(cfg.numel, generator=g, device="cuda") * cfg.coeff_std
              for _ in range(cfg.degree + 1)]
    for t, out, w in zip(cfg.targets, outs, ws):
        tau = t / cfg.time_scale
        quad = (coeffs[0].double() + coeffs[1].double() * tau + coeffs[2].double() * tau * tau)
        dev = (out.double() - quad).abs().max().item()
        bound = 6 * cfg.noise_std * float(np.abs(w).sum()) + 1e-5
        assert dev <= bound, (t, dev, bound)
    cache.close()
