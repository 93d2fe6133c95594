"""The interleaved history layout on the GPU, through the C ABI.

The same history held in chunk-interleaved lanes instead of contiguous slots:
the pushed entries read back bit for bit (ragged segments, zeroed padding,
FIFO order), predictions agree with the oracle on the same stored inputs
under the floored bound and with the slot layout's predictions bit for bit
(the arithmetic and its order are the same), for every history size and
storage type, every workload (every element at a reduced size, sampled at
full size), several targets per pass, the residual form and the online stage
driven by the offline table.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_23429_amd as cheb
from synth import CONFIGS, make_history, split_segments, by_name
from tests.gpu_util import check_parity, say, to_host_bits

pytestmark = pytest.mark.gpu

DT = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}
INT = {"bf16": torch.int16, "f16": torch.int16, "f32": torch.int32}


def _bits_equal(a, b, dtype):
    return torch.equal(a.view(INT[dtype]), b.view(INT[dtype]))


def _rand_segs(seg, dtype, seed):
    out = []
    for k, m in enumerate(seg):
        g = torch.Generator(device="cuda")
        g.manual_seed(seed * 97 + k)
        out.append(torch.randn(m, generator=g, device="cuda").to(DT[dtype]))
    return out


def _pair(n, dtype, seg):
    return (cheb.ChebCache(n, DT[dtype], seg, layout="slots"),
            cheb.ChebCache(n, DT[dtype], seg, layout="interleaved"))


# Segment mixes: ragged sizes inside a chunk, across chunk boundaries, and
# an entry that is not a whole number of chunks.
RAGGED = [13, 1, 8, 1_000_003, 0, 4096 * 3 + 7, 16384 * 2 + 5]


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
def test_interleaved_entries_fifo_and_padding(dtype):
    n = 4
    sl, il = _pair(n, dtype, RAGGED)
    pushed = []
    ts = [999.0, 979.0, 959.0, 939.0, 919.0, 899.0, 879.0]
    vec = 4 if dtype == "f32" else 8
    for i, t in enumerate(ts):
        say(f"interleaved ring dtype={dtype} push {i}")
        segs = _rand_segs(RAGGED, dtype, i)
        sl.push(t, segs)
        il.push(t, segs)
        pushed.append((t, segs))
        torch.cuda.synchronize()
        held = pushed[-n:]
        assert il.history().tolist() == [p[0] for p in held]
        for age, (_, psegs) in enumerate(held):
            flat = to_host_bits(il.entry(age))
            assert flat.size == il.slot_numel
            for s, (off, m) in enumerate(zip(il.seg_offset, il.seg_numel)):
                assert np.array_equal(flat[off:off + m], to_host_bits(psegs[s])), (i, age, s)
                pad_end = off + -(-m // vec) * vec
                assert np.all(flat[off + m:pad_end] == 0), "padding not zeroed"
    for target in (859.0, 700.0):
        o1, w1 = sl.extrapolate_at(target)
        o2, w2 = il.extrapolate_at(target)
        torch.cuda.synchronize()
        assert np.array_equal(w1, w2)
        assert _bits_equal(o1, o2, dtype), target
        w_or = oracle.weights_row(il.history(), target)
        got = to_host_bits(o2)
        hosts = [to_host_bits(il.entry(a)) for a in range(n)]
        for s, (off, m) in enumerate(zip(il.seg_offset, il.seg_numel)):
            check_parity(got[off:off + m], [h[off:off + m] for h in hosts], w_or, dtype,
                         f"seg{s} t={target}")
    sl.close()
    il.close()


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("n", range(1, 9))
def test_interleaved_every_history_size(dtype, n):
    seg = [70_001, 16384 * 3, 9]
    sl, il = _pair(n, dtype, seg)
    nodes = [float(100 - 7 * k) for k in range(n + 2)]
    for i, t in enumerate(nodes):
        segs = _rand_segs(seg, dtype, 1000 * n + i)
        sl.push(t, segs)
        il.push(t, segs)
    held = nodes[-n:]
    rng = np.random.default_rng(n)
    targets = [held[-1] - 7 * rng.uniform(0.2, 2.0) for _ in range(3)]
    outs_s, _ = sl.extrapolate_at_multi(targets)
    outs_i, w = il.extrapolate_at_multi(targets)
    torch.cuda.synchronize()
    hosts = [to_host_bits(il.entry(a)) for a in range(n)]
    for m, t in enumerate(targets):
        assert _bits_equal(outs_s[m], outs_i[m], dtype), (n, t)
        check_parity(to_host_bits(outs_i[m]), hosts, oracle.weights_row(held, t), dtype,
                     f"n={n} t={t:.3f}")
    sl.close()
    il.close()


def test_interleaved_multi_target_equals_single():
    cfg = by_name("flux_dev_1024").shrunk(2_000_000)
    entries = make_history(cfg, "cuda")
    il = cheb.ChebCache(cfg.n_hist, torch.bfloat16, cfg.seg_numel, layout="interleaved")
    for x, e in zip(cfg.nodes, entries):
        il.push(x, split_segments(e, cfg))
    targets = [0.48, 0.46, 0.44, 0.42, 0.40, 0.38, 0.36, 0.34]
    for m in range(1, 9):
        outs, _ = il.extrapolate_at_multi(targets[:m])
        torch.cuda.synchronize()
        for k in range(m):
            single, _ = il.extrapolate_at(targets[k])
            torch.cuda.synchronize()
            assert _bits_equal(outs[k], single, "bf16"), (m, k)
    il.close()


def test_interleaved_arena_not_on_a_64k_boundary():
    """An arena that is 256-byte aligned but not 64 KiB aligned: the library
    starts the lanes at the next 64 KiB boundary inside it."""
    seg = [300_000, 17]
    need = cheb.cheb_cache_arena_bytes_ex(5, cheb.CHEB_BF16, seg, cheb.CHEB_LAYOUT_INTERLEAVED)
    big = torch.empty(need + 65536, dtype=torch.uint8, device="cuda")
    shift = (256 - big.data_ptr() % 65536) % 65536 or 256
    arena = big[shift:shift + need]
    assert arena.data_ptr() % 256 == 0 and arena.data_ptr() % 65536 != 0
    il = cheb.ChebCache(5, torch.bfloat16, seg, arena=arena, layout="interleaved")
    sl = cheb.ChebCache(5, torch.bfloat16, seg)
    for i, t in enumerate([0.9, 0.8, 0.7, 0.6, 0.5]):
        segs = _rand_segs(seg, "bf16", 50 + i)
        il.push(t, segs)
        sl.push(t, segs)
    o1, _ = il.extrapolate_at(0.45)
    o2, _ = sl.extrapolate_at(0.45)
    torch.cuda.synchronize()
    assert _bits_equal(o1, o2, "bf16")
    for a in range(5):
        assert _bits_equal(il.entry(a), sl.entry(a), "bf16"), a
    il.close()
    sl.close()


@pytest.mark.parametrize("cfg", CONFIGS, ids=lambda c: c.name)
def test_interleaved_workload_small_all_elements(cfg):
    small = cfg.shrunk(600_000)
    say(f"interleaved workload {cfg.name} (small, {small.numel} elems)")
    entries = make_history(small, "cuda")
    il = cheb.ChebCache(small.n_hist, DT[small.dtype], small.seg_numel, layout="interleaved")
    for x, e in zip(small.nodes, entries):
        il.push(x, split_segments(e, small))
    hosts = [to_host_bits(e) for e in entries]
    for t in small.targets:
        out, _ = il.extrapolate_at(t)
        torch.cuda.synchronize()
        check_parity(to_host_bits(out), hosts, oracle.weights_row(small.nodes, t), small.dtype,
                     f"{cfg.name} t={t}")
    il.close()


def _sample_indices(numel, seg_offsets, seg_numel, count, seed):
    rng = np.random.default_rng(seed)
    idx = [rng.integers(0, numel, size=count), np.arange(min(4096, numel)),
           np.arange(max(0, numel - 4096), numel)]
    for off, m in zip(seg_offsets, seg_numel):
        idx.append(np.arange(off, off + min(16, m)))
        idx.append(np.arange(max(off, off + m - 16), off + m))
    return np.unique(np.concatenate(idx))


@pytest.mark.parametrize("cfg", [c for c in CONFIGS if c.name != "tiny"], ids=lambda c: c.name)
def test_interleaved_workload_full_size(cfg):
    """Full cache shape in the launch shape the benchmark times: every element
    equal bit for bit to the slot layout's prediction, and a sample (random
    elements, both ends of the cache and of every segment) against the
    oracle."""
    cheb.cheb_set_launch_config(**cheb.DEFAULT_LAUNCH_CONFIG)
    say(f"interleaved workload {cfg.name} full size: {cfg.numel} x {cfg.n_hist}")
    entries = make_history(cfg, "cuda")
    il = cheb.ChebCache(cfg.n_hist, DT[cfg.dtype], cfg.seg_numel, layout="interleaved")
    sl = cheb.ChebCache(cfg.n_hist, DT[cfg.dtype], cfg.seg_numel)
    for x, e in zip(cfg.nodes, entries):
        il.push(x, split_segments(e, cfg))
        sl.push(x, split_segments(e, cfg))
    idx = _sample_indices(cfg.numel, il.seg_offset, il.seg_numel, 1 << 19, cfg.seed)
    idx_t = torch.from_numpy(idx).to("cuda")
    hosts = [to_host_bits(e.index_select(0, idx_t)) for e in entries]
    o_il, o_sl = il.new_output(), sl.new_output()
    for t in cfg.targets:
        il.extrapolate_at(t, o_il)
        sl.extrapolate_at(t, o_sl)
        torch.cuda.synchronize()
        assert _bits_equal(o_il, o_sl, cfg.dtype), t
        e, nw = check_parity(to_host_bits(o_il.index_select(0, idx_t)), hosts,
                             oracle.weights_row(cfg.nodes, t), cfg.dtype, f"{cfg.name} t={t}")
        say(f"  t={t}: floored error {e:.3e}")
    il.close()
    sl.close()
    del entries, o_il, o_sl
    torch.cuda.empty_cache()


RES_TOL = 1e-5


@pytest.mark.parametrize("case", [("dit", lambda: by_name("dit_xl2_256").scaled_blocks(16, 4)),
                                  ("flux", lambda: by_name("flux_dev_1024").scaled_blocks(32, 3)),
                                  ("tiny", lambda: by_name("tiny"))], ids=lambda c: c[0])
def test_interleaved_residual_apply(case):
    cfg = case[1]()
    res_off, res_n = cfg.residual_map()
    entries = make_history(cfg, "cuda")
    il = cheb.ChebCache(cfg.n_hist, DT[cfg.dtype], cfg.seg_numel, layout="interleaved")
    sl = cheb.ChebCache(cfg.n_hist, DT[cfg.dtype], cfg.seg_numel)
    for x, e in zip(cfg.nodes, entries):
        il.push(x, split_segments(e, cfg))
        sl.push(x, split_segments(e, cfg))
    t = cfg.targets[-1]
    w = cheb.cheb_precompute_weights(il.history(), [t])[0]
    g = torch.Generator(device="cuda")
    g.manual_seed(9)
    x_in = torch.randn(res_n, generator=g, device="cuda")
    a, b = torch.empty_like(x_in), torch.empty_like(x_in)
    il.residual_apply(w, res_off, a, x_in)
    sl.residual_apply(w, res_off, b, x_in)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    exp, mag = oracle.residual([to_host_bits(e) for e in entries], oracle.weights_row(cfg.nodes, t),
                               il.seg_offset, il.seg_numel, res_off, res_n,
                               x_in=x_in.cpu().numpy(), dtype=cfg.dtype)
    err = oracle.parity_error(a.cpu().numpy().astype(np.float64), exp, mag)[0]
    say(f"interleaved residual {case[0]}: floored error {err:.3e}")
    assert err <= RES_TOL
    il.close()
    sl.close()


def test_interleaved_online_stage_from_table():
    """50 steps of Algorithm 1 from the offline table: full steps push,
    runs of skipped steps are predicted in one pass; every prediction equals
    the slot layout's bit for bit and the oracle's under the bound."""
    cfg = by_name("flux_dev_1024").shrunk(400_000)
    T, n = 50, cfg.n_hist
    x = 1.0 - np.arange(T) / 50.0
    table = cheb.ChebTable(T, 1, 1, 6, n, x, cheb.CHEB_SHORT_LOWER)
    il = cheb.ChebCache(n, torch.bfloat16, cfg.seg_numel, layout="interleaved")
    sl = cheb.ChebCache(n, torch.bfloat16, cfg.seg_numel)
    runs = dict(table.runs())
    host = {}
    s, k, checked = 0, 0, 0
    while s < T:
        if not table.step(s)[0]:
            e = make_history(cfg, "cuda", nodes=[x[s]], seed=cfg.seed + s)[0]
            il.push(float(x[s]), split_segments(e, cfg))
            sl.push(float(x[s]), split_segments(e, cfg))
            host[s] = to_host_bits(e)
            s += 1
            continue
        c = runs[s]
        oi = il.extrapolate_steps(table, s, c)
        os_ = sl.extrapolate_steps(table, s, c)
        torch.cuda.synchronize()
        for j in range(c):
            assert _bits_equal(oi[j], os_[j], "bf16"), s + j
            kind, nodes_j, w_j = oracle.table_row(T, 1, 1, 6, n, x, cheb.CHEB_SHORT_LOWER, s + j)
            assert kind == 1
            check_parity(to_host_bits(oi[j]), [host[q] for q in nodes_j], w_j, "bf16",
                         f"step {s + j}")
            checked += 1
        s += c
    assert checked > 0
    il.close()
    sl.close()
    table.close()


def test_interleaved_refuses_fused_push():
    il = cheb.ChebCache(3, torch.bfloat16, [1000], layout="interleaved")
    with pytest.raises(cheb.ChebError) as e:
        il.begin_push()
    assert e.value.code == cheb._binding.CHEB_E_INVAL
    il.close()
