"""Residual application on a skipped step (block equation of Section 3.1
with every module output predicted) and the collapsed history, through the
C ABI, against the oracle's plain per-segment fp64 definition."""
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle
import paper_2608_23429_amd as cheb
from synth import CONFIGS, make_history, split_segments, by_name
from tests.gpu_util import say, to_host_bits

pytestmark = pytest.mark.gpu

DT = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}
RES_TOL = 1e-5      # fp64 accumulation, one fp32 rounding of the result
# Collapsed history: each entry r_k is the fp64 sum of one full step's module
# outputs rounded once to fp32, so |r_k - exact_k| <= 2^-24 |exact_k| <=
# 2^-24 sum_s |F_k[s]|; the prediction adds sum_k |w_k| of that, at most
# 2^-24 times the oracle's magnitude S, and rounds the fp64 result once to
# fp32 (2^-24 |o|).  Against max(|o|, 10^-3 S) the floored error is at most
# (1 + 10^3) * 2^-24 = 6.0e-5.
COLLAPSED_TOL = 1e-4


def _check(got, expect, mag, tol, label):
    e = oracle.parity_error(np.asarray(got, dtype=np.float64), expect, mag)[0]
    say(f"  {label}: floored error {e:.3e}")
    assert e <= tol, (label, e)
    return e


def _fill(cfg, nodes, seed_shift=0):
    entries = make_history(cfg, "cuda", nodes=nodes, seed=cfg.seed + seed_shift)
    cache = cheb.ChebCache(len(nodes), DT[cfg.dtype], cfg.seg_numel)
    for x, e in zip(nodes, entries):
        cache.push(x, split_segments(e, cfg))
    return entries, cache


def _x_in(n, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return torch.randn(n, generator=g, device="cuda") * 3.0


SMALL = [
    ("dit", lambda: by_name("dit_xl2_256").scaled_blocks(16, 4)),
    ("pixart", lambda: by_name("pixart_sigma_1024").scaled_blocks(64, 3)),
    ("flux", lambda: by_name("flux_dev_1024").scaled_blocks(32, 3)),
    ("tiny", lambda: by_name("tiny")),
    ("pixart_f16", lambda: replace(by_name("pixart_sigma_1024").scaled_blocks(64, 3), dtype="f16")),
]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: c[0])
def test_residual_apply_small(case):
    cfg = case[1]()
    res_off, res_n = cfg.residual_map()
    entries, cache = _fill(cfg, cfg.nodes)
    hosts = [to_host_bits(e) for e in entries]
    t = cfg.targets[-1]
    w = cheb.cheb_precompute_weights(cache.history(), [t])[0]
    x_in = _x_in(res_n, 7)
    x_out = torch.empty_like(x_in)
    say(f"residual {case[0]}: {len(cfg.segments)} segments, residual {res_n}")
    cache.residual_apply(w, res_off, x_out, x_in)
    torch.cuda.synchronize()
    w_or = oracle.weights_row(cfg.nodes, t)
    exp, mag = oracle.residual(hosts, w_or, cache.seg_offset, cache.seg_numel, res_off, res_n,
                               x_in=x_in.cpu().numpy(), dtype=cfg.dtype)
    _check(x_out.cpu().numpy(), exp, mag, RES_TOL, "with x_in")
    # no x_in, and in place
    cache.residual_apply(w, res_off, x_out, None)
    torch.cuda.synchronize()
    exp0, mag0 = oracle.residual(hosts, w_or, cache.seg_offset, cache.seg_numel, res_off, res_n,
                                 dtype=cfg.dtype)
    _check(x_out.cpu().numpy(), exp0, mag0, RES_TOL, "x_in = NULL")
    y = x_in.clone()
    cache.residual_apply(w, res_off, y, y)
    torch.cuda.synchronize()
    _check(y.cpu().numpy(), exp, mag, RES_TOL, "in place")
    cache.close()


def test_residual_more_segments_than_one_launch_holds():
    """300 segments over one residual: the covering list is split across
    launches that accumulate in place."""
    L = 4096
    cfg = by_name("dit_xl2_256").with_segments([(1, 4, 1024)] * 300)
    entries, cache = _fill(cfg, cfg.nodes)
    w = cheb.cheb_precompute_weights(cache.history(), [cfg.targets[0]])[0]
    x_out = torch.empty(L, dtype=torch.float32, device="cuda")
    cache.residual_apply(w, [0] * 300, x_out, None)
    torch.cuda.synchronize()
    exp, mag = oracle.residual([to_host_bits(e) for e in entries],
                               oracle.weights_row(cfg.nodes, cfg.targets[0]),
                               cache.seg_offset, cache.seg_numel, [0] * 300, L)
    _check(x_out.cpu().numpy(), exp, mag, RES_TOL, "300 segments")
    cache.close()


def test_residual_partial_coverage_and_unmapped_segments():
    """Segments covering different parts of the residual, one left out."""
    cfg = by_name("pixart_sigma_1024").with_segments([(64, 8), (32, 8), (16, 8), (64, 8), (8, 8)])
    res_off = [0, 256, 128, 0, -1]
    L = 64 * 8
    entries, cache = _fill(cfg, cfg.nodes)
    w = cheb.cheb_precompute_weights(cache.history(), [cfg.targets[1]])[0]
    x_in = _x_in(L, 3)
    x_out = torch.empty_like(x_in)
    cache.residual_apply(w, res_off, x_out, x_in)
    torch.cuda.synchronize()
    exp, mag = oracle.residual([to_host_bits(e) for e in entries],
                               oracle.weights_row(cfg.nodes, cfg.targets[1]),
                               cache.seg_offset, cache.seg_numel, res_off, L,
                               x_in=x_in.cpu().numpy())
    _check(x_out.cpu().numpy(), exp, mag, RES_TOL, "partial coverage")
    cache.close()


@pytest.mark.parametrize("case", SMALL[:3] + SMALL[4:], ids=lambda c: c[0])
def test_collapsed_history_equals_full_form(case):
    """Push-time reduction into a residual-sized fp32 ring, then the skipped
    step's residual from it, against the oracle on the full history."""
    cfg = case[1]()
    res_off, res_n = cfg.residual_map()
    entries = make_history(cfg, "cuda")
    hist = cheb.ResidualHistory(cfg.n_hist, res_off, res_n)
    for x, e in zip(cfg.nodes, entries):
        hist.push(x, split_segments(e, cfg))
    # the reduction alone: one entry against the oracle with w = [1]
    lay = cheb.cheb_cache_layout(1, cheb.CHEB_BF16, cfg.seg_numel)
    seg_off = [int(o) for o in lay["seg_offset"]]
    red = hist.cache.entry(cfg.n_hist - 1)[:res_n].cpu().numpy()
    exp1, mag1 = oracle.residual([to_host_bits(entries[-1])], [1.0], seg_off, cfg.seg_numel,
                                 res_off, res_n, dtype=cfg.dtype)
    _check(red, exp1, mag1, RES_TOL, "push-time reduction")
    x_in = _x_in(res_n, 11)
    for t in cfg.targets:
        x_out = torch.empty_like(x_in)
        hist.predict(t, x_out, x_in)
        torch.cuda.synchronize()
        exp, mag = oracle.residual([to_host_bits(e) for e in entries],
                                   oracle.weights_row(cfg.nodes, t), seg_off, cfg.seg_numel,
                                   res_off, res_n, x_in=x_in.cpu().numpy(), dtype=cfg.dtype)
        _check(x_out.cpu().numpy(), exp, mag, COLLAPSED_TOL, f"collapsed t={t}")
    hist.close()


# Entries rounded once to fp32 from an exact fp64 difference: per element the
# error is at most 2^-24 * sum_k |w_k| |d_k| (entries) plus 2^-24 |o| (the
# output), so the floored error stays below (1 + 10^3) * 2^-24 = 6.0e-5.
DIFF_TOL = 1e-4


@pytest.mark.parametrize("case", SMALL[:3], ids=lambda c: c[0])
def test_collapsed_history_from_residual_difference(case):
    """The collapsed entry taken as x_after - x_before of a full step's
    block stack (ResidualHistory.push_difference): each entry is the
    oracle's exact difference rounded once to fp32, bit for bit, and by the
    block equation the oracle's sum of the step's module outputs up to the
    fp32 rounding of x_after; the prediction against the oracle's
    x_in + sum_k w_k (x_after_k - x_before_k) in fp64."""
    cfg = case[1]()
    res_off, res_n = cfg.residual_map()
    entries = make_history(cfg, "cuda")
    lay = cheb.cheb_cache_layout(1, cheb.CHEB_BF16, cfg.seg_numel)
    seg_off = [int(o) for o in lay["seg_offset"]]
    befores, afters = [], []
    for k, e in enumerate(entries):
        xb = _x_in(res_n, 100 + k)
        full, _ = oracle.residual([to_host_bits(e)], [1.0], seg_off, cfg.seg_numel, res_off, res_n,
                                  x_in=xb.cpu().numpy())
        befores.append(xb)
        afters.append(torch.from_numpy(full.astype(np.float32)).to("cuda"))
    diff = cheb.ResidualHistory(cfg.n_hist, res_off, res_n)
    red = cheb.ResidualHistory(cfg.n_hist, res_off, res_n)
    for x, e, xa, xb in zip(cfg.nodes, entries, afters, befores):
        diff.push_difference(x, xa, xb)
        red.push(x, split_segments(e, cfg))
    torch.cuda.synchronize()
    hosts_a = [a.cpu().numpy() for a in afters]
    hosts_b = [b.cpu().numpy() for b in befores]
    for k in range(cfg.n_hist):
        d = diff.cache.entry(k)[:res_n].cpu().numpy()
        # the entry is the exact difference rounded once to fp32: bit for bit
        exact, _ = oracle.residual([hosts_a[k], hosts_b[k]], [1.0, -1.0], [0], [res_n], [0], res_n,
                                   dtype="f32")
        assert np.array_equal(d.view(np.uint32), exact.astype(np.float32).view(np.uint32)), k
        # and, by the block equation, the sum of the step's module outputs up
        # to the fp32 rounding of x_after
        outs_sum, _ = oracle.residual([to_host_bits(entries[k])], [1.0], seg_off, cfg.seg_numel,
                                      res_off, res_n)
        scale = float((np.abs(hosts_a[k]) + np.abs(hosts_b[k])).max())
        assert np.max(np.abs(d - outs_sum)) <= 3 * 2.0 ** -24 * scale, k
        r = red.cache.entry(k)[:res_n].cpu().numpy()
        assert np.max(np.abs(r - outs_sum)) <= 2.0 ** -24 * np.abs(outs_sum).max() + 1e-30, k
    x_in = _x_in(res_n, 12)
    for t in cfg.targets:
        x_out = torch.empty_like(x_in)
        _, w = diff.predict(t, x_out, x_in)
        torch.cuda.synchronize()
        w_or = oracle.weights_row(cfg.nodes, t)
        exp, mag = oracle.residual(hosts_a + hosts_b, np.concatenate([w_or, -w_or]), [0], [res_n],
                                   [0], res_n, x_in=x_in.cpu().numpy(), dtype="f32")
        _check(x_out.cpu().numpy(), exp, mag, DIFF_TOL, f"difference-form t={t}")
    with pytest.raises(cheb.ChebError):
        diff.push_difference(0.0, afters[0][:-4], befores[0][:-4])
    diff.close()
    red.close()


def _compact_problem(cfg, entries, res_off, res_n, seg_off, idx):
    """Sampled residual elements idx: per segment, the source value each
    sampled element receives (zero where the segment does not cover it), so
    the oracle evaluates the same sum on a compact layout."""
    m = idx.size
    cols = []
    for s, (so, sn, ro) in enumerate(zip(seg_off, cfg.seg_numel, res_off)):
        src = np.full(m, -1, dtype=np.int64)
        if ro >= 0:
            inside = (idx >= ro) & (idx < ro + sn)
            src[inside] = so + idx[inside] - ro
        cols.append(src)
    compact = []
    for e in entries:
        vals = []
        for src in cols:
            take = torch.from_numpy(np.where(src >= 0, src, 0)).to("cuda")
            v = e.index_select(0, take)
            v = torch.where(torch.from_numpy(src >= 0).to("cuda"), v, torch.zeros_like(v))
            vals.append(v)
        compact.append(to_host_bits(torch.cat(vals)))
    n_seg = len(cols)
    return compact, [s * m for s in range(n_seg)], [m] * n_seg, [0] * n_seg, m


@pytest.mark.parametrize("cfg", [c for c in CONFIGS if c.name != "tiny"], ids=lambda c: c.name)
def test_residual_full_size_sampled(cfg):
    res_off, res_n = cfg.residual_map()
    entries, cache = _fill(cfg, cfg.nodes)
    t = cfg.targets[0]
    w = cheb.cheb_precompute_weights(cache.history(), [t])[0]
    x_in = _x_in(res_n, 5)
    x_out = torch.empty_like(x_in)
    say(f"residual {cfg.name} full size: {len(cfg.segments)} segments, residual {res_n}")
    cache.residual_apply(w, res_off, x_out, x_in)
    torch.cuda.synchronize()
    rng = np.random.default_rng(cfg.seed)
    idx = np.unique(np.concatenate([rng.integers(0, res_n, 20000), np.arange(64),
                                    np.arange(res_n - 64, res_n)]))
    comp, so, sn, ro, m = _compact_problem(cfg, entries, res_off, res_n, cache.seg_offset, idx)
    exp, mag = oracle.residual(comp, oracle.weights_row(cfg.nodes, t), so, sn, ro, m,
                               x_in=x_in.cpu().numpy()[idx])
    _check(x_out.cpu().numpy()[idx], exp, mag, RES_TOL, f"{cfg.name} sampled")
    cache.close()
    del entries
    torch.cuda.empty_cache()
