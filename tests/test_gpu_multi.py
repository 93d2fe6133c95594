"""Multi-target prediction (every skipped step between two full steps from
one pass over the history) against the oracle and against the single-target
path, through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_23429_amd as cheb
from synth import CONFIGS, make_history, split_segments
from tests.gpu_util import check_parity, say, to_host_bits

pytestmark = pytest.mark.gpu

DT = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}


def _rand(n, numel, dtype, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return [torch.randn(numel, generator=g, device="cuda").to(DT[dtype]) for _ in range(n)]


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("n_src", [1, 3, 6, 8])
def test_combine_multi_all_output_counts(dtype, n_src):
    rng = np.random.default_rng(n_src)
    for n_out in range(1, 9):
        for numel in [5, 8 * 1024 + 3, 1_000_001]:
            say(f"multi dtype={dtype} n_src={n_src} n_out={n_out} numel={numel}")
            srcs = _rand(n_src, numel, dtype, seed=numel + n_src)
            x = np.arange(n_src, dtype=float)
            w = np.stack([oracle.weights_row(x, n_src - 1 + rng.uniform(0.2, 3.0))
                          for _ in range(n_out)])
            outs = [torch.empty(numel, dtype=DT[dtype], device="cuda") for _ in range(n_out)]
            cheb.combine_multi(srcs, w, outs)
            torch.cuda.synchronize()
            hosts = [to_host_bits(s) for s in srcs]
            for m in range(n_out):
                check_parity(to_host_bits(outs[m]), hosts, w[m], dtype, f"out {m}")
                # same arithmetic, same order as the single-target kernel: bit for bit
                single = torch.empty_like(outs[m])
                cheb.combine(srcs, w[m], single)
                torch.cuda.synchronize()
                assert torch.equal(single.view(torch.int32 if dtype == "f32" else torch.int16),
                                   outs[m].view(torch.int32 if dtype == "f32" else torch.int16))


@pytest.mark.parametrize("cfg", CONFIGS, ids=lambda c: c.name)
def test_workload_all_targets_one_pass(cfg):
    """Full cache shape: every target of the workload from one launch,
    sampled against the oracle."""
    say(f"multi workload {cfg.name}: {len(cfg.targets)} targets in one pass")
    entries = make_history(cfg, "cuda")
    cache = cheb.ChebCache(cfg.n_hist, DT[cfg.dtype], cfg.seg_numel)
    for x, e in zip(cfg.nodes, entries):
        cache.push(x, split_segments(e, cfg))
    outs, w = cache.extrapolate_at_multi(cfg.targets)
    torch.cuda.synchronize()
    rng = np.random.default_rng(cfg.seed)
    idx = np.unique(np.concatenate([rng.integers(0, cfg.numel, 1 << 19),
                                    np.arange(min(cfg.numel, 2048)),
                                    np.arange(cfg.numel - 2048, cfg.numel)]))
    it = torch.from_numpy(idx).to("cuda")
    hosts = [to_host_bits(e.index_select(0, it)) for e in entries]
    for m, t in enumerate(cfg.targets):
        w_or = oracle.weights_row(cfg.nodes, t)
        assert np.max(np.abs(w[m] - w_or)) <= 1e-12 * max(1.0, np.abs(w_or).sum()) ** 2
        check_parity(to_host_bits(outs[m].index_select(0, it)), hosts, w_or, cfg.dtype,
                     f"{cfg.name} t={t}")
    cache.close()
    del entries, outs, cache
    torch.cuda.empty_cache()
