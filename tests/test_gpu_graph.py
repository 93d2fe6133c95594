"""Skipped-step predictions captured in a HIP graph (torch.cuda.CUDAGraph)
and replayed: the library only launches kernels (no allocation, no memset),
so captured predictions replay to the same bits as eager ones, which are
checked against the oracle first.  Every replay is checked, with eager work
and synchronisation in between.  Pushes
are not captured: they update host-side ring state at call time."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_23429_amd as cheb
from synth import CONFIGS, make_history, split_segments, by_name
from tests.gpu_util import check_parity, to_host_bits

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg", [by_name("tiny"), by_name("flux_dev_1024").shrunk(2_000_000)], ids=["tiny", "flux_small"])
def test_predictions_replay_from_a_graph(cfg):
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    entries = make_history(cfg, "cuda")
    cache = cheb.ChebCache(cfg.n_hist, dt, cfg.seg_numel)
    for x, e in zip(cfg.nodes, entries):
        cache.push(x, split_segments(e, cfg))
    torch.cuda.synchronize()
    eager = [cache.extrapolate_at(t)[0].clone() for t in cfg.targets]
    eager_multi = cache.extrapolate_at_multi(cfg.targets)[0]
    torch.cuda.synchronize()
    hosts = [to_host_bits(e) for e in entries]
    for t, e, em in zip(cfg.targets, eager, eager_multi):
        w = oracle.weights_row(cfg.nodes, t)
        check_parity(to_host_bits(e), hosts, w, cfg.dtype, f"eager t={t}")
        check_parity(to_host_bits(em), hosts, w, cfg.dtype, f"eager multi t={t}")
    outs = [cache.new_output() for _ in cfg.targets]
    outs_multi = [cache.new_output() for _ in cfg.targets]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g):
            for t, o in zip(cfg.targets, outs):
                cache.extrapolate_at(t, o)
            cache.extrapolate_at_multi(cfg.targets, outs_multi)
    torch.cuda.current_stream().wait_stream(side)
    view = torch.int16 if dt == torch.bfloat16 else torch.int32
    for rep in range(4):
        for o in outs + outs_multi:
            o.zero_()                               # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for o, e in zip(outs, eager):
            assert torch.equal(o.view(view), e.view(view)), rep
        for o, e in zip(outs_multi, eager_multi):
            assert torch.equal(o.view(view), e.view(view)), rep
    del g
    cache.close()
