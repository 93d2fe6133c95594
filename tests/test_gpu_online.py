"""The online stage end to end (Algorithm 1): a sampler-shaped loop over T
steps; full steps push their features into the ring, each run of skipped
steps is predicted from the table in one pass; every prediction is checked
against the oracle's own simulation of Algorithm 1 on the same stored
features."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_23429_amd as cheb
from synth import CONFIGS, make_history, split_segments, by_name
from tests.gpu_util import check_parity, say, to_host_bits

pytestmark = pytest.mark.gpu

DT = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}

# (workload, T, s0, s1, r, n, policy, abscissa of step s)
CASES = [
    ("flux_dev_1024", 50, 1, 1, 6, 6, cheb.CHEB_SHORT_LOWER, lambda s: 1.0 - s / 50.0),
    ("flux_dev_1024", 50, 1, 1, 6, 2, cheb.CHEB_SHORT_FULL, lambda s: 1.0 - s / 50.0),
    ("dit_xl2_256", 50, 1, 1, 3, 3, cheb.CHEB_SHORT_LOWER, lambda s: 980.0 - 20.0 * s),
    ("pixart_sigma_1024", 20, 2, 1, 4, 6, cheb.CHEB_SHORT_FULL, lambda s: 999.0 - 50.0 * s),
    ("tiny", 30, 0, 0, 3, 4, cheb.CHEB_SHORT_LOWER, lambda s: 999.0 - 20.0 * s),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}_r{c[4]}_n{c[5]}_p{c[6]}")
def test_online_stage(case):
    name, T, s0, s1, r, n, policy, absc = case
    cfg = [c for c in CONFIGS if c.name == name][0].shrunk(250_000)
    x = np.array([absc(s) for s in range(T)])
    table = cheb.ChebTable(T, s0, s1, r, n, x, policy)
    full_steps = [s for s in range(T) if not table.step(s)[0]]
    say(f"online {name}: T={T} r={r} n={n} policy={policy}, {len(full_steps)} full steps, "
        f"{cfg.numel} elements")
    feats = make_history(cfg, "cuda", nodes=x[full_steps])
    feat_of = dict(zip(full_steps, feats))
    host_of = {s: to_host_bits(f) for s, f in feat_of.items()}
    cache = cheb.ChebCache(n, DT[cfg.dtype], cfg.seg_numel)
    runs = dict(table.runs())
    predicted = 0
    s = 0
    while s < T:
        pred, _, _ = table.step(s)
        if not pred:
            cache.push(x[s], split_segments(feat_of[s], cfg))
            s += 1
            continue
        count = runs[s]
        outs = cache.extrapolate_steps(table, s, count)
        torch.cuda.synchronize()
        for m in range(count):
            kind, nodes, w = oracle.table_row(T, s0, s1, r, n, x, policy, s + m)
            assert kind == 1
            check_parity(to_host_bits(outs[m]), [host_of[j] for j in nodes], w, cfg.dtype,
                         f"{name} step {s + m}")
            predicted += 1
        s += count
    assert predicted == T - len(full_steps)
    cache.close()
    table.close()


def test_table_row_must_match_ring():
    """A table built for another abscissa grid is refused before launch."""
    cfg = by_name("flux_dev_1024").shrunk(50_000)
    x = 1.0 - np.arange(20) / 20.0
    table = cheb.ChebTable(20, 1, 1, 4, 2, x)
    cache = cheb.ChebCache(2, torch.bfloat16, cfg.seg_numel)
    feats = make_history(cfg, "cuda", nodes=[0.99, 0.95])        # not the table's abscissae
    for t, f in zip([0.99, 0.95], feats):
        cache.push(t, split_segments(f, cfg))
    with pytest.raises(cheb.ChebError) as e:
        cache.extrapolate_steps(table, 2, 2)
    assert e.value.code == cheb._binding.CHEB_E_MISMATCH
    cache.close()
