"""The online stage inside a sampler loop over real (random-weight) DiT
blocks: each block adds a gated attention output and a gated MLP output to
the residual stream (Section 3.1, block equation), with the gates depending
on the timestep.  Full steps, chosen by the offline table (Section 3.3
schedule), run the blocks and write every module output straight into the
ring slot (fused push), and feed the collapsed history with
x_after - x_before; skipped steps predict the block stack's output from the
cache (Algorithm 1, online stage) in both residual forms, and the sampler
goes on from the per-module prediction.  Every prediction is checked against
the oracle on host copies of the stored module outputs."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_23429_amd as cheb
from tests.gpu_util import say, to_host_bits

pytestmark = pytest.mark.gpu

N_TOK, DIM, HEADS, BLOCKS = 128, 256, 4, 3
RES_TOL = 1e-5       # fp64 accumulation of exactly decoded bf16 values, one fp32 rounding
DIFF_TOL = 1e-4      # entries rounded once to fp32: (1 + 10^3) 2^-24 floored


def _params(seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)

    def mat(r, c):
        return torch.randn(r, c, generator=g, device="cuda") / math.sqrt(r)
    return [dict(qkv=mat(DIM, 3 * DIM), o=mat(DIM, DIM), w1=mat(DIM, 4 * DIM),
                 w2=mat(4 * DIM, DIM), ga=0.3 + 0.1 * b, gm=0.2 + 0.1 * b)
            for b in range(BLOCKS)]


def _norm(x):
    return (x - x.mean(-1, keepdim=True)) / torch.sqrt(x.var(-1, unbiased=False, keepdim=True) + 1e-6)


def _attn(p, h):
    q, k, v = (h @ p["qkv"]).split(DIM, dim=-1)
    d = DIM // HEADS
    q = q.reshape(N_TOK, HEADS, d).transpose(0, 1).contiguous()
    k = k.reshape(N_TOK, HEADS, d).transpose(0, 1).contiguous()
    v = v.reshape(N_TOK, HEADS, d).transpose(0, 1).contiguous()
    a = torch.softmax(torch.matmul(q, k.transpose(1, 2).contiguous()) / math.sqrt(d), dim=-1)
    return torch.matmul(a, v).transpose(0, 1).reshape(N_TOK, DIM) @ p["o"]


def _forward(params, x0, t, slot_views):
    """The block stack at timestep t; every gated module output is rounded to
    bf16 once, written into its slot view, and added (as stored) to the
    residual stream.  Returns the stack's output."""
    x = x0.clone()
    for b, p in enumerate(params):
        gate_a = p["ga"] * (1.0 + 0.5 * math.sin(3.0 * t))
        gate_m = p["gm"] * (1.0 + 0.5 * math.cos(2.0 * t))
        for j, out in enumerate((gate_a * _attn(p, _norm(x)),
                                 gate_m * (torch.nn.functional.gelu(_norm(x) @ p["w1"]) @ p["w2"]))):
            stored = slot_views[2 * b + j]
            stored.copy_(out.reshape(-1))                  # bf16, into the ring slot
            x = x + stored.float().reshape(N_TOK, DIM)
    return x


def _check(got, expect, mag, tol, label):
    e = oracle.parity_error(np.asarray(got, dtype=np.float64), expect, mag)[0]
    say(f"  {label}: floored error {e:.3e}")
    assert e <= tol, (label, e)


@pytest.mark.parametrize("r,n", [(3, 3), (4, 4)])
def test_sampler_loop_with_dit_blocks(r, n):
    T = 16
    sigma = 1.0 - np.arange(T) / T
    table = cheb.ChebTable(T, 1, 1, r, n, sigma, cheb.CHEB_SHORT_FULL)
    params = _params(7)
    seg_numel = [N_TOK * DIM] * (2 * BLOCKS)
    res_off, res_n = [0] * (2 * BLOCKS), N_TOK * DIM
    cache = cheb.ChebCache(n, torch.bfloat16, seg_numel)
    hist = cheb.ResidualHistory(n, res_off, res_n)
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    x = torch.randn(N_TOK, DIM, generator=g, device="cuda")
    host_feats, host_after, host_before, held = {}, {}, {}, []
    predicted = 0
    for s in range(T):
        t = float(sigma[s])
        x0 = x + 0.1 * t                                    # timestep embedding
        if not table.step(s)[0]:
            slot = cache.begin_push()
            xl = _forward(params, x0, t, cache.segment_views(slot))
            cache.commit(t)
            hist.push_difference(t, xl.reshape(-1), x0.reshape(-1))
            torch.cuda.synchronize()
            host_feats[t] = to_host_bits(slot[:cache.slot_numel])
            host_after[t] = xl.reshape(-1).cpu().numpy()
            host_before[t] = x0.reshape(-1).cpu().numpy()
            held = (held + [t])[-n:]
        else:
            pred, nodes, _ = table.step(s)
            assert [float(sigma[j]) for j in nodes] == held == cache.history().tolist()
            w = cheb.cheb_precompute_weights(held, [t])[0]
            x_mod = torch.empty(res_n, device="cuda")
            cache.residual_apply(w, res_off, x_mod, x0.reshape(-1))
            x_col = torch.empty(res_n, device="cuda")
            hist.predict(t, x_col, x0.reshape(-1))
            torch.cuda.synchronize()
            w_or = oracle.weights_row(held, t)
            xin = x0.reshape(-1).cpu().numpy()
            seg_off = cache.seg_offset
            exp, mag = oracle.residual([host_feats[h] for h in held], w_or, seg_off, seg_numel,
                                       res_off, res_n, x_in=xin)
            _check(x_mod.cpu().numpy(), exp, mag, RES_TOL, f"r={r} n={n} step {s} per-module")
            exp2, mag2 = oracle.residual([host_after[h] for h in held] + [host_before[h] for h in held],
                                         np.concatenate([w_or, -w_or]), [0], [res_n], [0], res_n,
                                         x_in=xin, dtype="f32")
            _check(x_col.cpu().numpy(), exp2, mag2, DIFF_TOL, f"r={r} n={n} step {s} collapsed")
            xl = x_mod.reshape(N_TOK, DIM)
            predicted += 1
        x = x - (1.0 / T) * xl                             # sampler update
    assert predicted == T - table.n_full and predicted > 0
    assert torch.isfinite(x).all()
    cache.close()
    hist.close()
    table.close()
