"""Seeded feature histories for the cache workloads.

Every element of every cached tensor follows its own random polynomial in the
normalised time variable tau, plus independent Gaussian noise at each history
entry:

    F_k[i] = sum_{d=0}^{D} c_d[i] * tau_k^d + noise_std * eta_k[i],
    c_d[i] ~ N(0, coeff_std^2),  eta_k[i] ~ N(0, 1),  tau_k = x_k / time_scale.

Draw order from one ``torch.Generator`` seeded with the workload seed:
c_0, ..., c_D (each over all elements), then eta_0, ..., eta_K.  Values are
formed in fp32 and stored in the cache's dtype with round-to-nearest-even
(torch's own conversion).  The same seed gives different values on CPU and on
a GPU (different generator engines); each run draws its inputs once and hands
the same stored values to both sides of a comparison.
"""
from typing import List, Optional, Sequence

import numpy as np
import torch

from .configs import Config

_TORCH_DTYPES = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}


def torch_dtype(cfg: Config) -> torch.dtype:
    return _TORCH_DTYPES[cfg.dtype]


def make_history(cfg: Config, device="cpu", nodes: Optional[Sequence[float]] = None,
                 time_scale: Optional[float] = None, seed: Optional[int] = None,
                 numel: Optional[int] = None) -> List[torch.Tensor]:
    """History entries oldest to newest, each a flat tensor of the cache's
    total element count (segments concatenated in cache order)."""
    nodes = cfg.nodes if nodes is None else tuple(nodes)
    time_scale = cfg.time_scale if time_scale is None else float(time_scale)
    seed = cfg.seed if seed is None else int(seed)
    E = cfg.numel if numel is None else int(numel)
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    coeffs = [torch.randn(E, generator=g, device=dev, dtype=torch.float32)
              .mul_(cfg.coeff_std) for _ in range(cfg.degree + 1)]
    out = []
    for x in nodes:
        tau = float(x) / time_scale
        val = coeffs[cfg.degree].clone()
        for d in range(cfg.degree - 1, -1, -1):        # Horner in fp32
            val.mul_(tau).add_(coeffs[d])
        eta = torch.randn(E, generator=g, device=dev, dtype=torch.float32)
        val.add_(eta, alpha=cfg.noise_std)
        del eta
        out.append(val.to(torch_dtype(cfg)))
        del val
    del coeffs
    return out


def make_history_f64(cfg: Config, numel: int, nodes: Optional[Sequence[float]] = None,
                     time_scale: Optional[float] = None, seed: Optional[int] = None):
    """Unrounded fp64 history on the CPU (numpy), with its ingredients.

    Returns (entries [K+1, numel], coeffs [D+1, numel], eta [K+1, numel],
    taus).  Used to check that a combination of the entries equals the
    polynomial at the target plus the combined noise.
    """
    nodes = cfg.nodes if nodes is None else tuple(nodes)
    time_scale = cfg.time_scale if time_scale is None else float(time_scale)
    seed = cfg.seed if seed is None else int(seed)
    rng = np.random.default_rng(seed)
    coeffs = rng.standard_normal((cfg.degree + 1, numel)) * cfg.coeff_std
    eta = rng.standard_normal((len(nodes), numel))
    taus = np.array([float(x) / time_scale for x in nodes])
    entries = np.empty((len(nodes), numel))
    for k, tau in enumerate(taus):
        val = coeffs[cfg.degree].copy()
        for d in range(cfg.degree - 1, -1, -1):
            val = val * tau + coeffs[d]
        entries[k] = val + cfg.noise_std * eta[k]
    return entries, coeffs, eta, taus


def split_segments(flat: torch.Tensor, cfg: Config) -> List[torch.Tensor]:
    """Views of one flat history entry as the cache's segment tensors."""
    views, off = [], 0
    for shape, n in zip(cfg.segments, cfg.seg_numel):
        views.append(flat[off:off + n].view(shape))
        off += n
    return views
