"""The five cache workloads the online stage is exercised and measured on.

Each workload is the set of cached DiT module outputs of one model at one
resolution (the tensors a full step writes into the history and a skipped
step predicts), a history of K+1 abscissae (oldest to newest) taken from the
sampler's schedule, and the target abscissae of the skipped steps that follow.

Feature values are synthetic: per element, a random polynomial in the
normalised time variable plus Gaussian noise (standard deviations as given).
They stand in for real activations of DiT-XL/2 (ImageNet class-conditional),
PixArt-Sigma (HPSv2 prompts) and FLUX.1-dev (DrawBench prompts); no dataset or
checkpoint is used.
"""
from dataclasses import dataclass, field, replace
from typing import List, Optional, Tuple

import math


@dataclass(frozen=True)
class Config:
    name: str
    index: int
    dtype: str                      # "bf16", "f16" or "f32": storage type of the cache
    segments: Tuple[Tuple[int, ...], ...]   # cached tensor shapes, in cache order
    segment_names: Tuple[str, ...]
    nodes: Tuple[float, ...]        # history abscissae, oldest to newest
    targets: Tuple[float, ...]      # skipped-step abscissae (primary reading)
    alt_nodes: Optional[Tuple[float, ...]] = None    # second reading, if any
    alt_targets: Optional[Tuple[float, ...]] = None
    time_scale: float = 1000.0      # tau = abscissa / time_scale in the generator
    degree: int = 2                 # degree of the per-element polynomial
    coeff_std: float = 1.0
    noise_std: float = 1e-3
    seed_base: int = 2025           # the paper's sampling seed

    @property
    def seed(self) -> int:
        return self.seed_base + self.index

    @property
    def n_hist(self) -> int:
        return len(self.nodes)

    @property
    def K(self) -> int:
        return len(self.nodes) - 1

    @property
    def elem_size(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def seg_numel(self) -> List[int]:
        return [math.prod(s) for s in self.segments]

    @property
    def numel(self) -> int:
        return sum(self.seg_numel)

    @property
    def bytes_per_step(self) -> int:
        """Algorithmic bytes of one skipped step: K+1 entries read, one written."""
        return (self.n_hist + 1) * self.numel * self.elem_size

    def with_segments(self, segments, names=None) -> "Config":
        segments = tuple(tuple(int(d) for d in s) for s in segments)
        if names is None:
            names = tuple(f"seg{i}" for i in range(len(segments)))
        return replace(self, segments=segments, segment_names=tuple(names))

    def residual_map(self):
        """Where each cached output adds into the residual stream, as
        (res_offset per segment, residual elements).  DiT and PixArt blocks
        add both outputs into the one token stream; FLUX double-stream
        blocks add text outputs into the text tokens (first) and image
        outputs into the image tokens (after them), single-stream blocks
        into the joint stream."""
        names = self.segment_names
        if any(n.startswith("double") for n in names):
            txt = [n for n, name in zip(self.seg_numel, names) if name.endswith(".txt")]
            img = [n for n, name in zip(self.seg_numel, names) if name.endswith(".img")]
            single = [n for n, name in zip(self.seg_numel, names) if name.startswith("single")]
            n_txt, n_img = txt[0], img[0]
            n_res = single[0] if single else n_txt + n_img
            assert n_txt + n_img == n_res, "joint stream is text + image tokens"
            offs = [n_txt if name.endswith(".img") else 0 for name in names]
            return offs, n_res
        n_res = self.seg_numel[0]
        assert all(n == n_res for n in self.seg_numel), "one residual stream"
        return [0] * len(names), n_res

    def scaled_blocks(self, token_div: int, max_blocks: int) -> "Config":
        """Same model structure with fewer blocks and fewer tokens (leading
        dimensions divided by token_div), so residual maps stay consistent."""
        segs, names = [], []
        for shape, name in zip(self.segments, self.segment_names):
            block = int("".join(ch for ch in name.split(".")[0] if ch.isdigit()) or 0)
            if block >= max_blocks:
                continue
            new = list(shape)
            new[-2] = max(1, new[-2] // token_div)
            segs.append(tuple(new))
            names.append(name)
        return self.with_segments(segs, names)

    def shrunk(self, max_numel: int) -> "Config":
        """Same history, schedule and generator on a smaller cache.

        Keeps the segment mix (one of each distinct shape, leading dimensions
        cut down) so the result stays ragged where the original is; used for
        parity cases the oracle finishes in seconds.
        """
        seen = []
        for s in self.segments:
            if s not in seen:
                seen.append(s)
        out = []
        budget = max(1, max_numel // max(1, len(seen)))
        for s in seen:
            s = list(s)
            while math.prod(s) > budget and any(d > 1 for d in s[:-1]):
                for i in range(len(s) - 1):
                    if s[i] > 1:
                        s[i] = (s[i] + 1) // 2
                        break
            out.append(tuple(s))
        return self.with_segments(out)


def _dit_segments(blocks, shape):
    segs, names = [], []
    for b in range(blocks):
        segs += [shape, shape]
        names += [f"block{b}.attn", f"block{b}.mlp"]
    return tuple(segs), tuple(names)


def _flux_segments():
    segs, names = [], []
    for b in range(19):
        segs += [(1, 4096, 3072), (1, 512, 3072)]
        names += [f"double{b}.img", f"double{b}.txt"]
    for b in range(38):
        segs.append((1, 4608, 3072))
        names.append(f"single{b}")
    return tuple(segs), tuple(names)


def _ddim50(step):          # DDIM, 50 steps over t in [0, 999]
    return 980.0 - 20.0 * step


def _dpm20(step):           # 20-step DPM-Solver-like grid over t in [0, 999]
    return 999.0 - 50.0 * step


def _flow50(step):          # 50-step flow matching, sigma from 1 to 0
    return 1.0 - step / 50.0


_dit256 = _dit_segments(28, (16, 256, 1152))
_dit512 = _dit_segments(28, (16, 1024, 1152))
_pix1024 = _dit_segments(28, (2, 4096, 1152))
_flux = _flux_segments()

CONFIGS: List[Config] = [
    # One fp32 tensor; four history entries 20 timesteps apart; the next
    # three timesteps are the targets (a second reading: one to three
    # node spacings ahead).
    Config(
        name="tiny", index=0, dtype="f32",
        segments=((2, 256, 1152),), segment_names=("feature",),
        nodes=(999.0, 979.0, 959.0, 939.0),
        targets=(938.0, 937.0, 936.0),
        alt_nodes=(999.0, 979.0, 959.0, 939.0),
        alt_targets=(919.0, 899.0, 879.0),
        degree=2, coeff_std=1.0, noise_std=1e-3,
    ),
    # DiT-XL/2 256x256, batch 8 doubled by classifier-free guidance:
    # 28 blocks x (attention, MLP) outputs of [16, 256, 1152].
    # Full steps 4, 8, ..., 20 of DDIM-50; skipped steps 21, 22, 23.
    Config(
        name="dit_xl2_256", index=1, dtype="bf16",
        segments=_dit256[0], segment_names=_dit256[1],
        nodes=tuple(_ddim50(s) for s in (4, 8, 12, 16, 20)),
        targets=tuple(_ddim50(s) for s in (21, 22, 23)),
        degree=3, coeff_std=1.0, noise_std=0.02,
    ),
    # DiT-XL/2 512x512: 28 blocks x 2 outputs of [16, 1024, 1152].
    # Full steps 5, 10, ..., 25 of DDIM-50; skipped steps 26..29.
    Config(
        name="dit_xl2_512", index=2, dtype="bf16",
        segments=_dit512[0], segment_names=_dit512[1],
        nodes=tuple(_ddim50(s) for s in (5, 10, 15, 20, 25)),
        targets=tuple(_ddim50(s) for s in (26, 27, 28, 29)),
        degree=3, coeff_std=1.0, noise_std=0.02,
    ),
    # PixArt-Sigma 1024x1024, batch 1 doubled by guidance: 28 blocks x
    # 2 outputs of [2, 4096, 1152].  Full steps from the paper's schedule
    # with T=20, s0=2, s1=1, r=4: {0,1,2,6,10,14,...}; the last six before
    # the skipped steps 15, 16, 17.  Second reading: uniform steps 0..20 by
    # 4 (step units), skipped steps 21..23.
    Config(
        name="pixart_sigma_1024", index=3, dtype="bf16",
        segments=_pix1024[0], segment_names=_pix1024[1],
        nodes=tuple(_dpm20(s) for s in (0, 1, 2, 6, 10, 14)),
        targets=tuple(_dpm20(s) for s in (15, 16, 17)),
        alt_nodes=(0.0, 4.0, 8.0, 12.0, 16.0, 20.0),
        alt_targets=(21.0, 22.0, 23.0),
        degree=4, coeff_std=0.5, noise_std=0.02,
    ),
    # FLUX.1-dev 1024x1024: 19 double-stream blocks (image [1,4096,3072],
    # text [1,512,3072]) and 38 single-stream blocks [1,4608,3072].
    # Full steps 2, 5, 10, 14, 20, 25 (intervals 3,5,4,6,5) of a 50-step
    # flow schedule in sigma; skipped steps 26..29.
    Config(
        name="flux_dev_1024", index=4, dtype="bf16",
        segments=_flux[0], segment_names=_flux[1],
        nodes=tuple(_flow50(s) for s in (2, 5, 10, 14, 20, 25)),
        targets=tuple(_flow50(s) for s in (26, 27, 28, 29)),
        time_scale=1.0,
        degree=4, coeff_std=0.5, noise_std=0.02,
    ),
]


def by_name(name: str) -> Config:
    for c in CONFIGS:
        if c.name == name or str(c.index) == str(name):
            return c
    raise KeyError(name)
