"""ChebBooster online stage on AMD MI355X (gfx950).

``libcheb.so`` (C ABI in ``include/cheb.h``) does all the work: fp64 host
weights, the device history ring, the full-step push and the skipped-step
prediction kernel.  This package is its Python face: the C entry points under
their own names (``_binding``) and a small tensor-level wrapper,
``ChebCache``, that takes torch tensors and streams and passes their
addresses through.  PyTorch provides device memory and streams only.
"""
from typing import List, Optional, Sequence

import numpy as np
import torch

from ._binding import (  # noqa: F401  (re-exported C entry points)
    CHEB_LAYOUT_INTERLEAVED, CHEB_LAYOUT_SLOTS, cheb_cache_arena_bytes_ex, cheb_cache_create_ex,
    cheb_cache_geometry, DEFAULT_LAUNCH_CONFIG,
    CHEB_BF16, CHEB_F16, CHEB_F32, CHEB_MAX_NODES, CHEB_MAX_OUTPUTS, CHEB_MAX_SLOTS, CHEB_RHO_ALTERNATING,
    CHEB_RHO_GENERAL, CHEB_SHORT_FULL, CHEB_TAYLOR, CHEB_SHORT_LOWER, ChebError, cheb_chebyshev_nodes,
    cheb_precompute_weights_variant,
    cheb_cache_abort_push, cheb_cache_arena_bytes, cheb_cache_begin_push, cheb_cache_commit, cheb_cache_create,
    cheb_cache_destroy,
    cheb_cache_dtype, cheb_cache_entry, cheb_cache_history, cheb_cache_layout, cheb_cache_push,
    cheb_cache_reset, cheb_cache_segment_offset, cheb_cache_slot_numel, cheb_combine,
    cheb_combine_multi, cheb_extrapolate, cheb_extrapolate_at, cheb_extrapolate_at_multi,
    cheb_extrapolate_multi, cheb_extrapolate_steps, cheb_get_launch_config, cheb_last_error,
    cheb_precompute_weights, cheb_residual_apply, cheb_residual_reduce, cheb_schedule,
    cheb_set_launch_config, cheb_table_build, cheb_table_build_mask,
    cheb_table_destroy, cheb_table_info, cheb_table_load, cheb_table_save, cheb_table_step,
    cheb_version,
)
from . import _binding

LIB_PATH = _binding.LIB_PATH

_DTYPES = {torch.bfloat16: CHEB_BF16, torch.float16: CHEB_F16, torch.float32: CHEB_F32}
_TORCH = {CHEB_BF16: torch.bfloat16, CHEB_F16: torch.float16, CHEB_F32: torch.float32}


def cheb_dtype(dtype: torch.dtype) -> int:
    try:
        return _DTYPES[dtype]
    except KeyError:
        raise ChebError(_binding.CHEB_E_DTYPE, f"unsupported dtype {dtype}") from None


def _stream_handle(stream: Optional[torch.cuda.Stream]) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _check_device_tensor(t: torch.Tensor, what: str):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ChebError(_binding.CHEB_E_INVAL, f"{what} must be a GPU tensor")
    if not t.is_contiguous():
        raise ChebError(_binding.CHEB_E_INVAL, f"{what} must be contiguous")


def combine(srcs: Sequence[torch.Tensor], w, out: torch.Tensor,
            stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """out = sum_k w[k] * srcs[k] (elementwise, one launch of cheb_combine)."""
    if len(srcs) == 0:
        raise ChebError(_binding.CHEB_E_INVAL, "no sources")
    dt = cheb_dtype(out.dtype)
    _check_device_tensor(out, "out")
    for i, s in enumerate(srcs):
        _check_device_tensor(s, f"srcs[{i}]")
        if s.dtype != out.dtype or s.numel() != out.numel():
            raise ChebError(_binding.CHEB_E_MISMATCH, f"srcs[{i}] differs from out in dtype or size")
    cheb_combine([s.data_ptr() for s in srcs], w, out.data_ptr(), out.numel(), dt,
                 _stream_handle(stream))
    return out


def combine_multi(srcs: Sequence[torch.Tensor], w, outs: Sequence[torch.Tensor],
                  stream: Optional[torch.cuda.Stream] = None):
    """outs[m] = sum_k w[m][k] * srcs[k], all outputs from one pass
    (one launch of cheb_combine_multi)."""
    if len(srcs) == 0 or len(outs) == 0:
        raise ChebError(_binding.CHEB_E_INVAL, "no sources or no outputs")
    dt = cheb_dtype(outs[0].dtype)
    for i, t in enumerate(list(srcs) + list(outs)):
        _check_device_tensor(t, f"tensor {i}")
        if t.dtype != outs[0].dtype or t.numel() != outs[0].numel():
            raise ChebError(_binding.CHEB_E_MISMATCH, f"tensor {i} differs in dtype or size")
    cheb_combine_multi([s.data_ptr() for s in srcs], w, [o.data_ptr() for o in outs],
                       outs[0].numel(), dt, _stream_handle(stream))
    return outs


def precompute_weights(hist_t, target_t) -> np.ndarray:
    return cheb_precompute_weights(hist_t, target_t)


class ChebTable:
    """The offline stage's weight table (schedule F, rows for every
    predicted step), built in the library or loaded from a file."""

    def __init__(self, T=None, s0=None, s1=None, r=None, n_hist=None, abscissa=None,
                 policy=CHEB_SHORT_FULL, _handle=None):
        if _handle is None:
            _handle = cheb_table_build(T, s0, s1, r, n_hist, abscissa, policy)
        self._h = _handle
        info = cheb_table_info(self._h)
        self.T, self.n_hist, self.policy, self.n_full = (
            info["T"], info["n_hist"], info["policy"], info["n_full"])

    @classmethod
    def from_mask(cls, is_full, n_hist, abscissa, policy=CHEB_SHORT_FULL):
        return cls(_handle=cheb_table_build_mask(is_full, n_hist, abscissa, policy))

    @classmethod
    def load(cls, path):
        return cls(_handle=cheb_table_load(path))

    def save(self, path):
        cheb_table_save(self._h, path)

    def step(self, s):
        return cheb_table_step(self._h, s)

    def runs(self):
        """Consecutive predicted steps sharing one history: [(first, count)],
        each cut to at most CHEB_MAX_OUTPUTS steps."""
        out, s = [], 0
        while s < self.T:
            pred, nodes, _ = self.step(s)
            if not pred:
                s += 1
                continue
            first = s
            while (s < self.T and s - first < CHEB_MAX_OUTPUTS and self.step(s)[0]
                   and self.step(s)[1] == nodes):
                s += 1
            out.append((first, s - first))
        return out

    @property
    def handle(self):
        return self._h

    def close(self):
        if getattr(self, "_h", None) is not None:
            cheb_table_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def residual_reduce(segments: Sequence[torch.Tensor], res_offset, x_out: torch.Tensor,
                    x_in: Optional[torch.Tensor] = None,
                    stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """x_out = x_in + the mapped sum of one step's module outputs."""
    dt = cheb_dtype(segments[0].dtype)
    for i, t in enumerate(segments):
        _check_device_tensor(t, f"segments[{i}]")
        if t.dtype != segments[0].dtype:
            raise ChebError(_binding.CHEB_E_MISMATCH, "segments differ in dtype")
    _check_device_tensor(x_out, "x_out")
    cheb_residual_reduce([t.data_ptr() for t in segments], [t.numel() for t in segments],
                         res_offset, dt, None if x_in is None else x_in.data_ptr(),
                         x_out.data_ptr(), x_out.numel(), _stream_handle(stream))
    return x_out


class ResidualHistory:
    """Collapsed history: per full step, only the block stack's total
    contribution to the residual stream (fp32), in a ring of n entries.  A
    skipped step's residual is x_in plus the prediction from these entries,
    which by linearity equals the sum of every module's prediction."""

    def __init__(self, n_slots: int, res_offset: Sequence[int], res_numel: int, device=None):
        self.res_offset = [int(o) for o in res_offset]
        self.res_numel = int(res_numel)
        self.cache = ChebCache(n_slots, torch.float32, [self.res_numel], device=device)

    def push(self, t: float, segments: Sequence[torch.Tensor],
             stream: Optional[torch.cuda.Stream] = None):
        slot = self.cache.begin_push()
        try:
            residual_reduce(segments, self.res_offset, slot[:self.res_numel], stream=stream)
        except Exception:
            self.cache.abort_push()
            raise
        self.cache.commit(t)

    def push_difference(self, t: float, x_after: torch.Tensor, x_before: torch.Tensor,
                        stream: Optional[torch.cuda.Stream] = None):
        """Entry taken from the residual stream itself.  A full step's block
        stack leaves x_after = x_before + (every module output added into
        the residual), so the entry is x_after - x_before: one launch of
        the combination kernel with weights (1, -1) over residual-sized fp32
        tensors, instead of a pass over every module output.  The difference
        is formed in fp64 and rounded once to fp32."""
        for name, x in (("x_after", x_after), ("x_before", x_before)):
            if x.dtype != torch.float32 or x.numel() != self.res_numel:
                raise ChebError(_binding.CHEB_E_MISMATCH,
                                f"{name} must be float32 with {self.res_numel} elements")
        slot = self.cache.begin_push()
        try:
            combine([x_after, x_before], [1.0, -1.0], slot[:self.res_numel], stream=stream)
        except Exception:
            self.cache.abort_push()
            raise
        self.cache.commit(t)

    def history(self):
        return self.cache.history()

    def predict(self, target_t: float, x_out: torch.Tensor, x_in: Optional[torch.Tensor] = None,
                stream: Optional[torch.cuda.Stream] = None):
        w = cheb_precompute_weights(self.history(), [target_t])[0]
        self.cache.residual_apply(w, [0], x_out, x_in, stream=stream)
        return x_out, w

    def close(self):
        self.cache.close()


_LAYOUTS = {"slots": CHEB_LAYOUT_SLOTS, "interleaved": CHEB_LAYOUT_INTERLEAVED}


class ChebCache:
    """The history ring of one feature set, over a torch-allocated arena.

    ``seg_numel`` lists the element counts of the cached tensors in cache
    order.  Outputs (and, in the slot layout, entries) share one flat
    layout; ``segment_views`` cuts a flat buffer into per-segment views.
    ``layout`` is "slots" (contiguous entries; fused push possible) or
    "interleaved" (entries cut into 32 KiB chunks taken in turn; filled by
    ``push``).
    """

    def __init__(self, n_slots: int, dtype: torch.dtype, seg_numel: Sequence[int],
                 device=None, arena: Optional[torch.Tensor] = None, layout: str = "slots"):
        self.n_slots = int(n_slots)
        self.dtype = dtype
        self.cdtype = cheb_dtype(dtype)
        self.seg_numel = [int(n) for n in seg_numel]
        if layout not in _LAYOUTS:
            raise ChebError(_binding.CHEB_E_INVAL, f"unknown layout {layout!r}")
        self.layout = layout
        lay = cheb_cache_layout(self.n_slots, self.cdtype, self.seg_numel)
        self.seg_offset = [int(o) for o in lay["seg_offset"]]
        self.slot_numel = int(lay["slot_numel"])
        self.slot_stride_bytes = int(lay["slot_stride_bytes"])
        self.arena_bytes = cheb_cache_arena_bytes_ex(self.n_slots, self.cdtype, self.seg_numel,
                                                     _LAYOUTS[layout])
        if arena is None:
            device = torch.device("cuda", torch.cuda.current_device()) if device is None else device
            arena = torch.empty(self.arena_bytes, dtype=torch.uint8, device=device)
        _check_device_tensor(arena, "arena")
        self.arena = arena
        self.device = arena.device
        self._h = cheb_cache_create_ex(self.n_slots, self.cdtype, self.seg_numel, _LAYOUTS[layout],
                                       arena.data_ptr(), arena.numel() * arena.element_size())
        _, self.chunk_elems, self.entry_stride_elems = cheb_cache_geometry(self._h)

    # -- lifetime ------------------------------------------------------------
    def close(self):
        if getattr(self, "_h", None) is not None:
            cheb_cache_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def handle(self):
        return self._h

    # -- buffers -------------------------------------------------------------
    def new_output(self) -> torch.Tensor:
        return torch.empty(self.slot_numel, dtype=self.dtype, device=self.device)

    def segment_views(self, flat: torch.Tensor, shapes=None) -> List[torch.Tensor]:
        views = []
        for s, (off, n) in enumerate(zip(self.seg_offset, self.seg_numel)):
            v = flat[off:off + n]
            views.append(v.view(shapes[s]) if shapes is not None else v)
        return views

    def _slot_tensor(self, addr: int) -> torch.Tensor:
        start = addr - self.arena.data_ptr()
        esz = torch.empty((), dtype=self.dtype).element_size()
        raw = self.arena[start:start + self.slot_numel * esz]
        return raw.view(self.dtype)

    def entry(self, idx: int) -> torch.Tensor:
        """The held entry of age index idx (0 = oldest) as a flat tensor: a
        view of its slot in the slot layout, a gathered copy of its chunks
        in the interleaved layout."""
        addr = cheb_cache_entry(self._h, idx)
        if self.layout == "slots":
            return self._slot_tensor(addr)
        esz = torch.empty((), dtype=self.dtype).element_size()
        start = (addr - self.arena.data_ptr()) // esz
        chunk, stride = self.chunk_elems, self.entry_stride_elems
        n_chunks = -(-self.slot_numel // chunk)
        if n_chunks == 0:
            return torch.empty(0, dtype=self.dtype, device=self.device)
        whole = self.arena.view(self.dtype)
        chunks = torch.as_strided(whole, (n_chunks, chunk), (stride, 1),
                                  storage_offset=whole.storage_offset() + start)
        return chunks.reshape(-1)[:self.slot_numel].clone()

    # -- the online stage ------------------------------------------------------
    def push(self, t: float, segments: Sequence[torch.Tensor],
             stream: Optional[torch.cuda.Stream] = None):
        if len(segments) != len(self.seg_numel):
            raise ChebError(_binding.CHEB_E_MISMATCH, "segment count differs from the layout")
        for i, (s, n) in enumerate(zip(segments, self.seg_numel)):
            _check_device_tensor(s, f"segments[{i}]")
            if s.dtype != self.dtype or s.numel() != n:
                raise ChebError(_binding.CHEB_E_MISMATCH, f"segments[{i}] differs from the layout")
        cheb_cache_push(self._h, t, [s.data_ptr() for s in segments], _stream_handle(stream))

    def begin_push(self) -> torch.Tensor:
        """Flat view of the slot the next entry occupies (fused push)."""
        return self._slot_tensor(cheb_cache_begin_push(self._h))

    def commit(self, t: float):
        cheb_cache_commit(self._h, t)

    def abort_push(self):
        """Close an open fused push without recording an entry; the entry
        its slot held stays dropped."""
        cheb_cache_abort_push(self._h)

    def reset(self):
        cheb_cache_reset(self._h)

    def history(self) -> np.ndarray:
        return cheb_cache_history(self._h)

    def _check_out(self, out: torch.Tensor):
        _check_device_tensor(out, "out")
        if out.dtype != self.dtype or out.numel() < self.slot_numel:
            raise ChebError(_binding.CHEB_E_MISMATCH, "out differs from the slot layout")

    def extrapolate(self, w, out: Optional[torch.Tensor] = None,
                    stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
        out = self.new_output() if out is None else out
        self._check_out(out)
        cheb_extrapolate(self._h, w, out.data_ptr(), _stream_handle(stream))
        return out

    def extrapolate_multi(self, w, outs: Optional[Sequence[torch.Tensor]] = None,
                          stream: Optional[torch.cuda.Stream] = None):
        w = np.asarray(w, dtype=np.float64).reshape(-1, self.n_slots)
        outs = [self.new_output() for _ in range(w.shape[0])] if outs is None else list(outs)
        for o in outs:
            self._check_out(o)
        cheb_extrapolate_multi(self._h, w, [o.data_ptr() for o in outs], _stream_handle(stream))
        return outs

    def extrapolate_at_multi(self, targets, outs: Optional[Sequence[torch.Tensor]] = None,
                             stream: Optional[torch.cuda.Stream] = None):
        targets = list(targets)
        outs = [self.new_output() for _ in targets] if outs is None else list(outs)
        for o in outs:
            self._check_out(o)
        w = cheb_extrapolate_at_multi(self._h, targets, [o.data_ptr() for o in outs],
                                      _stream_handle(stream), n_slots=self.n_slots)
        return outs, w

    def extrapolate_steps(self, table: "ChebTable", first_step: int, n_steps: int = 1,
                          outs: Optional[Sequence[torch.Tensor]] = None,
                          stream: Optional[torch.cuda.Stream] = None):
        outs = [self.new_output() for _ in range(n_steps)] if outs is None else list(outs)
        for o in outs:
            self._check_out(o)
        cheb_extrapolate_steps(self._h, table.handle, first_step, [o.data_ptr() for o in outs],
                               _stream_handle(stream))
        return outs

    def residual_apply(self, w, res_offset, x_out: torch.Tensor,
                       x_in: Optional[torch.Tensor] = None,
                       stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
        """x_out = x_in + the block stack's predicted module outputs (one pass)."""
        _check_device_tensor(x_out, "x_out")
        if x_out.dtype != torch.float32:
            raise ChebError(_binding.CHEB_E_DTYPE, "the residual is float32")
        if x_in is not None:
            _check_device_tensor(x_in, "x_in")
            if x_in.dtype != torch.float32 or x_in.numel() != x_out.numel():
                raise ChebError(_binding.CHEB_E_MISMATCH, "x_in differs from x_out")
        cheb_residual_apply(self._h, w, res_offset, x_out.numel(),
                            None if x_in is None else x_in.data_ptr(), x_out.data_ptr(),
                            _stream_handle(stream))
        return x_out

    def extrapolate_at(self, target_t: float, out: Optional[torch.Tensor] = None,
                       stream: Optional[torch.cuda.Stream] = None):
        out = self.new_output() if out is None else out
        self._check_out(out)
        w = cheb_extrapolate_at(self._h, target_t, out.data_ptr(), _stream_handle(stream),
                                n_slots=self.n_slots)
        return out, w


__all__ = [n for n in dir() if n.startswith("cheb_")] + [
    "ChebCache", "ChebTable", "ChebError", "ResidualHistory", "residual_reduce", "combine", "combine_multi", "precompute_weights", "CHEB_BF16",
    "CHEB_F32", "CHEB_MAX_SLOTS", "CHEB_MAX_OUTPUTS", "CHEB_MAX_NODES", "LIB_PATH"]
