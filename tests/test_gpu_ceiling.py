"""The benchmark's stream-ceiling kernels (bench_ceiling.hip) move the bytes
they are credited with: each reading kind's output is the XOR of exactly the
vectors it should read (contiguous streams, or the lanes of the interleaved
layout), the write-only kind writes every vector, the window kind wraps its
stores into the window, and the read-only kinds leave the destination
untouched.  Small sizes with a ragged last block, in both launch shapes
(1024-lane blocks, and 64-lane blocks under an occupancy cap)."""
import ctypes
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "bench_ceiling.so")


def _lib():
    if not os.path.exists(LIB):
        pytest.fail("bench_ceiling.so is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB)
    lib.ceiling_stream.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_void_p), ctypes.c_int,
                                   ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                   ctypes.c_int, ctypes.c_void_p]
    lib.ceiling_stream.restype = ctypes.c_int
    return lib


def _run(lib, kind, srcs, n_src, dst, n_vec, window=0, waves=0):
    arr = (ctypes.c_void_p * max(1, len(srcs)))(*[s.data_ptr() for s in srcs]) if srcs else None
    rc = lib.ceiling_stream(kind, arr, n_src, dst.data_ptr(), n_vec, window, waves,
                            torch.cuda.current_stream().cuda_stream)
    assert rc == 0, rc
    torch.cuda.synchronize()


def _vectors(n_vec, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return torch.randint(-2 ** 31, 2 ** 31 - 1, (n_vec, 4), generator=g, device="cuda",
                         dtype=torch.int32)


N_VEC = 3 * 2048 + 517           # three whole 32 KiB chunks and a part


WAVES = [0, 8, 3, 32]


@pytest.mark.parametrize("waves", WAVES)
def test_contiguous_kinds(waves):
    lib = _lib()
    srcs = [_vectors(N_VEC, 10 + k) for k in range(6)]
    x = srcs[0].clone()
    for s in srcs[1:]:
        x ^= s
    out = torch.zeros(N_VEC, 4, dtype=torch.int32, device="cuda")
    _run(lib, 1, srcs, 6, out, N_VEC, waves=waves)          # 6 reads, 1 write
    assert torch.equal(out, x)
    _run(lib, 1, srcs[:1], 1, out, N_VEC, waves=waves)      # copy
    assert torch.equal(out, srcs[0])
    out.zero_()
    _run(lib, 0, srcs, 6, out, N_VEC, waves=waves)          # read only: no store
    assert not out.any()
    _run(lib, 3, [], 1, out, N_VEC, waves=waves)            # write only
    idx = torch.arange(N_VEC, device="cuda", dtype=torch.int32)
    assert torch.equal(out[:, 0], idx) and not out[:, 1:].any()


@pytest.mark.parametrize("waves", WAVES)
def test_interleaved_kinds(waves):
    lib = _lib()
    n = 6
    chunks = -(-N_VEC // 2048)
    region = _vectors(chunks * n * 2048, 77)
    lanes = region.view(chunks, n, 2048, 4)
    x = lanes[:, 0].reshape(-1, 4)[:N_VEC].clone()
    for k in range(1, n):
        x ^= lanes[:, k].reshape(-1, 4)[:N_VEC]
    out = torch.zeros(N_VEC, 4, dtype=torch.int32, device="cuda")
    _run(lib, 2, [region], n, out, N_VEC, waves=waves)
    assert torch.equal(out, x)
    out.zero_()
    _run(lib, 4, [region], n, out, N_VEC, waves=waves)      # read only: no store
    assert not out.any()
    window = 1024
    _run(lib, 5, [region], n, out, N_VEC, window, waves)    # stores wrap into the window
    assert not out[window:].any()
    # several vectors land on each window slot and any of them may be the
    # last written, so check that every slot holds one that maps to it
    got = out[:window].cpu().numpy()
    xs = x.cpu().numpy()
    for j in range(0, window, 97):
        cands = xs[j::window]
        assert any(np.array_equal(got[j], c) for c in cands), j


def test_refused_arguments():
    lib = _lib()
    out = torch.zeros(16, 4, dtype=torch.int32, device="cuda")
    srcs = [_vectors(16, 1)]
    arr = (ctypes.c_void_p * 1)(srcs[0].data_ptr())
    assert lib.ceiling_stream(6, arr, 1, out.data_ptr(), 16, 0, 0, None) == -1
    assert lib.ceiling_stream(1, arr, 9, out.data_ptr(), 16, 0, 0, None) == -1
    assert lib.ceiling_stream(5, arr, 1, out.data_ptr(), 16, 3, 0, None) == -1   # not a power of 2
    assert lib.ceiling_stream(5, arr, 1, out.data_ptr(), 16, 32, 0, None) == -1  # past n_vec
    assert lib.ceiling_stream(1, arr, 1, out.data_ptr(), 16, 0, 2, None) == -1   # cap too low
    assert lib.ceiling_stream(1, arr, 1, out.data_ptr(), 16, 0, 33, None) == -1  # cap too high


def test_lds_per_cu_reported():
    """The occupancy cap divides the LDS the runtime reports per compute
    unit; gfx950 has 160 KiB."""
    lib = _lib()
    lib.ceiling_lds_per_cu.restype = ctypes.c_int
    lds = lib.ceiling_lds_per_cu()
    assert lds >= 64 * 1024, lds
    if "gfx950" in torch.cuda.get_device_properties(0).gcnArchName:
        assert lds == 160 * 1024, lds
