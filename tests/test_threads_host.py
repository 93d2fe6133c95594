"""Host calls from several threads at once (no GPU): error messages are
per thread, weight rows and tables built concurrently equal those built
alone, and the launch shape is read and written under a lock.  ctypes drops
the interpreter lock around each foreign call, so the calls overlap."""
import threading

import numpy as np

import paper_2608_23429_amd as cheb
from paper_2608_23429_amd import _binding as B

THREADS = 8
ITERS = 400


def _run(worker):
    errors = []

    def wrap(i):
        try:
            worker(i)
        except Exception as e:          # collected and re-raised below
            errors.append(e)

    ts = [threading.Thread(target=wrap, args=(i,)) for i in range(THREADS)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    if errors:
        raise errors[0]


def test_error_messages_are_per_thread():
    def worker(i):
        dup = 1000.0 + i                        # a value only this thread uses
        h = np.array([dup, 3.0, dup])
        t = np.array([5.0])
        w = np.empty((1, 3))
        good = np.array([1.0, 2.0, 4.0 + i])
        for _ in range(ITERS):
            rc = B.LIB.cheb_precompute_weights(B._dptr(h), 3, B._dptr(t), 1, B._dptr(w))
            assert rc == B.CHEB_E_DUPNODE
            msg = cheb.cheb_last_error()
            assert f"({dup:.17g})" in msg, msg
            cheb.cheb_precompute_weights(good, [8.0])
            assert cheb.cheb_last_error() == ""
    _run(worker)


def test_weights_and_tables_built_concurrently_match():
    x = 1.0 - np.arange(50) / 50.0
    ref_w = cheb.cheb_precompute_weights(x[[2, 5, 10, 14, 20, 25]], x[26:30])
    ref_t = cheb.ChebTable(50, 1, 1, 6, 6, x, cheb.CHEB_SHORT_LOWER)
    ref_rows = [ref_t.step(s) for s in range(50)]

    def worker(i):
        for _ in range(ITERS // 8):
            w = cheb.cheb_precompute_weights(x[[2, 5, 10, 14, 20, 25]], x[26:30])
            assert np.array_equal(w, ref_w)
            t = cheb.ChebTable(50, 1, 1, 6, 6, x, cheb.CHEB_SHORT_LOWER)
            for s in range(0, 50, 7):
                a, b = t.step(s), ref_rows[s]
                assert a[0] == b[0] and a[1] == b[1] and np.array_equal(a[2], b[2])
            t.close()
    _run(worker)
    ref_t.close()


def test_launch_shape_updates_are_whole():
    """Concurrent set/get of the launch shape never returns a mix of two
    settings."""
    shapes = [dict(block=256, unroll=4, nontemporal=1, blocks_per_cu=0, waves_per_cu=12),
              dict(block=512, unroll=2, nontemporal=0, blocks_per_cu=2, waves_per_cu=-1),
              dict(block=64, unroll=1, nontemporal=1, blocks_per_cu=0, waves_per_cu=0)]
    old = cheb.cheb_get_launch_config()

    def worker(i):
        for k in range(ITERS):
            cheb.cheb_set_launch_config(**shapes[(i + k) % 3])
            got = cheb.cheb_get_launch_config()
            assert got in shapes, got
    try:
        _run(worker)
    finally:
        cheb.cheb_set_launch_config(**old)
