"""Offline stage through the C ABI (host only): schedule, weight table,
serialisation and the table/ring consistency checks, against the oracle's
Algorithm-1 simulation."""
import os

import numpy as np
import pytest

import oracle
import paper_2608_23429_amd as cheb
from paper_2608_23429_amd import _binding as B

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
FAKE_ARENA = 1 << 40


def _wtol(w, factor=16.0):
    s = float(np.abs(w).sum())
    return factor * max(1, len(w)) * 2.0 ** -53 * s * max(s, 1.0)


def _sampler_grid(rng, T, top=1000.0):
    """Decreasing timesteps whose spacing varies by at most 3x, as in a
    sampler's schedule (the rows stay well inside fp64's resolution)."""
    gaps = rng.uniform(0.5, 1.5, size=T) * (top / max(T, 1))
    return (top - np.concatenate([[0.0], np.cumsum(gaps[:-1])]))


def test_schedule_matches_golden_and_oracle():
    with open(os.path.join(GOLDEN, "full_schedule.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            head, tail = line.split(":")
            kind, T, s0, s1, r = head.split()
            mask = cheb.cheb_schedule(int(T), int(s0), int(s1), int(r))
            if kind == "set":
                assert np.flatnonzero(mask).tolist() == [int(v) for v in tail.split()]
            else:
                assert int(mask.sum()) == int(tail)
    rng = np.random.default_rng(1)
    for _ in range(200):
        T, s0, s1, r = int(rng.integers(1, 80)), int(rng.integers(0, 6)), int(rng.integers(0, 6)), int(rng.integers(1, 9))
        assert np.array_equal(cheb.cheb_schedule(T, s0, s1, r), oracle.full_schedule(T, s0, s1, r))


def _compare_table(T, s0, s1, r, n, x, policy):
    t = cheb.ChebTable(T, s0, s1, r, n, x, policy)
    n_full = 0
    for s in range(T):
        pred, nodes, w = t.step(s)
        kind, onodes, ow = oracle.table_row(T, s0, s1, r, n, x, policy, s)
        assert pred == bool(kind), (T, s0, s1, r, n, policy, s)
        n_full += 0 if pred else 1
        assert nodes == onodes, (s, nodes, onodes)
        if pred:
            assert np.max(np.abs(w - ow)) <= _wtol(ow), (s, w, ow)
    assert t.n_full == n_full
    return t


@pytest.mark.parametrize("policy", [B.CHEB_SHORT_FULL, B.CHEB_SHORT_LOWER])
def test_table_matches_oracle_simulation(policy):
    rng = np.random.default_rng(10 + policy)
    for _ in range(60):
        T = int(rng.integers(2, 60))
        s0, s1, r = int(rng.integers(0, 5)), int(rng.integers(0, 5)), int(rng.integers(1, 8))
        n = int(rng.integers(1, 9))
        x = _sampler_grid(rng, T)
        _compare_table(T, s0, s1, r, n, x, policy)


def test_paper_schedules():
    """The full-step counts the paper's FLOPs columns imply (Table 1,
    DiT-XL/2 DDIM-50, H=3: 18/14/12 for r=3/4/5; Table 2, FLUX 50 steps, H=2:
    12/10 for r=5/6) with s0 = s1 = 1.  For H=3 they hold when the steps
    before three entries exist predict from fewer (CHEB_SHORT_LOWER); running
    those steps in full adds one full step."""
    t_ddim = 980.0 - 20.0 * np.arange(50)
    for r, full in [(3, 18), (4, 14), (5, 12)]:
        assert _compare_table(50, 1, 1, r, 3, t_ddim, B.CHEB_SHORT_LOWER).n_full == full
        assert _compare_table(50, 1, 1, r, 3, t_ddim, B.CHEB_SHORT_FULL).n_full == full + 1
    sigma = 1.0 - np.arange(50) / 50.0
    for r, full in [(5, 12), (6, 10)]:
        for policy in (B.CHEB_SHORT_FULL, B.CHEB_SHORT_LOWER):
            assert _compare_table(50, 1, 1, r, 2, sigma, policy).n_full == full


def test_table_save_load_roundtrip(tmp_path):
    x = 1.0 - np.arange(50) / 50.0
    t = cheb.ChebTable(50, 1, 1, 6, 6, x, B.CHEB_SHORT_LOWER)
    path = os.path.join(tmp_path, "flux.chebtable")
    t.save(path)
    u = cheb.ChebTable.load(path)
    assert (u.T, u.n_hist, u.policy, u.n_full) == (t.T, t.n_hist, t.policy, t.n_full)
    for s in range(50):
        a, b = t.step(s), u.step(s)
        assert a[0] == b[0] and a[1] == b[1]
        assert np.array_equal(a[2], b[2])             # bit for bit (hex floats)


@pytest.mark.parametrize("mangle", [
    lambda txt: "notatable 1\n" + txt.split("\n", 1)[1],
    lambda txt: txt.replace("n_hist 6", "n_hist 99"),
    lambda txt: txt.replace("step 7 ", "step 8 ", 1),
    lambda txt: txt.replace(" predict 2 ", " predict 9 ", 1),
    lambda txt: txt.rsplit("\n", 3)[0],
    lambda txt: txt.replace(" predict 6 ", " predict 6 99 0x1p+0 ", 1),
])
def test_table_load_rejects_malformed(tmp_path, mangle):
    x = 1.0 - np.arange(50) / 50.0
    t = cheb.ChebTable(50, 1, 1, 6, 6, x, B.CHEB_SHORT_LOWER)
    good = os.path.join(tmp_path, "good")
    t.save(good)
    bad = os.path.join(tmp_path, "bad")
    with open(good) as f, open(bad, "w") as g:
        g.write(mangle(f.read()))
    with pytest.raises(cheb.ChebError) as e:
        cheb.ChebTable.load(bad)
    assert e.value.code == B.CHEB_E_IO
    with pytest.raises(cheb.ChebError) as e:
        cheb.ChebTable.load(os.path.join(tmp_path, "missing"))
    assert e.value.code == B.CHEB_E_IO


def test_table_errors():
    x = np.arange(10.0)
    for args, code in [((0, 0, 0, 1, 2, x[:0]), B.CHEB_E_INVAL), ((10, 0, 0, 0, 2, x), B.CHEB_E_INVAL),
                       ((10, 0, 0, 2, 9, x), B.CHEB_E_INVAL), ((10, -1, 0, 2, 2, x), B.CHEB_E_INVAL)]:
        with pytest.raises(cheb.ChebError) as e:
            cheb.cheb_table_build(*args)
        assert e.value.code == code
    xs = x.copy()
    xs[3] = np.nan
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_table_build(10, 0, 0, 2, 2, xs)
    assert e.value.code == B.CHEB_E_NONFINITE
    xd = x.copy()
    xd[4] = xd[2]                                   # full steps 2 and 4 collide
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_table_build(10, 0, 0, 2, 2, xd)
    assert e.value.code == B.CHEB_E_DUPNODE
    with pytest.raises(cheb.ChebError) as e:
        cheb.cheb_table_build(10, 0, 0, 2, 2, x, 3)
    assert e.value.code == B.CHEB_E_INVAL


def test_table_with_an_ill_conditioned_row_is_refused():
    """Three full steps a thousandth apart predicting a step 500 away: the
    row's sum |w| (about 2.5e11) is past what fp64 resolves to fp32
    accuracy, so the build fails instead of storing it."""
    x = np.array([1000.0, 999.999, 999.998, 500.0, 400.0])
    mask = np.array([True, True, True, False, True])
    kind, _, ow = oracle.table_row_mask(mask, 3, x, B.CHEB_SHORT_FULL, 3)
    assert kind == 1 and 3 * 2.0 ** -53 * np.abs(ow).sum() > 2.0 ** -24
    with pytest.raises(cheb.ChebError) as e:
        cheb.ChebTable.from_mask(mask, 3, x, B.CHEB_SHORT_FULL)
    assert e.value.code == B.CHEB_E_NONFINITE


def test_extrapolate_steps_checks_ring_against_row():
    """Row selection (the history must hold the row's nodes) is checked on
    the host before anything is enqueued."""
    x = 999.0 - 50.0 * np.arange(20)
    t = cheb.ChebTable(20, 2, 1, 4, 3, x)           # full {0,1,2,6,10,14,18,19}
    lay = cheb.cheb_cache_layout(3, B.CHEB_BF16, [4096])
    h = cheb.cheb_cache_create(3, B.CHEB_BF16, [4096], FAKE_ARENA, lay["arena_bytes"])
    out = [FAKE_ARENA + (1 << 34) + k * (1 << 20) for k in range(4)]

    def push(step):
        cheb.cheb_cache_begin_push(h)
        cheb.cheb_cache_commit(h, x[step])

    def code(first, outs):
        with pytest.raises(cheb.ChebError) as e:
            cheb.cheb_extrapolate_steps(h, t.handle, first, outs)
        return e.value.code

    push(0)
    push(1)
    assert code(3, out[:3]) == B.CHEB_E_NOTREADY            # H = {0, 1}, needs 3
    push(2)
    assert code(6, out[:1]) == B.CHEB_E_INVAL               # step 6 is a full step
    assert code(5, out[:2]) == B.CHEB_E_INVAL               # 5, 6: 6 is full
    push(6)
    assert code(3, out[:1]) == B.CHEB_E_MISMATCH            # ring holds {1, 2, 6}
    assert code(17, out[:3]) == B.CHEB_E_INVAL              # runs past the table
    assert code(7, out[:0]) == B.CHEB_E_INVAL               # no outputs
    cheb.cheb_cache_destroy(h)


def test_mask_tables_match_oracle_and_roundtrip(tmp_path):
    rng = np.random.default_rng(77)
    for policy in (B.CHEB_SHORT_FULL, B.CHEB_SHORT_LOWER):
        for _ in range(40):
            T = int(rng.integers(2, 50))
            mask = rng.random(T) < rng.uniform(0.1, 0.6)
            n = int(rng.integers(1, 7))
            x = _sampler_grid(rng, T, 1.0)
            t = cheb.ChebTable.from_mask(mask, n, x, policy)
            for s in range(T):
                pred, nodes, w = t.step(s)
                kind, onodes, ow = oracle.table_row_mask(mask, n, x, policy, s)
                assert pred == bool(kind) and nodes == onodes
                if pred:
                    assert np.max(np.abs(w - ow)) <= _wtol(ow)
    # F itself as a mask gives the grid table
    x = 980.0 - 20.0 * np.arange(50)
    a = cheb.ChebTable(50, 1, 1, 3, 3, x, B.CHEB_SHORT_LOWER)
    b = cheb.ChebTable.from_mask(cheb.cheb_schedule(50, 1, 1, 3), 3, x, B.CHEB_SHORT_LOWER)
    for s in range(50):
        assert a.step(s)[1] == b.step(s)[1]
        assert np.array_equal(a.step(s)[2], b.step(s)[2])
    # Chebyshev-placed full steps over 50 steps, saved and loaded
    cheb_steps = np.unique(np.rint(cheb.cheb_chebyshev_nodes(12, 1, 0, 49)).astype(int))
    mask = np.zeros(50, dtype=bool)
    mask[cheb_steps] = True
    t = cheb.ChebTable.from_mask(mask, 4, x, B.CHEB_SHORT_LOWER)
    path = os.path.join(tmp_path, "cheb_nodes.chebtable")
    t.save(path)
    u = cheb.ChebTable.load(path)
    for s in range(50):
        assert t.step(s)[1] == u.step(s)[1] and np.array_equal(t.step(s)[2], u.step(s)[2])
