"""Generator invariants: valid streams, the recipe's shapes, determinism."""
import numpy as np
import pytest

from paper_1904_03409_amd import workloads as wk


def _depth(ops):
    return np.vstack([np.zeros((1, ops.shape[1]), np.int64), np.cumsum(ops.astype(np.int64), axis=0)])


@pytest.mark.parametrize("name", ["tiny", "parser", "large", "deep"])
def test_pointer_never_negative_and_ops_valid(name):
    wl = wk.make(name)
    assert wl.ops.dtype == np.int8 and wl.ops.shape == (wl.T, wl.B)
    assert set(np.unique(wl.ops)).issubset({-1, 0, 1})
    assert _depth(wl.ops).min() == 0
    assert wl.x.shape == (wl.T, wl.B, wl.I) and wl.W.shape == (wl.I, 4 * wl.H) and wl.U.shape == (wl.H, 4 * wl.H)
    assert wl.dh_top.shape == (wl.T, wl.B, wl.H)


@pytest.mark.parametrize("name,nlo,nhi", [("parser", 10, 60), ("large", 20, 120)])
def test_arc_standard_shape(name, nlo, nhi):
    wl = wk.make(name)
    d = _depth(wl.ops)
    nmax = 0
    for b in range(wl.B):
        col = wl.ops[:, b].astype(np.int64)
        n = int((col == 1).sum())
        assert nlo <= n <= nhi
        assert int((col == -1).sum()) == n - 1
        nmax = max(nmax, n)
        L = 2 * n - 1
        assert np.all(col[L:] == 0) and np.all(col[:L] != 0)       # holds only as trailing padding
        pops = np.where(col == -1)[0]
        assert np.all(d[pops, b] >= 2)                                # a reduce needs two items
        assert d[L, b] == 1
    assert wl.T == 2 * nmax


def test_tiny_shape():
    wl = wk.make("tiny")
    assert wl.T == 64 and wl.B == 8
    for b in range(wl.B):
        col = wl.ops[:, b]
        nz = np.nonzero(col)[0]
        L = nz[-1] + 1
        assert L <= 64 and np.all(col[:L] != 0)
    assert np.all(wl.b == 0) and np.abs(wl.W).max() <= 0.1


def test_deep_shape():
    wl = wk.make("deep")
    st = wl.op_stats()
    assert wl.T == 1024 and st["hold"] == 0.0
    assert 400 <= st["max_depth"] <= 700


def test_same_seed_same_bytes():
    a, b = wk.make("parser"), wk.make("parser")
    for k in ("ops", "x", "W", "U", "b", "h0", "c0", "dh_top"):
        assert getattr(a, k).tobytes() == getattr(b, k).tobytes()
    c = wk.make("parser", seed=7)
    assert c.x.tobytes() != a.x.tobytes()


def test_arc_hybrid_streams_follow_the_transition_table():
    """Stack and buffer streams of one sentence: the n words enter the buffer first (the
    stack holds), then every shift is a stack push and a buffer pop, every arc a stack pop
    and a buffer hold; neither stack underflows; the buffer ends empty and one item stays
    on the stack."""
    rng = np.random.default_rng(0)
    for _ in range(200):
        n = int(rng.integers(1, 30))
        st, bu = wk.ops_arc_hybrid_streams(rng, n)
        assert len(st) == len(bu) == 3 * n - 1
        assert np.all(bu[:n] == 1) and np.all(st[:n] == 0)
        tr_s, tr_b = st[n:], bu[n:]
        assert np.all((tr_s == 1) == (tr_b == -1))      # shift
        assert np.all((tr_s == -1) == (tr_b == 0))      # left-arc / right-arc
        assert (tr_s == 1).sum() == n and (tr_s == -1).sum() == n - 1
        ds, db = np.cumsum(st.astype(int)), np.cumsum(bu.astype(int))
        assert ds.min() >= 0 and db.min() >= 0
        assert ds[-1] == 1 and db[-1] == 0


def test_hybrid_workload_is_a_doubled_batch():
    w = wk.make("hybrid", B=6)
    assert w.B == 12 and w.ops.shape == (w.T, 12)
    depth = np.cumsum(w.ops.astype(np.int64), axis=0)
    assert depth.min() >= 0
    assert np.all(depth[-1, :6] == 1) and np.all(depth[-1, 6:] == 0)
    # the buffer half starts with pushes while the stack half holds
    assert np.all(w.ops[0, :6] == 0) and np.all(w.ops[0, 6:] == 1)
