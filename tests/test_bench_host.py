"""Host-side logic of the benchmark (no GPU): the Amdahl fit of the batch sweep and the
fixed-length workloads it runs on."""
import numpy as np

import bench
from paper_1904_03409_amd import workloads as wk


def test_amdahl_fit_recovers_the_parallel_fraction():
    for P in (0.5, 0.99, 0.9992):
        bs = [1, 2, 4, 8, 16, 32, 64, 128, 256]
        S = [1.0 / ((1.0 - P) + P / b) for b in bs]
        p_fit, each = bench.amdahl_fit(bs, S)
        assert abs(p_fit - P) < 1e-12
        assert all(abs(v - P) < 1e-12 for v in each.values())


def test_amdahl_matches_the_papers_figures():
    # a 60.8x speed-up at a batch of 64 is a parallel fraction of 99.92% (to the printed digits)
    _, each = bench.amdahl_fit([1, 64], [1.0, 60.8])
    assert abs(each[64] - 0.9992) < 5e-5


def test_sweep_workloads_have_fixed_length_and_hold_padding():
    for B in (1, 4, 64):
        wl = wk.make("parser", B=B, T=120)
        assert wl.T == 120 and wl.ops.shape == (120, B)
        depth = np.cumsum(wl.ops.astype(np.int64), axis=0)
        assert depth.min() >= 0
        # the padded tail is holds only
        last = [np.nonzero(wl.ops[:, b])[0].max() for b in range(B)]
        assert all(np.all(wl.ops[l + 1:, b] == 0) for b, l in enumerate(last))
    # without the override the recipe is unchanged
    a, b = wk.make("parser"), wk.make("parser", T=None)
    assert a.T == b.T and np.array_equal(a.ops, b.ops) and np.array_equal(a.x, b.x)


def test_kernel_hash_ignores_comments_not_code():
    """Stored counter readings stay valid across comment edits, not across code edits."""
    from bench import strip_comments
    a = "int f(int x) { return x + 1; } // add one\n/* block\n comment */ int g;"
    b = "int f(int x) {\n  return x + 1;   // different words\n}\nint g;"
    c = "int f(int x) { return x + 2; } int g;"
    assert strip_comments(a) == strip_comments(b)
    assert strip_comments(a) != strip_comments(c)
