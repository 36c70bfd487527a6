"""The GPU-vs-oracle comparison rule (CPU)."""
from oracle.compare import compare

O = [[((1, 2, 0), -1.0, 2), ((1, 0), -1.5, 2)]]


def test_identical_passes():
    r = compare(O, [1.0], O)
    assert r.ok and r.n_exact == 1


def test_score_within_tolerance():
    g = [[((1, 2, 0), -1.00005, 2), ((1, 0), -1.5, 2)]]
    assert compare(O, [1.0], g, score_tol=1e-4).ok
    assert not compare(O, [1.0], g, score_tol=1e-5).ok


def test_token_mismatch_fails_without_tie():
    g = [[((1, 3, 0), -1.0, 2), ((1, 0), -1.5, 2)]]
    assert not compare(O, [1e-3], g).ok


def test_order_and_status_matter():
    assert not compare(O, [1.0], [list(reversed(O[0]))]).ok
    assert not compare(O, [1.0], [[((1, 2, 0), -1.0, 3), ((1, 0), -1.5, 2)]]).ok
    assert not compare(O, [1.0], [O[0][:1]]).ok


def test_near_tie_excuses_mismatch():
    g = [[((1, 3, 0), -1.0, 2)]]
    r = compare(O, [5e-5], g, inputs=[7])
    assert r.ok and r.n_excused == 1 and r.excused == [7]


def test_score_error_on_identical_outputs_is_never_excused():
    # Same tokens, statuses and order, but a score off by more than the
    # tolerance: a near tie cannot explain it, whatever the logged margin.
    g = [[((1, 2, 0), -1.01, 2), ((1, 0), -1.5, 2)]]
    r = compare(O, [1e-9], g)
    assert not r.ok and r.n_excused == 0
