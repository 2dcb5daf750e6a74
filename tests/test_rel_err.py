"""The value checker behind every float parity test: oracle.rel_err (the
infinity-norm relative error, max|y - r| / max|r|) and oracle.rel_err_tiles
(the same per 32 x 32 output tile), pinned on the CPU by cases whose value is
fixed by the definition, and by planted mistakes that each must fail a case."""
import numpy as np
import pytest

import oracle

INF = float("inf")


def _cases():
    r = np.array([[3.0, -4.0], [1.0, 2.0]])
    yield "one element up", r + np.array([[0.0, 0.0], [0.5, 0.0]]), r, 0.5 / 4.0
    yield "one element down (the difference's sign)", r - np.array([[0.0, 0.0], [0.5, 0.0]]), r, 0.5 / 4.0
    yield "scale is the reference's, not the result's", 2.0 * r, r, 1.0
    neg = np.array([[-10.0, 1.0]])
    yield "largest magnitude is negative", np.array([[-10.0, 1.5]]), neg, 0.05
    yield "exact match", r.copy(), r, 0.0
    yield "all-zero reference, zero result", np.zeros((3, 3)), np.zeros((3, 3)), 0.0
    yield "all-zero reference, nonzero result", np.eye(3) * 1e-30, np.zeros((3, 3)), INF
    yield "empty", np.zeros((0, 4)), np.zeros((0, 4)), 0.0
    y = r.copy()
    y[0, 0] = np.nan
    yield "NaN in the result", y, r, INF
    y = r.copy()
    y[1, 1] = np.inf
    yield "Inf in the result", y, r, INF
    yield "shape mismatch", r[:1], r, INF


def _tile_cases():
    g = np.random.default_rng(3)
    r = g.normal(size=(70, 90))          # ragged: 3 x 3 tiles of 32 x 32
    big = r.copy()
    big[:32, :32] *= 1000.0              # one tile dominates the global maximum
    y = big.copy()
    y[64:, 64:] += 0.01                  # an error confined to the ragged corner tile
    corner = np.max(np.abs(r[64:, 64:]))
    yield "error confined to one small tile", y, big, 0.01 / corner
    y = r.copy()
    yield "exact", y, r, 0.0
    z = r.copy()
    z[32:64, 32:64] = 0.0
    y = z.copy()
    y[40, 40] = 1e-6
    yield "all-zero tile with a nonzero result", y, z, INF
    y = r.copy()
    y[69, 89] = np.nan
    yield "NaN in the last ragged element", y, r, INF


@pytest.mark.parametrize("name,y,r,want", list(_cases()), ids=lambda v: v if isinstance(v, str) else "")
def test_rel_err_cases(name, y, r, want):
    got = oracle.rel_err(y, r)
    if want == INF:
        assert got == INF
    else:
        assert got == pytest.approx(want, rel=1e-12, abs=0.0)


@pytest.mark.parametrize("name,y,r,want", list(_tile_cases()), ids=lambda v: v if isinstance(v, str) else "")
def test_rel_err_tiles_cases(name, y, r, want):
    got = oracle.rel_err_tiles(y, r)
    if want == INF:
        assert got == INF
    else:
        assert got == pytest.approx(want, rel=1e-12, abs=0.0)
    # the global measure hides the confined error; the tile-wise one does not
    if name.startswith("error confined"):
        assert oracle.rel_err(y, r) < 1e-4 < got


def test_rel_err_tiles_equals_global_on_one_tile():
    g = np.random.default_rng(4)
    r = g.normal(size=(20, 30))
    y = r + g.normal(size=r.shape) * 1e-3
    assert oracle.rel_err_tiles(y, r) == pytest.approx(oracle.rel_err(y, r), rel=1e-15)


# ---- planted mistakes: each must fail at least one case ------------------------

def _m_no_abs(y, r):
    return float(np.max(y - r) / np.max(np.abs(r)))


def _m_scale_from_y(y, r):
    return float(np.max(np.abs(y - r)) / np.max(np.abs(y)))


def _m_scale_signed(y, r):
    return float(np.max(np.abs(y - r)) / np.max(r))


def _m_mean_not_max(y, r):
    return float(np.mean(np.abs(y - r)) / np.max(np.abs(r)))


def _m_zero_ref_is_ok(y, r):
    s = np.max(np.abs(r)) if r.size else 0.0
    return 0.0 if s == 0 else float(np.max(np.abs(y - r)) / s)


def _m_nan_passes(y, r):
    y = np.nan_to_num(np.asarray(y, np.float64), nan=0.0, posinf=0.0)
    return oracle.rel_err(y, r)


def _m_elementwise(y, r):
    return float(np.max(np.abs(y - r) / np.maximum(np.abs(r), 1e-300)))


MUTANTS = [_m_no_abs, _m_scale_from_y, _m_scale_signed, _m_mean_not_max, _m_zero_ref_is_ok,
           _m_nan_passes, _m_elementwise]


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda f: f.__name__[3:])
def test_mutants_fail_a_case(mutant):
    failed = []
    for name, y, r, want in _cases():
        try:
            with np.errstate(all="ignore"):
                got = mutant(np.asarray(y, np.float64), np.asarray(r, np.float64))
        except (ValueError, ZeroDivisionError):
            failed.append(name)
            continue
        ok = (got == INF) if want == INF else (got == pytest.approx(want, rel=1e-12, abs=0.0))
        if not ok:
            failed.append(name)
    assert failed, "planted mistake %s passed every case" % mutant.__name__
