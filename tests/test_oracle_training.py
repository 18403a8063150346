"""Pins for the oracle's dead-unit record and targeted re-initialisation: brute force over
tiny batches, special cases that reduce to known values (lam = 0 keeps W, lam = 1
replaces it by the scaled draw, lam = 1/2 is the midpoint), an invariant (live units
untouched, every result between the old weight and the draw) and the variance of the
re-initialised weights in closed form."""
import numpy as np

from oracle import bf16, training


def brute_active(Z):
    T, f = len(Z), len(Z[0])
    out = []
    for n in range(f):
        hit = False
        for t in range(T):
            if Z[t][n] > 0:
                hit = True
        out.append(hit)
    return out


def test_active_units_brute_force():
    r = np.random.default_rng(3)
    for T, f in [(1, 1), (3, 7), (9, 40)]:
        Z = r.normal(size=(T, f))
        Z[:, ::5] = -np.abs(Z[:, ::5])          # some columns never positive
        assert list(training.active_units(Z)) == brute_active(Z.tolist())


def test_active_units_special_values():
    Z = np.array([[0.0, -0.0, np.nan, 1e-45, -np.inf, np.inf],
                  [-1.0, 0.0, -2.0, -1.0, -1.0, -1.0]])
    assert list(training.active_units(Z)) == [False, False, False, True, False, True]
    assert training.active_units(np.zeros((0, 4))).tolist() == [False] * 4


def test_last_active_and_dead_units():
    last = np.array([-1, 3, 5, 2], dtype=np.int64)
    got = training.update_last_active(last, [True, False, True, False], 5)
    assert got.tolist() == [5, 3, 5, 2]
    assert training.dead_units(got, 5).tolist() == [False, True, False, True]
    # a unit active at the current step is never dead; before any activity all are dead
    assert training.dead_units(np.full(3, -1), 0).all()


def test_reinit_special_cases():
    r = np.random.default_rng(4)
    W = r.normal(size=(6, 5)) * 0.02
    nz = r.normal(size=(6, 5))
    dead = np.array([True, False, True, False, False])
    same = training.reinit_dead(W, dead, 0.0, 0.02, nz)
    assert np.array_equal(same, W)
    full = training.reinit_dead(W, dead, 1.0, 0.02, nz)
    assert np.array_equal(full[:, dead], 0.02 * nz[:, dead])
    assert np.array_equal(full[:, ~dead], W[:, ~dead])
    mid = training.reinit_dead(W, dead, 0.5, 0.02, nz)
    assert np.allclose(mid[:, dead], (W[:, dead] + 0.02 * nz[:, dead]) / 2, rtol=0, atol=1e-17)
    # rows as units (a transposed copy) give the transposed result
    rows = training.reinit_dead(W.T, dead, 0.3, 0.02, nz.T, units_on_rows=True)
    assert np.array_equal(rows, training.reinit_dead(W, dead, 0.3, 0.02, nz).T)


def test_reinit_between_old_and_draw():
    r = np.random.default_rng(5)
    W = r.normal(size=(50, 20)) * 0.02
    nz = r.normal(size=(50, 20))
    dead = r.random(20) < 0.5
    out = training.reinit_dead(W, dead, 0.1, 0.02, nz)
    lo = np.minimum(W, 0.02 * nz) - 1e-18
    hi = np.maximum(W, 0.02 * nz) + 1e-18
    assert ((out >= lo) & (out <= hi)).all()
    assert np.array_equal(out[:, ~dead], W[:, ~dead])


def test_reinit_variance_closed_form():
    # W at its initial distribution N(0, s^2) and an independent draw: the result has
    # variance ((1 - lam)^2 + lam^2) s^2
    r = np.random.default_rng(6)
    s, lam = 0.02, 0.1
    W = r.normal(size=(4000, 50)) * s
    nz = r.normal(size=(4000, 50))
    out = training.reinit_dead(W, np.ones(50, dtype=bool), lam, s, nz)
    want = ((1 - lam) ** 2 + lam ** 2) * s * s
    assert abs(out.var() / want - 1) < 0.01


def test_reinit_bf16_rounding():
    r = np.random.default_rng(7)
    W = bf16.round_to_bf16_value(r.normal(size=(8, 9)) * 0.02)
    nz = r.normal(size=(8, 9))
    dead = np.ones(9, dtype=bool)
    out = training.reinit_dead(W, dead, 0.1, 0.02, nz, bf16_out=True)
    assert np.array_equal(out, bf16.round_to_bf16_value(out))
    exact = training.reinit_dead(W, dead, 0.1, 0.02, nz)
    # within half a bf16 unit in the last place of the exact value
    ulp = np.ldexp(1.0, np.frexp(np.abs(exact))[1] - 8)
    assert (np.abs(out - exact) <= ulp / 2 + 1e-30).all()
