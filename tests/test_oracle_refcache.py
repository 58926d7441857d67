"""Pins of the adaptive reference cache oracle (Sec. 3.4): closed forms at the
threshold extremes, a hand-worked example, the release sequence, hold-count
invariants under random multi-step writes, and the residual's error bound."""
import numpy as np
import pytest

from oracle.refcache import NONE, REFERENCE, RESIDUAL, RefCache, cosine, step_update


def _rows(rng, L, D):
    return rng.standard_normal((L, D)).astype(np.float32)


def test_cosine_special_cases():
    a = np.array([3.0, 4.0], np.float32)
    assert cosine(a, a) == pytest.approx(1.0, abs=1e-15)
    assert cosine(a, -a) == pytest.approx(-1.0, abs=1e-15)
    assert cosine(np.array([1.0, 0.0]), np.array([0.0, 2.0])) == 0.0
    assert cosine(np.zeros(2), a) == 0.0 and cosine(a, np.zeros(2)) == 0.0


def test_tau_below_minus_one_keeps_one_reference_per_chain():
    # every similarity exceeds tau < -1: a chain's first written token is its
    # only reference, every later token a residual against it
    rng = np.random.default_rng(0)
    L, D, w = 40, 16, 8
    c = RefCache(L, D, w, tau=-2.0, dtype="f32")
    c.write(np.arange(L), _rows(rng, L, D))
    assert c.live_refs() == L // w
    assert list(np.flatnonzero(c.kind == REFERENCE)) == list(range(0, L, w))
    assert (c.kind[np.arange(L) % w != 0] == RESIDUAL).all()
    c.check_holds()


def test_tau_above_one_stores_every_token():
    # no similarity exceeds 1.5: every written token is a reference, read back exactly
    rng = np.random.default_rng(1)
    L, D, w = 24, 8, 6
    y = _rows(rng, L, D)
    for dtype in ("f32", "bf16"):
        c = RefCache(L, D, w, tau=1.5, dtype=dtype)
        c.write(np.arange(L), y)
        assert c.live_refs() == L
        assert (c.kind == REFERENCE).all()
        from oracle.cache import cast_act
        assert np.array_equal(c.read(), cast_act(y, dtype))
        c.check_holds()


def test_hand_worked_chain():
    # chain of 4: e1, close to e1, e2, close to e2 (tau 0.9):
    # cos((0.9, 0.1), e1) = 0.9939 -> residual; cos(e2, e1) = 0 -> new reference;
    # cos((0.1, 0.9), e2) = 0.9939 -> residual
    y = np.array([[1, 0], [0.9, 0.1], [0, 1], [0.1, 0.9]], np.float32)
    c = RefCache(4, 2, 4, tau=0.9, dtype="f32")
    c.write(np.arange(4), y)
    assert list(c.kind) == [REFERENCE, RESIDUAL, REFERENCE, RESIDUAL]
    assert c.ref_of[1] == c.ref_of[0] and c.ref_of[3] == c.ref_of[2] != c.ref_of[0]
    assert c.live_refs() == 2
    # the residual (-0.1, 0.1) has amax 0.1: codes -127, 127, read back within half a step
    assert list(c.codes[1]) == [-127, 127]
    assert np.allclose(c.read([1])[0], y[1], atol=0.1 / 254 + 1e-7)
    c.check_holds()


def test_identical_rows_give_zero_residuals():
    y = np.tile(np.array([[0.5, -1.5, 2.0]], np.float32), (6, 1))
    c = RefCache(6, 3, 3, tau=0.99, dtype="f32")
    c.write(np.arange(6), y)
    assert list(c.kind) == [REFERENCE, RESIDUAL, RESIDUAL] * 2
    assert (c.scale[c.kind == RESIDUAL] == 0).all() and (c.codes == 0).all()
    assert np.array_equal(c.read(), y)


def test_release_sequence():
    # one chain: t0 reference, t1 t2 residuals of it
    y = np.array([[1, 0], [1, 0.01], [1, -0.01]], np.float32)
    c = RefCache(3, 2, 3, tau=0.9, dtype="f32")
    c.write([0, 1, 2], y)
    r0 = int(c.ref_of[0])
    assert c.holds[r0] == 4                      # 3 entries + the chain
    # rewrite t0 with something orthogonal: its old entry drops, the chain
    # moves to the new reference, r0 survives for t1 and t2
    c.write([0], np.array([[0, 1]], np.float32))
    assert c.kind[0] == REFERENCE and int(c.ref_of[0]) != r0
    assert r0 in c.refs and c.holds[r0] == 2
    assert c.live_refs() == 2
    # rewriting t1 and t2 against the new reference (orthogonal to them:
    # both become references themselves) releases r0
    c.write([1, 2], y[1:])
    assert r0 not in c.refs
    c.check_holds()


@pytest.mark.parametrize("tau", [0.0, 0.3, 0.6])
def test_random_multi_step_invariants(tau):
    rng = np.random.default_rng(int(tau * 10) + 5)
    L, D, w = 60, 12, 10
    base = _rows(rng, w, D)
    c = RefCache(L, D, w, tau=tau, dtype="bf16")
    stored = {}
    for step in range(6):
        k = L if step == 0 else int(rng.integers(1, L))
        idx = np.sort(rng.choice(L, k, replace=False))
        # rows drift around a per-position base so that similarities vary
        y = (base[idx % w] + rng.standard_normal((k, D)) * (0.2 + 0.3 * step)).astype(np.float32)
        c.write(idx, y)
        c.check_holds()
        for j, l in enumerate(idx):
            stored[int(l)] = y[j]
        # every token reads back its last written output within its residual's bound
        got = c.read()
        for l in range(L):
            want = stored[l]
            if c.kind[l] == REFERENCE:
                from oracle.cache import round_bf16
                assert np.array_equal(got[l], round_bf16(want))
            else:
                # half a quantization step, then the bf16 rounding of the output
                half = 0.5 * float(c.scale[l]) * (1 + 1e-5)
                bound = half + 2.0 ** -8 * (np.abs(want) + half) + 1e-30
                assert (np.abs(got[l] - want) <= bound).all()


def test_step_update_fuses_fresh_and_cached():
    rng = np.random.default_rng(3)
    L, D, w = 20, 6, 5
    c = RefCache(L, D, w, tau=0.2, dtype="f32")
    x0 = _rows(rng, L, D)
    y0 = _rows(rng, L, D)
    y, xref = step_update(c, x0, np.arange(L), y0, np.zeros((L, D), np.float32))
    assert np.array_equal(y, y0) and np.array_equal(xref, x0)
    before = c.read()
    idx = np.array([2, 7, 11])
    x1 = _rows(rng, L, D)
    y1 = _rows(rng, 3, D)
    y, xref = step_update(c, x1, idx, y1, xref)
    assert np.array_equal(y[idx], y1)
    rest = np.setdiff1d(np.arange(L), idx)
    assert np.array_equal(y[rest], before[rest])
    assert np.array_equal(xref[idx], x1[idx]) and np.array_equal(xref[rest], x0[rest])
    assert (c.kind != NONE).all()


def test_threshold_is_strict():
    # cos(e1, (1, 1, 1, 1)) = 1 / 2 exactly (norms 1 and 2): equal to tau -> a new
    # reference; a threshold just below -> residual
    y = np.array([[1, 0, 0, 0], [1, 1, 1, 1]], np.float32)
    c = RefCache(2, 4, 2, tau=0.5, dtype="f32")
    c.write([0, 1], y)
    assert c.sims[1] == 0.5
    assert list(c.kind) == [REFERENCE, REFERENCE]
    c = RefCache(2, 4, 2, tau=0.4999, dtype="f32")
    c.write([0, 1], y)
    assert list(c.kind) == [REFERENCE, RESIDUAL]


def test_threshold_is_the_fp32_value():
    # the boundary takes tau as an fp32: 0.3 means 0.30000001192...
    assert RefCache(2, 4, 2, tau=0.3, dtype="f32").tau == float(np.float32(0.3))


def test_current_reference_persists_across_writes():
    # a later write that starts mid-chain compares against the chain's
    # reference from the earlier write instead of starting a new one
    c = RefCache(4, 2, 4, tau=0.9, dtype="f32")
    c.write([0], np.array([[1, 0]], np.float32))
    c.write([2], np.array([[1, 0.05]], np.float32))
    assert c.kind[2] == RESIDUAL and c.ref_of[2] == c.ref_of[0]
    assert c.live_refs() == 1
