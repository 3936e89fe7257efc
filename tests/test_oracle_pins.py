"""Pins for the CPU oracle of the exchange step (no GPU needed).

Each test checks the oracle against something other than itself: values
derived by hand (golden files), closed forms, exact rational arithmetic with
the rounding points of IEEE-754 single precision, a library optimizer, and
the forward error bound of the fp32 evaluation.  Together they are chosen so
that a dropped term, a wrong sign, a mixed-up index or a changed rounding
point in the oracle fails at least one test.
"""

import math
import os
from fractions import Fraction

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

f32 = np.float32


def _hx(s):
    return float.fromhex(s)


def _one_elem_step(oracle_mod, gs, w, m, lr, mu, wd, nesterov, steps=1):
    grads = [np.array([g], dtype=np.float32) for g in gs]
    wa = np.array([w], dtype=np.float32)
    ma = np.array([m], dtype=np.float32)
    out = []
    for _ in range(steps):
        oracle_mod.step_flat(grads, wa, ma, lr, mu, wd, nesterov)
        out.append((wa.copy(), ma.copy()))
    return out


def _bits(a):
    return np.asarray(a, dtype=np.float32).view(np.uint32)


# --------------------------------------------------------------------------
# Golden: worked example (hand-derived dyadic values).
# --------------------------------------------------------------------------

def _read_worked_example():
    inputs = None
    expect = {"nesterov": {}, "plain": {}}
    with open(os.path.join(GOLDEN, "worked_example.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "inputs":
                inputs = [float(t) for t in tok[1:]]
            else:
                expect[tok[0]][int(tok[1])] = (float(tok[2]), float(tok[3]))
    return inputs, expect


@pytest.mark.parametrize("mode", ["nesterov", "plain"])
def test_worked_example(oracle_mod, mode):
    (g0, g1, w0, m0, lr, mu, wd), expect = _read_worked_example()
    out = _one_elem_step(oracle_mod, [g0, g1], w0, m0, lr, mu, wd, mode == "nesterov", steps=3)
    for t, (w, m) in enumerate(out, start=1):
        ew, em = expect[mode][t]
        assert _bits(w)[0] == _bits(ew), (mode, t, w, ew)
        assert _bits(m)[0] == _bits(em), (mode, t, m, em)


def test_worked_example_mean_reading_fails_pin(oracle_mod):
    """The pin distinguishes a sum from a mean: with lr halved (the mean of
    two workers) the first Nesterov step would differ from the golden value."""
    (g0, g1, w0, m0, lr, mu, wd), expect = _read_worked_example()
    out = _one_elem_step(oracle_mod, [g0 / 2, g1 / 2], w0, m0, lr, mu, wd, True, steps=1)
    assert out[0][0][0] != expect["nesterov"][1][0]


# --------------------------------------------------------------------------
# Golden: rounding points (summation order, fused multiply-adds, subnormals).
# --------------------------------------------------------------------------

def _read_rounding_cases():
    cases = []
    with open(os.path.join(GOLDEN, "rounding_points.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            name, nest, n = tok[0], int(tok[1]), int(tok[2])
            vals = [_hx(t) for t in tok[3:]]
            gs = vals[:n]
            w, m, lr, mu, wd, ew, em = vals[n:n + 7]
            assert len(vals) == n + 7, name
            cases.append((name, bool(nest), gs, w, m, lr, mu, wd, ew, em))
    return cases


ROUNDING_CASES = _read_rounding_cases()


@pytest.mark.parametrize("case", ROUNDING_CASES, ids=[c[0] for c in ROUNDING_CASES])
def test_rounding_points(oracle_mod, case):
    name, nest, gs, w, m, lr, mu, wd, ew, em = case
    for v in gs + [w, m, lr, mu, wd, ew, em]:
        assert float(f32(v)) == v, f"{name}: fixture value {v!r} is not an fp32 value"
    (wo, mo), = _one_elem_step(oracle_mod, gs, w, m, lr, mu, wd, nest)
    assert _bits(wo)[0] == _bits(ew), (name, wo[0].hex() if hasattr(wo[0], 'hex') else wo, ew)
    assert _bits(mo)[0] == _bits(em), (name, mo, em)


# --------------------------------------------------------------------------
# Identical gradients: N copies of g sum to N*g.
# --------------------------------------------------------------------------

@pytest.mark.parametrize("n_workers", [1, 2, 3, 4, 7, 8, 16])
def test_identical_gradients_sum_exactly(oracle_mod, n_workers):
    rng = np.random.default_rng(100 + n_workers)
    # dyadic gradients k * 2^-12 with |k| < 2^11: every partial sum of up to
    # 16 copies needs at most 15 significant bits, so fp32 sums them exactly
    k = rng.integers(-(1 << 11) + 1, 1 << 11, size=257)
    g = (k * 2.0 ** -12).astype(np.float32)
    grads = [g.copy() for _ in range(n_workers)]
    # lr = -1, mu = wd = 0, w = 0 leaves w' = m' = s
    w = np.zeros_like(g)
    m = np.zeros_like(g)
    oracle_mod.step_flat(grads, w, m, -1.0, 0.0, 0.0, False)
    expect = (k * n_workers * 2.0 ** -12).astype(np.float32)
    assert np.array_equal(_bits(m), _bits(expect))
    assert np.array_equal(_bits(w), _bits(expect))


@pytest.mark.parametrize("nesterov", [True, False])
def test_identical_gradients_equal_one_worker_with_scaled_gradient(oracle_mod, nesterov):
    rng = np.random.default_rng(7)
    n_workers = 8
    k = rng.integers(-(1 << 11) + 1, 1 << 11, size=300)
    g = (k * 2.0 ** -12).astype(np.float32)
    w0 = rng.standard_normal(300).astype(np.float32) * f32(0.05)
    m0 = rng.standard_normal(300).astype(np.float32) * f32(0.01)
    wa, ma = w0.copy(), m0.copy()
    oracle_mod.step_flat([g] * n_workers, wa, ma, 0.1, 0.9, 1e-4, nesterov)
    wb, mb = w0.copy(), m0.copy()
    oracle_mod.step_flat([(g * f32(n_workers)).astype(np.float32)], wb, mb, 0.1, 0.9, 1e-4, nesterov)
    assert np.array_equal(_bits(wa), _bits(wb))
    assert np.array_equal(_bits(ma), _bits(mb))


# --------------------------------------------------------------------------
# Zero gradient: weights decay only through weight decay and momentum,
# following a closed-form linear recurrence.
# --------------------------------------------------------------------------

def _zero_grad_matrix(lr, mu, wd, nesterov):
    """[w; m] after one step with zero gradient is A @ [w; m]:
    plain:    w' = (1 - lr*wd) w - lr*mu m,        m' = wd w + mu m
    nesterov: w' = (1 - lr*wd*(1+mu)) w - lr*mu^2 m, m' = wd w + mu m"""
    if nesterov:
        return np.array([[1 - lr * wd * (1 + mu), -lr * mu * mu], [wd, mu]], dtype=np.float64)
    return np.array([[1 - lr * wd, -lr * mu], [wd, mu]], dtype=np.float64)


@pytest.mark.parametrize("nesterov", [True, False])
def test_zero_gradient_closed_form(oracle_mod, nesterov):
    lr, mu, wd = float(f32(0.1)), float(f32(0.9)), float(f32(0.05))
    rng = np.random.default_rng(11)
    n, steps, n_workers = 97, 12, 3
    w0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    A = _zero_grad_matrix(lr, mu, wd, nesterov)

    # double-precision oracle against the matrix power, nearly exactly
    w64, m64 = w0.astype(np.float64), np.zeros(n)
    zeros64 = [np.zeros(n) for _ in range(n_workers)]
    # fp32 oracle against the same closed form within its rounding error
    w32, m32 = w0.copy(), np.zeros(n, dtype=np.float32)
    zeros32 = [np.zeros(n, dtype=np.float32) for _ in range(n_workers)]
    for t in range(1, steps + 1):
        oracle_mod.step_flat(zeros64, w64, m64, lr, mu, wd, nesterov, dtype=np.float64)
        oracle_mod.step_flat(zeros32, w32, m32, lr, mu, wd, nesterov)
        At = np.linalg.matrix_power(A, t)
        ew = At[0, 0] * w0.astype(np.float64)
        em = At[1, 0] * w0.astype(np.float64)
        scale_w = np.abs(w0).astype(np.float64)
        assert np.all(np.abs(w64 - ew) <= 1e-14 * scale_w + 1e-300)
        assert np.all(np.abs(m64 - em) <= 1e-14 * scale_w * wd * 20 + 1e-300)
        # each step rounds a handful of times at about 2^-24 relative
        assert np.all(np.abs(w32 - ew) <= 8 * t * 2.0 ** -24 * scale_w)
        assert np.all(np.abs(m32 - em) <= 8 * t * 2.0 ** -24 * scale_w * wd * 20)


def test_zero_gradient_single_step_by_hand(oracle_mod):
    # lr = 0.5, mu = 0.5, wd = 0.25, w = 1: m' = wd*w = 0.25;
    # Nesterov w' = 1 - 0.5*0.25*1.5 = 0.8125; plain w' = 1 - 0.5*0.25 = 0.875
    (wn, mn), = _one_elem_step(oracle_mod, [0.0, 0.0], 1.0, 0.0, 0.5, 0.5, 0.25, True)
    (wp, mp), = _one_elem_step(oracle_mod, [0.0, 0.0], 1.0, 0.0, 0.5, 0.5, 0.25, False)
    assert (wn[0], mn[0], wp[0], mp[0]) == (0.8125, 0.25, 0.875, 0.25)


# --------------------------------------------------------------------------
# Special cases.
# --------------------------------------------------------------------------

def _rand_case(seed, n_workers=4, n=513):
    rng = np.random.default_rng(seed)
    grads = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for _ in range(n_workers)]
    w = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-2).astype(np.float32)
    return grads, w, m


def test_zero_momentum_makes_nesterov_flag_irrelevant(oracle_mod):
    grads, w, m = _rand_case(1)
    wa, ma, wb, mb = w.copy(), m.copy(), w.copy(), m.copy()
    oracle_mod.step_flat(grads, wa, ma, 0.1, 0.0, 1e-4, True)
    oracle_mod.step_flat(grads, wb, mb, 0.1, 0.0, 1e-4, False)
    assert np.array_equal(_bits(wa), _bits(wb)) and np.array_equal(_bits(ma), _bits(mb))


@pytest.mark.parametrize("nesterov", [True, False])
def test_zero_lr_leaves_weights_and_updates_momentum(oracle_mod, nesterov):
    grads, w, m = _rand_case(2)
    wa, ma = w.copy(), m.copy()
    oracle_mod.step_flat(grads, wa, ma, 0.0, 0.9, 1e-4, nesterov)
    assert np.array_equal(_bits(wa), _bits(w))
    assert not np.array_equal(_bits(ma), _bits(m))


def test_plain_sgd_on_dyadic_values_is_exact(oracle_mod):
    # mu = wd = 0: w' = w - lr*s; with dyadic values of few bits all exact
    rng = np.random.default_rng(3)
    n_workers, n = 5, 200
    gk = rng.integers(-1000, 1000, size=(n_workers, n))
    wk = rng.integers(-1000, 1000, size=n)
    grads = [(gk[j] * 2.0 ** -10).astype(np.float32) for j in range(n_workers)]
    w = (wk * 2.0 ** -10).astype(np.float32)
    m = np.zeros(n, dtype=np.float32)
    oracle_mod.step_flat(grads, w, m, 0.25, 0.0, 0.0, False)
    s = gk.sum(axis=0) * 2.0 ** -10
    assert np.array_equal(m, s.astype(np.float32))
    assert np.array_equal(w, (wk * 2.0 ** -10 - 0.25 * s).astype(np.float32))


# --------------------------------------------------------------------------
# Keys and workers are addressed correctly: distinct codes per (worker, key).
# --------------------------------------------------------------------------

def test_key_and_worker_indexing(oracle_mod):
    n_workers, sizes = 3, [5, 1, 17, 8]
    grads = []
    for j in range(n_workers):
        row = []
        for k, n in enumerate(sizes):
            i = np.arange(n)
            # worker j contributes 2^(8j) * (k*64 + i + 1) * 2^-30: the sum
            # over workers is (1 + 2^8 + 2^16) * code, exact in fp32
            row.append(((k * 64 + i + 1) * 2.0 ** (8 * j - 30)).astype(np.float32))
        grads.append(row)
    weights = [np.zeros(n, dtype=np.float32) for n in sizes]
    moms = [np.zeros(n, dtype=np.float32) for n in sizes]
    oracle_mod.step(grads, weights, moms, -1.0, 0.0, 0.0, False)
    for k, n in enumerate(sizes):
        code = (k * 64 + np.arange(n) + 1).astype(np.float64)
        expect = (code * (1 + 2 ** 8 + 2 ** 16) * 2.0 ** -30).astype(np.float32)
        assert np.array_equal(moms[k], expect), k
        assert np.array_equal(weights[k], expect), k


# --------------------------------------------------------------------------
# Exact rational arithmetic with IEEE single-precision rounding points.
# --------------------------------------------------------------------------

def round_to_f32(x: Fraction) -> float:
    """Round an exact rational to the nearest fp32 value, ties to even,
    with gradual underflow (IEEE 754 binary32: 24-bit significand, minimum
    normal exponent -126, subnormal quantum 2^-149)."""
    if x == 0:
        return 0.0
    sign = -1.0 if x < 0 else 1.0
    a = -x if x < 0 else x
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    elif Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)
    q = Fraction(2) ** (e - 23)
    n = a / q
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    r = fl * q
    if r >= Fraction(2) ** 128:
        return sign * math.inf
    return sign * float(r)


def test_round_to_f32_matches_numpy_conversion():
    rng = np.random.default_rng(5)
    xs = np.concatenate([rng.standard_normal(2000),
                         rng.standard_normal(500) * 1e-40,   # subnormal range
                         rng.standard_normal(500) * 1e30,
                         [1 + 2.0 ** -24, 1 + 3 * 2.0 ** -24, -(1 + 2.0 ** -24), 2.0 ** -150, 3 * 2.0 ** -150]])
    for x in xs:
        assert round_to_f32(Fraction(float(x))) == float(np.float32(x)), x


def _exact_step(gs, w, m, lr, mu, wd, nesterov):
    F = lambda v: Fraction(float(v))
    s = F(gs[0])
    for g in gs[1:]:
        s = Fraction(round_to_f32(s + F(g)))
    d = Fraction(round_to_f32(F(wd) * F(w) + s))
    m1 = Fraction(round_to_f32(F(mu) * F(m) + d))
    u = Fraction(round_to_f32(F(mu) * m1 + d)) if nesterov else m1
    w1 = round_to_f32(-F(lr) * u + F(w))
    return w1, float(m1)


@pytest.mark.parametrize("n_workers", [1, 2, 3, 4, 5, 16])
@pytest.mark.parametrize("nesterov", [True, False])
def test_exact_rational_bruteforce(oracle_mod, n_workers, nesterov):
    rng = np.random.default_rng(1000 * n_workers + nesterov)
    n = 17
    lr, mu, wd = float(f32(0.1)), float(f32(0.9)), float(f32(1e-4))
    grads_steps = [[(rng.standard_normal(n) * 1e-2).astype(np.float32) for _ in range(n_workers)]
                   for _ in range(2)]
    w = (rng.standard_normal(n) * 0.05).astype(np.float32)
    m = np.zeros(n, dtype=np.float32)
    ew, em = [float(v) for v in w], [0.0] * n
    for grads in grads_steps:
        oracle_mod.step_flat(grads, w, m, lr, mu, wd, nesterov)
        for i in range(n):
            ew[i], em[i] = _exact_step([g[i] for g in grads], ew[i], em[i], lr, mu, wd, nesterov)
        assert np.array_equal(w, np.array(ew, dtype=np.float32))
        assert np.array_equal(m, np.array(em, dtype=np.float32))


# --------------------------------------------------------------------------
# Library optimizer: torch.optim.SGD (momentum, no dampening, coupled weight
# decay, Nesterov) on the aggregated gradient.
# --------------------------------------------------------------------------

def _torch_sgd_run(grads_steps, w0, lr, mu, wd, nesterov):
    torch = pytest.importorskip("torch")
    p = torch.nn.Parameter(torch.from_numpy(w0.astype(np.float64).copy()))
    opt = torch.optim.SGD([p], lr=lr, momentum=mu, dampening=0.0, weight_decay=wd,
                          nesterov=nesterov)
    out = []
    for grads in grads_steps:
        s = np.zeros(w0.size, dtype=np.float64)
        for g in grads:
            s = s + g.astype(np.float64)
        p.grad = torch.from_numpy(s)
        opt.step()
        buf = opt.state[p]["momentum_buffer"].detach().numpy().copy()
        out.append((p.detach().numpy().copy(), buf))
    return out


def _fp32_error_bound(grads_steps, w0, lr, mu, wd, nesterov):
    """First-order forward error bound of the fp32 step sequence, per
    element, with unit roundoff u = 2^-24: the left-fold sum of N terms errs
    by at most (N-1) u sum|g|; each fused multiply-add adds u times its
    result's magnitude and carries the operands' errors forward."""
    u = 2.0 ** -24
    n = w0.size
    w = w0.astype(np.float64)
    m = np.zeros(n)
    Ew, Em = np.zeros(n), np.zeros(n)
    for grads in grads_steps:
        g = np.array([x.astype(np.float64) for x in grads])
        s = g.sum(axis=0)
        Es = (len(grads) - 1) * u * np.abs(g).sum(axis=0)
        d = s + wd * w
        Ed = Es + wd * Ew + u * np.abs(d)
        m1 = mu * m + d
        Em1 = mu * Em + Ed + u * np.abs(m1)
        if nesterov:
            uu = d + mu * m1
            Eu = Ed + mu * Em1 + u * np.abs(uu)
        else:
            uu, Eu = m1, Em1
        w1 = w - lr * uu
        Ew = Ew + lr * Eu + u * np.abs(w1)
        w, m, Em = w1, m1, Em1
    return Ew, Em


@pytest.mark.parametrize("nesterov", [True, False])
def test_against_torch_sgd(oracle_mod, nesterov):
    rng = np.random.default_rng(21 + nesterov)
    n_workers, n, steps = 8, 4099, 10
    lr, mu, wd = float(f32(0.1)), float(f32(0.9)), float(f32(1e-4))
    grads_steps = [[(rng.standard_normal(n) * 1e-3).astype(np.float32) for _ in range(n_workers)]
                   for _ in range(steps)]
    w0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    ref = _torch_sgd_run(grads_steps, w0, lr, mu, wd, nesterov)

    w64, m64 = w0.astype(np.float64), np.zeros(n)
    w32, m32 = w0.copy(), np.zeros(n, dtype=np.float32)
    for t, grads in enumerate(grads_steps):
        oracle_mod.step_flat([g.astype(np.float64) for g in grads], w64, m64, lr, mu, wd, nesterov,
                             dtype=np.float64)
        oracle_mod.step_flat(grads, w32, m32, lr, mu, wd, nesterov)
        rw, rm = ref[t]
        # double-precision oracle agrees with torch to double rounding
        assert np.all(np.abs(w64 - rw) <= 1e-12 * (np.abs(rw) + 1e-3))
        assert np.all(np.abs(m64 - rm) <= 1e-12 * (np.abs(rm) + 1e-3))
    # fp32 oracle within its forward error bound of the library result
    Ew, Em = _fp32_error_bound(grads_steps, w0, lr, mu, wd, nesterov)
    rw, rm = ref[-1]
    assert np.all(np.abs(w32 - rw) <= 2 * Ew + 1e-15)
    assert np.all(np.abs(m32 - rm) <= 2 * Em + 1e-15)
    # and within the 1e-6 relative tolerance (floored at the key's rms)
    rms_w, rms_m = np.sqrt(np.mean(rw ** 2)), np.sqrt(np.mean(rm ** 2))
    assert np.max(np.abs(w32 - rw) / np.maximum(np.abs(rw), rms_w)) < 1e-6
    assert np.max(np.abs(m32 - rm) / np.maximum(np.abs(rm), rms_m)) < 1e-6


# --------------------------------------------------------------------------
# fp32 oracle within the forward error bound of the fp64 oracle, at the
# scale of the evaluation workloads (16 workers, 10 steps).
# --------------------------------------------------------------------------

@pytest.mark.parametrize("nesterov", [True, False])
def test_fp32_within_error_bound_of_fp64(oracle_mod, nesterov):
    rng = np.random.default_rng(31 + nesterov)
    n_workers, n, steps = 16, 2053, 10
    lr, mu, wd = float(f32(0.1)), float(f32(0.9)), float(f32(1e-4))
    grads_steps = [[(rng.standard_normal(n) * 1e-3).astype(np.float32) for _ in range(n_workers)]
                   for _ in range(steps)]
    w0 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    w64, m64 = w0.astype(np.float64), np.zeros(n)
    w32, m32 = w0.copy(), np.zeros(n, dtype=np.float32)
    for grads in grads_steps:
        oracle_mod.step_flat([g.astype(np.float64) for g in grads], w64, m64, lr, mu, wd, nesterov,
                             dtype=np.float64)
        oracle_mod.step_flat(grads, w32, m32, lr, mu, wd, nesterov)
    Ew, Em = _fp32_error_bound(grads_steps, w0, lr, mu, wd, nesterov)
    assert np.all(np.abs(w32 - w64) <= 2 * Ew + 1e-15)
    assert np.all(np.abs(m32 - m64) <= 2 * Em + 1e-15)


# --------------------------------------------------------------------------
# Argument checks.
# --------------------------------------------------------------------------

def test_oracle_rejects_mismatched_lengths(oracle_mod):
    with pytest.raises(ValueError):
        oracle_mod.step_flat([np.zeros(3, np.float32)], np.zeros(4, np.float32),
                             np.zeros(4, np.float32), 0.1, 0.9, 0.0, True)
    with pytest.raises(ValueError):
        oracle_mod.step([], [np.zeros(4, np.float32)], [np.zeros(4, np.float32)], 0.1, 0.9, 0.0, True)


def test_oracle_empty_key_is_a_no_op(oracle_mod):
    w = np.zeros(0, np.float32)
    oracle_mod.step_flat([np.zeros(0, np.float32)] * 2, w, np.zeros(0, np.float32), 0.1, 0.9, 0.0, True)
    assert w.size == 0
