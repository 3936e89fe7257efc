"""Pins of the oracle's pluggable optimizers (paper section 3.2.2: the
aggregators and optimizers are extensible): plain SGD and Adam.

Each pin checks the oracle against something other than its own formula:
hand-derived dyadic examples (tests/golden), closed forms of the
algorithm on special inputs, an exact scaling symmetry, a special case that
reduces to the momentum oracle, and torch's own optimizers within a
rounding tolerance.
"""

import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module")
def oracle_lib():
    return oracle.OracleLib(oracle.build(force=False))


def _bits(a):
    return np.asarray(a, np.float32).view(np.uint32)


def _read(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def _fold(grads):
    """Left fold in fp32, worker 0 first (numpy float32 additions are
    correctly rounded)."""
    s = grads[0].astype(np.float32).copy()
    for g in grads[1:]:
        s = (s + g).astype(np.float32)
    return s


# ---------------------------------------------------------------- plain SGD

def test_sgd_worked_example(oracle_lib):
    rows = _read("worked_example_sgd.txt")
    g0, g1, w0, lr, wd = (float(x) for x in rows[0][1:])
    w = [np.array([w0], np.float32)]
    for step, expect in rows[1:]:
        oracle_lib.step_sgd([[np.array([g0], np.float32)], [np.array([g1], np.float32)]], w, lr, wd)
        assert w[0][0] == np.float32(float(expect)), f"step {step}"


@pytest.mark.parametrize("nesterov", [True, False])
def test_sgd_equals_momentum_with_zero_momentum(oracle_lib, nesterov):
    """With mu = 0 the momentum form's W update is d itself, so its weights
    must equal the stateless SGD's bit for bit."""
    rng = np.random.default_rng(7)
    n, sizes = 5, (1, 7, 300)
    w_a = [rng.standard_normal(k).astype(np.float32) for k in sizes]
    w_b = [x.copy() for x in w_a]
    moms = [np.zeros(k, np.float32) for k in sizes]
    for _ in range(4):
        grads = [[(rng.standard_normal(k) * 1e-2).astype(np.float32) for k in sizes] for _ in range(n)]
        oracle_lib.step_sgd(grads, w_a, 0.1, 1e-4)
        oracle_lib.step(grads, w_b, moms, 0.1, 0.0, 1e-4, nesterov)
    for a, b in zip(w_a, w_b):
        assert np.array_equal(_bits(a), _bits(b))


def test_sgd_zero_gradient_closed_form(oracle_lib):
    """g = 0: w_t = w0 (1 - lr wd)^t."""
    rng = np.random.default_rng(8)
    w0 = rng.standard_normal(64).astype(np.float32)
    w = [w0.copy()]
    lr, wd = np.float32(0.1), np.float32(0.01)
    for t in range(1, 31):
        oracle_lib.step_sgd([[np.zeros(64, np.float32)]], w, lr, wd)
        exact = w0.astype(np.float64) * (1.0 - float(lr) * float(wd)) ** t
        assert np.all(np.abs(w[0] - exact) <= t * 2.0 ** -23 * np.abs(exact) + 1e-30)


def test_sgd_identical_gradients_equal_one_worker_with_the_sum(oracle_lib):
    """N copies of a dyadic gradient with few significant bits sum exactly,
    so the step equals a one-worker step on N * g."""
    rng = np.random.default_rng(9)
    g = (rng.integers(-2 ** 10, 2 ** 10, 100) * 2.0 ** -12).astype(np.float32)
    w0 = rng.standard_normal(100).astype(np.float32)
    for n in (2, 3, 8, 16):
        a, b = [w0.copy()], [w0.copy()]
        oracle_lib.step_sgd([[g] for _ in range(n)], a, 0.1, 1e-4)
        oracle_lib.step_sgd([[(g * n).astype(np.float32)]], b, 0.1, 1e-4)
        assert np.array_equal(_bits(a[0]), _bits(b[0])), n


def test_sgd_against_torch(oracle_lib):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(10)
    w0 = rng.standard_normal(257).astype(np.float32)
    w = [w0.copy()]
    p = torch.nn.Parameter(torch.from_numpy(w0.copy()))
    opt = torch.optim.SGD([p], lr=0.1, momentum=0.0, weight_decay=1e-4)
    for _ in range(5):
        grads = [(rng.standard_normal(257) * 1e-2).astype(np.float32) for _ in range(4)]
        oracle_lib.step_sgd([[g] for g in grads], w, 0.1, 1e-4)
        p.grad = torch.from_numpy(_fold(grads))
        opt.step()
    ref = p.detach().numpy()
    assert np.max(np.abs(w[0] - ref) / np.maximum(np.abs(ref), 1e-3)) < 1e-6


# --------------------------------------------------------------------- Adam

def _adam(oracle_lib, grads_per_key, w, m, v, lr, b1, b2, eps, wd, t):
    oracle_lib.step_adam(grads_per_key, w, m, v, lr, b1, b2, eps, wd, t)


@pytest.mark.parametrize("case", ["A", "B"])
def test_adam_worked_example(oracle_lib, case):
    rows = _read("worked_example_adam.txt")
    g0, g1, w0, lr, b1, b2 = (float(x) for x in rows[0][1:])
    row = next(r for r in rows[1:] if r[0] == case)
    wd, eps, ew, em, ev = (float(x) for x in row[1:])
    w, m, v = [np.array([w0], np.float32)], [np.zeros(1, np.float32)], [np.zeros(1, np.float32)]
    _adam(oracle_lib, [[np.array([g0], np.float32)], [np.array([g1], np.float32)]], w, m, v,
          lr, b1, b2, eps, wd, 1)
    assert (w[0][0], m[0][0], v[0][0]) == (np.float32(ew), np.float32(em), np.float32(ev))


def _adam_update_bound(q, w):
    # a dozen roundings of relative size 2^-24 on the update, one on w
    return 2.0 ** -20 * np.abs(q) + 2.0 ** -23 * np.abs(w) + 1e-30


@pytest.mark.parametrize("eps", [1e-8, 1e-3])
def test_adam_first_step_closed_form(oracle_lib, eps):
    """Step 1 from zero moments, wd = 0: the bias-corrected moments are g and
    g^2, so the update is lr * g / (|g| + eps)."""
    rng = np.random.default_rng(11)
    g = (rng.standard_normal(500) * 1e-3).astype(np.float32)
    w0 = rng.standard_normal(500).astype(np.float32)
    lr, b1, b2 = 1e-3, 0.9, 0.999
    w, m, v = [w0.copy()], [np.zeros(500, np.float32)], [np.zeros(500, np.float32)]
    _adam(oracle_lib, [[g]], w, m, v, lr, b1, b2, eps, 0.0, 1)
    gd = g.astype(np.float64)
    q = float(np.float32(lr)) * gd / (np.abs(gd) + float(np.float32(eps)))
    exact = w0.astype(np.float64) - q
    assert np.all(np.abs(w[0] - exact) <= _adam_update_bound(q, exact))


def test_adam_constant_gradient_closed_form(oracle_lib):
    """A constant gradient keeps the bias-corrected moments at g and g^2 at
    every step, so after t steps w = w0 - t * lr * g / (|g| + eps)."""
    rng = np.random.default_rng(12)
    g = (rng.standard_normal(300) * 1e-2).astype(np.float32)
    w0 = rng.standard_normal(300).astype(np.float32)
    lr, b1, b2, eps = 1e-3, 0.9, 0.999, 1e-6
    w, m, v = [w0.copy()], [np.zeros(300, np.float32)], [np.zeros(300, np.float32)]
    gd = g.astype(np.float64)
    q = float(np.float32(lr)) * gd / (np.abs(gd) + float(np.float32(eps)))
    for t in range(1, 21):
        _adam(oracle_lib, [[g]], w, m, v, lr, b1, b2, eps, 0.0, t)
        exact = w0.astype(np.float64) - t * q
        # per step: the update's rounding, and one rounding of w
        assert np.all(np.abs(w[0] - exact) <= t * (2.0 ** -19 * np.abs(q) + 2.0 ** -23 * (np.abs(w0) + 1))), t


@pytest.mark.parametrize("scale_exp", [6, -5])
def test_adam_is_exactly_invariant_to_power_of_two_gradient_scale(oracle_lib, scale_exp):
    """With eps = 0 and wd = 0, scaling every gradient by 2^k scales m by 2^k
    and v by 4^k exactly and leaves w bit for bit unchanged (the square root
    of the second moment cancels the scale)."""
    rng = np.random.default_rng(13)
    c = np.float32(2.0 ** scale_exp)
    sizes = (9, 200)
    w0 = [rng.standard_normal(k).astype(np.float32) for k in sizes]
    wa, wb = [x.copy() for x in w0], [x.copy() for x in w0]
    ma, va = [np.zeros(k, np.float32) for k in sizes], [np.zeros(k, np.float32) for k in sizes]
    mb, vb = [np.zeros(k, np.float32) for k in sizes], [np.zeros(k, np.float32) for k in sizes]
    for t in range(1, 5):
        grads = [[(rng.standard_normal(k) * 1e-3).astype(np.float32) for k in sizes] for _ in range(3)]
        scaled = [[(x * c).astype(np.float32) for x in wg] for wg in grads]
        _adam(oracle_lib, grads, wa, ma, va, 1e-3, 0.9, 0.999, 0.0, 0.0, t)
        _adam(oracle_lib, scaled, wb, mb, vb, 1e-3, 0.9, 0.999, 0.0, 0.0, t)
        for k in range(len(sizes)):
            assert np.array_equal(_bits(wa[k]), _bits(wb[k])), (t, k)
            assert np.array_equal(_bits((ma[k] * c).astype(np.float32)), _bits(mb[k])), (t, k)
            assert np.array_equal(_bits((va[k] * c * c).astype(np.float32)), _bits(vb[k])), (t, k)


def test_adam_zero_lr_updates_moments_only(oracle_lib):
    rng = np.random.default_rng(14)
    w0 = rng.standard_normal(50).astype(np.float32)
    grads = [[(rng.standard_normal(50) * 1e-2).astype(np.float32)] for _ in range(2)]
    w, m, v = [w0.copy()], [np.zeros(50, np.float32)], [np.zeros(50, np.float32)]
    _adam(oracle_lib, grads, w, m, v, 0.0, 0.9, 0.999, 1e-8, 1e-2, 1)
    assert np.array_equal(_bits(w[0]), _bits(w0))
    assert np.all(m[0] != 0) and np.all(v[0] > 0)


def test_adam_with_zero_beta1_keeps_the_gradient_as_first_moment(oracle_lib):
    """b1 = 0: c1 = 1 and m' = d exactly; with wd = 0, d is the fp32 sum."""
    rng = np.random.default_rng(15)
    grads = [(rng.standard_normal(40) * 1e-2).astype(np.float32) for _ in range(5)]
    w, m, v = [rng.standard_normal(40).astype(np.float32)], [np.ones(40, np.float32)], [np.zeros(40, np.float32)]
    _adam(oracle_lib, [[g] for g in grads], w, m, v, 1e-3, 0.0, 0.999, 1e-8, 0.0, 3)
    assert np.array_equal(_bits(m[0]), _bits(_fold(grads)))


def test_adam_against_torch(oracle_lib):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(16)
    w0 = rng.standard_normal(333).astype(np.float32)
    w, m, v = [w0.copy()], [np.zeros(333, np.float32)], [np.zeros(333, np.float32)]
    p = torch.nn.Parameter(torch.from_numpy(w0.copy()))
    lr, b1, b2, eps, wd = 1e-3, 0.9, 0.999, 1e-8, 1e-2
    f32 = lambda x: float(np.float32(x))   # the hyperparameters are fp32 values on both sides
    opt = torch.optim.Adam([p], lr=f32(lr), betas=(f32(b1), f32(b2)), eps=f32(eps),
                           weight_decay=f32(wd))
    for t in range(1, 8):
        grads = [(rng.standard_normal(333) * 1e-2).astype(np.float32) for _ in range(4)]
        _adam(oracle_lib, [[g] for g in grads], w, m, v, lr, b1, b2, eps, wd, t)
        p.grad = torch.from_numpy(_fold(grads))
        opt.step()
    st = opt.state[p]

    def rel(x, ref):   # relative error with the rms of the reference as floor
        ref = ref.astype(np.float64)
        return np.max(np.abs(x - ref) / np.maximum(np.abs(ref), np.sqrt(np.mean(ref ** 2))))

    assert rel(w[0], p.detach().numpy()) < 1e-6
    assert rel(m[0], st["exp_avg"].numpy()) < 1e-5
    assert rel(v[0], st["exp_avg_sq"].numpy()) < 1e-5


def test_adam_rejects_bad_arguments(oracle_lib):
    g = [[np.zeros(3, np.float32)]]
    for kw in (dict(t=0), dict(b1=1.0), dict(b2=-0.1)):
        a = dict(t=1, b1=0.9, b2=0.999)
        a.update(kw)
        w, m, v = [np.zeros(3, np.float32)], [np.zeros(3, np.float32)], [np.zeros(3, np.float32)]
        with pytest.raises(ValueError):
            _adam(oracle_lib, g, w, m, v, 1e-3, a["b1"], a["b2"], 1e-8, 0.0, a["t"])


# ------------------------------------------------------- planted mistakes
# Each mistake is planted in a copy of the oracle's C source (CPU only) and
# must make at least one pin above fail.

SGD_START = "int oracle_step_sgd_f32("
ADAM_START = "static void adam_scalars("

OPT_MUTANTS = [
    ("sgd_update_sign", "sgd", "w[i] = fmaf(-lr, d, w[i]);", "w[i] = fmaf(lr, d, w[i]);"),
    ("sgd_weight_decay_dropped", "sgd", "float d = fmaf(wd, w[i], s);", "float d = s;"),
    ("sgd_sum_is_mean", "sgd", "float d = fmaf(wd, w[i], s);",
     "float d = fmaf(wd, w[i], s / (float)num_workers);"),
    ("sgd_update_unfused", "sgd", "w[i] = fmaf(-lr, d, w[i]);", "{ float t = lr * d; w[i] = w[i] - t; }"),
    ("adam_no_bias_correction_1", "adam",
     "*k1 = (float)((double)lr / (1.0 - pow((double)b1, (double)step)));", "*k1 = lr;"),
    ("adam_no_bias_correction_2", "adam",
     "*k2 = (float)(1.0 / (1.0 - pow((double)b2, (double)step)));", "*k2 = 1.0f;"),
    ("adam_second_moment_not_squared", "adam", "float dd = d * d;", "float dd = fabsf(d);"),
    ("adam_no_sqrt", "adam", "float den = sqrtf(vn * k2) + eps;", "float den = vn * k2 + eps;"),
    ("adam_eps_inside_sqrt", "adam", "float den = sqrtf(vn * k2) + eps;", "float den = sqrtf(vn * k2 + eps);"),
    ("adam_first_moment_undamped", "adam", "float mn = fmaf(b1, m[i], c1 * d);", "float mn = fmaf(b1, m[i], d);"),
    ("adam_betas_swapped", "adam", "float vn = fmaf(b2, v[i], c2 * dd);", "float vn = fmaf(b1, v[i], c1 * dd);"),
    ("adam_update_sign", "adam", "w[i] = w[i] - q;", "w[i] = w[i] + q;"),
    ("adam_weight_decay_decoupled", "adam", "float d = fmaf(wd, w[i], s);", "float d = s;"),
    ("adam_step_off_by_one", "adam", "adam_scalars(lr, b1, b2, step, &c1, &c2, &k1, &k2);",
     "adam_scalars(lr, b1, b2, step + 1, &c1, &c2, &k1, &k2);"),
    ("adam_moment_not_stored", "adam", "m[i] = mn;", "m[i] = d;"),
]


def _plant_opt(src, which, old, new):
    start = src.index(SGD_START if which == "sgd" else ADAM_START)
    end = src.index(ADAM_START) if which == "sgd" else len(src)
    body = src[start:end]
    assert body.count(old) == 1, f"mutation anchor not unique: {old!r}"
    return src[:start] + body.replace(old, new) + src[end:]


def _opt_pin_calls():
    calls = [("sgd_worked", test_sgd_worked_example),
             ("sgd_zero_grad", test_sgd_zero_gradient_closed_form),
             ("sgd_identical", test_sgd_identical_gradients_equal_one_worker_with_the_sum),
             ("adam_zero_lr", test_adam_zero_lr_updates_moments_only),
             ("adam_beta1_zero", test_adam_with_zero_beta1_keeps_the_gradient_as_first_moment),
             ("adam_constant", test_adam_constant_gradient_closed_form)]
    for nest in (True, False):
        calls.append((f"sgd_mu0[{nest}]", lambda o, nest=nest: test_sgd_equals_momentum_with_zero_momentum(o, nest)))
    for case in ("A", "B"):
        calls.append((f"adam_worked[{case}]", lambda o, case=case: test_adam_worked_example(o, case)))
    for eps in (1e-8, 1e-3):
        calls.append((f"adam_first[{eps}]", lambda o, eps=eps: test_adam_first_step_closed_form(o, eps)))
    for k in (6, -5):
        calls.append((f"adam_scale[{k}]", lambda o, k=k: test_adam_is_exactly_invariant_to_power_of_two_gradient_scale(o, k)))
    return calls


@pytest.mark.parametrize("mutant", OPT_MUTANTS, ids=[m[0] for m in OPT_MUTANTS])
def test_planted_optimizer_mistake_is_caught(tmp_path, mutant):
    name, which, old, new = mutant
    with open(oracle.SRC) as f:
        src = f.read()
    cpath = tmp_path / f"{name}.c"
    cpath.write_text(_plant_opt(src, which, old, new))
    o = oracle.OracleLib(oracle.build(force=True, src=str(cpath), out=str(tmp_path / f"lib{name}.so")))
    caught = []
    for pin_name, call in _opt_pin_calls():
        try:
            call(o)
        except AssertionError:
            caught.append(pin_name)
    assert caught, f"no pin caught the planted mistake {name}"
