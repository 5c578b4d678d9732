"""Pins for the CPU oracle, against things other than itself.

* every primitive's adjoint against a complex-step derivative of a separate
  forward-only evaluator (tests/cstep.py), with asymmetric shapes and distinct
  weights so a transposed operand, a wrong sign or a dropped term fails;
* closed forms (exponential-decay gradient; RK4 on a linear ODE is
  multiplication by the stability polynomial; logistic sensitivity at r = 0);
* invariants (exact zero gradient at the generating parameters of
  noise-free data);
* the Kalman filter likelihood against the dense Gaussian likelihood of the
  stacked observations (prediction-error decomposition), with a complex-step
  gradient through the dense formula;
* central finite differences on tiny random programs away from branch ties;
* edge cases: clamps, abs at 0, select ties and NaN predicates, empty loops,
  error handling, thread-count determinism.
"""
import math
import struct

import numpy as np
import pytest

import cstep
from conftest import lane_rel_err, rel_err
from workloads import bytecode as B
from workloads import configs, randtree
from workloads.bytecode import Asm


def run(oracle_mod, bc, params, obs=(), **kw):
    return oracle_mod.run(bc, np.atleast_2d(np.asarray(params, float)),
                          np.asarray(obs, float), **kw)


def check_vs_cstep(oracle_mod, bc, theta, obs=(), tol=1e-12):
    loss, g, _ = run(oracle_mod, bc, [theta], obs)
    want_loss = cstep.loss(bc, theta, list(obs))
    want = cstep.gradient(bc, theta, list(obs))
    assert rel_err(loss[0], want_loss) <= 1e-13, (loss[0], want_loss)
    err = lane_rel_err(g, [want])
    assert err.max() <= tol, (g[0], want, err)
    return g[0]


# ---------------------------------------------------------------- primitives
UNARY = [(B.NEG, 0.7), (B.EXP, 0.3), (B.LOG, 1.7), (B.SQRT, 2.3), (B.SIN, 0.4),
         (B.COS, 0.9), (B.ABS, -1.3), (B.ABS, 0.8)]


@pytest.mark.parametrize("op,x", UNARY)
def test_unary_scalar_adjoint(oracle_mod, op, x):
    A = Asm(2, 0)
    A.param(0).raw(op).param(1).mul().halt()
    check_vs_cstep(oracle_mod, A.bytes(), [x, -1.7])


BINARY = [B.ADD, B.SUB, B.MUL, B.DIV, B.POW]


@pytest.mark.parametrize("op", BINARY)
def test_binary_scalar_adjoint(oracle_mod, op):
    A = Asm(3, 0)
    A.param(0).param(1).raw(op).param(2).mul().halt()
    check_vs_cstep(oracle_mod, A.bytes(), [1.3, 0.6, -0.8])


def _mat(A, r, c, base):
    for i in range(r * c):
        A.param(base + i)
    A.pack(r, c)


def _weights(A, r, c, seed):
    rng = np.random.default_rng(seed)
    for v in rng.uniform(-1.5, 1.5, r * c):
        A.push(float(v))
    A.pack(r, c)


def _theta(n, seed, lo=-1.0, hi=1.0):
    return list(np.random.default_rng(seed).uniform(lo, hi, n))


@pytest.mark.parametrize("m,k,n", [(2, 3, 2), (4, 4, 4), (4, 4, 1), (2, 4, 4), (4, 2, 2),
                                   (1, 2, 2), (3, 1, 2)])
def test_matmul_adjoint(oracle_mod, m, k, n):
    A = Asm(m * k + n * k, 0)
    _mat(A, m, k, 0)
    _mat(A, k, n, m * k)
    A.matmul()
    _weights(A, m, n, 7)
    A.dot().halt()
    check_vs_cstep(oracle_mod, A.bytes(), _theta(m * k + n * k, 1))


def test_matmul_forward_value(oracle_mod):
    """(2x3)(3x2) product read back element by element against numpy."""
    X = np.arange(1.0, 7.0).reshape(2, 3) / 7.0
    Y = np.arange(2.0, 8.0).reshape(3, 2) / 5.0
    Z = X @ Y
    for i in range(2):
        for j in range(2):
            A = Asm(12, 0)
            _mat(A, 2, 3, 0)
            _mat(A, 3, 2, 6)
            A.matmul().index(i, j).halt()
            loss, _, _ = run(oracle_mod, A.bytes(), [list(X.ravel()) + list(Y.ravel())])
            assert abs(loss[0] - Z[i, j]) <= 1e-15 * abs(Z[i, j]) + 1e-300


@pytest.mark.parametrize("what", ["transpose", "trace", "outer", "dot", "index",
                                  "add", "sub", "hadamard", "ediv", "smul", "muls",
                                  "divs", "eexp", "esin", "elog"])
def test_matrix_misc_adjoint(oracle_mod, what):
    A = Asm(13, 0)
    if what == "transpose":
        _mat(A, 2, 3, 0); A.transpose(); _weights(A, 3, 2, 3); A.dot()
    elif what == "trace":
        _mat(A, 3, 3, 0); A.trace(); A.param(9).mul()
    elif what == "outer":
        _mat(A, 3, 1, 0); _mat(A, 2, 1, 3); A.outer(); _weights(A, 3, 2, 4); A.dot()
    elif what == "dot":
        _mat(A, 2, 3, 0); _mat(A, 2, 3, 6); A.dot()
    elif what == "index":
        _mat(A, 2, 3, 0); A.index(1, 2); A.param(0).mul()
    elif what in ("add", "sub", "hadamard", "ediv"):
        op = {"add": B.ADD, "sub": B.SUB, "hadamard": B.MUL, "ediv": B.DIV}[what]
        _mat(A, 2, 3, 0); _mat(A, 2, 3, 6); A.raw(op); _weights(A, 2, 3, 5); A.dot()
    elif what == "smul":
        A.param(12); _mat(A, 2, 3, 0); A.mul(); _weights(A, 2, 3, 6); A.dot()
    elif what == "muls":
        _mat(A, 2, 3, 0); A.param(12); A.mul(); _weights(A, 2, 3, 6); A.dot()
    elif what == "divs":
        _mat(A, 2, 3, 0); A.param(12); A.div(); _weights(A, 2, 3, 6); A.dot()
    elif what in ("eexp", "esin", "elog"):
        op = {"eexp": B.EXP, "esin": B.SIN, "elog": B.LOG}[what]
        _mat(A, 2, 3, 0); A.raw(op); _weights(A, 2, 3, 8); A.dot()
    A.halt()
    lo = 0.2 if what in ("elog", "ediv") else -1.0
    check_vs_cstep(oracle_mod, A.bytes(), _theta(13, 2, lo, 1.3))


@pytest.mark.parametrize("n", [1, 2])
@pytest.mark.parametrize("op", ["inv", "det", "logdet"])
def test_small_linalg_adjoint(oracle_mod, n, op):
    A = Asm(n * n + 1, 0)
    _mat(A, n, n, 0)
    getattr(A, op)()
    if op == "inv":
        _weights(A, n, n, 11)
        A.dot()
    else:
        A.param(n * n).mul()
    A.halt()
    theta = [1.4, 0.3, -0.2, 0.9, 0.7][: n * n] + [1.1]
    if n == 1:
        theta = [1.6, 1.1]
    check_vs_cstep(oracle_mod, A.bytes(), theta)


def test_inverse_value(oracle_mod):
    M = np.array([[1.4, 0.3], [-0.2, 0.9]])
    Mi = np.linalg.inv(M)
    for i in range(2):
        for j in range(2):
            A = Asm(4, 0)
            _mat(A, 2, 2, 0)
            A.inv().index(i, j).halt()
            loss, _, _ = run(oracle_mod, A.bytes(), [M.ravel()])
            assert abs(loss[0] - Mi[i, j]) <= 4e-16 * np.abs(Mi).max()


# ---------------------------------------------------------------- edge cases
def _log_prog(op):
    A = Asm(1, 0)
    A.param(0).raw(op).halt()
    return A.bytes()


@pytest.mark.parametrize("op", [B.LOG, B.SQRT])
def test_clamp(oracle_mod, op):
    bc = _log_prog(op)
    f = math.log if op == B.LOG else math.sqrt
    loss, g, _ = run(oracle_mod, bc, [[1e-9], [-1.0], [1e-8], [2e-8]])
    assert np.all(loss[:3] == f(1e-8))
    assert np.all(g[:3, 0] == 0.0)          # at or below the clamp: no gradient
    d = 1.0 / 2e-8 if op == B.LOG else 1.0 / (2.0 * math.sqrt(2e-8))
    assert rel_err(g[3, 0], d) <= 1e-15


def test_abs_at_zero(oracle_mod):
    A = Asm(1, 0)
    A.param(0).abs().halt()
    loss, g, _ = run(oracle_mod, A.bytes(), [[0.0], [-2.0], [3.0]])
    assert list(g[:, 0]) == [0.0, -1.0, 1.0]
    assert list(loss) == [0.0, 2.0, 3.0]


def _select_prog():
    """loss = theta0 < theta1 ? exp(1000*theta2) : 2*theta2"""
    A = Asm(3, 0)
    A.param(0).param(1).iflt()
    A.push(1000.0).param(2).mul().exp()
    A.else_()
    A.push(2.0).param(2).mul()
    A.endif().halt()
    return A.bytes()


def test_select_tie_nan_and_gating(oracle_mod):
    bc = _select_prog()
    P = [[1.0, 1.0, 5.0],            # tie -> else arm
         [float("nan"), 1.0, 5.0],   # unordered -> else arm
         [0.5, 1.0, 0.001],          # taken arm
         [2.0, 1.0, 5.0]]            # else arm; then-arm would overflow
    loss, g, m = run(oracle_mod, bc, P, margin=True)
    assert loss[0] == 10.0 and loss[1] == 10.0 and loss[3] == 10.0
    assert rel_err(loss[2], math.exp(1.0)) <= 1e-15
    assert list(g[0]) == [0.0, 0.0, 2.0] and list(g[1]) == [0.0, 0.0, 2.0]
    assert rel_err(g[2, 2], 1000.0 * math.exp(1.0)) <= 1e-14
    assert g[2, 0] == 0.0 and g[2, 1] == 0.0       # predicate carries no gradient
    assert m[0] == 0.0 and m[2] == pytest.approx(0.5)


def test_param_and_const_loss(oracle_mod):
    A = Asm(2, 0)
    A.param(1).halt()
    loss, g, _ = run(oracle_mod, A.bytes(), [[3.0, 4.0]])
    assert loss[0] == 4.0 and list(g[0]) == [0.0, 1.0]
    A = Asm(2, 0)
    A.push(2.5).halt()
    loss, g, _ = run(oracle_mod, A.bytes(), [[3.0, 4.0]])
    assert loss[0] == 2.5 and list(g[0]) == [0.0, 0.0]


def test_empty_loop_nested_strides_and_shuffles(oracle_mod):
    A = Asm(2, 12)
    A.push(0.0).storel(0)
    A.loop(0).param(0).storel(0).endloop()        # never runs
    A.loop(3).loop(4)
    A.loadl(0).obs(0, 1, 4).param(1).mul().add().storel(0)   # obs[k_in + 4 k_out]
    A.endloop().endloop()
    A.loadl(0).param(0).swap().over().drop().mul().halt()    # theta0 * acc
    obs = np.arange(12.0) + 1.0
    loss, g, _ = run(oracle_mod, A.bytes(), [[2.0, 0.5]], obs)
    s = obs.sum()
    assert loss[0] == 2.0 * 0.5 * s
    assert list(g[0]) == [0.5 * s, 2.0 * s]


@pytest.mark.parametrize("prog,code", [
    (b"XXXX" + bytes(20), 2),
    (Asm(1, 0).param(0).loop(2).halt().bytes(), 2),          # unterminated LOOP
    (Asm(1, 0).param(0).else_().halt().bytes(), 2),          # ELSE without IFLT
    (Asm(1, 0).add().halt().bytes(), 3),                     # stack underflow
    (Asm(1, 1).obs(5).halt().bytes(), 3),                    # obs index out of range
    (Asm(1, 0).param(0).param(0).halt().bytes(), 3),         # two values at HALT
    (Asm(1, 0).param(3).halt().bytes(), 3),                  # bad param index
    (Asm(1, 0).param(0).param(0).pack(1, 2).param(0).add().halt().bytes(), 3),  # shapes
])
def test_errors(oracle_mod, prog, code):
    with pytest.raises(oracle_mod.OracleError) as e:
        run(oracle_mod, prog, [[1.0]], [0.0] if b"NDVB" == prog[:4] and
            struct.unpack_from("<I", prog, 12)[0] == 1 else [])
    assert e.value.code == code


def test_thread_count_determinism(oracle_mod):
    w = configs.lotka_volterra(L=37, T=40)
    a = oracle_mod.run(w.bytecode, w.params, w.obs, threads=1)
    b = oracle_mod.run(w.bytecode, w.params, w.obs, threads=7)
    assert a[0].tobytes() == b[0].tobytes() and a[1].tobytes() == b[1].tobytes()


# ---------------------------------------------------------------- config 1
def test_exp_decay_closed_form(oracle_mod):
    w = configs.exp_decay(L=16)
    n = 64
    t, y = w.obs[:n], w.obs[n:]
    loss, g, _ = oracle_mod.run(w.bytecode, w.params, w.obs)
    for l, (a, b, c) in enumerate(w.params):
        e = [math.exp(-b * ti) for ti in t]
        r = [a * ei + c - yi for ei, yi in zip(e, y)]
        want_loss = sum(ri * ri for ri in r) / n
        want = [2.0 / n * sum(ri * ei for ri, ei in zip(r, e)),
                -2.0 / n * sum(ri * a * ti * ei for ri, ti, ei in zip(r, t, e)),
                2.0 / n * sum(r)]
        assert rel_err(loss[l], want_loss) <= 1e-13
        assert lane_rel_err(g[l], want).max() <= 1e-12


def test_exp_decay_zero_gradient_at_truth(oracle_mod):
    n = 64
    t = np.linspace(0.0, 5.0, n)
    a, b, c = 2.0, 0.7, 0.3
    y = [a * math.exp(-(b * ti)) + c for ti in t]     # same operation order as the program
    loss, g, _ = run(oracle_mod, configs.exp_decay_program(n), [[a, b, c]], list(t) + y)
    assert loss[0] == 0.0
    assert np.all(g == 0.0)


def test_exp_decay_cstep(oracle_mod):
    w = configs.exp_decay(L=3, n=8)
    for l in range(3):
        check_vs_cstep(oracle_mod, w.bytecode, list(w.params[l]), list(w.obs), tol=1e-12)


# ---------------------------------------------------------------- config 2
def test_logistic_invariant_at_truth(oracle_mod):
    T = 60
    truth = [2.0, 10.0, 0.5, 0.2]
    y = configs.logistic_truth_path(truth, T)
    loss, g, _ = run(oracle_mod, configs.logistic_program(T), [truth], y)
    assert g[0, 0] == 0.0 and g[0, 1] == 0.0 and g[0, 2] == 0.0
    assert rel_err(g[0, 3], T / truth[3]) <= 1e-13
    want = T * (math.log(truth[3]) + configs.HALF_LN_2PI)
    assert rel_err(loss[0], want) <= 1e-13


def test_logistic_sensitivity_at_zero_rate(oracle_mod):
    """r = 0 freezes x_k = x0 and d x_k / d r = k dt x0 (1 - x0/K)."""
    T, dt = 50, 0.01
    K, x0, sig = 7.0, 1.3, 0.4
    y = np.random.default_rng(3).uniform(0.5, 2.0, T)
    loss, g, _ = run(oracle_mod, configs.logistic_program(T), [[0.0, K, x0, sig]], y)
    s = [(k + 1) * dt * x0 * (1.0 - x0 / K) for k in range(T)]
    want_r = sum((x0 - yk) / sig ** 2 * sk for yk, sk in zip(y, s))
    want_x0 = sum((x0 - yk) / sig ** 2 for yk in y)
    want_sig = sum(-(x0 - yk) ** 2 / sig ** 3 + 1.0 / sig for yk in y)
    assert lane_rel_err(g[0, [0, 2, 3]], [want_r, want_x0, want_sig]).max() <= 1e-12
    assert g[0, 1] == 0.0                       # K enters only multiplied by r = 0


def test_logistic_cstep(oracle_mod):
    w = configs.logistic(L=2, T=30)
    for l in range(2):
        check_vs_cstep(oracle_mod, w.bytecode, list(w.params[l]), list(w.obs), tol=1e-11)


# ---------------------------------------------------------------- config 3
def _rk4_R(z):
    return 1 + z + z * z / 2 + z ** 3 / 6 + z ** 4 / 24


def _rk4_dR(z):
    return 1 + z + z * z / 2 + z ** 3 / 6


def test_lotka_volterra_decoupled_closed_form(oracle_mod):
    """beta = delta = 0: RK4 on x' = a x is x_n = x0 R(a h)^n."""
    T, h = 30, 0.02
    al, ga, x0, y0 = 0.9, 1.2, 1.1, 0.7
    obs = np.random.default_rng(5).uniform(0.5, 2.0, 2 * T)
    loss, g, _ = run(oracle_mod, configs.lotka_volterra_program(T), [[al, 0.0, ga, 0.0, x0, y0]], obs)
    zx, zy = al * h, -ga * h
    xs = [x0 * _rk4_R(zx) ** (k + 1) for k in range(T)]
    ys = [y0 * _rk4_R(zy) ** (k + 1) for k in range(T)]
    rx = [xk - obs[2 * k] for k, xk in enumerate(xs)]
    ry = [yk - obs[2 * k + 1] for k, yk in enumerate(ys)]
    want_loss = (sum(r * r for r in rx) + sum(r * r for r in ry)) / (2 * T)
    d_al = sum(rx[k] * x0 * (k + 1) * _rk4_R(zx) ** k * _rk4_dR(zx) * h for k in range(T)) / T
    d_x0 = sum(rx[k] * _rk4_R(zx) ** (k + 1) for k in range(T)) / T
    d_ga = sum(ry[k] * y0 * (k + 1) * _rk4_R(zy) ** k * _rk4_dR(zy) * (-h) for k in range(T)) / T
    d_y0 = sum(ry[k] * _rk4_R(zy) ** (k + 1) for k in range(T)) / T
    assert rel_err(loss[0], want_loss) <= 1e-12
    assert lane_rel_err(g[0, [0, 2, 4, 5]], [d_al, d_ga, d_x0, d_y0]).max() <= 1e-11


def test_lotka_volterra_invariant_at_truth(oracle_mod):
    T = 80
    truth = [1.0, 0.5, 1.0, 0.5, 1.0, 0.5]
    path = configs.lv_truth_path(truth, T)
    loss, g, _ = run(oracle_mod, configs.lotka_volterra_program(T), [truth], path.reshape(-1))
    assert loss[0] == 0.0
    assert np.all(g == 0.0)


def test_lotka_volterra_cstep(oracle_mod):
    w = configs.lotka_volterra(L=2, T=12)
    for l in range(2):
        check_vs_cstep(oracle_mod, w.bytecode, list(w.params[l]), list(w.obs), tol=1e-11)


# ---------------------------------------------------------------- config 4
def _lu_logdet_quad(S, r):
    """ln det S and r^T S^-1 r by Gaussian elimination without pivoting;
    analytic in the entries, so it carries a complex step."""
    n = len(S)
    A = [list(row) for row in S]
    b = list(r)
    for k in range(n):
        for i in range(k + 1, n):
            f = A[i][k] / A[k][k]
            for j in range(k, n):
                A[i][j] = A[i][j] - f * A[k][j]
            b[i] = b[i] - f * b[k]
    logdet = sum(np.log(A[k][k]) for k in range(n))
    x = [0] * n
    for i in reversed(range(n)):
        x[i] = (b[i] - sum(A[i][j] * x[j] for j in range(i + 1, n))) / A[i][i]
    quad = sum(r[i] * x[i] for i in range(n))
    return logdet, quad


def _dense_kalman_nll(theta, ys):
    """-ln N(y_1..T; m, Sigma) of the stacked observations of the model
    x_0 ~ N(x0, P0), x_k = F x_{k-1} + w_k, y_k = H x_k + v_k."""
    T = len(ys)
    dtype = complex if any(isinstance(v, complex) for v in theta) else float
    th = np.array(theta, dtype=dtype)
    dt = th[0]
    F = np.array([[1, 0, dt, 0], [0, 1, 0, dt], [0, 0, 1, 0], [0, 0, 0, 1]], dtype=dtype)
    Q = np.diag(th[1:5])
    H = np.array([[1, 0, 0, 0], [0, 1, 0, 0]], dtype=dtype)
    R = np.diag(th[5:7])
    x0 = th[7:11]
    P0 = th[11] * np.eye(4, dtype=dtype)
    Fp = [np.eye(4, dtype=dtype)]
    for _ in range(T):
        Fp.append(F @ Fp[-1])
    n = 2 * T
    S = np.zeros((n, n), dtype=dtype)
    m = np.zeros(n, dtype=dtype)
    for k in range(1, T + 1):
        m[2 * k - 2:2 * k] = H @ Fp[k] @ x0
        for l in range(1, T + 1):
            C = Fp[k] @ P0 @ Fp[l].T
            for j in range(1, min(k, l) + 1):
                C = C + Fp[k - j] @ Q @ Fp[l - j].T
            blk = H @ C @ H.T
            if k == l:
                blk = blk + R
            S[2 * k - 2:2 * k, 2 * l - 2:2 * l] = blk
    r = np.asarray(ys, dtype=dtype).reshape(-1) - m
    logdet, quad = _lu_logdet_quad(S.tolist(), list(r))
    return 0.5 * (logdet + quad + n * math.log(2 * math.pi))


@pytest.mark.parametrize("T", [1, 2, 4])
def test_kalman_prediction_error_decomposition(oracle_mod, T):
    w = configs.kalman(L=3, T=T)
    ys = w.obs.reshape(T, 2)
    loss, g, _ = oracle_mod.run(w.bytecode, w.params, w.obs)
    h = 1e-30
    for l in range(3):
        th = list(w.params[l])
        want = _dense_kalman_nll(th, ys)
        assert rel_err(loss[l], float(np.real(want))) <= 1e-11
        grad = []
        for p in range(12):
            tc = [complex(v) for v in th]
            tc[p] = complex(th[p], h)
            grad.append(np.imag(_dense_kalman_nll(tc, ys)) / h)
        assert lane_rel_err(g[l], grad).max() <= 1e-8


def test_kalman_cstep(oracle_mod):
    w = configs.kalman(L=2, T=6)
    for l in range(2):
        check_vs_cstep(oracle_mod, w.bytecode, list(w.params[l]), list(w.obs), tol=1e-11)


# ---------------------------------------------------------------- config 5
def _tiny_trees(k=6):
    w = configs.random_programs(n_prog=k, L=2, n=3, seed=77)
    return w


def test_random_trees_cstep_and_fd(oracle_mod):
    w = _tiny_trees()
    for i, bc in enumerate(w.programs):
        P = w.n_params_each[i]
        params = w.params[i][:, :P]
        loss, g, m = oracle_mod.run(bc, params, w.obs, margin=True)
        for l in range(2):
            if m[l] < 1e-6:
                continue                      # too close to a branch flip to pin
            want = cstep.gradient(bc, list(params[l]), list(w.obs))
            assert lane_rel_err(g[l], want).max() <= 1e-10, (i, l)
            fd = []
            for p in range(P):
                hp = 1e-6 * max(1.0, abs(params[l, p]))
                th = np.array([params[l]] * 2)
                th[0, p] += hp
                th[1, p] -= hp
                lp, _, mp = oracle_mod.run(bc, th, w.obs, grad=False, margin=True)
                fd.append((lp[0] - lp[1]) / (2 * hp))
            assert lane_rel_err(g[l], fd).max() <= 1e-5, (i, l, g[l], fd)


def test_random_tree_zero_gradient_at_hidden_constants(oracle_mod):
    w = configs.random_programs(n_prog=1, L=1, n=16, seed=5005)
    tree, c = w.meta["hidden_tree"]
    xs = w.obs[:16]
    ys = [randtree.evaluate(tree, c, float(x)) for x in xs]
    bc = configs.tree_program(tree, len(c), 16)
    loss, g, _ = run(oracle_mod, bc, [c], list(xs) + ys)
    assert loss[0] == 0.0
    assert np.all(g == 0.0)
