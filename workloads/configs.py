"""The five synthetic workloads: bytecode programs, observations and lane
parameter populations, all seeded.

Each builder returns a :class:`Workload`.  Sizes default to the full
benchmark shapes and can be shrunk for tests; shrinking changes only the
counts (steps, lanes, observations), never the structure of the program.

Program text is written in the stack bytecode of :mod:`workloads.bytecode`.
Data synthesis (simulating each model at its generating parameters and adding
noise) is the workload's ground truth, computed here with numpy; it is not the
method under test.

RNG: ``numpy.random.Generator(PCG64(SeedSequence(seed)))``; the seed sequence
is spawned into three children used for (data noise, lane parameters,
programs) in that order.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from .bytecode import Asm
from . import randtree

HALF_LN_2PI = 0.5 * math.log(2.0 * math.pi)
LN_2PI = math.log(2.0 * math.pi)


@dataclass
class Workload:
    name: str
    bytecode: bytes                 # single-program workloads
    obs: np.ndarray                 # float64 [n_obs]
    params: np.ndarray              # float64 [L, P] (or [n_prog, L, P_max])
    truth: Optional[np.ndarray] = None
    programs: List[bytes] = field(default_factory=list)   # cfg5 only
    n_params_each: List[int] = field(default_factory=list)
    meta: dict = field(default_factory=dict)

    @property
    def L(self) -> int:
        return self.params.shape[-2]


def _rngs(seed: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(3)]


# --------------------------------------------------------------------------
# config 1: exponential decay y = a exp(-b t) + c, MSE
# --------------------------------------------------------------------------
def exp_decay_program(n: int) -> bytes:
    """obs = [t_0..t_{n-1}, y_0..y_{n-1}]; params (a, b, c); loss = mean r^2."""
    A = Asm(3, 2 * n)
    A.param(0).storel(0).param(1).storel(1).param(2).storel(2)
    A.push(0.0).storel(3)
    A.loop(n)
    A.loadl(3)                                  # acc
    A.loadl(0).loadl(1).obs(0, 1).mul().neg().exp().mul()   # a * exp(-(b t))
    A.loadl(2).add()                            # + c
    A.obs(n, 1).sub()                           # - y
    A.dup().mul()                               # r^2
    A.add().storel(3)                           # acc + r^2
    A.endloop()
    A.loadl(3).push(1.0 / n).mul().halt()
    return A.bytes()


def exp_decay_term_program() -> bytes:
    """One data point of the exponential-decay loss, for the flattened data
    axis: obs = [t, y] of the lane's point; params (a, b, c); term = r^2 with
    r = a * exp(-(b t)) + c - y, the same operations in the same order as one
    trip of exp_decay_program's loop."""
    A = Asm(3, 2)
    A.param(0).param(1).obs(0).mul().neg().exp().mul()
    A.param(2).add()
    A.obs(1).sub()
    A.dup().mul()
    return A.halt().bytes()


def exp_decay(L: int = 256, n: int = 64, seed: int = 1001, noise: float = 0.01):
    r_data, r_lane, _ = _rngs(seed)
    t = np.linspace(0.0, 5.0, n)
    truth = np.array([2.0, 0.7, 0.3])
    y = truth[0] * np.exp(-truth[1] * t) + truth[2] + r_data.normal(0.0, noise, n)
    params = r_lane.uniform(0.1, 3.0, size=(L, 3))
    return Workload("exp_decay", exp_decay_program(n), np.concatenate([t, y]),
                    np.ascontiguousarray(params), truth,
                    meta=dict(n_obs_points=n, L=L, seed=seed))


# --------------------------------------------------------------------------
# config 2: logistic growth, forward Euler, Gaussian NLL
# --------------------------------------------------------------------------
def logistic_program(T: int, dt: float = 0.01) -> bytes:
    """params (r, K, x0, sigma); obs[k] observes the state after step k+1."""
    A = Asm(4, T)
    A.param(0).storel(0).param(1).storel(1).param(2).storel(2).param(3).storel(3)
    A.push(0.0).storel(4)
    A.loop(T)
    # x <- x + ((dt*r)*x) * (1 - x/K)
    A.loadl(2)
    A.push(dt).loadl(0).mul().loadl(2).mul()
    A.push(1.0).loadl(2).loadl(1).div().sub()
    A.mul().add().storel(2)
    # nll <- nll + ((x - y)^2 / ((2 sigma) sigma) + ln sigma + ln(2 pi)/2)
    A.loadl(4)
    A.loadl(2).obs(0, 1).sub().dup().mul()
    A.push(2.0).loadl(3).mul().loadl(3).mul().div()
    A.loadl(3).log().add()
    A.push(HALF_LN_2PI).add()
    A.add().storel(4)
    A.endloop()
    A.loadl(4).halt()
    return A.bytes()


def logistic_truth_path(theta, T, dt=0.01):
    r, K, x0 = theta[0], theta[1], theta[2]
    x = x0
    out = np.empty(T)
    for k in range(T):
        x = x + dt * r * x * (1.0 - x / K)
        out[k] = x
    return out


def logistic(L: int = 4096, T: int = 500, seed: int = 2002):
    r_data, r_lane, _ = _rngs(seed)
    truth = np.array([2.0, 10.0, 0.5, 0.2])
    y = logistic_truth_path(truth, T) + r_data.normal(0.0, truth[3], T)
    params = truth[None, :] * 10.0 ** r_lane.uniform(-0.5, 0.5, size=(L, 4))
    return Workload("logistic_euler", logistic_program(T), y,
                    np.ascontiguousarray(params), truth,
                    meta=dict(T=T, L=L, seed=seed, dt=0.01))


# --------------------------------------------------------------------------
# config 3: Lotka-Volterra, RK4, MSE on both states
# --------------------------------------------------------------------------
def lotka_volterra_program(T: int, h: float = 0.02) -> bytes:
    """params (alpha, beta, gamma, delta, x0, y0); obs interleaved
    (x_1, y_1, x_2, y_2, ...), obs pair k observes the state after step k+1."""
    A = Asm(6, 2 * T)
    AL, BE, GA, DE, X, Y, ACC = 0, 1, 2, 3, 4, 5, 6
    K = [(7, 8), (9, 10), (11, 12), (13, 14)]
    XS, YS, XY = 15, 16, 17
    for i in range(6):
        A.param(i).storel(i)
    A.push(0.0).storel(ACC)

    def f(kx, ky):
        A.loadl(XS).loadl(YS).mul().storel(XY)
        A.loadl(AL).loadl(XS).mul().loadl(BE).loadl(XY).mul().sub().storel(kx)
        A.loadl(DE).loadl(XY).mul().loadl(GA).loadl(YS).mul().sub().storel(ky)

    def stage_input(coef, kx, ky):
        A.loadl(X).push(coef).loadl(kx).mul().add().storel(XS)
        A.loadl(Y).push(coef).loadl(ky).mul().add().storel(YS)

    A.loop(T)
    A.loadl(X).storel(XS).loadl(Y).storel(YS)
    f(*K[0])
    stage_input(h / 2.0, *K[0])
    f(*K[1])
    stage_input(h / 2.0, *K[1])
    f(*K[2])
    stage_input(h, *K[2])
    f(*K[3])
    for comp, s in ((0, X), (1, Y)):
        A.loadl(s).push(h / 6.0)
        A.loadl(K[0][comp]).push(2.0).loadl(K[1][comp]).mul().add()
        A.push(2.0).loadl(K[2][comp]).mul().add()
        A.loadl(K[3][comp]).add()
        A.mul().add().storel(s)
    A.loadl(ACC)
    A.loadl(X).obs(0, 2).sub().dup().mul().add()
    A.loadl(Y).obs(1, 2).sub().dup().mul().add()
    A.storel(ACC)
    A.endloop()
    A.loadl(ACC).push(1.0 / (2.0 * T)).mul().halt()
    return A.bytes()


def lv_truth_path(theta, T, h=0.02):
    al, be, ga, de, x, y = [float(v) for v in theta]
    out = np.empty((T, 2))

    def f(x, y):
        xy = x * y
        return al * x - be * xy, de * xy - ga * y
    for k in range(T):
        k1 = f(x, y)
        k2 = f(x + h / 2 * k1[0], y + h / 2 * k1[1])
        k3 = f(x + h / 2 * k2[0], y + h / 2 * k2[1])
        k4 = f(x + h * k3[0], y + h * k3[1])
        x = x + h / 6 * (k1[0] + 2 * k2[0] + 2 * k3[0] + k4[0])
        y = y + h / 6 * (k1[1] + 2 * k2[1] + 2 * k3[1] + k4[1])
        out[k] = (x, y)
    return out


def lotka_volterra(L: int = 65536, T: int = 1000, seed: int = 3003):
    r_data, r_lane, _ = _rngs(seed)
    truth = np.array([1.0, 0.5, 1.0, 0.5, 1.0, 0.5])
    path = lv_truth_path(truth, T) + r_data.normal(0.0, 0.05, (T, 2))
    params = truth[None, :] * r_lane.uniform(0.5, 1.5, size=(L, 6))
    return Workload("lotka_volterra_rk4", lotka_volterra_program(T),
                    path.reshape(-1).copy(), np.ascontiguousarray(params), truth,
                    meta=dict(T=T, L=L, seed=seed, h=0.02))


# --------------------------------------------------------------------------
# config 4: 4-state constant-velocity Kalman filter, NLL
# --------------------------------------------------------------------------
def kalman_program(T: int, branch_tail: bool = False) -> bytes:
    """params (dt, q1..q4, r1, r2, x0_1..x0_4, s); obs interleaved 2-D
    measurements.  Filter: predict, innovation, update in the standard
    P+ = (I - K H) P- form.  branch_tail: the NLL is then reshaped by a
    numeric branch on dt (one of two chains of six multiply-adds; a test
    program with skippable arms)."""
    A = Asm(12, 2 * T)
    F, Ft, Q, H, Ht, R, X, P, I4, NLL = range(10)
    XM, PM, V, S, SI, KG = 10, 11, 12, 13, 14, 15
    # F(dt) row-major
    for i in range(4):
        for j in range(4):
            if (i, j) in ((0, 2), (1, 3)):
                A.param(0)
            else:
                A.push(1.0 if i == j else 0.0)
    A.pack(4, 4).storel(F)
    A.loadl(F).transpose().storel(Ft)
    for i in range(4):
        for j in range(4):
            if i == j:
                A.param(1 + i)
            else:
                A.push(0.0)
    A.pack(4, 4).storel(Q)
    for i in range(2):
        for j in range(4):
            A.push(1.0 if i == j else 0.0)
    A.pack(2, 4).storel(H)
    A.loadl(H).transpose().storel(Ht)
    A.param(5).push(0.0).push(0.0).param(6).pack(2, 2).storel(R)
    for i in range(4):
        A.param(7 + i)
    A.pack(4, 1).storel(X)
    for i in range(4):
        for j in range(4):
            A.push(1.0 if i == j else 0.0)
    A.pack(4, 4).storel(I4)
    A.loadl(I4).param(11).mul().storel(P)
    A.push(0.0).storel(NLL)
    A.loop(T)
    A.loadl(F).loadl(X).matmul().storel(XM)
    A.loadl(F).loadl(P).matmul().loadl(Ft).matmul().loadl(Q).add().storel(PM)
    A.obs(0, 2).obs(1, 2).pack(2, 1)
    A.loadl(H).loadl(XM).matmul().sub().storel(V)
    A.loadl(H).loadl(PM).matmul().loadl(Ht).matmul().loadl(R).add().storel(S)
    A.loadl(S).inv().storel(SI)
    A.loadl(PM).loadl(Ht).matmul().loadl(SI).matmul().storel(KG)
    A.loadl(XM).loadl(KG).loadl(V).matmul().add().storel(X)
    A.loadl(I4).loadl(KG).loadl(H).matmul().sub().loadl(PM).matmul().storel(P)
    A.loadl(NLL)
    A.loadl(S).logdet()
    A.loadl(V).transpose().loadl(SI).matmul().loadl(V).matmul()
    A.add().push(2.0 * LN_2PI).add().push(0.5).mul()
    A.add().storel(NLL)
    A.endloop()
    if branch_tail:
        A.param(0).push(0.1).iflt()
        for _ in range(6):
            A.loadl(NLL).loadl(NLL).param(1).mul().push(1e-3).mul().add().storel(NLL)
        A.else_()
        for _ in range(6):
            A.loadl(NLL).loadl(NLL).param(5).mul().push(2e-3).mul().add().storel(NLL)
        A.endif()
    A.loadl(NLL).halt()
    return A.bytes()


KALMAN_TRUTH = np.array([0.1, 1e-4, 1e-4, 1e-3, 1e-3, 1e-2, 1e-2,
                         0.0, 0.0, 1.0, 0.5, 1.0])


def kalman_matrices(theta):
    dt = theta[0]
    F = np.array([[1, 0, dt, 0], [0, 1, 0, dt], [0, 0, 1, 0], [0, 0, 0, 1]], float)
    Q = np.diag(theta[1:5])
    H = np.array([[1, 0, 0, 0], [0, 1, 0, 0]], float)
    R = np.diag(theta[5:7])
    x0 = np.array(theta[7:11], float)
    P0 = theta[11] * np.eye(4)
    return F, Q, H, R, x0, P0


def kalman(L: int = 16384, T: int = 200, seed: int = 4004):
    r_data, r_lane, _ = _rngs(seed)
    truth = KALMAN_TRUTH.copy()
    F, Q, H, R, x0, P0 = kalman_matrices(truth)
    x = r_data.multivariate_normal(x0, P0)
    ys = np.empty((T, 2))
    for k in range(T):
        x = F @ x + r_data.multivariate_normal(np.zeros(4), Q)
        ys[k] = H @ x + r_data.multivariate_normal(np.zeros(2), R)
    params = np.empty((L, 12))
    pos = [0, 1, 2, 3, 4, 5, 6, 11]
    params[:, pos] = truth[pos][None, :] * 10.0 ** r_lane.uniform(-0.5, 0.5, (L, len(pos)))
    params[:, 7:11] = truth[7:11][None, :] + r_lane.uniform(-0.5, 0.5, (L, 4))
    return Workload("kalman_cv4", kalman_program(T), ys.reshape(-1).copy(),
                    np.ascontiguousarray(params), truth,
                    meta=dict(T=T, L=L, seed=seed))


# --------------------------------------------------------------------------
# config 5: population of random expression programs, MSE
# --------------------------------------------------------------------------
def tree_program(tree, n_params: int, n: int) -> bytes:
    """obs = [x_0..x_{n-1}, y_0..y_{n-1}]; loss = mean (tree(x) - y)^2."""
    A = Asm(n_params, 2 * n)
    A.push(0.0).storel(0)
    A.loop(n)
    A.loadl(0)
    randtree.emit(A, tree)
    A.obs(n, 1).sub().dup().mul()
    A.add().storel(0)
    A.endloop()
    A.loadl(0).push(1.0 / n).mul().halt()
    return A.bytes()


def tree_term_program(tree, n_params: int) -> bytes:
    """One data point of a tree program's loss, for the flattened data axis:
    obs = [x, y] of the lane's point; term = (tree(x) - y)^2, the same
    operations in the same order as one trip of tree_program's loop."""
    A = Asm(n_params, 2)
    randtree.emit(A, tree, x_obs=(0,))
    A.obs(1).sub().dup().mul()
    return A.halt().bytes()


def points_of(obs: np.ndarray, n: int, width: int = 2) -> np.ndarray:
    """Observations [f_0..f_{n-1}, g_0..g_{n-1}, ...] as point-major rows
    [[f_0, g_0, ...], ...] (the layout of the flattened data axis)."""
    return np.ascontiguousarray(np.asarray(obs, dtype=np.float64).reshape(width, n).T)


def random_programs(n_prog: int = 1024, L: int = 1024, n: int = 128,
                    seed: int = 5005, noise: float = 0.1):
    r_data, r_lane, r_prog = _rngs(seed)
    hidden, hidden_c = randtree.hidden_tree(r_prog)
    xs = r_data.uniform(-2.0, 2.0, n)
    ys = np.array([randtree.evaluate(hidden, hidden_c, float(x)) for x in xs])
    ys = ys + r_data.normal(0.0, noise, n)
    trees, counts = [], []
    stats = dict(rejected=0)
    while len(trees) < n_prog:
        t = randtree.grow(r_prog)
        nc = randtree.n_consts(t)
        if not randtree.acceptable(t):
            stats["rejected"] += 1
            continue
        trees.append(t)
        counts.append(nc)
    pmax = 8
    params = np.zeros((n_prog, L, pmax))
    for i, nc in enumerate(counts):
        params[i, :, :nc] = r_lane.uniform(-2.0, 2.0, (L, nc))
    progs = [tree_program(t, c, n) for t, c in zip(trees, counts)]
    w = Workload("random_programs", progs[0], np.concatenate([xs, ys]),
                 np.ascontiguousarray(params), None, programs=progs,
                 n_params_each=counts,
                 meta=dict(n_prog=n_prog, L=L, n=n, seed=seed,
                           hidden=randtree.to_str(hidden, hidden_c),
                           **stats))
    w.meta["trees"] = trees
    w.meta["hidden_tree"] = (hidden, hidden_c)
    return w


# Programs whose numeric branches have heavy arms (eight value elements or
# more each side that is heavy), for wave-level branch skipping: the same
# lanes ordered by the branch's predicate (the waves decide alike and skip
# arms) or interleaved (every wave runs both arms).
_HA = ("pexp", ("ppow", ("add", ("x",), ("c", 2)), ("sin", ("mul", ("c", 3), ("x",)))))
_HB = ("plog", ("add", ("pdiv", ("c", 4), ("x",)), ("ppow", ("x",), ("c", 2))))
_HC = ("pdiv", ("pexp", ("mul", ("c", 2), ("c", 3))), ("plog", ("sub", ("c", 4), ("pexp", ("c", 3)))))
BRANCH_TREES = [
    # predicate c0 < c1, arms depend on x
    ("add", ("iflt", ("c", 0), ("c", 1), _HA, _HB), ("x",)),
    # a branch that does not depend on x: later loop trips repeat its values
    ("mul", ("ppow", ("x",), ("iflt", ("c", 0), ("c", 1), _HC, ("c", 4))), ("sin", ("x",))),
    # a select reading another select of the same predicate
    ("iflt", ("c", 0), ("c", 1), ("c", 2), ("iflt", ("c", 0), ("c", 1), _HA, _HB)),
    # predicate x < c0 (lanes ordered by c0 decide alike on most trips)
    ("iflt", ("x",), ("c", 0), ("sin", _HA), _HB),
]


def branch_population(case: int = 0, L: int = 65536, n: int = 128, seed: int = 6006, order: str = "sorted"):
    """Tree program BRANCH_TREES[case] (mean squared error over n points) on L
    lanes of parameters uniform in [-2, 2], ordered so that consecutive lanes
    decide the branch alike ("sorted") or alternately ("mixed"), or with c0
    moved so that every lane takes the first arm ("all_then") or the second
    ("all_else"); meta["order"] maps lane i to its index in the unordered
    draw."""
    tree = BRANCH_TREES[case]
    nc = randtree.n_consts(tree)
    r_data, r_lane, _ = _rngs(seed)
    xs = r_data.uniform(-2.0, 2.0, n)
    ys = r_data.uniform(-1.0, 1.0, n)
    p = r_lane.uniform(-2.0, 2.0, (L, nc))
    if order in ("all_then", "all_else"):
        then = order == "all_then"
        if case == 3:   # x < c0 with x in [-2, 2]
            p[:, 0] = 2.5 if then else -2.5
        else:           # c0 < c1
            p[:, 0] = p[:, 1] - 1.0 if then else p[:, 1] + 1.0
    key = p[:, 0] if case == 3 else (p[:, 0] < p[:, 1]).astype(np.float64)
    idx = np.argsort(key, kind="stable")
    if order in ("all_then", "all_else"):
        idx = np.arange(L)
    elif order == "mixed":
        half = L // 2
        mixed = np.empty(L, dtype=np.int64)
        mixed[0:2 * half:2] = idx[:half]
        mixed[1:2 * half:2] = idx[half:2 * half]
        if L % 2:
            mixed[-1] = idx[-1]
        idx = mixed
    elif order != "sorted":
        raise ValueError(order)
    return Workload("branch_population", tree_program(tree, nc, n), np.concatenate([xs, ys]),
                    np.ascontiguousarray(p[idx]), None,
                    meta=dict(case=case, L=L, n=n, seed=seed, order_kind=order, order=idx, tree=tree))


BUILDERS = {
    "exp_decay": exp_decay,
    "logistic_euler": logistic,
    "lotka_volterra_rk4": lotka_volterra,
    "kalman_cv4": kalman,
    "random_programs": random_programs,
}

# index order of the five benchmark configurations
ORDER = ["exp_decay", "logistic_euler", "lotka_volterra_rk4", "kalman_cv4",
         "random_programs"]


def build(name: str, **kw) -> Workload:
    return BUILDERS[name](**kw)
