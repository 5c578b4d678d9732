"""Seeded random expression trees for the program-population workload.

The paper's randomized differential tester draws typed scalar programs and
keeps them in a smooth, in-range domain by wrapping denominators and log/sqrt
arguments to 1 + x^2 and squashing exp arguments (Section "From buckets to
phases", correctness paragraph).  The generator here follows that recipe with
protected forms; the squash is a sine:

    pdiv(a, b) = a / (1 + b*b)        ppow(a, b) = (1 + a*a) ** sin(b)
    pexp(a)    = exp(sin(a))          plog(a)    = log(1 + a*a)
    iflt(a, b, c, d) = c if a < b else d      (a per-lane select)

plus add, sub, mul, sin.  Grow: a node at depth d is a leaf with probability
d/8 (always at depth 8); a leaf is the observation x or a fresh constant with
probability 1/2 each; the nine operators are drawn uniformly.  Structural
acceptance: 2..8 constants, at least one x, at most 60 tape ops per
observation term, and a magnitude bound (interval propagation with
|x|, |c| <= 2) no larger than 1e100 so that squared residuals stay finite.

Trees are tuples: ("x",), ("c", j), (op, child, ...).
"""
from __future__ import annotations

import math

OPS = ["add", "sub", "mul", "pdiv", "ppow", "sin", "pexp", "plog", "iflt"]
ARITY = {"add": 2, "sub": 2, "mul": 2, "pdiv": 2, "ppow": 2,
         "sin": 1, "pexp": 1, "plog": 1, "iflt": 4}
MAX_DEPTH = 8


def grow(rng, depth: int = 0, counter=None):
    if counter is None:
        counter = [0]
    if depth >= MAX_DEPTH or (depth > 0 and rng.random() < depth / MAX_DEPTH):
        if rng.random() < 0.5:
            return ("x",)
        j = counter[0]
        counter[0] += 1
        return ("c", j)
    op = OPS[int(rng.integers(len(OPS)))]
    kids = tuple(grow(rng, depth + 1, counter) for _ in range(ARITY[op]))
    return (op,) + kids


def n_consts(t) -> int:
    if t[0] == "c":
        return 1
    if t[0] == "x":
        return 0
    return sum(n_consts(k) for k in t[1:])


def n_x(t) -> int:
    if t[0] == "x":
        return 1
    if t[0] == "c":
        return 0
    return sum(n_x(k) for k in t[1:])


_TAPE_COST = {"add": 1, "sub": 1, "mul": 1, "pdiv": 4, "ppow": 5, "sin": 1,
              "pexp": 2, "plog": 4, "iflt": 1}


def tape_ops(t) -> int:
    """Tape ops one evaluation of the tree emits (leaves, wrappers, selects)."""
    if t[0] in ("x", "c"):
        return 1
    return _TAPE_COST[t[0]] + sum(tape_ops(k) for k in t[1:])


def bound(t) -> float:
    """Upper bound on |value| for |x|, |c| <= 2."""
    op = t[0]
    if op in ("x", "c"):
        return 2.0
    b = [bound(k) for k in t[1:]]
    if op in ("add", "sub"):
        return b[0] + b[1]
    if op == "mul":
        return b[0] * b[1]
    if op == "pdiv":
        return b[0]
    if op == "ppow":
        return 1.0 + b[0] * b[0]
    if op == "sin":
        return 1.0
    if op == "pexp":
        return math.e
    if op == "plog":
        return math.log1p(b[0] * b[0]) if b[0] < 1e150 else 2.0 * math.log(b[0]) + 1.0
    if op == "iflt":
        return max(b[2], b[3])
    raise ValueError(op)


def acceptable(t) -> bool:
    nc = n_consts(t)
    return (2 <= nc <= 8 and n_x(t) >= 1 and tape_ops(t) <= 60
            and bound(t) <= 1e100)


def hidden_tree(rng):
    """First acceptable tree of the program stream, with constants ~U(-2, 2)
    drawn right after it; it generates the observations."""
    while True:
        t = grow(rng)
        if acceptable(t):
            c = rng.uniform(-2.0, 2.0, n_consts(t))
            return t, [float(v) for v in c]


def evaluate(t, consts, x: float) -> float:
    """Plain evaluation, used only to synthesize observations."""
    op = t[0]
    if op == "x":
        return x
    if op == "c":
        return consts[t[1]]
    v = [evaluate(k, consts, x) for k in t[1:]] if op != "iflt" else None
    if op == "add":
        return v[0] + v[1]
    if op == "sub":
        return v[0] - v[1]
    if op == "mul":
        return v[0] * v[1]
    if op == "pdiv":
        return v[0] / (1.0 + v[1] * v[1])
    if op == "ppow":
        return math.pow(1.0 + v[0] * v[0], math.sin(v[1]))
    if op == "sin":
        return math.sin(v[0])
    if op == "pexp":
        return math.exp(math.sin(v[0]))
    if op == "plog":
        return math.log(1.0 + v[0] * v[0])
    if op == "iflt":
        a = evaluate(t[1], consts, x)
        b = evaluate(t[2], consts, x)
        return evaluate(t[3], consts, x) if a < b else evaluate(t[4], consts, x)
    raise ValueError(op)


def emit(A, t, x_obs=(0, 1)):
    """Append postfix bytecode evaluating the tree for the current loop
    counter (x = OBS 0 with stride 1, constant j = PARAM j); x_obs gives the
    OBS word's base and strides (x_obs=(0,) reads obs[0] outside any loop)."""
    op = t[0]
    if op == "x":
        A.obs(*x_obs)
        return
    if op == "c":
        A.param(t[1])
        return
    k = t[1:]
    if op in ("add", "sub", "mul"):
        emit(A, k[0], x_obs)
        emit(A, k[1], x_obs)
        getattr(A, op)()
    elif op == "pdiv":
        emit(A, k[0], x_obs)
        A.push(1.0)
        emit(A, k[1], x_obs)
        A.dup().mul().add().div()
    elif op == "ppow":
        A.push(1.0)
        emit(A, k[0], x_obs)
        A.dup().mul().add()
        emit(A, k[1], x_obs)
        A.sin().pow()
    elif op == "sin":
        emit(A, k[0], x_obs)
        A.sin()
    elif op == "pexp":
        emit(A, k[0], x_obs)
        A.sin().exp()
    elif op == "plog":
        A.push(1.0)
        emit(A, k[0], x_obs)
        A.dup().mul().add().log()
    elif op == "iflt":
        emit(A, k[0], x_obs)
        emit(A, k[1], x_obs)
        A.iflt()
        emit(A, k[2], x_obs)
        A.else_()
        emit(A, k[3], x_obs)
        A.endif()
    else:
        raise ValueError(op)


def to_str(t, consts=None) -> str:
    op = t[0]
    if op == "x":
        return "x"
    if op == "c":
        return f"{consts[t[1]]:.6g}" if consts is not None else f"c{t[1]}"
    return f"{op}(" + ", ".join(to_str(k, consts) for k in t[1:]) + ")"
