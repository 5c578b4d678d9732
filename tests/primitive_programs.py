"""Small programs that exercise every primitive of the bytecode once (scalar
unary and binary ops, matrix products of several shapes, transposes, traces,
outer products, elementwise matrix ops, 1x1 and 2x2 inverse, determinant and
log-determinant, a numeric select with a tie, a NaN predicate and an
overflowing untaken arm, the log/sqrt clamp and |x| at 0), each with a few
parameter rows.  Shared by the oracle pins and the GPU parity tests.
"""
import numpy as np

from workloads.bytecode import Asm


def primitive_programs():
    import test_oracle_pins as T
    out = []
    for op, x in T.UNARY:
        A = Asm(2, 0)
        A.param(0).raw(op).param(1).mul().halt()
        out.append((A.bytes(), [[x, -1.7], [x * 0.5, 2.0]]))
    for op in T.BINARY:
        A = Asm(3, 0)
        A.param(0).param(1).raw(op).param(2).mul().halt()
        out.append((A.bytes(), [[1.3, 0.6, -0.8], [0.7, 1.9, 1.1]]))
    for m, k, n in [(2, 3, 2), (4, 4, 4), (4, 4, 1), (2, 4, 4), (4, 2, 2), (1, 2, 2), (3, 1, 2)]:
        A = Asm(m * k + n * k, 0)
        T._mat(A, m, k, 0)
        T._mat(A, k, n, m * k)
        A.matmul()
        T._weights(A, m, n, 7)
        A.dot().halt()
        out.append((A.bytes(), [T._theta(m * k + n * k, s) for s in (1, 2)]))
    for what in ["transpose", "trace", "outer", "dot", "index", "add", "sub", "hadamard", "ediv",
                 "smul", "muls", "divs", "eexp", "esin", "elog"]:
        A = Asm(13, 0)
        if what == "transpose":
            T._mat(A, 2, 3, 0); A.transpose(); T._weights(A, 3, 2, 3); A.dot()
        elif what == "trace":
            T._mat(A, 3, 3, 0); A.trace(); A.param(9).mul()
        elif what == "outer":
            T._mat(A, 3, 1, 0); T._mat(A, 2, 1, 3); A.outer(); T._weights(A, 3, 2, 4); A.dot()
        elif what == "dot":
            T._mat(A, 2, 3, 0); T._mat(A, 2, 3, 6); A.dot()
        elif what == "index":
            T._mat(A, 2, 3, 0); A.index(1, 2); A.param(0).mul()
        elif what in ("add", "sub", "hadamard", "ediv"):
            from workloads import bytecode as B
            op = {"add": B.ADD, "sub": B.SUB, "hadamard": B.MUL, "ediv": B.DIV}[what]
            T._mat(A, 2, 3, 0); T._mat(A, 2, 3, 6); A.raw(op); T._weights(A, 2, 3, 5); A.dot()
        elif what == "smul":
            A.param(12); T._mat(A, 2, 3, 0); A.mul(); T._weights(A, 2, 3, 6); A.dot()
        elif what == "muls":
            T._mat(A, 2, 3, 0); A.param(12); A.mul(); T._weights(A, 2, 3, 6); A.dot()
        elif what == "divs":
            T._mat(A, 2, 3, 0); A.param(12); A.div(); T._weights(A, 2, 3, 6); A.dot()
        else:
            from workloads import bytecode as B
            op = {"eexp": B.EXP, "esin": B.SIN, "elog": B.LOG}[what]
            T._mat(A, 2, 3, 0); A.raw(op); T._weights(A, 2, 3, 8); A.dot()
        A.halt()
        lo = 0.2 if what in ("elog", "ediv") else -1.0
        out.append((A.bytes(), [T._theta(13, s, lo, 1.3) for s in (2, 3)]))
    for n in (1, 2):
        for op in ("inv", "det", "logdet"):
            A = Asm(n * n + 1, 0)
            T._mat(A, n, n, 0)
            getattr(A, op)()
            if op == "inv":
                T._weights(A, n, n, 11)
                A.dot()
            else:
                A.param(n * n).mul()
            A.halt()
            th = [1.4, 0.3, -0.2, 0.9][: n * n] + [1.1] if n == 2 else [1.6, 1.1]
            out.append((A.bytes(), [th, [v * 0.9 for v in th]]))
    out.append((T._select_prog(), [[1.0, 1.0, 5.0], [np.nan, 1.0, 5.0], [0.5, 1.0, 0.001], [2.0, 1.0, 5.0]]))
    out.append((T._log_prog(0x19), [[1e-9], [-1.0], [1e-8], [2e-8]]))
    out.append((T._log_prog(0x1A), [[1e-9], [-1.0], [1e-8], [2e-8]]))
    A = Asm(1, 0)
    A.param(0).abs().halt()
    out.append((A.bytes(), [[0.0], [-2.0], [3.0]]))
    return out


