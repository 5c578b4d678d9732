"""Forward-only NDVB evaluator over complex numbers, used to pin the oracle.

Complex-step differentiation (Squire & Trapp 1998; Martins, Sturdza & Alonso
2003): for a real-analytic f, f'(x) = Im f(x + i h) / h + O(h^2) with no
subtractive cancellation, so h = 1e-30 gives derivatives to machine
precision.  This evaluator knows only the *forward* meaning of each bytecode
word; it has no adjoint rules, no tape and no code in common with the oracle,
so agreement between the two checks the oracle's reverse sweep.

Non-analytic points are handled the way the method defines them: abs
continues as +x or -x by the sign of the real part (derivative 0 at exactly
0), the sqrt/log clamp becomes a constant below 1e-8, and a numeric IFLT
compares real parts (Property 1: the predicate carries no gradient).
"""
from __future__ import annotations

import cmath
import struct

from workloads import bytecode as B

EPS = 1e-8


class M:
    """Small row-major matrix of complex numbers."""
    __slots__ = ("r", "c", "e")

    def __init__(self, r, c, e):
        self.r, self.c, self.e = r, c, list(e)

    @staticmethod
    def s(x):
        return M(1, 1, [x])

    def scalar(self):
        return self.r == 1 and self.c == 1


def _clamp(x):
    return complex(EPS, 0.0) if x.real < EPS else x


def _abs(x):
    if x.real > 0:
        return x
    if x.real < 0:
        return -x
    return complex(0.0, 0.0)


def _mm(a, b):
    out = []
    for i in range(a.r):
        for j in range(b.c):
            out.append(sum(a.e[i * a.c + p] * b.e[p * b.c + j] for p in range(a.c)))
    return M(a.r, b.c, out)


def _t(a):
    return M(a.c, a.r, [a.e[i * a.c + j] for j in range(a.c) for i in range(a.r)])


def _det(a):
    if a.r == 1:
        return a.e[0]
    if a.r == 2:
        return a.e[0] * a.e[3] - a.e[1] * a.e[2]
    raise ValueError("det: only 1x1 and 2x2")


def _inv(a):
    d = _det(a)
    if a.r == 1:
        return M(1, 1, [1.0 / d])
    return M(2, 2, [a.e[3] / d, -a.e[1] / d, -a.e[2] / d, a.e[0] / d])


def evaluate(bc: bytes, theta, obs):
    """Return the (complex) loss of one lane with parameter vector theta."""
    n_params, n_obs, n_instr, n_consts = B.parse_header(bc)
    code = [struct.unpack_from("<BBHI", bc, 24 + 8 * k) for k in range(n_instr)]
    consts = struct.unpack_from(f"<{n_consts}d", bc, 24 + 8 * n_instr)
    # block matching
    match, st = {}, []
    for pc, (op, a, b, imm) in enumerate(code):
        if op in (B.LOOP, B.IFLT):
            st.append(pc)
        elif op == B.ELSE:
            match[st[-1]] = pc
            st[-1] = pc
        elif op == B.ENDIF:
            match[st.pop()] = pc
        elif op == B.ENDLOOP:
            o = st.pop()
            match[o] = pc
            match[pc] = o
    stack, loc, loops = [], {}, []
    pc = 0
    elem1 = {B.NEG: lambda x: -x, B.EXP: cmath.exp, B.LOG: lambda x: cmath.log(_clamp(x)),
             B.SQRT: lambda x: cmath.sqrt(_clamp(x)), B.SIN: cmath.sin,
             B.COS: cmath.cos, B.ABS: _abs}
    while True:
        op, a, b, imm = code[pc]
        if op == B.HALT:
            assert len(stack) == 1 and stack[0].scalar()
            return stack[0].e[0]
        if op == B.PUSH:
            stack.append(M.s(complex(consts[imm])))
        elif op == B.PARAM:
            stack.append(M.s(complex(theta[imm])))
        elif op == B.OBS:
            idx = imm
            for d in range(a):
                stride = struct.unpack("<i", struct.pack("<I", code[pc + 1 + d][3]))[0]
                idx += stride * loops[-1 - d][2]
            stack.append(M.s(complex(obs[idx])))
            pc += a
        elif op == B.LOADL:
            stack.append(loc[imm])
        elif op == B.STOREL:
            loc[imm] = stack.pop()
        elif op == B.DUP:
            stack.append(stack[-1])
        elif op == B.OVER:
            stack.append(stack[-2])
        elif op == B.SWAP:
            stack[-1], stack[-2] = stack[-2], stack[-1]
        elif op == B.DROP:
            stack.pop()
        elif op in (B.ADD, B.SUB, B.MUL, B.DIV):
            y = stack.pop()
            x = stack.pop()
            f = {B.ADD: lambda p, q: p + q, B.SUB: lambda p, q: p - q,
                 B.MUL: lambda p, q: p * q, B.DIV: lambda p, q: p / q}[op]
            if (x.r, x.c) == (y.r, y.c):
                stack.append(M(x.r, x.c, [f(p, q) for p, q in zip(x.e, y.e)]))
            elif y.scalar():
                stack.append(M(x.r, x.c, [f(p, y.e[0]) for p in x.e]))
            elif x.scalar() and op == B.MUL:
                stack.append(M(y.r, y.c, [x.e[0] * q for q in y.e]))
            else:
                raise ValueError("shape")
        elif op in elem1:
            x = stack.pop()
            stack.append(M(x.r, x.c, [elem1[op](v) for v in x.e]))
        elif op == B.POW:
            y = stack.pop()
            x = stack.pop()
            stack.append(M.s(cmath.exp(y.e[0] * cmath.log(x.e[0]))))
        elif op == B.DOT:
            y = stack.pop()
            x = stack.pop()
            stack.append(M.s(sum(p * q for p, q in zip(x.e, y.e))))
        elif op == B.MATMUL:
            y = stack.pop()
            x = stack.pop()
            stack.append(_mm(x, y))
        elif op == B.TRANSPOSE:
            stack.append(_t(stack.pop()))
        elif op == B.TRACE:
            x = stack.pop()
            stack.append(M.s(sum(x.e[i * x.c + i] for i in range(x.r))))
        elif op == B.INV:
            stack.append(_inv(stack.pop()))
        elif op == B.DET:
            stack.append(M.s(_det(stack.pop())))
        elif op == B.LOGDET:
            stack.append(M.s(cmath.log(_clamp(_det(stack.pop())))))
        elif op == B.OUTER:
            y = stack.pop()
            x = stack.pop()
            stack.append(M(x.r, y.r, [p * q for p in x.e for q in y.e]))
        elif op == B.PACK:
            n = a * b
            vals = [v.e[0] for v in stack[-n:]]
            del stack[-n:]
            stack.append(M(a, b, vals))
        elif op == B.INDEX:
            x = stack.pop()
            stack.append(M.s(x.e[a * x.c + b]))
        elif op == B.LOOP:
            if imm == 0:
                pc = match[pc] + 1
                continue
            loops.append([pc + 1, imm, 0])
        elif op == B.ENDLOOP:
            loops[-1][2] += 1
            if loops[-1][2] < loops[-1][1]:
                pc = loops[-1][0]
                continue
            loops.pop()
        elif op == B.IFLT:
            y = stack.pop()
            x = stack.pop()
            if not (x.e[0].real < y.e[0].real):
                pc = match[pc] + 1
                continue
        elif op == B.ELSE:
            pc = match[pc] + 1
            continue
        elif op == B.ENDIF:
            pass
        else:
            raise ValueError(f"opcode {op:#x}")
        pc += 1


def gradient(bc: bytes, theta, obs, h: float = 1e-30):
    """Complex-step gradient of the loss with respect to every parameter."""
    theta = [float(t) for t in theta]
    out = []
    for p in range(len(theta)):
        th = [complex(t) for t in theta]
        th[p] = complex(theta[p], h)
        out.append(evaluate(bc, th, obs).imag / h)
    return out


def loss(bc: bytes, theta, obs) -> float:
    return evaluate(bc, [complex(t) for t in theta], obs).real
