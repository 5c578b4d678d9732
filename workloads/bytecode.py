"""Stack-bytecode format ("NDVB") and a small assembler.

The paper's second client is a stack-bytecode VM with a linear instruction
stream and an explicit operand stack (Section "Generality", second-client
paragraph): PUSH, LOAD, the four arithmetic operators, NEG, EXP, LOG, SIN, COS,
DUP, a counted LOOP, a conditional BRANCH and DOT.  The format below keeps that
dispatch model and widens the instruction set to cover every numeric primitive
of the adjoint table (Appendix "Implemented numeric primitives", table
tab:adjoints) plus the structural words the five synthetic workloads need
(locals, PACK/INDEX for building small matrices from scalars, IFLT for a
numeric two-way branch).

This module only *encodes* programs: it holds no arithmetic of the method.
Every consumer (the trace producer, the reference tape encoder, the CPU
oracle) parses these bytes with its own parser.

Binary layout (little-endian)::

    header   : b"NDVB", u32 version(=1), u32 n_params, u32 n_obs,
               u32 n_instr, u32 n_consts                      (24 bytes)
    code     : n_instr x 8-byte words {u8 op, u8 a, u16 b, u32 imm}
    consts   : n_consts x f64

Instruction semantics (a is the value below b on the stack):

    PUSH k          push const[k]                      (imm = k)
    PARAM i         push theta_i                       (imm = i)
    OBS             push obs[base + sum_d stride_d * counter_d]
                    imm = base, a = number n of OBSX words that follow;
                    OBSX word d (d = 0 is the innermost enclosing LOOP)
                    carries stride_d as a signed 32-bit imm
    LOADL j/STOREL j  push / pop-into local j          (imm = j)
    DUP SWAP DROP OVER  stack shuffles (no numeric work)
    ADD SUB MUL DIV     a (op) b; ADD/SUB elementwise on equal shapes; MUL/DIV
                    scalar*scalar, matrix*scalar, scalar*matrix, matrix/scalar,
                    or elementwise on equal shapes
    NEG EXP LOG SQRT SIN COS ABS   elementwise
    POW             a ** b, scalars only
    DOT             sum_i a_i * b_i over equal shapes  -> scalar
    MATMUL          (m x k)(k x n) -> m x n
    TRANSPOSE TRACE INV DET LOGDET   (INV/DET/LOGDET: 1x1 or 2x2)
    OUTER           (m x 1)(n x 1) -> m x n
    PACK            pop a*b scalars (a = rows, b = cols), first pushed is
                    element (0,0), row-major
    INDEX           matrix -> scalar element (a, b)
    LOOP n ... ENDLOOP     counted loop (imm = n >= 0)
    IFLT ... ELSE ... ENDIF   pops b then a; runs the first arm when a < b
                    (strict; unordered compares take the ELSE arm)
    HALT            end; the stack must hold exactly one scalar (the loss)
"""
from __future__ import annotations

import struct
from dataclasses import dataclass, field
from typing import List

import numpy as np

MAGIC = b"NDVB"
VERSION = 1

# opcode numbers of the bytecode format
HALT = 0x00
PUSH = 0x01
PARAM = 0x02
OBS = 0x03
OBSX = 0x04
LOADL = 0x05
STOREL = 0x06
DUP = 0x07
SWAP = 0x08
DROP = 0x09
OVER = 0x0A
ADD = 0x10
SUB = 0x11
MUL = 0x12
DIV = 0x13
NEG = 0x14
EXP = 0x18
LOG = 0x19
SQRT = 0x1A
SIN = 0x1B
COS = 0x1C
POW = 0x1D
ABS = 0x1E
DOT = 0x20
MATMUL = 0x21
TRANSPOSE = 0x22
INV = 0x23
DET = 0x24
LOGDET = 0x25
TRACE = 0x26
OUTER = 0x27
PACK = 0x28
INDEX = 0x29
LOOP = 0x30
ENDLOOP = 0x31
IFLT = 0x32
ELSE = 0x33
ENDIF = 0x34

NAMES = {v: k for k, v in dict(globals()).items()
         if k.isupper() and isinstance(v, int) and k not in ("VERSION",)}

_SIMPLE = {
    "dup": DUP, "swap": SWAP, "drop": DROP, "over": OVER,
    "add": ADD, "sub": SUB, "mul": MUL, "div": DIV, "neg": NEG,
    "exp": EXP, "log": LOG, "sqrt": SQRT, "sin": SIN, "cos": COS,
    "pow": POW, "abs": ABS, "dot": DOT, "matmul": MATMUL,
    "transpose": TRANSPOSE, "inv": INV, "det": DET, "logdet": LOGDET,
    "trace": TRACE, "outer": OUTER, "endloop": ENDLOOP, "iflt": IFLT,
    "else_": ELSE, "endif": ENDIF, "halt": HALT,
}


@dataclass
class Program:
    """An assembled program: code words, constant pool, declared sizes."""
    n_params: int
    n_obs: int
    code: List[tuple] = field(default_factory=list)   # (op, a, b, imm)
    consts: List[float] = field(default_factory=list)

    def to_bytes(self) -> bytes:
        out = bytearray(MAGIC)
        out += struct.pack("<5I", VERSION, self.n_params, self.n_obs,
                           len(self.code), len(self.consts))
        for op, a, b, imm in self.code:
            out += struct.pack("<BBHI", op & 0xFF, a & 0xFF, b & 0xFFFF,
                               imm & 0xFFFFFFFF)
        out += np.asarray(self.consts, dtype="<f8").tobytes()
        return bytes(out)


class Asm:
    """Tiny assembler: one method per instruction, constants interned by bit
    pattern so the pool stays small and deterministic."""

    def __init__(self, n_params: int, n_obs: int):
        self.p = Program(n_params, n_obs)
        self._cidx = {}

    def _emit(self, op, a=0, b=0, imm=0):
        self.p.code.append((op, a, b, imm))
        return self

    def const_index(self, value: float) -> int:
        key = struct.pack("<d", float(value))
        if key not in self._cidx:
            self._cidx[key] = len(self.p.consts)
            self.p.consts.append(float(value))
        return self._cidx[key]

    def push(self, value: float):
        return self._emit(PUSH, imm=self.const_index(value))

    def param(self, i: int):
        return self._emit(PARAM, imm=i)

    def obs(self, base: int, *strides: int):
        """OBS with strides for the enclosing loops, innermost first."""
        self._emit(OBS, a=len(strides), imm=base)
        for s in strides:
            self._emit(OBSX, imm=s & 0xFFFFFFFF)
        return self

    def loadl(self, j: int):
        return self._emit(LOADL, imm=j)

    def storel(self, j: int):
        return self._emit(STOREL, imm=j)

    def pack(self, rows: int, cols: int):
        return self._emit(PACK, a=rows, b=cols)

    def index(self, i: int, j: int):
        return self._emit(INDEX, a=i, b=j)

    def loop(self, n: int):
        return self._emit(LOOP, imm=n)

    def raw(self, op, a=0, b=0, imm=0):
        return self._emit(op, a, b, imm)

    def __getattr__(self, name):
        if name in _SIMPLE:
            op = _SIMPLE[name]
            return lambda: self._emit(op)
        raise AttributeError(name)

    def program(self) -> Program:
        return self.p

    def bytes(self) -> bytes:
        return self.p.to_bytes()


def parse_header(bc: bytes):
    """Return (n_params, n_obs, n_instr, n_consts) of an NDVB blob."""
    if bc[:4] != MAGIC:
        raise ValueError("not an NDVB blob")
    ver, n_params, n_obs, n_instr, n_consts = struct.unpack_from("<5I", bc, 4)
    if ver != VERSION:
        raise ValueError("unsupported NDVB version")
    return n_params, n_obs, n_instr, n_consts
