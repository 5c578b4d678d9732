"""Reference tape encoder -- TEST INFRASTRUCTURE ONLY.

An independent Python implementation of the trace producer's output format,
used to check the native trace producer byte for byte.  It walks the stack
bytecode once with *symbolic* values (slot ids and shapes, never numbers):
every numeric word appends one tape op and pushes a fresh write-once slot
(paper Section 3.4: a define-by-run tape over numeric payloads only);
structural words (locals, shuffles, loops) append nothing; a counted LOOP is
unrolled because its trip count is structural (Section 3.3: the evaluator's
control is resolved, the object program stays data).  A numeric IFLT traces
both arms and merges every stack position and local the arms left different
with one per-lane SELECT (Section 6: lane-masked divergent control); an IFLT
whose two operands are both constant slots is structural and resolves here.

Tape layout (little-endian)::

    header : b"NDVT", u32 version(=1), n_params, n_obs, n_ops, n_consts,
             n_aux, loss_slot                                   (32 bytes)
    consts : n_consts x u64  fp64 bit patterns, bytecode constants in order
             of first use
    aux    : n_aux x u32     PACK element slot lists
    ops    : n_ops x 24 B    {u16 opcode, u8 rows, u8 cols,
                              u32 a, u32 b, u32 c, u32 d, u32 imm}

Op k defines slot k.  Opcodes reuse the bytecode numbers for the numeric
words; CONST = 0x01 (imm = tape const index), PARAM = 0x02 (imm = i),
OBS = 0x03 (imm = resolved index), PACK (a = aux offset, b = count),
INDEX (a = source, imm = flattened element), SELECT = 0x40 (a < b ? c : d).
No folding, no common-subexpression elimination, unused fields zero.
"""
from __future__ import annotations

import struct

from workloads import bytecode as B

T_SELECT = 0x40
MAX_OPS = 1 << 26

UNARY = {B.NEG, B.EXP, B.LOG, B.SQRT, B.SIN, B.COS, B.ABS, B.TRANSPOSE,
         B.TRACE, B.INV, B.DET, B.LOGDET}
BINARY = {B.ADD, B.SUB, B.MUL, B.DIV, B.POW, B.DOT, B.MATMUL, B.OUTER}

E_BYTECODE = 2
E_STRUCT_DIVERGE = 3


class TapeError(Exception):
    def __init__(self, code, msg):
        super().__init__(msg)
        self.code = code


def _shape(op, sa, sb):
    (ra, ca), (rb, cb) = sa, sb if sb is not None else (None, None)
    if op in (B.ADD, B.SUB):
        if sa != sb:
            return None
        return sa
    if op == B.MUL:
        if sa == sb:
            return sa
        if sa == (1, 1):
            return sb
        if sb == (1, 1):
            return sa
        return None
    if op == B.DIV:
        if sa == sb or sb == (1, 1):
            return sa
        return None
    if op in (B.NEG, B.EXP, B.LOG, B.SQRT, B.SIN, B.COS, B.ABS):
        return sa
    if op == B.POW:
        return (1, 1) if sa == (1, 1) and sb == (1, 1) else None
    if op == B.DOT:
        return (1, 1) if sa == sb else None
    if op == B.MATMUL:
        return (ra, cb) if ca == rb else None
    if op == B.TRANSPOSE:
        return (ca, ra)
    if op == B.TRACE:
        return (1, 1) if ra == ca else None
    if op == B.INV:
        return sa if ra == ca and ra in (1, 2) else None
    if op in (B.DET, B.LOGDET):
        return (1, 1) if ra == ca and ra in (1, 2) else None
    if op == B.OUTER:
        return (ra, rb) if ca == 1 and cb == 1 else None
    return None


class _Tracer:
    def __init__(self, bc: bytes):
        try:
            self.n_params, self.n_obs, n_instr, n_consts = B.parse_header(bc)
        except ValueError as e:
            raise TapeError(E_BYTECODE, str(e))
        if len(bc) != 24 + 8 * n_instr + 8 * n_consts:
            raise TapeError(E_BYTECODE, "NDVB size mismatch")
        self.code = [struct.unpack_from("<BBHI", bc, 24 + 8 * k) for k in range(n_instr)]
        self.cbits = [struct.unpack_from("<Q", bc, 24 + 8 * n_instr + 8 * k)[0]
                      for k in range(n_consts)]
        self.cvals = [struct.unpack_from("<d", bc, 24 + 8 * n_instr + 8 * k)[0]
                      for k in range(n_consts)]
        self.match = self._match()
        self.ops = []          # (opcode, rows, cols, a, b, c, d, imm)
        self.shapes = []
        self.aux = []
        self.pool = {}         # bytecode const index -> tape const index
        self.pool_bits = []

    def _match(self):
        m, st = {}, []
        pc = 0
        while pc < len(self.code):
            op, a = self.code[pc][0], self.code[pc][1]
            if op in (B.LOOP, B.IFLT):
                st.append(pc)
            elif op == B.ELSE:
                if not st or self.code[st[-1]][0] != B.IFLT:
                    raise TapeError(E_BYTECODE, "ELSE without IFLT")
                m[st[-1]] = pc
                st[-1] = pc
            elif op == B.ENDIF:
                if not st or self.code[st[-1]][0] != B.ELSE:
                    raise TapeError(E_BYTECODE, "ENDIF without ELSE")
                m[st.pop()] = pc
            elif op == B.ENDLOOP:
                if not st or self.code[st[-1]][0] != B.LOOP:
                    raise TapeError(E_BYTECODE, "ENDLOOP without LOOP")
                m[st.pop()] = pc
            elif op == B.OBS:
                for d in range(1, a + 1):
                    if pc + d >= len(self.code) or self.code[pc + d][0] != B.OBSX:
                        raise TapeError(E_BYTECODE, "missing OBSX word")
                pc += a
            pc += 1
        if st:
            raise TapeError(E_BYTECODE, "unterminated block")
        return m

    def emit(self, opcode, shape, a=0, b=0, c=0, d=0, imm=0):
        if len(self.ops) >= MAX_OPS:
            raise TapeError(E_BYTECODE, "tape too large")
        self.ops.append((opcode, shape[0], shape[1], a, b, c, d, imm))
        self.shapes.append(shape)
        return len(self.ops) - 1

    def run(self):
        stack, loc = [], {}
        counters = []
        end = self._block(0, len(self.code), stack, loc, counters, top=True)
        return end

    def _pop(self, stack, n=1):
        if len(stack) < n:
            raise TapeError(E_BYTECODE, "stack underflow")
        out = stack[-n:]
        del stack[-n:]
        return out

    def _block(self, pc, stop, stack, loc, counters, top=False):
        """Trace words [pc, stop); returns the loss slot at HALT (top level)."""
        while pc < stop:
            op, a, b, imm = self.code[pc]
            if op == B.HALT:
                if not top:
                    raise TapeError(E_BYTECODE, "HALT inside a block")
                if len(stack) != 1 or self.shapes[stack[0]] != (1, 1):
                    raise TapeError(E_BYTECODE, "HALT needs one scalar")
                return stack[0]
            if op == B.PUSH:
                if imm >= len(self.cvals):
                    raise TapeError(E_BYTECODE, "bad const index")
                if imm not in self.pool:
                    self.pool[imm] = len(self.pool_bits)
                    self.pool_bits.append(self.cbits[imm])
                stack.append(self.emit(B.PUSH, (1, 1), imm=self.pool[imm]))
            elif op == B.PARAM:
                if imm >= self.n_params:
                    raise TapeError(E_BYTECODE, "bad param index")
                stack.append(self.emit(B.PARAM, (1, 1), imm=imm))
            elif op == B.OBS:
                if a > len(counters):
                    raise TapeError(E_BYTECODE, "OBS stride beyond loop depth")
                idx = imm
                for dd in range(a):
                    s = struct.unpack("<i", struct.pack("<I", self.code[pc + 1 + dd][3]))[0]
                    idx += s * counters[-1 - dd]
                if not 0 <= idx < self.n_obs:
                    raise TapeError(E_BYTECODE, "obs index out of range")
                stack.append(self.emit(B.OBS, (1, 1), imm=idx))
                pc += a
            elif op == B.OBSX:
                raise TapeError(E_BYTECODE, "stray OBSX word")
            elif op == B.LOADL:
                if imm not in loc:
                    raise TapeError(E_BYTECODE, "unset local")
                stack.append(loc[imm])
            elif op == B.STOREL:
                loc[imm] = self._pop(stack)[0]
            elif op == B.DUP:
                stack.append(self._pop(stack)[0])
                stack.append(stack[-1])
            elif op == B.OVER:
                x, y = self._pop(stack, 2)
                stack += [x, y, x]
            elif op == B.SWAP:
                x, y = self._pop(stack, 2)
                stack += [y, x]
            elif op == B.DROP:
                self._pop(stack)
            elif op in UNARY or op in BINARY:
                args = self._pop(stack, 2 if op in BINARY else 1)
                sh = _shape(op, self.shapes[args[0]],
                            self.shapes[args[1]] if len(args) == 2 else None)
                if sh is None:
                    raise TapeError(E_BYTECODE, "shape error")
                stack.append(self.emit(op, sh, a=args[0], b=args[1] if len(args) == 2 else 0))
            elif op == B.PACK:
                if not (1 <= a <= 4 and 1 <= b <= 4):
                    raise TapeError(E_BYTECODE, "bad PACK shape")
                els = self._pop(stack, a * b)
                if any(self.shapes[s] != (1, 1) for s in els):
                    raise TapeError(E_BYTECODE, "PACK of a non-scalar")
                off = len(self.aux)
                self.aux += els
                stack.append(self.emit(B.PACK, (a, b), a=off, b=a * b))
            elif op == B.INDEX:
                src = self._pop(stack)[0]
                r, c = self.shapes[src]
                if a >= r or b >= c:
                    raise TapeError(E_BYTECODE, "INDEX out of range")
                stack.append(self.emit(B.INDEX, (1, 1), a=src, imm=a * c + b))
            elif op == B.LOOP:
                end = self.match[pc]
                counters.append(0)
                for k in range(imm):
                    counters[-1] = k
                    self._block(pc + 1, end, stack, loc, counters)
                counters.pop()
                pc = end
            elif op == B.IFLT:
                els_pc = self.match[pc]
                end = self.match[els_pc]
                xa, xb = self._pop(stack, 2)
                if self.shapes[xa] != (1, 1) or self.shapes[xb] != (1, 1):
                    raise TapeError(E_BYTECODE, "IFLT on a non-scalar")
                if self.ops[xa][0] == B.PUSH and self.ops[xb][0] == B.PUSH:
                    va = self.cvals[self._bc_const(self.ops[xa][7])]
                    vb = self.cvals[self._bc_const(self.ops[xb][7])]
                    if va < vb:
                        self._block(pc + 1, els_pc, stack, loc, counters)
                    else:
                        self._block(els_pc + 1, end, stack, loc, counters)
                else:
                    s0, l0 = list(stack), dict(loc)
                    self._block(pc + 1, els_pc, stack, loc, counters)
                    s1, l1 = list(stack), dict(loc)
                    stack[:] = s0
                    loc.clear()
                    loc.update(l0)
                    self._block(els_pc + 1, end, stack, loc, counters)
                    s2, l2 = list(stack), dict(loc)
                    if len(s1) != len(s2):
                        raise TapeError(E_STRUCT_DIVERGE, "arms leave different stack depths")
                    merged = []
                    for x, y in zip(s1, s2):
                        if self.shapes[x] != self.shapes[y]:
                            raise TapeError(E_STRUCT_DIVERGE, "arms leave different shapes")
                        merged.append(x if x == y else
                                      self.emit(T_SELECT, self.shapes[x], a=xa, b=xb, c=x, d=y))
                    newloc = {}
                    for j in sorted(set(l1) | set(l2)):
                        if j not in l1 or j not in l2:
                            raise TapeError(E_STRUCT_DIVERGE, "local set in one arm only")
                        x, y = l1[j], l2[j]
                        if self.shapes[x] != self.shapes[y]:
                            raise TapeError(E_STRUCT_DIVERGE, "arms leave different shapes")
                        newloc[j] = x if x == y else self.emit(T_SELECT, self.shapes[x],
                                                               a=xa, b=xb, c=x, d=y)
                    stack[:] = merged
                    loc.clear()
                    loc.update(newloc)
                pc = end
            elif op in (B.ELSE, B.ENDIF, B.ENDLOOP):
                raise TapeError(E_BYTECODE, "unexpected block word")
            else:
                raise TapeError(E_BYTECODE, f"unknown opcode {op:#x}")
            pc += 1
        if top:
            raise TapeError(E_BYTECODE, "missing HALT")
        return None

    def _bc_const(self, pool_idx):
        for k, v in self.pool.items():
            if v == pool_idx:
                return k
        raise KeyError(pool_idx)


def encode(bc: bytes) -> bytes:
    """Bytecode -> tape bytes (raises TapeError with a status code)."""
    t = _Tracer(bc)
    loss = t.run()
    out = bytearray(b"NDVT")
    out += struct.pack("<7I", 1, t.n_params, t.n_obs, len(t.ops), len(t.pool_bits),
                       len(t.aux), loss)
    out += struct.pack(f"<{len(t.pool_bits)}Q", *t.pool_bits)
    out += struct.pack(f"<{len(t.aux)}I", *t.aux)
    for o in t.ops:
        out += struct.pack("<HBB5I", *o)
    return bytes(out)


def decode(tape: bytes):
    """Parse tape bytes into (header dict, consts bits, aux, ops list)."""
    if tape[:4] != b"NDVT":
        raise ValueError("not a tape")
    ver, n_params, n_obs, n_ops, n_consts, n_aux, loss = struct.unpack_from("<7I", tape, 4)
    off = 32
    consts = list(struct.unpack_from(f"<{n_consts}Q", tape, off))
    off += 8 * n_consts
    aux = list(struct.unpack_from(f"<{n_aux}I", tape, off))
    off += 4 * n_aux
    ops = [struct.unpack_from("<HBB5I", tape, off + 24 * k) for k in range(n_ops)]
    return dict(version=ver, n_params=n_params, n_obs=n_obs, n_ops=n_ops,
                n_consts=n_consts, n_aux=n_aux, loss_slot=loss), consts, aux, ops
