"""The reference tape encoder against hand-written expectations.

These fix the tape format (the contract the native trace producer is checked
against byte for byte): op order, slot numbering, the const pool in order of
first use with unchanged bit patterns, PACK operand lists, the placement and
operands of SELECT ops after a numeric branch, structural resolution of a
branch on two constants, and the error classes.
"""
import struct

import pytest

from oracle import tape_ref as TR
from workloads import bytecode as B
from workloads import configs
from workloads.bytecode import Asm


def ops_of(bc):
    hdr, consts, aux, ops = TR.decode(TR.encode(bc))
    return hdr, consts, aux, ops


def test_scalar_program():
    A = Asm(2, 3)
    A.param(0).push(2.5).mul().obs(1).add().push(2.5).div().halt()
    hdr, consts, aux, ops = ops_of(A.bytes())
    assert hdr["n_ops"] == 7 and hdr["loss_slot"] == 6 and hdr["n_consts"] == 1
    assert consts == [struct.unpack("<Q", struct.pack("<d", 2.5))[0]]
    assert ops == [
        (B.PARAM, 1, 1, 0, 0, 0, 0, 0),
        (B.PUSH, 1, 1, 0, 0, 0, 0, 0),
        (B.MUL, 1, 1, 0, 1, 0, 0, 0),
        (B.OBS, 1, 1, 0, 0, 0, 0, 1),
        (B.ADD, 1, 1, 2, 3, 0, 0, 0),
        (B.PUSH, 1, 1, 0, 0, 0, 0, 0),      # no CSE: a fresh slot per PUSH
        (B.DIV, 1, 1, 4, 5, 0, 0, 0),
    ]


def test_const_pool_first_use_order_and_bits():
    A = Asm(1, 0)
    A.push(1.0).push(-0.0).push(float("inf")).add().add().push(1.0).mul().halt()
    bc = A.bytes()
    hdr, consts, aux, ops = ops_of(bc)
    n_instr = struct.unpack_from("<I", bc, 16)[0]
    bc_bits = [struct.unpack_from("<Q", bc, 24 + 8 * n_instr + 8 * k)[0] for k in range(3)]
    assert consts == bc_bits
    assert [o[7] for o in ops if o[0] == B.PUSH] == [0, 1, 2, 0]


def test_pack_matmul_index():
    A = Asm(4, 0)
    A.param(0).param(1).param(2).param(3).pack(2, 2).dup().matmul().index(1, 0).halt()
    hdr, consts, aux, ops = ops_of(A.bytes())
    assert aux == [0, 1, 2, 3]
    assert ops[4] == (B.PACK, 2, 2, 0, 4, 0, 0, 0)
    assert ops[5] == (B.MATMUL, 2, 2, 4, 4, 0, 0, 0)
    assert ops[6] == (B.INDEX, 1, 1, 5, 0, 0, 0, 2)


def test_numeric_branch_emits_selects_for_stack_and_locals():
    A = Asm(3, 0)
    A.param(2).storel(0)            # local 0 = slot 0
    A.param(0).param(1).iflt()      # slots 1, 2
    A.loadl(0).exp().push(1.0)      # then: slot 3 = exp, slot 4 = const
    A.loadl(0).sin().storel(0)      # slot 5 = sin -> local 0
    A.else_()
    A.loadl(0).push(1.0)            # else: stack [slot0, slot6]; local 0 unchanged
    A.endif()
    A.add().loadl(0).add().halt()
    hdr, consts, aux, ops = ops_of(A.bytes())
    sel = [(k, o) for k, o in enumerate(ops) if o[0] == TR.T_SELECT]
    # stack position 0 (then slot 3 vs else slot 0), position 1 (4 vs 6), then local 0 (5 vs 0)
    assert [o[3:7] for _, o in sel] == [(1, 2, 3, 0), (1, 2, 4, 6), (1, 2, 5, 0)]
    assert [k for k, _ in sel] == [7, 8, 9]


def test_constant_branch_is_structural():
    A = Asm(1, 0)
    A.push(1.0).push(2.0).iflt().param(0).exp().else_().param(0).sin().endif().halt()
    hdr, consts, aux, ops = ops_of(A.bytes())
    assert [o[0] for o in ops] == [B.PUSH, B.PUSH, B.PARAM, B.EXP]
    assert not any(o[0] == TR.T_SELECT for o in ops)


def test_branch_divergence_is_an_error():
    A = Asm(1, 0)
    A.param(0).param(0).iflt().param(0).param(0).else_().param(0).endif().add().halt()
    with pytest.raises(TR.TapeError) as e:
        TR.encode(A.bytes())
    assert e.value.code == TR.E_STRUCT_DIVERGE
    A = Asm(1, 0)
    A.param(0).param(0).iflt().param(0).param(0).pack(1, 2).else_().param(0).param(0).pack(2, 1) \
        .endif().dup().dot().halt()
    with pytest.raises(TR.TapeError) as e:
        TR.encode(A.bytes())
    assert e.value.code == TR.E_STRUCT_DIVERGE


def test_loop_unrolling_and_obs_strides():
    A = Asm(1, 6)
    A.push(0.0).loop(2).loop(3).obs(0, 1, 3).add().endloop().endloop().halt()
    hdr, consts, aux, ops = ops_of(A.bytes())
    assert [o[7] for o in ops if o[0] == B.OBS] == [0, 1, 2, 3, 4, 5]
    assert hdr["n_ops"] == 1 + 6 * 2


@pytest.mark.parametrize("name,kw,expect", [
    ("exp_decay", dict(L=1), 3 + 1 + 64 * 10 + 2),
    ("logistic_euler", dict(L=1, T=500), 4 + 1 + 500 * 20),
    ("lotka_volterra_rk4", dict(L=1, T=20), 6 + 1 + 20 * 74 + 2),
])
def test_op_counts(name, kw, expect):
    w = configs.build(name, **kw)
    hdr, _, _, _ = ops_of(w.bytecode)
    assert hdr["n_ops"] == expect


def test_errors():
    for bc in (b"NOPE" + bytes(20), Asm(1, 0).param(0).loop(1).halt().bytes(),
               Asm(1, 0).add().halt().bytes(), Asm(1, 2).obs(2).halt().bytes(),
               Asm(1, 0).param(0).param(0).halt().bytes()):
        with pytest.raises(TR.TapeError) as e:
            TR.encode(bc)
        assert e.value.code == TR.E_BYTECODE
