"""Device walker, host side (no GPU): validation and structural measurement
of stack bytecode (ndvm_walk_measure, the checks ndvm_walk_prepare applies).

The node bound must cover every node a walk can record: the tape the trace
producer builds for the same program records both arms of every branch and
one SELECT per merged value, and per parameter use a PARAM op where the
walker reuses one node per parameter, so the walker records at most
(tape ops - parameter uses + parameters) nodes; the bound is checked against
that on every benchmark program and on random programs."""
import numpy as np
import pytest

from workloads import configs
from workloads.bytecode import Asm

nd = pytest.importorskip("paper_2607_03574_amd")


def _tape_ops(bc):
    tape = nd.tape_build(bc)
    n_ops = int.from_bytes(tape[16:20], "little")
    # PARAM ops of the tape: op records follow the header, pool and aux
    n_pool = int.from_bytes(tape[20:24], "little")
    n_aux = int.from_bytes(tape[24:28], "little")
    off = 32 + 8 * n_pool + 4 * n_aux
    codes = np.frombuffer(tape[off:off + 24 * n_ops], dtype=np.uint8).reshape(n_ops, 24)[:, :2]
    code = codes[:, 0].astype(np.int64) | (codes[:, 1].astype(np.int64) << 8)
    return n_ops, int((code == 0x02).sum())


@pytest.mark.parametrize("name,kw", [("exp_decay", {}), ("logistic_euler", dict(L=4)),
                                     ("lotka_volterra_rk4", dict(L=4, T=20))])
def test_node_bound_covers_the_walk(name, kw):
    w = configs.build(name, **kw)
    info = nd.walk_measure(w.bytecode)
    n_ops, param_uses = _tape_ops(w.bytecode)
    assert info["n_nodes"] >= n_ops - param_uses + info["n_params"]
    assert info["n_nodes"] <= 2 * n_ops + 16


def test_node_bound_on_random_programs():
    w = configs.random_programs(n_prog=200, L=2, n=16, seed=5)
    for q, bc in enumerate(w.programs):
        info = nd.walk_measure(bc)
        n_ops, param_uses = _tape_ops(bc)
        assert info["n_nodes"] >= n_ops - param_uses + info["n_params"], q
        assert info["depth"] >= 1 and info["n_locals"] == 1


def test_matrix_programs_are_unsupported():
    w = configs.kalman(L=2, T=2)
    with pytest.raises(nd.NdvmError) as e:
        nd.walk_measure(w.bytecode)
    assert e.value.status == nd.E_UNSUPPORTED


@pytest.mark.parametrize("bc,status", [
    # arms leaving different depths
    (Asm(2, 0).param(0).param(1).iflt().push(1.0).push(2.0).else_().push(3.0).endif().halt().bytes(),
     "E_STRUCT_DIVERGE"),
    # a local set in one arm only
    (Asm(2, 0).param(0).param(1).iflt().push(1.0).storel(0).else_().endif().param(0).halt().bytes(),
     "E_STRUCT_DIVERGE"),
    # constant operands do not exempt the arms (the tape path would resolve this branch)
    (Asm(1, 0).push(1.0).push(2.0).iflt().param(0).param(0).else_().param(0).endif().halt().bytes(),
     "E_STRUCT_DIVERGE"),
    (Asm(1, 0).loadl(0).halt().bytes(), "E_BYTECODE"),                       # unset local
    (Asm(1, 0).param(0).add().halt().bytes(), "E_BYTECODE"),                 # underflow
    (Asm(1, 0).param(0).param(0).halt().bytes(), "E_BYTECODE"),              # HALT needs one value
    (Asm(1, 0).param(3).halt().bytes(), "E_BYTECODE"),                       # bad param index
    (Asm(1, 2).loop(3).obs(0, 1).drop().endloop().param(0).halt().bytes(), "E_BYTECODE"),   # obs 0..2 of 2
    (Asm(1, 0).param(0).halt().bytes()[:-1], "E_BYTECODE"),                  # size mismatch
])
def test_rejected_programs(bc, status):
    with pytest.raises(nd.NdvmError) as e:
        nd.walk_measure(bc)
    assert e.value.status == getattr(nd, status), nd.last_error()


def test_loops_are_measured_without_unrolling():
    # a loop body that deepens the stack: depth and nodes grow with the trips
    bc = Asm(1, 0).param(0).loop(60).push(1.0).endloop().loop(60).add().endloop().halt().bytes()
    info = nd.walk_measure(bc)
    assert info["depth"] == 61
    assert info["n_nodes"] >= 60 + 60 + 1
    with pytest.raises(nd.NdvmError):
        # deeper than the walker's operand stack limit (64)
        nd.walk_measure(Asm(1, 0).param(0).loop(70).push(1.0).endloop().loop(70).add().endloop().halt().bytes())
    info = nd.walk_measure(Asm(1, 3).push(0.0).storel(0).loop(3).loadl(0).obs(0, 1).add().storel(0).endloop()
                           .loadl(0).halt().bytes())
    assert info["n_loops"] == 1 and info["depth"] == 2 and info["n_nodes"] == 1 + 1 + 3 * 2


def test_nesting_is_measured():
    bc = (Asm(2, 0).param(0).param(1).iflt()
          .param(0).param(1).iflt().push(1.0).else_().push(2.0).endif()
          .else_().push(3.0).endif().halt().bytes())
    info = nd.walk_measure(bc)
    assert info["n_frames"] == 2 and info["n_params"] == 2
