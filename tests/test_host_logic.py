"""Host-side logic of libndvm, no GPU needed.

* the native trace producer matches the reference encoder byte for byte on
  every benchmark program (and the SHA-256 goldens written from the reference
  encoder), including error classes;
* the C-ABI library loads and exports every symbol include/ndvm.h declares;
  host-detectable argument errors are reported before any GPU work;
* the scheduler's device programs, run through the shared instruction
  handlers by the host emulator (bounds- and initialisation-checked), agree
  with the oracle at several register budgets (forcing many checkpoint
  segments) -- a check of the host logic, not a parity claim for the GPU.
"""
import ctypes
import hashlib
import json
import os
import re

import numpy as np
import pytest

import emu
from fusion_cases import fusion_programs
from conftest import ROOT, lane_rel_err, rel_err
from oracle import tape_ref
from workloads import bytecode as B
from workloads import configs
from workloads.bytecode import Asm

nd = pytest.importorskip("paper_2607_03574_amd")


def test_library_exports_every_declared_symbol():
    hdr = open(os.path.join(ROOT, "include", "ndvm.h")).read()
    declared = sorted(set(re.findall(r"\b(ndvm_\w+)\s*\(", hdr)))
    assert len(declared) >= 11
    lib = ctypes.CDLL(nd.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(nd.EXPORTS) == declared


@pytest.mark.parametrize("name", configs.ORDER[:4])
def test_tape_bit_exact_and_golden(name):
    w = configs.build(name, L=1)
    tape = nd.tape_build(w.bytecode)
    assert tape == tape_ref.encode(w.bytecode)
    gold = json.load(open(os.path.join(ROOT, "tests", "golden", "tape_sha256.json")))
    assert hashlib.sha256(tape).hexdigest() == gold[name]
    assert nd.tape_build(w.bytecode) == tape          # deterministic


def test_random_program_tapes_golden():
    w = configs.random_programs(L=1)
    h = hashlib.sha256()
    for i, bc in enumerate(w.programs):
        t = nd.tape_build(bc)
        if i < 48:
            assert t == tape_ref.encode(bc)
        h.update(t)
    gold = json.load(open(os.path.join(ROOT, "tests", "golden", "tape_sha256.json")))
    assert h.hexdigest() == gold["random_programs"]


def test_tape_constants_keep_bytecode_bit_patterns():
    A = Asm(1, 0)
    A.push(-0.0).push(float("nan")).push(5e-324).add().add().param(0).mul().halt()
    bc = A.bytes()
    hdr, consts, aux, ops = tape_ref.decode(nd.tape_build(bc))
    import struct
    n_instr = struct.unpack_from("<I", bc, 16)[0]
    want = [struct.unpack_from("<Q", bc, 24 + 8 * n_instr + 8 * k)[0] for k in range(3)]
    assert consts == want


UNIT_PROGRAMS = [
    Asm(3, 0).param(2).storel(0).param(0).param(1).iflt().loadl(0).exp().push(1.0).loadl(0).sin()
    .storel(0).else_().loadl(0).push(1.0).endif().add().loadl(0).add().halt().bytes(),
    Asm(1, 0).push(1.0).push(2.0).iflt().param(0).exp().else_().param(0).sin().endif().halt().bytes(),
    Asm(1, 6).push(0.0).loop(2).loop(3).obs(0, 1, 3).add().endloop().endloop().halt().bytes(),
    Asm(4, 0).param(0).param(1).param(2).param(3).pack(2, 2).dup().matmul().index(1, 0).halt().bytes(),
]


@pytest.mark.parametrize("k", range(len(UNIT_PROGRAMS)))
def test_unit_tapes_bit_exact(k):
    bc = UNIT_PROGRAMS[k]
    assert nd.tape_build(bc) == tape_ref.encode(bc)


@pytest.mark.parametrize("bc,code", [
    (b"NOPE" + bytes(20), nd.E_BYTECODE),
    (Asm(1, 0).param(0).loop(1).halt().bytes(), nd.E_BYTECODE),
    (Asm(1, 0).add().halt().bytes(), nd.E_BYTECODE),
    (Asm(1, 2).obs(2).halt().bytes(), nd.E_BYTECODE),
    (Asm(1, 0).param(0).param(0).halt().bytes(), nd.E_BYTECODE),
    (Asm(1, 0).param(0).param(0).iflt().param(0).param(0).else_().param(0).endif().add().halt().bytes(),
     nd.E_STRUCT_DIVERGE),
])
def test_trace_errors_match_reference(bc, code):
    with pytest.raises(nd.NdvmError) as e:
        nd.tape_build(bc)
    assert e.value.status == code
    with pytest.raises(tape_ref.TapeError) as r:
        tape_ref.encode(bc)
    assert r.value.code == code


def test_malformed_tape_rejected_before_gpu_work():
    w = configs.exp_decay(L=1, n=4)
    tape = bytearray(nd.tape_build(w.bytecode))
    for bad in (bytes(tape[:-1]), b"XXXX" + bytes(tape[4:])):
        with pytest.raises(nd.NdvmError) as e:
            nd.tape_upload(bad, stream=0)
        assert e.value.status == nd.E_TAPE
    # forward reference in an op record
    hdr, consts, aux, ops = tape_ref.decode(bytes(tape))
    off = 32 + 8 * hdr["n_consts"] + 4 * hdr["n_aux"] + 24 * (len(ops) - 1) + 4
    t2 = bytearray(tape)
    t2[off:off + 4] = (len(ops) + 5).to_bytes(4, "little")
    with pytest.raises(nd.NdvmError) as e:
        nd.tape_upload(bytes(t2), stream=0)
    assert e.value.status == nd.E_TAPE
    with pytest.raises(nd.NdvmError) as e:
        nd.tape_upload(bytes(tape), policy=99, stream=0)
    assert e.value.status == nd.E_UNSUPPORTED


def test_batch_upload_rejects_a_malformed_tape_before_gpu_work():
    # the first failing tape is named; no handle is returned; the batch is
    # validated on the host before anything is copied to the device
    good = nd.tape_build(configs.exp_decay(L=1, n=4).bytecode)
    bad = good[:-1]
    with pytest.raises(nd.NdvmError) as e:
        nd.tape_upload_many([good, good, bad, good, bad], stream=0)
    assert e.value.status == nd.E_TAPE
    assert "tape 2" in str(e.value)
    assert nd.tape_upload_many([], stream=0) == []
    lib = ctypes.CDLL(nd.LIB_PATH)
    assert lib.ndvm_tape_upload_many(None, None, -1, 0, None, None) == nd.E_ARG
    assert lib.ndvm_tape_upload_many(None, None, 1, 0, None, None) == nd.E_ARG
    arr = (ctypes.c_char_p * 1)(good)
    lens = (ctypes.c_size_t * 1)(len(good))
    out = (ctypes.c_void_p * 1)()
    assert lib.ndvm_tape_upload_many(arr, lens, 1, 77, None, out) == nd.E_UNSUPPORTED


CASES = [("exp_decay", dict(L=9)), ("logistic_euler", dict(L=9, T=60)),
         ("lotka_volterra_rk4", dict(L=9, T=25)), ("kalman_cv4", dict(L=9, T=12))]


@pytest.mark.parametrize("name,kw", CASES)
@pytest.mark.parametrize("budget", [320, 48, 12])
def test_emulated_programs_match_oracle(oracle_mod, name, kw, budget):
    w = configs.build(name, **kw)
    tape = nd.tape_build(w.bytecode)
    lo, go, _ = oracle_mod.run(w.bytecode, w.params, w.obs)
    le, ge, st = emu.run(tape, w.params, w.obs, True, budget)
    lf, _, _ = emu.run(tape, w.params, w.obs, False, budget)
    assert rel_err(le, lo).max() <= 1e-13
    assert rel_err(lf, lo).max() <= 1e-13
    assert lane_rel_err(ge, go).max() <= 1e-13
    if budget < 100 and name != "exp_decay":
        assert st["n_segments"] > 1


@pytest.mark.parametrize("name,kw", CASES)
@pytest.mark.parametrize("budget", [320, 48])
def test_emulated_save_policy_equals_recompute(oracle_mod, name, kw, budget):
    """The save policy (every value an adjoint rule reads stored, nothing
    recomputed) gives the recompute policy's bits, and recomputes nothing."""
    w = configs.build(name, **kw)
    tape = nd.tape_build(w.bytecode)
    lr, gr, _ = emu.run(tape, w.params, w.obs, True, budget)
    ls, gs, st = emu.run(tape, w.params, w.obs, True, budget, save=True)
    assert lr.tobytes() == ls.tobytes() and gr.tobytes() == gs.tobytes()
    assert st["recompute_ops"] <= st["fwd_ops"] // 10 + 64   # observation reloads only
    lo, go, _ = oracle_mod.run(w.bytecode, w.params, w.obs)
    assert lane_rel_err(gs, go).max() <= 1e-13


def test_emulated_random_programs_match_oracle(oracle_mod):
    w = configs.random_programs(n_prog=24, L=8, n=8, seed=99)
    for i, bc in enumerate(w.programs):
        P = w.n_params_each[i]
        p = w.params[i][:, :P]
        lo, go, m = oracle_mod.run(bc, p, w.obs, margin=True)
        le, ge, _ = emu.run(nd.tape_build(bc), p, w.obs, True, 24)
        ok = m > 1e-9
        assert rel_err(le[ok], lo[ok]).max(initial=0) <= 1e-13
        assert lane_rel_err(ge[ok], go[ok]).max(initial=0) <= 1e-12


@pytest.mark.parametrize("seed", [3, 8])
def test_emulated_branch_skipping_is_exact(oracle_mod, seed):
    """Branch arms behind skip tests: every lane skips the arms it does not
    take (the most skipping any wave could do); every value a skipped arm
    would form is NaN for that lane.  Results must equal, bit for bit, the
    run of both arms and the program without skip tests, at two register
    budgets and under both policies, and the oracle wherever no branch is
    near a tie."""
    w = configs.random_programs(n_prog=120, L=16, n=8, seed=seed)
    n_arms = 0
    for i, bc in enumerate(w.programs):
        P = w.n_params_each[i]
        p = np.ascontiguousarray(w.params[i][:, :P])
        tape = nd.tape_build(bc)
        lo, go, m = oracle_mod.run(bc, p, w.obs, margin=True)
        ok = m > 1e-9
        for budget in (320, 24):
            for save in (False, True):
                la, ga, _ = emu.run(tape, p, w.obs, True, budget, save=save, arms="all", skip=False)
                lb, gb, st = emu.run(tape, p, w.obs, True, budget, save=save, arms="all", skip=True)
                lc, gc, _ = emu.run(tape, p, w.obs, True, budget, save=save)
                np.testing.assert_array_equal(lc, la, err_msg=f"program {i} budget {budget} save {save}")
                np.testing.assert_array_equal(gc, ga, err_msg=f"program {i} budget {budget} save {save}")
                np.testing.assert_array_equal(lb, la, err_msg=f"program {i} budget {budget} save {save}")
                np.testing.assert_array_equal(gb, ga, err_msg=f"program {i} budget {budget} save {save}")
                assert rel_err(lb[ok], lo[ok]).max(initial=0) <= 1e-13
                assert lane_rel_err(gb[ok], go[ok]).max(initial=0) <= 1e-12
                n_arms += st["n_skips"]
    assert n_arms > 0


@pytest.mark.parametrize("tree", [
    ("iflt", ("x",), ("x",), ("c", 0), ("iflt", ("x",), ("x",), ("x",), ("c", 1))),
    ("iflt", ("x",), ("c", 2), ("c", 0), ("iflt", ("x",), ("c", 2), ("c", 3), ("c", 1))),
    ("iflt", ("x",), ("c", 2), ("iflt", ("x",), ("c", 2), ("c", 3), ("c", 1)), ("c", 0)),
    ("iflt", ("x",), ("x",), ("sub", ("c", 0), ("x",)), ("iflt", ("x",), ("x",), ("x",), ("c", 1))),
    ("mul", ("iflt", ("c", 0), ("c", 1), ("pdiv", ("c", 2), ("c", 3)), ("c", 4)),
     ("iflt", ("c", 0), ("c", 1), ("pdiv", ("c", 2), ("c", 3)), ("x",))),
])
def test_emulated_nested_and_repeated_branches(oracle_mod, tree):
    """A select reading another select of the same predicate, a branch whose
    arm values recur after it (duplicates), exact ties: skipping and not
    skipping agree bit for bit and with the oracle."""
    from workloads import randtree
    nc = randtree.n_consts(tree)
    rng = np.random.default_rng(7)
    n = 8
    obs = np.concatenate([rng.uniform(-2, 2, n), rng.uniform(-1, 1, n)])
    p = rng.uniform(-2, 2, (16, nc))
    bc = configs.tree_program(tree, nc, n)
    lo, go, _ = oracle_mod.run(bc, p, obs)
    for budget in (320, 12):
        for save in (False, True):
            for skip in (False, True):
                le, ge, _ = emu.run(nd.tape_build(bc), p, obs, True, budget, save=save, arms="all", skip=skip)
                assert rel_err(le, lo).max() <= 1e-13, (budget, save, skip)
                assert lane_rel_err(ge, go).max() <= 1e-12, (budget, save, skip)


@pytest.mark.parametrize("case", range(len(configs.BRANCH_TREES)))
def test_branch_population_programs_have_skippable_arms(oracle_mod, case):
    """The programs the GPU skipping tests and the skipping study run have
    arms the BRANCH_SKIP option marks; ordered and interleaved lanes, with
    per-lane skipping, give the oracle's results."""
    for order in ("sorted", "mixed", "all_then", "all_else"):
        w = configs.branch_population(case, L=64, n=8, order=order)
        tape = nd.tape_build(w.bytecode)
        lo, go, _ = oracle_mod.run(w.bytecode, w.params, w.obs)
        for save in (False, True):
            le, ge, st = emu.run(tape, w.params, w.obs, True, 320, save=save, arms="option")
            assert st["n_skips"] > 0
            assert rel_err(le, lo).max() <= 1e-13
            assert lane_rel_err(ge, go).max() <= 1e-12


def test_emulated_edge_programs(oracle_mod):
    progs = [
        (Asm(3, 0).param(0).param(1).iflt().push(1000.0).param(2).mul().exp().else_().push(2.0)
         .param(2).mul().endif().halt().bytes(),
         [[1.0, 1.0, 5.0], [np.nan, 1.0, 5.0], [0.5, 1.0, 0.001], [2.0, 1.0, 5.0]]),
        (Asm(1, 0).param(0).log().halt().bytes(), [[1e-9], [-1.0], [1e-8], [2e-8]]),
        (Asm(1, 0).param(0).sqrt().halt().bytes(), [[1e-9], [4.0]]),
        (Asm(1, 0).param(0).abs().halt().bytes(), [[0.0], [-2.0], [3.0]]),
        (Asm(2, 0).param(1).halt().bytes(), [[3.0, 4.0]]),
        (Asm(2, 0).push(2.5).halt().bytes(), [[3.0, 4.0]]),
    ]
    for bc, params in progs:
        lo, go, _ = oracle_mod.run(bc, params, [])
        le, ge, _ = emu.run(nd.tape_build(bc), params, [], True, 8)
        np.testing.assert_array_equal(le, lo)
        np.testing.assert_array_equal(ge, go)


def test_schedule_is_deterministic():
    w = configs.lotka_volterra(L=3, T=15)
    tape = nd.tape_build(w.bytecode)
    a = emu.run(tape, w.params, w.obs, True, 40)
    b = emu.run(tape, w.params, w.obs, True, 40)
    assert a[0].tobytes() == b[0].tobytes() and a[1].tobytes() == b[1].tobytes() and a[2] == b[2]


def test_emulated_wide_program_beyond_packed_register_fields(oracle_mod):
    # 17000 parameters put the register file far past any LDS budget (the
    # tail spills to workspace rows) and register byte offsets past 16 bits;
    # the gradient of sum_i p_i p_(i+1) is p_(i-1) + p_(i+1)
    P = 17000
    A = Asm(P, 0)
    A.param(0).param(1).mul()
    for i in range(1, P - 1):
        A.param(i).param(i + 1).mul().add()
    bc = A.halt().bytes()
    rng = np.random.default_rng(5)
    params = rng.uniform(-1, 1, (2, P))
    le, ge, st = emu.run(nd.tape_build(bc), params, [], True, 320)
    lo, go, _ = oracle_mod.run(bc, params, [])
    assert st["n_regs"] > 2 ** 15
    np.testing.assert_allclose(le, lo, rtol=1e-12)
    want = np.zeros_like(params)
    want[:, :-1] += params[:, 1:]
    want[:, 1:] += params[:, :-1]
    np.testing.assert_array_equal(ge, go)
    np.testing.assert_allclose(ge, want, rtol=0, atol=0)


# form numbers of the device program format (slot.h)
HOT_FORMS = set(range(1, 32))
COLD_FORMS = {40, 41, 42, 43}
END = 63
INDEX_X = {25, 26, 27, 28, 29, 43}      # LDOBS LDPARAM LDCONST CKST CKLD STGRAD
NO_A = {28, 42, 43}                     # CKST STLOSS STGRAD (register a is read)


@pytest.mark.parametrize("name,kw", CASES)
def test_device_program_encoding(name, kw):
    """The encoded program: known forms only, END once followed by END padding,
    register fields as byte offsets of whole 16-lane registers inside the
    register file, slot flags only where a slot exists, and the one-hot
    dispatch bits (10: MAC, 11: ACC, 12: MSUB, 13: DOTB or DOTBACC) set
    exactly on their forms (the kernel dispatches on these bits alone)."""
    w = configs.build(name, **kw)
    tape = nd.tape_build(w.bytecode)
    budget = 48
    _, _, st = emu.run(tape, w.params[:1], w.obs, True, budget)
    headers, words = emu.program(tape, True, budget)
    forms = headers & 63
    n = int(np.argmax(forms == END)) + 1
    assert n == st["n_instr"]
    assert set(forms[n:len(words)].tolist()) <= {END}
    assert set(forms[:n].tolist()) <= HOT_FORMS | COLD_FORMS | {END}
    bit = lambda b: ((headers[:n] >> b) & 1).astype(bool)
    np.testing.assert_array_equal(bit(10), forms[:n] == 1)
    np.testing.assert_array_equal(bit(11), forms[:n] == 2)
    np.testing.assert_array_equal(bit(12), forms[:n] == 30)
    np.testing.assert_array_equal(bit(13), (forms[:n] == 18) | (forms[:n] == 19))
    stride = 16 * 8
    for k in range(n - 1):
        f = int(forms[k])
        regs = words[k, :, 0:1] if f in INDEX_X else words[k, :, [0, 2, 3]].T
        if f in (1, 2, 3, 4, 5, 6, 30, 31):   # every field of these forms names a register
            regs = words[k]
        assert (regs % stride == 0).all(), (k, f)
        assert (regs // stride < st["n_regs"] + 8).all(), (k, f)
    # all four slots of every executed instruction carry a micro-op
    assert st["n_uops"] <= 4 * st["n_instr"]


def test_bench_traffic_only_for_matching_kernel_sources(tmp_path, monkeypatch):
    import bench
    sha = bench.kernel_sources_sha256()
    (tmp_path / "ndvm_replay_logistic_euler_L4096.md").write_text(
        f"text\n\n    traffic_bytes_per_launch: 12345\n    kernel_sources_sha256: {sha}\n")
    (tmp_path / "ndvm_replay_kalman_cv4_L16384.md").write_text(
        "    traffic_bytes_per_launch: 999\n    kernel_sources_sha256: " + "0" * 64 + "\n")
    (tmp_path / "ndvm_replay_logistic_euler_L4096_save.md").write_text(
        f"    policy: save\n    traffic_bytes_per_launch: 777\n    kernel_sources_sha256: {sha}\n")
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.profiled_traffic("logistic_euler") == 12345.0
    assert bench.profiled_traffic("logistic_euler", "save") == 777.0
    assert bench.profiled_traffic("kalman_cv4") is None      # counters of another kernel build
    assert bench.profiled_traffic("exp_decay") is None       # no summary


def test_emulated_product_folding_is_bit_exact(oracle_mod):
    rng = np.random.default_rng(21)
    for bc, P, must in fusion_programs():
        params = rng.uniform(-2, 2, (6, P))
        params[0, :] = 0.0                      # signed zeros: +0 * +0 - +0
        params[1, :] = -0.0
        lo, go, _ = oracle_mod.run(bc, params, [])
        tape = nd.tape_build(bc)
        for budget in (320, 8):
            le, ge, _ = emu.run(tape, params, [], True, budget)
            np.testing.assert_array_equal(le, lo)
            np.testing.assert_array_equal(ge, go)
        headers, _ = emu.program(tape, True, 320)
        forms = set((headers & 63).tolist())
        assert must <= forms, (must, forms)
