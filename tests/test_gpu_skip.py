"""GPU: numeric branches whose arms a wave skips when all of its lanes decide
the branch the other way (the BRANCH_SKIP option: one ballot per arm,
Section 6 lane masking taken per wave).  A lane's result must not depend on
its wave neighbours: the same lanes are run ordered by the branch's
predicate (waves decide alike and skip arms) and interleaved (waves are mixed
and run both arms), under both save policies, and without the option; all
results must agree bit for bit and pass the oracle's parity rules.  Lanes
that all take one arm (every wave skips the other) must equal the run
without the option bit for bit."""
import numpy as np
import pytest

from conftest import record
from parity import judge
from workloads import configs

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def nd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_03574_amd as m
    return m


def _run(nd, w, policy):
    tape = nd.tape_upload(nd.tape_build(w.bytecode), policy)
    p = torch.tensor(w.params, device="cuda")
    o = torch.tensor(w.obs, device="cuda")
    loss, g = nd.grad(tape, p, o)
    torch.cuda.synchronize()
    # back to the order of the unordered draw
    order = w.meta["order"]
    gl = np.empty_like(loss.cpu().numpy())
    gg = np.empty_like(g.cpu().numpy())
    gl[order] = loss.cpu().numpy()
    gg[order] = g.cpu().numpy()
    return gl, gg


@pytest.mark.parametrize("case", range(len(configs.BRANCH_TREES)))
def test_lane_results_independent_of_wave_neighbours(nd, oracle_mod, case):
    L, n = 1024, 16
    skip = nd.POLICY_RECOMPUTE | nd.BRANCH_SKIP
    runs = {}
    for name, order, policy in (("sorted", "sorted", skip), ("mixed", "mixed", skip),
                                ("plain", "sorted", nd.POLICY_RECOMPUTE),
                                ("save", "mixed", nd.POLICY_SAVE | nd.BRANCH_SKIP)):
        w = configs.branch_population(case, L=L, n=n, order=order)
        runs[name] = _run(nd, w, policy)
    for other in ("mixed", "plain", "save"):
        np.testing.assert_array_equal(runs["sorted"][0], runs[other][0], err_msg=other)
        np.testing.assert_array_equal(runs["sorted"][1], runs[other][1], err_msg=other)
    # every lane (so every wave) takes one arm: the other arm is skipped
    # throughout, in both sweeps
    for order in ("all_then", "all_else"):
        w = configs.branch_population(case, L=L, n=n, order=order)
        a = _run(nd, w, skip)
        b = _run(nd, w, nd.POLICY_RECOMPUTE)
        np.testing.assert_array_equal(a[0], b[0], err_msg=order)
        np.testing.assert_array_equal(a[1], b[1], err_msg=order)
        r = judge(oracle_mod, w.bytecode, w.params, w.obs, a[0], a[1])
        record("skip_uniform_population", case=case, order=order, **r)
    w = configs.branch_population(case, L=L, n=n, order="sorted")
    p = np.empty_like(w.params)
    p[w.meta["order"]] = w.params
    r = judge(oracle_mod, w.bytecode, p, w.obs, runs["sorted"][0], runs["sorted"][1])
    record("skip_wave_neighbours", case=case, **r)


def test_random_programs_with_skipping_equal_without(nd):
    """The random-program population (1,024 programs of 1,024 lanes, one
    launch) uploaded with the option gives, bit for bit, the results of the
    uploads without it (those are judged against the oracle program by
    program in the full-size parity test)."""
    w = configs.random_programs()
    p = torch.tensor(w.params, device="cuda")
    o = torch.tensor(w.obs, device="cuda")
    out = []
    for policy in (nd.POLICY_RECOMPUTE, nd.POLICY_RECOMPUTE | nd.BRANCH_SKIP):
        tapes = [nd.tape_upload(nd.tape_build(bc), policy) for bc in w.programs]
        loss, grad = nd.grad_many(tapes, p, o)
        torch.cuda.synchronize()
        out.append((loss.cpu().numpy(), grad.cpu().numpy()))
        del tapes
    np.testing.assert_array_equal(out[0][0], out[1][0])
    np.testing.assert_array_equal(out[0][1], out[1][1])


def _ode_with_branch_program(T, h=0.02):
    """Lotka-Volterra RK4 MSE (as the workload) whose loss is reshaped after
    the loop by a numeric branch on alpha (one of two chains of six
    multiply-adds): a reverse-sweep-dominated program with skippable arms."""
    from workloads.bytecode import Asm
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
    A.loadl(AL).push(1.0).iflt()
    for _ in range(6):
        A.loadl(ACC).loadl(ACC).loadl(X).mul().push(1e-3).mul().add().storel(ACC)
    A.else_()
    for _ in range(6):
        A.loadl(ACC).loadl(ACC).loadl(Y).mul().push(2e-3).mul().add().storel(ACC)
    A.endif()
    A.loadl(ACC).push(1.0 / (2.0 * T)).mul().halt()
    return A.bytes()


def test_skipping_under_the_adjoint_first_dispatch(nd, oracle_mod):
    """A program whose instructions are led by the linear adjoint rule, with
    frequent multiply-subtracts and a skippable branch, runs the replay
    variant that tests the adjoint rule first and skips arms; lanes sorted by
    the branch's predicate (waves skip an arm) and interleaved give the same
    results bit for bit as the upload without skipping, and pass the
    oracle's parity rules.  At 16,384 lanes (four waves per CU on a 256-CU
    GPU) the launch budget is 320 registers; the mix holds from 80 to 640
    (at 1,280, a one-wave-per-CU budget, multiply-adds lead)."""
    import emu
    T, L = 40, 16384
    bc = _ode_with_branch_program(T)
    tape = nd.tape_build(bc)
    for budget in (80, 160, 320, 640):
        headers, _ = emu.program(tape, True, budget, arms="option")
        forms = headers & 63
        n = int(np.argmax(forms == 63)) + 1
        n_mac, n_acc, n_msub = (int(np.sum(forms[:n] == f)) for f in (1, 2, 30))
        assert n_acc > n_mac and 16 * n_msub >= n, (budget, n, n_mac, n_acc, n_msub)
        assert np.sum(forms[:n] == 32) > 0
    rng = np.random.default_rng(7007)
    truth = np.array([1.0, 0.5, 1.0, 0.5, 1.0, 0.5])
    obs = (configs.lv_truth_path(truth, T) + rng.normal(0.0, 0.05, (T, 2))).reshape(-1).copy()
    params = truth[None, :] * rng.uniform(0.5, 1.5, size=(L, 6))
    order = np.argsort(params[:, 0], kind="stable")
    o = torch.tensor(obs, device="cuda")
    out = {}
    for name, p_host, policy in (("sorted", params[order], nd.POLICY_RECOMPUTE | nd.BRANCH_SKIP),
                                 ("sorted_plain", params[order], nd.POLICY_RECOMPUTE),
                                 ("mixed", params, nd.POLICY_RECOMPUTE | nd.BRANCH_SKIP)):
        t = nd.tape_upload(tape, policy)
        loss, g = nd.grad(t, torch.tensor(np.ascontiguousarray(p_host), device="cuda"), o)
        torch.cuda.synchronize()
        out[name] = (loss.cpu().numpy(), g.cpu().numpy())
    np.testing.assert_array_equal(out["sorted"][0], out["sorted_plain"][0])
    np.testing.assert_array_equal(out["sorted"][1], out["sorted_plain"][1])
    inv = np.empty_like(order)
    inv[order] = np.arange(L)
    np.testing.assert_array_equal(out["sorted"][0][inv], out["mixed"][0])
    np.testing.assert_array_equal(out["sorted"][1][inv], out["mixed"][1])
    r = judge(oracle_mod, bc, params, obs, out["mixed"][0], out["mixed"][1])
    record("skip_adjoint_first", **r)


def test_skipping_under_the_block_dispatch(nd, oracle_mod):
    """The Kalman filter with a branch on dt after its loop: a program whose
    instructions are a quarter block dots runs the replay variant that tests
    multiply-add and the block dots first and skips arms; lanes sorted by dt
    (waves skip an arm) and interleaved give the same results bit for bit as
    the upload without skipping, and pass the oracle's parity rules (the mix
    holds at budgets 160 to 640 registers; 16,384 lanes give 320 on a 256-CU
    GPU)."""
    import emu
    T, L = 40, 16384
    bc = configs.kalman_program(T, branch_tail=True)
    tape = nd.tape_build(bc)
    for budget in (160, 320, 640):
        headers, _ = emu.program(tape, True, budget, arms="option")
        forms = headers & 63
        n = int(np.argmax(forms == 63)) + 1
        n_mac, n_acc = int(np.sum(forms[:n] == 1)), int(np.sum(forms[:n] == 2))
        n_block = int(np.sum((forms[:n] == 18) | (forms[:n] == 19)))
        assert 4 * n_block >= n and n_mac >= n_acc, (budget, n, n_mac, n_acc, n_block)
        assert np.sum(forms[:n] == 32) > 0
    w = configs.kalman(L=L, T=T)
    params, obs = w.params, w.obs
    order = np.argsort(params[:, 0], kind="stable")
    o = torch.tensor(obs, device="cuda")
    out = {}
    for name, p_host, policy in (("sorted", params[order], nd.POLICY_RECOMPUTE | nd.BRANCH_SKIP),
                                 ("sorted_plain", params[order], nd.POLICY_RECOMPUTE),
                                 ("mixed", params, nd.POLICY_RECOMPUTE | nd.BRANCH_SKIP)):
        t = nd.tape_upload(tape, policy)
        loss, g = nd.grad(t, torch.tensor(np.ascontiguousarray(p_host), device="cuda"), o)
        torch.cuda.synchronize()
        out[name] = (loss.cpu().numpy(), g.cpu().numpy())
    np.testing.assert_array_equal(out["sorted"][0], out["sorted_plain"][0])
    np.testing.assert_array_equal(out["sorted"][1], out["sorted_plain"][1])
    inv = np.empty_like(order)
    inv[order] = np.arange(L)
    np.testing.assert_array_equal(out["sorted"][0][inv], out["mixed"][0])
    np.testing.assert_array_equal(out["sorted"][1][inv], out["mixed"][1])
    r = judge(oracle_mod, bc, params, obs, out["mixed"][0], out["mixed"][1])
    record("skip_block_dispatch", **r)
