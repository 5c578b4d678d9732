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
