"""The two save policies on the GPU (Section 3.4: the reverse sweep reads the
payloads the forward sweep produced; NDVM_POLICY_SAVE stores every value an
adjoint rule reads, NDVM_POLICY_RECOMPUTE stores segment inputs and
recomputes).  A recomputed value is the same operations on the same inputs
as the stored one, so both policies give the same bits; the save policy is
also judged against the oracle at full size."""
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


def run(nd, bc, params, obs, policy):
    tape = nd.tape_upload(nd.tape_build(bc), policy=policy)
    loss, g = nd.grad(tape, torch.tensor(np.ascontiguousarray(params), device="cuda"),
                      torch.tensor(obs, device="cuda"))
    torch.cuda.synchronize()
    return loss.cpu().numpy(), g.cpu().numpy()


CASES = [("exp_decay", dict()), ("logistic_euler", dict(L=300)), ("lotka_volterra_rk4", dict(L=130)),
         ("kalman_cv4", dict(L=200)), ("kalman_cv4", dict(L=16384)), ("lotka_volterra_rk4", dict(L=65536))]


@pytest.mark.parametrize("name,kw", CASES)
def test_policies_bit_identical(nd, name, kw):
    w = configs.build(name, **kw)
    a = run(nd, w.bytecode, w.params, w.obs, nd.POLICY_RECOMPUTE)
    b = run(nd, w.bytecode, w.params, w.obs, nd.POLICY_SAVE)
    assert a[0].tobytes() == b[0].tobytes() and a[1].tobytes() == b[1].tobytes()


@pytest.mark.parametrize("name", ["kalman_cv4", "logistic_euler"])
def test_save_policy_full_size_vs_oracle(nd, oracle_mod, name):
    w = configs.build(name)
    gl, gg = run(nd, w.bytecode, w.params, w.obs, nd.POLICY_SAVE)
    r = judge(oracle_mod, w.bytecode, w.params, w.obs, gl, gg)
    record(f"save_policy_full_size[{name}]", workload=name, L=int(w.params.shape[0]), **r)
    assert r["n_strict"] == r["n_lanes"]


def test_save_policy_random_programs(nd, oracle_mod):
    w = configs.random_programs(n_prog=24, L=100, n=128, seed=77)
    tr = [nd.tape_upload(nd.tape_build(bc), policy=nd.POLICY_RECOMPUTE) for bc in w.programs]
    ts = [nd.tape_upload(nd.tape_build(bc), policy=nd.POLICY_SAVE) for bc in w.programs]
    p = torch.tensor(w.params, device="cuda")
    o = torch.tensor(w.obs, device="cuda")
    l1, g1 = nd.grad_many(tr, p, o)
    l2, g2 = nd.grad_many(ts, p, o)
    torch.cuda.synchronize()
    assert torch.equal(l1, l2) and torch.equal(g1, g2)
    for q, bc in enumerate(w.programs):
        P = w.n_params_each[q]
        judge(oracle_mod, bc, w.params[q][:, :P], w.obs, l2[q].cpu().numpy(), g2[q, :, :P].cpu().numpy())
