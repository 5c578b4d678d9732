"""The allocation-free gradient entry point (ndvm_grad_noalloc), through the
C ABI: its results equal ndvm_grad's bit for bit (the same kernels, the static
scratch array instead of a caller workspace) on two calls in a row, the second
with a smaller input, and again after the array holds another program's
rows; a launch that needs more than the array is rejected before anything is
enqueued."""
import numpy as np
import pytest

from parity import compare
from workloads import configs

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

SENT = -7.25


@pytest.fixture(scope="module")
def nd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_03574_amd as m
    return m


def _call_both(nd, w, L):
    tape = nd.tape_upload(nd.tape_build(w.bytecode))
    p = torch.tensor(w.params[:L], device="cuda")
    o = torch.tensor(w.obs, device="cuda")
    need = nd.workspace_bytes(tape, L, True)            # preparation: schedules and uploads
    assert 0 < need <= nd.NOALLOC_SCRATCH_BYTES
    l0, g0 = nd.grad(tape, p, o)
    P = p.shape[1]
    l1 = torch.full((L,), SENT, dtype=torch.float64, device="cuda")
    g1 = torch.full((L, P), SENT, dtype=torch.float64, device="cuda")
    torch.cuda.synchronize()
    nd.grad_noalloc(tape, p, o, l1, g1)
    torch.cuda.synchronize()
    return tape, (l0, g0), (l1, g1)


@pytest.mark.parametrize("name,kw,L2", [("kalman_cv4", dict(L=300, T=30), 97),
                                         ("lotka_volterra_rk4", dict(L=1000, T=60), 130),
                                         ("logistic_euler", dict(L=4096), 65)])
def test_noalloc_equals_grad_two_calls(nd, oracle_mod, name, kw, L2):
    w = configs.build(name, **kw)
    L = w.params.shape[0]
    _, (l0, g0), (l1, g1) = _call_both(nd, w, L)
    assert torch.equal(l1, l0) and torch.equal(g1, g0)
    # second call in a row, smaller input (the array keeps the first call's rows)
    _, (l2, g2), (l3, g3) = _call_both(nd, w, L2)
    assert torch.equal(l3, l2) and torch.equal(g3, g2)
    ol, og, _ = oracle_mod.run(w.bytecode, w.params[:L2], w.obs)
    compare(l3.cpu().numpy(), g3.cpu().numpy(), ol, og)


def test_noalloc_rejects_launch_beyond_scratch(nd):
    """Kalman, 200 steps, 16384 lanes: about 1.9 GB of checkpoint rows."""
    w = configs.kalman(L=16384)
    tape = nd.tape_upload(nd.tape_build(w.bytecode))
    L = w.params.shape[0]
    need = nd.workspace_bytes(tape, L, True)
    assert need > nd.NOALLOC_SCRATCH_BYTES
    p = torch.tensor(w.params, device="cuda")
    o = torch.tensor(w.obs, device="cuda")
    l1 = torch.full((L,), SENT, dtype=torch.float64, device="cuda")
    g1 = torch.full((L, 12), SENT, dtype=torch.float64, device="cuda")
    with pytest.raises(nd.NdvmError) as e:
        nd.grad_noalloc(tape, p, o, l1, g1)
    assert e.value.status == nd.E_NOMEM and "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert torch.all(l1 == SENT) and torch.all(g1 == SENT)
