"""GPU parity of the flattened data axis (ndvm_grad_points) against its oracle
(oracle/flatten.py), through the C ABI.

Every per-point term and term gradient the replay writes (read back from the
workspace) is judged against the per-lane oracle on that point (tests/parity.py
rules), and the fold is checked bit for bit against a sequential ascending
fold of those GPU terms; the final loss and gradient are compared with the
flattened oracle.  Exponential decay at its benchmark size (256 x 64), one
tree program at its benchmark size (1024 x 128), ragged shapes, error paths.
"""
import numpy as np
import pytest

from parity import compare, judge
from workloads import configs

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def nd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_03574_amd as m
    return m


def run_points(nd, term_bc, params, points, scale):
    tape = nd.tape_upload(nd.tape_build(term_bc))
    p = torch.tensor(np.ascontiguousarray(params), device="cuda")
    pts = torch.tensor(np.ascontiguousarray(points), device="cuda")
    L, P = p.shape
    N = pts.shape[0]
    need = nd.workspace_bytes_points(tape, L, N)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    loss, grad = nd.grad_points(tape, p, pts, scale, workspace=ws)
    torch.cuda.synchronize()
    wsd = ws.view(torch.float64)
    F = L * N
    terms = wsd[need // 8 - F * (1 + P): need // 8 - F * P].cpu().numpy().reshape(L, N)
    tgrad = wsd[need // 8 - F * P:].cpu().numpy().reshape(L, N, P)
    return loss.cpu().numpy(), grad.cpu().numpy(), terms, tgrad


def check(nd, oracle_mod, term_bc, params, points, scale):
    from oracle import flatten
    gl, gg, terms, tgrad = run_points(nd, term_bc, params, points, scale)
    L, N = terms.shape
    tot = dict(n_lanes=0, n_strict=0, n_ill_conditioned=0, n_libm_sensitive=0, n_other_arm=0)
    for i in range(N):
        r = judge(oracle_mod, term_bc, params, points[i], terms[:, i], tgrad[:, i, :])
        for k in tot:
            tot[k] += r[k]
    # the fold, bit for bit, from the GPU's own terms
    acc = np.zeros(L)
    accg = np.zeros_like(gg)
    for i in range(N):
        acc = acc + terms[:, i]
        accg = accg + tgrad[:, i, :]
    np.testing.assert_array_equal(gl, acc * scale)
    np.testing.assert_array_equal(gg, accg * scale)
    if tot["n_strict"] == tot["n_lanes"]:
        ol, og = flatten.run_points(term_bc, params, points, scale)
        compare(gl, gg, ol, og)
    return tot


def test_exp_decay_full_size(nd, oracle_mod):
    w = configs.exp_decay()
    n = 64
    pts = configs.points_of(w.obs, n)
    tot = check(nd, oracle_mod, configs.exp_decay_term_program(), w.params, pts, 1.0 / n)
    assert tot["n_lanes"] == 256 * 64
    # the flattened loss equals the unflattened replay's within the bar
    tape = nd.tape_upload(nd.tape_build(w.bytecode))
    lu, _ = nd.grad(tape, torch.tensor(w.params, device="cuda"), torch.tensor(w.obs, device="cuda"))
    gl, _, _, _ = run_points(nd, configs.exp_decay_term_program(), w.params, pts, 1.0 / n)
    compare(gl, None, lu.cpu().numpy(), None)


@pytest.mark.parametrize("q", [0, 437])
def test_tree_program_full_size(nd, oracle_mod, q):
    w = configs.random_programs()
    P = w.n_params_each[q]
    term = configs.tree_term_program(w.meta["trees"][q], P)
    pts = configs.points_of(w.obs, 128)
    tot = check(nd, oracle_mod, term, w.params[q][:, :P], pts, 1.0 / 128)
    assert tot["n_lanes"] == 1024 * 128
    assert tot["n_other_arm"] <= tot["n_lanes"] // 50


@pytest.mark.parametrize("L,N", [(1, 1), (1, 64), (37, 13), (65, 2), (3, 200)])
def test_ragged_shapes(nd, oracle_mod, L, N):
    w = configs.exp_decay(L=L, n=N)
    pts = configs.points_of(w.obs, N)
    check(nd, oracle_mod, configs.exp_decay_term_program(), w.params, pts, 1.0 / N)


def test_points_argument_errors(nd):
    term = configs.exp_decay_term_program()
    tape = nd.tape_upload(nd.tape_build(term))
    L, N = 20, 10
    p = torch.ones((L, 3), dtype=torch.float64, device="cuda")
    pts = torch.ones((N, 2), dtype=torch.float64, device="cuda")
    loss = torch.full((L,), 5.5, dtype=torch.float64, device="cuda")
    g = torch.full((L, 3), 5.5, dtype=torch.float64, device="cuda")
    need = nd.workspace_bytes_points(tape, L, N)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    base = [tape.handle, p.data_ptr(), L, 3, pts.data_ptr(), N, 2, 0.1, loss.data_ptr(), g.data_ptr(), 3,
            ws.data_ptr(), need, s]

    def call(**kw):
        a = list(base)
        for k, v in kw.items():
            a[int(k[1:])] = v
        return nd._grad_points(*a)

    for what, kw, want in [("null tape", dict(a0=None), nd.E_ARG), ("null params", dict(a1=None), nd.E_ARG),
                           ("negative L", dict(a2=-1), nd.E_ARG), ("ld_p < P", dict(a3=2), nd.E_ARG),
                           ("null points", dict(a4=None), nd.E_ARG), ("no points", dict(a5=0), nd.E_ARG),
                           ("ld_pt < D", dict(a6=1), nd.E_ARG), ("null loss", dict(a8=None), nd.E_ARG),
                           ("null grad", dict(a9=None), nd.E_ARG), ("ld_g < P", dict(a10=2), nd.E_ARG),
                           ("workspace too small", dict(a12=need - 8), nd.E_NOMEM),
                           ("point count never prepared", dict(a5=N * 4096 * 64, a12=0), nd.E_ARG)]:
        st = call(**kw)
        assert st == want, (what, st, nd.last_error())
    torch.cuda.synchronize()
    assert torch.all(loss == 5.5) and torch.all(g == 5.5)
    assert call() == nd.OK
