"""The C ABI's error paths and stream behaviour, on the GPU, through the raw
ctypes entry points (no binding-side checks in between).

Every argument error of ndvm_forward / ndvm_grad / ndvm_grad_many is reported
synchronously with its status (NDVM_E_ARG; NDVM_E_NOMEM for a workspace that
is too small) and enqueues nothing: the outputs keep the sentinel they were
filled with.  A compute call for a lane count whose device program was never
prepared by the sizing call fails instead of scheduling.  Calls on a side
stream without a caller workspace give bit-identical results to calls on the
current stream.  A many-program launch that mixes a spilling program with
small ones matches the oracle and each program's own single-program launch.
A program whose registers do not fit the budget of an all-resident launch
runs in rounds of waves rather than spilling.
"""
import ctypes

import numpy as np
import pytest

from parity import compare, judge
from workloads import configs
from workloads.bytecode import Asm

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def nd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_03574_amd as m
    return m


SENT = 12345.5


def _bufs(nd, w, L):
    tape = nd.tape_upload(nd.tape_build(w.bytecode))
    P = w.params.shape[1]
    p = torch.tensor(w.params[:L], device="cuda")
    o = torch.tensor(w.obs, device="cuda")
    loss = torch.full((L,), SENT, dtype=torch.float64, device="cuda")
    g = torch.full((L, P), SENT, dtype=torch.float64, device="cuda")
    need = nd.workspace_bytes(tape, L, True)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    return tape, p, o, loss, g, ws, need, P


def _grad_raw(nd, tape, p, L, ld_p, o, n_obs, loss, g, ld_g, ws, nbytes):
    return nd._grad(tape.handle if tape is not None else None, p, L, ld_p, o, n_obs, loss, g, ld_g, ws, nbytes,
                    torch.cuda.current_stream().cuda_stream)


def test_grad_and_forward_argument_errors(nd):
    w = configs.logistic(L=100, T=30)
    L = 100
    tape, p, o, loss, g, ws, need, P = _bufs(nd, w, L)
    pp, op, lp, gp, wp = p.data_ptr(), o.data_ptr(), loss.data_ptr(), g.data_ptr(), ws.data_ptr()
    n_obs = o.numel()
    cases = [
        ("null tape", (None, pp, L, P, op, n_obs, lp, gp, P, wp, need), nd.E_ARG),
        ("null params", (tape, None, L, P, op, n_obs, lp, gp, P, wp, need), nd.E_ARG),
        ("null loss", (tape, pp, L, P, op, n_obs, None, gp, P, wp, need), nd.E_ARG),
        ("null grad", (tape, pp, L, P, op, n_obs, lp, None, P, wp, need), nd.E_ARG),
        ("null obs", (tape, pp, L, P, None, n_obs, lp, gp, P, wp, need), nd.E_ARG),
        ("negative L", (tape, pp, -1, P, op, n_obs, lp, gp, P, wp, need), nd.E_ARG),
        ("ld_p < P", (tape, pp, L, P - 1, op, n_obs, lp, gp, P, wp, need), nd.E_ARG),
        ("ld_g < P", (tape, pp, L, P, op, n_obs, lp, gp, P - 1, wp, need), nd.E_ARG),
        ("n_obs mismatch", (tape, pp, L, P, op, n_obs - 1, lp, gp, P, wp, need), nd.E_ARG),
        ("workspace too small", (tape, pp, L, P, op, n_obs, lp, gp, P, wp, need - 8), nd.E_NOMEM),
        ("null workspace", (tape, pp, L, P, op, n_obs, lp, gp, P, None, need), nd.E_NOMEM),
    ]
    for what, args, want in cases:
        st = _grad_raw(nd, *args)
        assert st == want, (what, st, nd.last_error())
        assert nd.last_error(), what
    # forward: the same argument rules
    fws = max(nd.workspace_bytes(tape, L, False), 8)
    fw = torch.empty(fws, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    for what, args, want in [
        ("null params", (tape.handle, None, L, P, op, n_obs, lp, fw.data_ptr(), fws, s), nd.E_ARG),
        ("ld_p < P", (tape.handle, pp, L, P - 1, op, n_obs, lp, fw.data_ptr(), fws, s), nd.E_ARG),
        ("n_obs mismatch", (tape.handle, pp, L, P, op, n_obs + 1, lp, fw.data_ptr(), fws, s), nd.E_ARG),
        ("negative L", (tape.handle, pp, -5, P, op, n_obs, lp, fw.data_ptr(), fws, s), nd.E_ARG),
        ("workspace too small", (tape.handle, pp, L, P, op, n_obs, lp, fw.data_ptr(), 0, s), nd.E_NOMEM),
    ]:
        st = nd._forward(*args)
        assert st == want, (what, st, nd.last_error())
    torch.cuda.synchronize()
    # nothing was enqueued by any failing call
    assert torch.all(loss == SENT) and torch.all(g == SENT)
    # the valid call then works
    assert _grad_raw(nd, tape, pp, L, P, op, n_obs, lp, gp, P, wp, need) == nd.OK
    torch.cuda.synchronize()
    assert not torch.any(loss == SENT)


def test_compute_call_without_preparation_fails(nd):
    """ndvm_grad for a lane count whose register budget was never sized
    returns NDVM_E_ARG (it does not schedule inside the compute call)."""
    w = configs.lotka_volterra(L=64, T=5)
    tape = nd.tape_upload(nd.tape_build(w.bytecode))
    L_small, L_big = 64, 64 * 256 * 12         # different waves per CU -> different budgets
    need_small = nd.workspace_bytes(tape, L_small, True)
    p = torch.ones((L_big, 6), dtype=torch.float64, device="cuda")
    o = torch.tensor(w.obs, device="cuda")
    loss = torch.full((L_big,), SENT, dtype=torch.float64, device="cuda")
    g = torch.full((L_big, 6), SENT, dtype=torch.float64, device="cuda")
    ws = torch.empty(need_small * 4096, dtype=torch.uint8, device="cuda")
    st = _grad_raw(nd, tape, p.data_ptr(), L_big, 6, o.data_ptr(), o.numel(), loss.data_ptr(), g.data_ptr(), 6,
                   ws.data_ptr(), ws.numel())
    assert st == nd.E_ARG and "ndvm_workspace_bytes" in nd.last_error()
    torch.cuda.synchronize()
    assert torch.all(loss == SENT)


def test_grad_many_argument_errors(nd):
    w = configs.random_programs(n_prog=3, L=40, n=128, seed=9)
    tapes = [nd.tape_upload(nd.tape_build(bc)) for bc in w.programs]
    n, L, Pm = w.params.shape
    p = torch.tensor(w.params, device="cuda")
    o = torch.tensor(w.obs, device="cuda")
    loss = torch.full((n, L), SENT, dtype=torch.float64, device="cuda")
    g = torch.full((n, L, Pm), SENT, dtype=torch.float64, device="cuda")
    need = nd.workspace_bytes_many(tapes, L)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    arr = (nd._vp * n)(*[t.handle for t in tapes])
    s = torch.cuda.current_stream().cuda_stream
    base = dict(tapes=arr, n=n, p=p.data_ptr(), L=L, ld_p=Pm, sp=L * Pm, o=o.data_ptr(), n_obs=o.numel(),
                loss=loss.data_ptr(), g=g.data_ptr(), ld_g=Pm, sg=L * Pm, ws=ws.data_ptr(), nb=need)

    def call(**kw):
        a = dict(base, **kw)
        return nd._grad_many(a["tapes"], a["n"], a["p"], a["L"], a["ld_p"], a["sp"], a["o"], a["n_obs"],
                             a["loss"], a["g"], a["ld_g"], a["sg"], a["ws"], a["nb"], s)

    with_null = (nd._vp * n)(tapes[0].handle, None, tapes[2].handle)
    for what, kw, want in [
        ("null tape list", dict(tapes=None), nd.E_ARG),
        ("null tape", dict(tapes=with_null), nd.E_ARG),
        ("negative n_prog", dict(n=-1), nd.E_ARG),
        ("null params", dict(p=None), nd.E_ARG),
        ("null grad", dict(g=None), nd.E_ARG),
        ("ld_g < P", dict(ld_g=1), nd.E_ARG),
        ("program stride too small", dict(sp=L * Pm - 1), nd.E_ARG),
        ("grad stride too small", dict(sg=L * Pm - 1), nd.E_ARG),
        ("n_obs mismatch", dict(n_obs=5), nd.E_ARG),
        ("workspace too small", dict(nb=need - 8), nd.E_NOMEM),
    ]:
        st = call(**kw)
        assert st == want, (what, st, nd.last_error())
    # a lane count with another register budget (more waves per CU) that was
    # never sized: the call fails before looking at the workspace or buffers
    L_big = 16 * 256 * 4
    pb = torch.zeros((n, L_big, Pm), dtype=torch.float64, device="cuda")
    lb = torch.full((n, L_big), SENT, dtype=torch.float64, device="cuda")
    gb = torch.full((n, L_big, Pm), SENT, dtype=torch.float64, device="cuda")
    st = call(p=pb.data_ptr(), L=L_big, sp=L_big * Pm, loss=lb.data_ptr(), g=gb.data_ptr(), sg=L_big * Pm)
    assert st == nd.E_ARG and "ndvm_workspace_bytes_many" in nd.last_error()
    torch.cuda.synchronize()
    assert torch.all(loss == SENT) and torch.all(g == SENT) and torch.all(lb == SENT)
    assert call() == nd.OK


def test_side_stream_without_workspace_matches_current_stream(nd):
    """grad / grad_many / forward on a side stream, temporaries allocated by
    the binding: bit-identical to the current-stream results."""
    w = configs.kalman(L=300, T=25)
    tape = nd.tape_upload(nd.tape_build(w.bytecode))
    p = torch.tensor(w.params, device="cuda")
    o = torch.tensor(w.obs, device="cuda")
    l0, g0 = nd.grad(tape, p, o)
    f0 = nd.forward(tape, p, o)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    for _ in range(3):
        l1, g1 = nd.grad(tape, p, o, stream=side)
        f1 = nd.forward(tape, p, o, stream=side)
        # churn the allocator on the current stream meanwhile
        junk = [torch.full((300 * 12,), 7.0, dtype=torch.float64, device="cuda") for _ in range(8)]
        del junk
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        assert torch.equal(l1, l0) and torch.equal(g1, g0) and torch.equal(f1, f0)
    wr = configs.random_programs(n_prog=4, L=50, n=128, seed=3)
    tapes = [nd.tape_upload(nd.tape_build(bc)) for bc in wr.programs]
    pr = torch.tensor(wr.params, device="cuda")
    orr = torch.tensor(wr.obs, device="cuda")
    lm0, gm0 = nd.grad_many(tapes, pr, orr)
    torch.cuda.synchronize()
    side.wait_stream(torch.cuda.current_stream())
    lm1, gm1 = nd.grad_many(tapes, pr, orr, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert torch.equal(lm1, lm0) and torch.equal(gm1, gm0)


def _wide_program(P):
    A = Asm(P, 0)
    A.param(0).param(1).mul()
    for i in range(1, P - 1):
        A.param(i).param(i + 1).mul().add()
    return A.halt().bytes()


def test_many_programs_mixing_a_spilling_program(nd, oracle_mod):
    """A 17,000-parameter program (registers far beyond the LDS budget, the
    spill variant) among small random programs in one launch: the per-program
    kernel variant; each program equals the oracle and its own single-program
    launch bit for bit.  Also the forward-only replay of the wide program."""
    P = 17000
    wide = _wide_program(P)
    small = [Asm(2, 0).param(0).param(1).mul().param(0).sin().add().halt().bytes(),
             Asm(3, 0).param(0).param(1).div().param(2).exp().mul().halt().bytes()]
    progs = [small[0], wide, small[1], small[0]]
    Ps = [2, P, 3, 2]
    L = 70
    rng = np.random.default_rng(4)
    params = np.zeros((len(progs), L, P))
    for q, Pq in enumerate(Ps):
        params[q, :, :Pq] = rng.uniform(-1, 1, (L, Pq))
    tapes = [nd.tape_upload(nd.tape_build(bc)) for bc in progs]
    pt = torch.tensor(params, device="cuda")
    o = torch.zeros(0, dtype=torch.float64, device="cuda")
    loss, grad = nd.grad_many(tapes, pt, o)
    torch.cuda.synchronize()
    for q, bc in enumerate(progs):
        Pq = Ps[q]
        ol, og, _ = oracle_mod.run(bc, params[q, :, :Pq], [])
        compare(loss[q].cpu().numpy(), grad[q, :, :Pq].cpu().numpy(), ol, og)
        l1, g1 = nd.grad(tapes[q], pt[q, :, :Pq].contiguous(), o)
        torch.cuda.synchronize()
        assert torch.equal(l1, loss[q]) and torch.equal(g1, grad[q, :, :Pq])
    fl = nd.forward(tapes[1], pt[1].contiguous(), o)
    torch.cuda.synchronize()
    ol, _, _ = oracle_mod.run(wide, params[1], [], grad=False)
    compare(fl.cpu().numpy(), None, ol, None)


def test_register_hungry_program_runs_in_rounds_instead_of_spilling(nd, oracle_mod):
    """A Kalman filter needs about 315 registers per lane.  At 32,768 lanes,
    every wave resident would leave a budget of 160 and push the rest to HBM
    rows; the launch instead keeps the program of 320 registers (the
    workspace holds the same rows per lane as at 16,384 lanes, none for
    spilled registers) and runs its waves in two rounds.  Results: bit for
    bit those of a 16,384-lane launch on the same lanes, and the oracle on a
    sample of lanes."""
    w = configs.build("kalman_cv4", L=32768, T=12)
    tape = nd.tape_upload(nd.tape_build(w.bytecode))
    assert nd.workspace_bytes(tape, 32768) == 2 * nd.workspace_bytes(tape, 16384)
    p = torch.tensor(w.params, device="cuda")
    o = torch.tensor(w.obs, device="cuda")
    lf, gf = nd.grad(tape, p, o)
    lh, gh = nd.grad(tape, p[16384:].contiguous(), o)
    torch.cuda.synchronize()
    assert torch.equal(lf[16384:], lh) and torch.equal(gf[16384:], gh)
    idx = np.r_[0:64, 16320:16448, 32704:32768]
    lo, go, _ = oracle_mod.run(w.bytecode, w.params[idx], w.obs)
    compare(lf.cpu().numpy()[idx], gf.cpu().numpy()[idx], lo, go)


def test_batch_upload_equals_single_uploads(nd):
    """Tapes uploaded together (validated and scheduled on all host threads)
    give the same device programs as tapes uploaded one by one: a
    many-program gradient over either set is bit-identical, and so is each
    tape's forward loss."""
    w = configs.random_programs(n_prog=40, L=64, n=16, seed=12)
    bs = [nd.tape_build(bc) for bc in w.programs]
    one = [nd.tape_upload(b) for b in bs]
    many = nd.tape_upload_many(bs)
    assert len(many) == len(one)
    p = torch.tensor(w.params, device="cuda")
    o = torch.tensor(w.obs, device="cuda")
    l1, g1 = nd.grad_many(one, p, o)
    l2, g2 = nd.grad_many(many, p, o)
    torch.cuda.synchronize()
    assert torch.equal(l1, l2) and torch.equal(g1, g2)
    for q in (0, 17, 39):
        P = w.n_params_each[q]
        pq = p[q, :, :P].contiguous()
        assert torch.equal(nd.forward(one[q], pq, o), nd.forward(many[q], pq, o))
