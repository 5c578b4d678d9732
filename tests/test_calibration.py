"""The calibration loop (Adam driving the exact per-lane gradients, as in the
paper's Kalman maximum-likelihood fit, Section "From buckets to phases").

CPU: the Adam oracle pinned to closed forms -- its first step from zero
moments is sign descent, a constant gradient moves every step by
lr*g/(|g|+eps), and a quadratic is driven to its minimum.  GPU: the Adam
kernel bit for bit against the oracle's step, a whole calibration against the
oracle's, and the autograd function against the replay's own gradient.
"""
import numpy as np
import pytest

from workloads import configs
from workloads.bytecode import Asm


def test_adam_first_step_is_sign_descent(oracle_mod):
    from oracle import adam
    rng = np.random.default_rng(7)
    p0 = rng.normal(size=(5, 3))
    g = rng.normal(size=(5, 3)) * 10.0 ** rng.integers(-6, 6, size=(5, 3))
    p = p0.copy()
    lr, eps = 1e-2, 1e-8
    adam.adam_step(p, g, np.zeros_like(p), np.zeros_like(p), 1, lr, eps=eps)
    want = p0 - lr * g / (np.abs(g) + eps)
    np.testing.assert_allclose(p, want, rtol=0, atol=4e-16 * lr + 1e-15 * np.abs(p0).max())


def test_adam_constant_gradient(oracle_mod):
    # loss = 2.5 p0 - 0.75 p1 + 1e-3 p2: the gradient is constant, so the
    # bias-corrected moments are g and g^2 and every step is lr*g/(|g|+eps)
    from oracle import adam
    c = [2.5, -0.75, 1e-3]
    A = Asm(3, 0)
    A.param(0).push(c[0]).mul()
    for k in (1, 2):
        A.param(k).push(c[k]).mul().add()
    bc = A.halt().bytes()
    p0 = np.array([[0.3, -1.2, 4.0], [1.0, 2.0, 3.0]])
    steps, lr, eps = 40, 1e-3, 1e-8
    p, hist = adam.calibrate(bc, p0, [], steps, lr, eps=eps)
    g = np.array(c)
    want = p0 - steps * lr * g / (np.abs(g) + eps)
    np.testing.assert_allclose(p, want, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(hist[0], p0 @ g, rtol=1e-15)


def test_adam_quadratic_reaches_minimum(oracle_mod):
    from oracle import adam
    A = Asm(1, 0)
    bc = A.param(0).push(3.0).sub().dup().mul().halt().bytes()   # (p - 3)^2
    p, hist = adam.calibrate(bc, np.array([[0.0], [10.0]]), [], 600, 0.05)
    assert np.all(np.abs(p[:, 0] - 3.0) < 1e-2)
    assert np.all(hist[-1] < 1e-3 * hist[0])


# ---------------------------------------------------------------- GPU
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def nd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_03574_amd as m
    return m


@pytest.mark.gpu
def test_adam_step_bitwise(nd, oracle_mod):
    from oracle import adam
    rng = np.random.default_rng(11)
    L, P = 1000, 7
    p0, g = rng.normal(size=(L, P)), rng.normal(size=(L, P)) * 10.0 ** rng.integers(-8, 3, size=(L, P))
    m0, v0 = rng.normal(size=(L, P)) * 0.1, rng.uniform(0, 1, size=(L, P))
    g[0, 0] = 0.0
    for t in (1, 3, 250):
        p, m, v = p0.copy(), m0.copy(), v0.copy()
        adam.adam_step(p, g, m, v, t, 1e-3, 0.9, 0.999, 1e-8)
        dp = torch.tensor(p0, device="cuda")
        dm, dv = torch.tensor(m0, device="cuda"), torch.tensor(v0, device="cuda")
        nd.adam_step(dp, torch.tensor(g, device="cuda"), dm, dv, t, 1e-3, 0.9, 0.999, 1e-8)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(dp.cpu().numpy(), p)
        np.testing.assert_array_equal(dm.cpu().numpy(), m)
        np.testing.assert_array_equal(dv.cpu().numpy(), v)


@pytest.mark.gpu
def test_adam_step_errors(nd):
    p = torch.zeros((4, 3), dtype=torch.float64, device="cuda")
    with pytest.raises(nd.NdvmError):
        nd.adam_step(p, p, p.clone(), p.clone(), 0, 1e-3)           # t < 1
    with pytest.raises(nd.NdvmError):
        nd.adam_step(p, p, p.clone(), p.clone(), 1, 1e-3, beta1=1.0)


@pytest.mark.gpu
@pytest.mark.parametrize("name,kw,steps,lr", [("kalman_cv4", dict(L=70, T=20), 12, 1e-6),
                                              ("logistic_euler", dict(L=70, T=60), 12, 1e-3),
                                              ("exp_decay", dict(L=70), 25, 1e-2)])
def test_calibration_matches_oracle(nd, oracle_mod, name, kw, steps, lr):
    from oracle import adam
    from paper_2607_03574_amd import torch_api
    w = configs.build(name, **kw)
    po, ho = adam.calibrate(w.bytecode, w.params, w.obs, steps, lr)
    tape = nd.tape_upload(nd.tape_build(w.bytecode))
    p = torch.tensor(w.params, device="cuda")
    hg = torch_api.calibrate(tape, p, torch.tensor(w.obs, device="cuda"), steps, lr)
    torch.cuda.synchronize()
    pg, hg = p.cpu().numpy(), hg.cpu().numpy()
    # the gradients agree to ~1e-15 relative; Adam's step is bounded by ~lr
    scale = np.maximum(np.abs(po), 1.0)
    assert np.all(np.abs(pg - po) <= 1e-11 * scale), np.abs(pg - po).max()
    np.testing.assert_allclose(hg, ho, rtol=1e-11, atol=0)
    assert np.mean(hg[-1] < hg[0]) > 0.9     # the fit makes progress for most lanes


@pytest.mark.gpu
def test_replay_loss_autograd(nd):
    from paper_2607_03574_amd import torch_api
    w = configs.build("kalman_cv4", L=40, T=10)
    tape = nd.tape_upload(nd.tape_build(w.bytecode))
    obs = torch.tensor(w.obs, device="cuda")
    p = torch.tensor(w.params, device="cuda", requires_grad=True)
    wts = torch.linspace(-1.0, 2.0, 40, dtype=torch.float64, device="cuda")
    loss = torch_api.replay_loss(tape, p, obs)
    (loss * wts).sum().backward()
    l2, g2 = nd.grad(tape, p.detach(), obs)
    torch.cuda.synchronize()
    assert torch.equal(loss.detach(), l2)
    assert torch.equal(p.grad, wts.unsqueeze(1) * g2)
