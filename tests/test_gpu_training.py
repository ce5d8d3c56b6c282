"""End to end: the library as a PyTorch optimiser in an autograd training
loop (the usage the README shows).  A small MLP (2-D weights and 1-D
biases) fits a smooth synthetic regression target; R-iKFAD with damping
(gamma > 0, friction on) must reduce the loss by a large factor and keep
every state tensor finite.  Adafactor-m, the paper's baseline, runs the
same loop.  This checks that the step optimises -- the parity tests check
that it computes the Table exactly."""
import pytest
import torch

from paper_2609_30342_amd import rikfad as R

from parity import log

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _problem():
    gen = torch.Generator(device="cuda:0").manual_seed(3)
    x = torch.randn((512, 16), generator=gen, device="cuda:0")
    w = torch.randn((16, 1), generator=gen, device="cuda:0") / 4.0
    y = torch.sin(2.0 * (x @ w)) + 0.5 * torch.cos(x[:, :1])
    torch.manual_seed(0)
    model = torch.nn.Sequential(torch.nn.Linear(16, 64), torch.nn.Tanh(),
                                torch.nn.Linear(64, 1)).to("cuda:0")
    params = list(model.parameters())
    for p in params:
        p.grad = torch.zeros_like(p)
    return model, params, x, y


def _train(model, params, x, y, opt, steps):
    losses = []
    for _ in range(steps):
        for p in params:
            p.grad.zero_()
        loss = torch.nn.functional.mse_loss(model(x), y)
        loss.backward()
        opt.step()
        losses.append(loss.item())
    return losses


def test_rikfad_trains_an_mlp():
    log("[case] training loop R-iKFAD")
    model, params, x, y = _problem()
    opt = R.RIKFAD(params, [p.grad for p in params], h=0.3, gamma=2.0, alpha=0.1, mu=1.0,
                   eps_stab=1e-8)
    losses = _train(model, params, x, y, opt, 300)
    log(f"[train] R-iKFAD loss {losses[0]:.4f} -> {losses[-1]:.4f}")
    assert losses[-1] < 0.2 * losses[0], (losses[0], losses[-1])
    opt.sync_momentum()
    for p, r, c in opt.state:
        assert torch.isfinite(p).all() and (r >= 0).all() and (c >= 0).all()
        assert torch.isfinite(r).all() and torch.isfinite(c).all()
    assert not opt.nonfinite()
    # the friction factors have been driven by the momentum
    assert max(float(r.sum()) for _, r, _ in opt.state) > 0.0
    opt.close()


def test_adafm_trains_an_mlp():
    log("[case] training loop Adafactor-m")
    model, params, x, y = _problem()
    opt = R.ADAFM(params, [p.grad for p in params], h=1e-2, beta1=0.9)
    losses = _train(model, params, x, y, opt, 300)
    log(f"[train] Adafactor-m loss {losses[0]:.4f} -> {losses[-1]:.4f}")
    assert losses[-1] < 0.2 * losses[0], (losses[0], losses[-1])
    opt.close()
