"""Autograd wrappers (PAMLinear, pam_matmul): forward and approximate-derivative
backward (Sec. 3.2, Table 1) against the CPU oracle, and a small training run."""
import numpy as np
import pytest

import pam_workloads as wl
from gpu_util import device, note
from oracle import pam_ref

pytestmark = pytest.mark.gpu


def close(got, ref, s, k, extra=0.0, what=""):
    got = np.asarray(got, np.float64)
    tol = pam_ref.gemm_tolerance(s, k) + extra
    err = np.abs(got - ref)
    assert np.all(err <= tol), f"{what}: max err {err.max():.3e}, worst ratio {(err / tol).max():.2f}"


def test_pam_linear_forward_backward_with_bias():
    import torch
    from paper_2305_17190_amd.autograd import pam_linear
    note("pam_linear 2x101x96 -> 72 with bias, forward + backward")
    dev = device()
    x = wl.random_matrix(202, 96, 301).reshape(2, 101, 96)
    w = wl.random_matrix(72, 96, 302, 0.05)
    bias = wl.random_matrix(1, 72, 303, 0.1).reshape(72)
    g = wl.random_matrix(202, 72, 304, 1e-3).reshape(2, 101, 72)
    xt = torch.from_numpy(x).to(dev).requires_grad_()
    wt = torch.from_numpy(w).to(dev).requires_grad_()
    bt = torch.from_numpy(bias).to(dev).requires_grad_()
    y = pam_linear(xt, wt, bt)
    y.backward(torch.from_numpy(g).to(dev))
    torch.cuda.synchronize()
    x2, g2 = x.reshape(202, 96), g.reshape(202, 72)
    c, s = pam_ref.pam_gemm_ref(x2, w, False, True)
    yref = c + bias.astype(np.float64)
    close(y.detach().cpu().numpy().reshape(202, 72), yref, s, 96, np.abs(yref) * 2.0 ** -23, "Y")
    c, s = pam_ref.pam_gemm_ref(g2, w)
    close(xt.grad.cpu().numpy().reshape(202, 96), c, s, 72, what="dX")
    c, s = pam_ref.pam_gemm_ref(g2, x2, True, False)
    close(wt.grad.cpu().numpy(), c, s, 202, what="dW")
    dbr = g2.astype(np.float64).sum(0)
    assert np.all(np.abs(bt.grad.cpu().numpy() - dbr) <= 1e-5 * np.sqrt(202) * np.abs(g2).sum(0) + 1e-30)


def test_pam_linear_module_and_partial_grads():
    import torch
    from paper_2305_17190_amd.autograd import PAMLinear
    note("PAMLinear module, grads of the weight only, non-contiguous input")
    dev = device()
    torch.manual_seed(0)
    lin = PAMLinear(64, 48, bias=False, device=dev)
    x = torch.from_numpy(wl.random_matrix(64, 130, 305)).to(dev).t()      # 130 x 64, rows strided
    y = lin(x)
    g = torch.from_numpy(wl.random_matrix(130, 48, 306)).to(dev)
    y.backward(g)
    xn, wn, gn = x.cpu().numpy(), lin.weight.detach().cpu().numpy(), g.cpu().numpy()
    c, s = pam_ref.pam_gemm_ref(xn, wn, False, True)
    close(y.detach().cpu().numpy(), c, s, 64, what="Y")
    c, s = pam_ref.pam_gemm_ref(gn, xn, True, False)
    close(lin.weight.grad.cpu().numpy(), c, s, 130, what="dW")


@pytest.mark.parametrize("batched", [True, False])
def test_pam_matmul_forward_backward(batched):
    import torch
    from paper_2305_17190_amd.autograd import pam_matmul
    note(f"pam_matmul batched={batched}, forward + backward")
    dev = device()
    nb = 3 if batched else 1
    a = wl.random_matrix(nb * 70, 40, 307).reshape(nb, 70, 40)
    b = wl.random_matrix(nb * 40, 33, 308).reshape(nb, 40, 33)
    g = wl.random_matrix(nb * 70, 33, 309).reshape(nb, 70, 33)
    at = torch.from_numpy(a if batched else a[0]).to(dev).requires_grad_()
    bt = torch.from_numpy(b if batched else b[0]).to(dev).requires_grad_()
    c = pam_matmul(at, bt)
    c.backward(torch.from_numpy(g if batched else g[0]).to(dev))
    cg = c.detach().cpu().numpy().reshape(nb, 70, 33)
    da = at.grad.cpu().numpy().reshape(nb, 70, 40)
    db = bt.grad.cpu().numpy().reshape(nb, 40, 33)
    for i in range(nb):
        r, s = pam_ref.pam_gemm_ref(a[i], b[i])
        close(cg[i], r, s, 40, what=f"C[{i}]")
        r, s = pam_ref.pam_gemm_ref(g[i], b[i], False, True)
        close(da[i], r, s, 33, what=f"dA[{i}]")
        r, s = pam_ref.pam_gemm_ref(a[i], g[i], True, False)
        close(db[i], r, s, 70, what=f"dB[{i}]")


def train_mlp(linear, dev, steps=400, lr=0.1):
    """Fit a random teacher MLP (64 -> 128 -> 16, ReLU) with plain SGD; returns
    the per-step losses.  ``linear(x, w, b)`` is the layer's product."""
    import torch
    g = torch.Generator(device="cpu").manual_seed(7)
    teacher1 = torch.randn(128, 64, generator=g) / 8
    teacher2 = torch.randn(16, 128, generator=g) / 11
    gi = torch.Generator(device="cpu").manual_seed(8)
    w1 = ((torch.rand(128, 64, generator=gi) * 2 - 1) / 8).to(dev).requires_grad_()
    b1 = ((torch.rand(128, generator=gi) * 2 - 1) / 8).to(dev).requires_grad_()
    w2 = ((torch.rand(16, 128, generator=gi) * 2 - 1) / 11.3).to(dev).requires_grad_()
    b2 = ((torch.rand(16, generator=gi) * 2 - 1) / 11.3).to(dev).requires_grad_()
    opt = torch.optim.SGD([w1, b1, w2, b2], lr=lr)
    losses = []
    for _ in range(steps):
        x = torch.randn(256, 64, generator=g)
        yt = torch.relu(x @ teacher1.t()) @ teacher2.t()
        x, yt = x.to(dev), yt.to(dev)
        y = linear(torch.relu(linear(x, w1, b1)), w2, b2)
        loss = ((y - yt) ** 2).mean()
        opt.zero_grad()
        loss.backward()
        opt.step()
        losses.append(loss.item())
    return np.array(losses)


def test_training_a_small_pam_mlp_reduces_the_loss():
    """A two-layer PAM MLP fits a random teacher MLP (synthetic regression) with
    plain SGD: every product of the student, forward and backward, is PAM.  The
    same run with ordinary float32 products is printed beside it."""
    import torch
    from paper_2305_17190_amd.autograd import pam_linear
    note("train a 64-128-16 MLP for 400 SGD steps, PAM products and float32 products")
    dev = device()
    pam_l = train_mlp(pam_linear, dev)
    ref_l = train_mlp(torch.nn.functional.linear, dev)
    first, last = pam_l[:10].mean(), pam_l[-10:].mean()
    print(f"[training] PAM loss {first:.4f} -> {last:.4f}; float32 loss {ref_l[:10].mean():.4f} -> "
          f"{ref_l[-10:].mean():.4f}")
    assert np.isfinite(last) and last < 0.5 * first, (first, last)


def train_attention(matmul, linear, dev, steps=300, lr=2.0):
    """Single-head self-attention student fitted to a fixed random teacher on
    synthetic sequences (batch 64, length 16, width 32), plain SGD."""
    import torch
    g = torch.Generator().manual_seed(11)
    d, seq, batch = 32, 16, 64

    def init(seed):
        gi = torch.Generator().manual_seed(seed)
        return [((torch.rand(d, d, generator=gi) * 2 - 1) / d ** 0.5) for _ in range(4)]

    teacher = [w.to(dev) for w in init(12)]
    student = [w.to(dev).requires_grad_() for w in init(13)]
    opt = torch.optim.SGD(student, lr=lr)

    def layer(x, ws, mm, lin):
        wq, wk, wv, wo = ws
        q, k, v = lin(x, wq), lin(x, wk), lin(x, wv)
        s = mm(q, k.transpose(1, 2)) * (1.0 / d ** 0.5)
        return lin(mm(torch.softmax(s, dim=-1), v), wo)

    losses = []
    for _ in range(steps):
        x = torch.randn(batch, seq, d, generator=g).to(dev)
        with torch.no_grad():
            yt = layer(x, teacher, torch.matmul, torch.nn.functional.linear)
        y = layer(x, student, matmul, linear)
        loss = ((y - yt) ** 2).mean()
        opt.zero_grad()
        loss.backward()
        opt.step()
        losses.append(loss.item())
    return np.array(losses)


def test_training_a_pam_attention_layer_reduces_the_loss():
    """Every product of the student, the projections and the batched Q K^T and
    P V products, forward and backward, is PAM (approximate derivative); the
    same run with float32 products is printed beside it."""
    import torch
    from paper_2305_17190_amd.autograd import pam_linear, pam_matmul
    note("train a single-head attention layer for 300 SGD steps, PAM products and float32 products")
    dev = device()
    pam_l = train_attention(pam_matmul, pam_linear, dev)
    ref_l = train_attention(torch.matmul, torch.nn.functional.linear, dev)
    first, last = pam_l[:10].mean(), pam_l[-10:].mean()
    print(f"[training] PAM loss {first:.5f} -> {last:.5f}; float32 loss {ref_l[:10].mean():.5f} -> "
          f"{ref_l[-10:].mean():.5f}")
    assert np.isfinite(last) and last < 0.5 * first, (first, last)
