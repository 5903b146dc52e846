"""Pins of the oracle's unit math (CPU only).

1. Central finite differences in float64: for every unit kind and head, the
   analytic backward of a random projection L = <y, R> matches
   (L(theta + h) - L(theta - h)) / 2h for every parameter and input element.
2. PyTorch CPU autograd in float64 (a library implementation independent of
   both the oracle and the HIP path) gives the same forward values and
   gradients for each unit kind.
3. Finite differences of the whole full-storage step on tiny networks.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import units as U
from oracle import nets

RTOL = 1e-6


def _rng(s=0):
    return np.random.default_rng(s)


def _err(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-30)


def _fd_check(fwd_scalar, arrays, analytic, n_probe=40, seed=0):
    """Compare analytic grads with central differences on up to n_probe
    entries of every array (all entries when the array is smaller)."""
    rng = _rng(seed)
    for name, arr in arrays.items():
        flat = arr.reshape(-1)
        idx = np.arange(flat.size) if flat.size <= n_probe else rng.choice(flat.size, n_probe, replace=False)
        num = np.zeros(len(idx))
        for j, k in enumerate(idx):
            old = flat[k]
            h = 1e-6 * max(1.0, abs(old))
            flat[k] = old + h
            lp = fwd_scalar()
            flat[k] = old - h
            lm = fwd_scalar()
            flat[k] = old
            num[j] = (lp - lm) / (2 * h)
        ana = analytic[name].reshape(-1)[idx]
        scale = max(np.max(np.abs(analytic[name])), 1e-12)
        assert np.max(np.abs(num - ana)) / scale < 1e-5, (name, np.max(np.abs(num - ana)) / scale)


def _unit_fd(unit, x, P, ext=None, seed=0, state_pair=False):
    rng = _rng(seed + 1)
    y0, s0, l0 = unit.fwd(x, P, ext)
    if state_pair:
        R = (rng.standard_normal(y0[0].shape), rng.standard_normal(y0[1].shape))

        def scalar():
            y, _, l = unit.fwd(x, P, ext)
            return float((y[0] * R[0]).sum() + (y[1] * R[1]).sum() + l)
        dx, grads = unit.bwd(R, x, y0, s0, P, ext)
        arrays = dict(P)
        arrays["x_h"], arrays["x_c"] = x[0], x[1]
        analytic = dict(grads)
        analytic["x_h"], analytic["x_c"] = dx[0], dx[1]
    else:
        R = rng.standard_normal(y0.shape)

        def scalar():
            y, _, _ = unit.fwd(x, P, ext)
            return float((y * R).sum())
        dx, grads = unit.bwd(R, x, y0, s0, P, ext)
        arrays = dict(P)
        arrays["x"] = x
        analytic = dict(grads)
        analytic["x"] = dx
    _fd_check(scalar, arrays, analytic, seed=seed)


def test_fd_mlp_block():
    rng = _rng(1)
    x = rng.standard_normal((3, 8))
    P = {"W": rng.standard_normal((8, 8)) * 0.5, "b": rng.standard_normal(8) * 0.1}
    _unit_fd(U.MLPBlock(), x, P)


def test_fd_stem3():
    rng = _rng(2)
    x = rng.random((2, 6, 6, 3))
    P = {"W": rng.standard_normal((4, 3, 3, 3)), "gamma": 1 + 0.1 * rng.standard_normal(4),
         "beta": 0.1 * rng.standard_normal(4)}
    _unit_fd(U.Stem3(), x, P)


@pytest.mark.parametrize("stride,cin,cout", [(1, 4, 4), (2, 4, 8)])
def test_fd_basic_block(stride, cin, cout):
    rng = _rng(3 + stride)
    x = rng.standard_normal((2, 6, 6, cin))
    P = {"W1": rng.standard_normal((cout, 3, 3, cin)) * 0.3, "gamma1": 1 + 0.1 * rng.standard_normal(cout),
         "beta1": 0.1 * rng.standard_normal(cout), "W2": rng.standard_normal((cout, 3, 3, cout)) * 0.3,
         "gamma2": 1 + 0.1 * rng.standard_normal(cout), "beta2": 0.1 * rng.standard_normal(cout)}
    _unit_fd(U.BasicBlock(stride, cin, cout), x, P)


def test_fd_stem7():
    rng = _rng(5)
    x = rng.random((2, 12, 12, 3))
    P = {"W": rng.standard_normal((4, 7, 7, 3)) * 0.2, "gamma": 1 + 0.1 * rng.standard_normal(4),
         "beta": 0.1 * rng.standard_normal(4)}
    _unit_fd(U.Stem7(), x, P)


@pytest.mark.parametrize("stride,proj", [(1, False), (2, True), (1, True)])
def test_fd_bottleneck(stride, proj):
    rng = _rng(6 + stride)
    cin, w = (8, 2) if not proj else (4, 3)
    cout = 4 * w if proj else cin
    x = rng.standard_normal((2, 6, 6, cin))
    P = {}
    for j, (co, k, ci) in enumerate([(w, 1, cin), (w, 3, w), (cout, 1, w)], 1):
        P[f"W{j}"] = rng.standard_normal((co, k, k, ci)) * 0.4
        P[f"gamma{j}"] = 1 + 0.1 * rng.standard_normal(co)
        P[f"beta{j}"] = 0.1 * rng.standard_normal(co)
    if proj:
        P["Wp"] = rng.standard_normal((cout, 1, 1, cin)) * 0.4
        P["gammap"] = 1 + 0.1 * rng.standard_normal(cout)
        P["betap"] = 0.1 * rng.standard_normal(cout)
    _unit_fd(U.Bottleneck(stride, cin, w, cout, proj), x, P)


def test_fd_lstm_step():
    rng = _rng(8)
    B, E, H, V = 3, 5, 4, 7
    P = {"W_x": rng.uniform(-0.5, 0.5, (E, 4 * H)), "W_h": rng.uniform(-0.5, 0.5, (H, 4 * H)),
         "b": rng.uniform(-0.5, 0.5, 4 * H), "W_o": rng.uniform(-0.5, 0.5, (H, V)),
         "b_o": rng.uniform(-0.5, 0.5, V)}
    ext = (rng.standard_normal((B, E)), rng.integers(0, V, B))
    x = (rng.standard_normal((B, H)) * 0.5, rng.standard_normal((B, H)) * 0.5)
    _unit_fd(U.LSTMStep(H, 1.0 / B), x, P, ext, state_pair=True)


def test_fd_heads():
    rng = _rng(9)
    x = rng.standard_normal((3, 5))
    t = rng.standard_normal((3, 5))
    loss, g = U.mse_head(x, t)
    _fd_check(lambda: float(U.mse_head(x, t)[0]), {"x": x}, {"x": g})
    xi = rng.standard_normal((4, 3, 3, 6))
    W = rng.standard_normal((6, 5))
    b = rng.standard_normal(5)
    lab = rng.integers(0, 5, 4)
    loss, g, grads = U.pool_fc_ce_head(xi, W, b, lab)
    _fd_check(lambda: float(U.pool_fc_ce_head(xi, W, b, lab)[0]), {"x": xi, "W": W, "b": b},
              {"x": g, "W": grads["W"], "b": grads["b"]})


# ---------------------------------------------------------------------------
# PyTorch float64 autograd cross-checks
# ---------------------------------------------------------------------------

def _t(a):
    return torch.tensor(np.asarray(a), dtype=torch.float64, requires_grad=True)


def _conv_t(x, W, stride, pad):
    # NHWC / [Co,KH,KW,Ci] -> torch NCHW / [Co,Ci,KH,KW]
    out = F.conv2d(x.permute(0, 3, 1, 2), W.permute(0, 3, 1, 2), stride=stride, padding=pad)
    return out.permute(0, 2, 3, 1)


def _bn_t(c, g, b):
    out = F.batch_norm(c.permute(0, 3, 1, 2), None, None, g, b, training=True, eps=U.EPS)
    return out.permute(0, 2, 3, 1)


def _compare_torch(unit, x, P, torch_fwd, seed):
    rng = _rng(seed)
    y, s, _ = unit.fwd(x, P)
    R = rng.standard_normal(y.shape)
    dx, grads = unit.bwd(R, x, y, s, P)
    tx = _t(x)
    tP = {k: _t(v) for k, v in P.items()}
    ty = torch_fwd(tx, tP)
    (ty * torch.tensor(R)).sum().backward()
    assert _err(y, ty.detach().numpy()) < 1e-12
    assert _err(dx, tx.grad.numpy()) < 1e-10
    for k in P:
        assert _err(grads[k], tP[k].grad.numpy()) < 1e-10, k


def test_torch_mlp():
    rng = _rng(11)
    x = rng.standard_normal((5, 7))
    P = {"W": rng.standard_normal((7, 7)), "b": rng.standard_normal(7)}
    _compare_torch(U.MLPBlock(), x, P, lambda x, P: x + torch.relu(x @ P["W"] + P["b"]), 1)


@pytest.mark.parametrize("stride,cin,cout", [(1, 3, 3), (2, 3, 6)])
def test_torch_basic_block(stride, cin, cout):
    rng = _rng(12)
    x = rng.standard_normal((3, 8, 8, cin))
    P = {"W1": rng.standard_normal((cout, 3, 3, cin)), "gamma1": rng.random(cout) + 0.5,
         "beta1": rng.standard_normal(cout), "W2": rng.standard_normal((cout, 3, 3, cout)),
         "gamma2": rng.random(cout) + 0.5, "beta2": rng.standard_normal(cout)}

    def fwd(x, P):
        r1 = torch.relu(_bn_t(_conv_t(x, P["W1"], stride, 1), P["gamma1"], P["beta1"]))
        b2 = _bn_t(_conv_t(r1, P["W2"], 1, 1), P["gamma2"], P["beta2"])
        sc = x[:, ::stride, ::stride, :]
        if cout > cin:
            sc = F.pad(sc, (0, cout - cin))
        return torch.relu(b2 + sc)
    _compare_torch(U.BasicBlock(stride, cin, cout), x, P, fwd, 2)


def test_torch_stem7():
    rng = _rng(13)
    x = rng.random((2, 16, 16, 3))
    P = {"W": rng.standard_normal((5, 7, 7, 3)), "gamma": rng.random(5) + 0.5, "beta": rng.standard_normal(5)}

    def fwd(x, P):
        r = torch.relu(_bn_t(_conv_t(x, P["W"], 2, 3), P["gamma"], P["beta"]))
        return F.max_pool2d(r.permute(0, 3, 1, 2), 3, 2, 1).permute(0, 2, 3, 1)
    _compare_torch(U.Stem7(), x, P, fwd, 3)


def test_torch_bottleneck_proj():
    rng = _rng(14)
    cin, w, cout, s = 6, 3, 12, 2
    x = rng.standard_normal((2, 8, 8, cin))
    P = {}
    for j, (co, k, ci) in enumerate([(w, 1, cin), (w, 3, w), (cout, 1, w)], 1):
        P[f"W{j}"] = rng.standard_normal((co, k, k, ci))
        P[f"gamma{j}"] = rng.random(co) + 0.5
        P[f"beta{j}"] = rng.standard_normal(co)
    P["Wp"] = rng.standard_normal((cout, 1, 1, cin))
    P["gammap"] = rng.random(cout) + 0.5
    P["betap"] = rng.standard_normal(cout)

    def fwd(x, P):
        r1 = torch.relu(_bn_t(_conv_t(x, P["W1"], 1, 0), P["gamma1"], P["beta1"]))
        r2 = torch.relu(_bn_t(_conv_t(r1, P["W2"], s, 1), P["gamma2"], P["beta2"]))
        b3 = _bn_t(_conv_t(r2, P["W3"], 1, 0), P["gamma3"], P["beta3"])
        sc = _bn_t(_conv_t(x, P["Wp"], s, 0), P["gammap"], P["betap"])
        return torch.relu(b3 + sc)
    _compare_torch(U.Bottleneck(s, cin, w, cout, True), x, P, fwd, 4)


def test_torch_lstm_step():
    rng = _rng(15)
    B, E, H, V = 4, 6, 5, 9
    P = {"W_x": rng.uniform(-0.3, 0.3, (E, 4 * H)), "W_h": rng.uniform(-0.3, 0.3, (H, 4 * H)),
         "b": rng.uniform(-0.3, 0.3, 4 * H), "W_o": rng.uniform(-0.3, 0.3, (H, V)),
         "b_o": rng.uniform(-0.3, 0.3, V)}
    x_t = rng.standard_normal((B, E))
    lab = rng.integers(0, V, B)
    h0, c0 = rng.standard_normal((B, H)), rng.standard_normal((B, H))
    unit = U.LSTMStep(H, 1.0 / B)
    (h, c), s, loss = unit.fwd((h0, c0), P, (x_t, lab))
    Rh, Rc = rng.standard_normal((B, H)), rng.standard_normal((B, H))
    (dh0, dc0), grads = unit.bwd((Rh, Rc), (h0, c0), (h, c), s, P, (x_t, lab))
    tP = {k: _t(v) for k, v in P.items()}
    th0, tc0 = _t(h0), _t(c0)
    th, tc = torch._VF.lstm_cell(torch.tensor(x_t), (th0, tc0), tP["W_x"].T, tP["W_h"].T, tP["b"],
                                 torch.zeros(4 * H, dtype=torch.float64))
    tl = F.cross_entropy(th @ tP["W_o"] + tP["b_o"], torch.tensor(lab), reduction="mean")
    assert abs(loss - tl.item()) < 1e-12
    assert _err(h, th.detach().numpy()) < 1e-12 and _err(c, tc.detach().numpy()) < 1e-12
    ((th * torch.tensor(Rh)).sum() + (tc * torch.tensor(Rc)).sum() + tl).backward()
    assert _err(dh0, th0.grad.numpy()) < 1e-10
    assert _err(dc0, tc0.grad.numpy()) < 1e-10
    for k in P:
        assert _err(grads[k], tP[k].grad.numpy()) < 1e-10, k


def test_torch_pool_fc_ce_and_mse():
    rng = _rng(16)
    x = rng.standard_normal((5, 4, 4, 7))
    W = rng.standard_normal((7, 11))
    b = rng.standard_normal(11)
    lab = rng.integers(0, 11, 5)
    loss, g, grads = U.pool_fc_ce_head(x, W, b, lab)
    tx, tW, tb = _t(x), _t(W), _t(b)
    tl = F.cross_entropy(tx.mean(dim=(1, 2)) @ tW + tb, torch.tensor(lab))
    tl.backward()
    assert abs(loss - tl.item()) < 1e-12
    assert _err(g, tx.grad.numpy()) < 1e-12
    assert _err(grads["W"], tW.grad.numpy()) < 1e-12 and _err(grads["b"], tb.grad.numpy()) < 1e-12
    y, t = rng.standard_normal((3, 4)), rng.standard_normal((3, 4))
    ty = _t(y)
    tl = F.mse_loss(ty, torch.tensor(t))
    tl.backward()
    loss, g = U.mse_head(y, t)
    assert abs(loss - tl.item()) < 1e-12 and _err(g, ty.grad.numpy()) < 1e-12


def test_bf16_round_matches_torch():
    rng = _rng(17)
    v = np.concatenate([rng.standard_normal(10000).astype(np.float32),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5e-3, 0.0], np.float32)])
    ours = U.bf16_round(v)
    ref = torch.tensor(v).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours, ref)


# ---------------------------------------------------------------------------
# whole-step finite differences on tiny networks
# ---------------------------------------------------------------------------

TINY = {
    "mlp": dict(kind="mlp", depth=4, width=8, batch=3, seed=21, w_var=0.1),
    "cnn": dict(kind="resnet_basic", blocks_per_stage=1, base=2, batch=2, image=8, classes=3, seed=22),
    "lstm": dict(kind="lstm", T=5, batch=2, input=3, hidden=4, vocab=5, seed=23),
    "bottleneck": dict(kind="resnet_bottleneck", stage_blocks=(1, 1), widths=(2, 3), expansion=2,
                       stem_channels=4, batch=2, image=16, classes=3, seed=24),
}


@pytest.mark.parametrize("name", list(TINY))
def test_fd_full_step(name):
    d = synth.make(TINY[name])
    chain = nets.Chain(d["structure"], d["params"])
    loss, grads = nets.full_storage_step(chain, d["input"], d["target"])
    params64 = chain.params

    def scalar():
        return float(nets.full_storage_step(chain, d["input"], d["target"])[0])
    _fd_check(scalar, params64, grads, n_probe=8, seed=5)
