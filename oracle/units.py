"""Unit math of the chain networks, written from their textbook definitions.

TEST INFRASTRUCTURE ONLY (see the package header).

Every function is plain NumPy, computed in the dtype of its inputs (float64 by
default).  Layouts are NHWC for images and [rows, features] for matrices.  Conv
weights are [Cout, KH, KW, Cin]; FC/MLP weights are [in, out].

Definitions used (the paper names the operators -- fully connected, sigmoid,
softmax, convolution, batch normalisation, activation, pooling (section 3,
Fig. 1; section 4.2) and LSTM (section 5.3) -- but not their formulas, so the
standard ones are written out):

* ReLU: max(z, 0); its derivative at 0 is taken as 0.
* Batch normalisation in training mode: per-channel mean and *biased* variance
  over N*H*W, eps = 1e-5, out = gamma * (x - mean) / sqrt(var + eps) + beta.
* Convolution: zero padding, cross-correlation, out[n,ho,wo,co] =
  sum_{kh,kw,ci} x[n, ho*s+kh-p, wo*s+kw-p, ci] * W[co,kh,kw,ci].
* Max pool 3x3/2 pad 1 (padding never wins); its gradient goes to the first
  maximum of the window in row-major (kh, kw) order.
* Softmax cross-entropy, max-subtracted; the loss is the mean over the rows
  that ``scale`` describes.
* LSTM gate order i, f, g, o:  c_t = f*c_{t-1} + i*g,  h_t = o*tanh(c_t).

Optional bf16 emulation (``Prec(bf16=True)``) rounds to bfloat16
(round-to-nearest-even on the float32 bit pattern) at the points where the GPU
stores bf16; all other arithmetic stays in the working dtype.

Parity: pinned by central finite differences in float64 on tiny shapes and by
PyTorch CPU autograd in float64 for each unit kind (tests/test_oracle_units.py).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

EPS = 1e-5


# --------------------------------------------------------------------------
# precision handling
# --------------------------------------------------------------------------

def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 value (ties to even), returned in x's dtype."""
    x = np.asarray(x)
    f = x.astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    u = (u + 0x7FFF + lsb) & 0xFFFF0000
    r = u.astype(np.uint32).view(np.float32)
    # NaN/Inf pass through unchanged (not expected in these workloads)
    r = np.where(np.isfinite(f), r, f)
    return r.astype(x.dtype if x.dtype != np.float32 else np.float32)


@dataclass
class Prec:
    """Working precision.  ``jitter`` (with ``rng``) multiplies every value by
    (1 + jitter * N(0, 1)) just before it is rounded to bf16: a model of the
    float32 accumulation error of another evaluation order, used only to
    measure how far such errors can move a result (conditioning)."""
    dtype: type = np.float64
    bf16: bool = False
    jitter: float = 0.0
    rng: object = None

    def cast(self, x):
        return np.asarray(x, dtype=self.dtype)

    def st(self, x):
        """A tensor the GPU stores in bf16 (activation or GEMM operand)."""
        if not self.bf16:
            return x
        if self.jitter:
            x = np.asarray(x) * (1.0 + self.jitter * self.rng.standard_normal(np.shape(x)))
        return bf16_round(x).astype(self.dtype)


F64 = Prec(np.float64, False)


# --------------------------------------------------------------------------
# elementary operators
# --------------------------------------------------------------------------

def relu(z):
    return np.maximum(z, 0)


def conv2d(x, W, stride, pad):
    """out[n,ho,wo,co] = sum_{kh,kw,ci} xpad[n, ho*s+kh, wo*s+kw, ci] W[co,kh,kw,ci]."""
    N, H, Wd, C = x.shape
    Co, KH, KW, Ci = W.shape
    assert Ci == C
    Ho = (H + 2 * pad - KH) // stride + 1
    Wo = (Wd + 2 * pad - KW) // stride + 1
    xp = np.pad(x, ((0, 0), (pad, pad), (pad, pad), (0, 0)))
    out = np.zeros((N, Ho, Wo, Co), dtype=x.dtype)
    for kh in range(KH):
        for kw in range(KW):
            patch = xp[:, kh:kh + stride * (Ho - 1) + 1:stride, kw:kw + stride * (Wo - 1) + 1:stride, :]
            out += (patch.reshape(-1, C) @ W[:, kh, kw, :].T).reshape(N, Ho, Wo, Co)
    return out


def conv2d_dgrad(dy, W, x_shape, stride, pad):
    """dL/dx of conv2d: every tap scatters dy * W back onto the input pixel it read."""
    N, H, Wd, C = x_shape
    Co, KH, KW, Ci = W.shape
    _, Ho, Wo, _ = dy.shape
    dxp = np.zeros((N, H + 2 * pad, Wd + 2 * pad, C), dtype=dy.dtype)
    d2 = dy.reshape(-1, Co)
    for kh in range(KH):
        for kw in range(KW):
            contrib = (d2 @ W[:, kh, kw, :]).reshape(N, Ho, Wo, C)
            dxp[:, kh:kh + stride * (Ho - 1) + 1:stride, kw:kw + stride * (Wo - 1) + 1:stride, :] += contrib
    return dxp[:, pad:pad + H, pad:pad + Wd, :]


def conv2d_wgrad(dy, x, W_shape, stride, pad):
    """dL/dW[co,kh,kw,ci] = sum_{n,ho,wo} dy[n,ho,wo,co] xpad[n,ho*s+kh,wo*s+kw,ci]."""
    Co, KH, KW, Ci = W_shape
    N, Ho, Wo, _ = dy.shape
    xp = np.pad(x, ((0, 0), (pad, pad), (pad, pad), (0, 0)))
    dW = np.zeros(W_shape, dtype=dy.dtype)
    d2 = dy.reshape(-1, Co)
    for kh in range(KH):
        for kw in range(KW):
            patch = xp[:, kh:kh + stride * (Ho - 1) + 1:stride, kw:kw + stride * (Wo - 1) + 1:stride, :]
            dW[:, kh, kw, :] = d2.T @ patch.reshape(-1, Ci)
    return dW


def bn_fwd(c, gamma, beta):
    axes = tuple(range(c.ndim - 1))
    mean = c.mean(axis=axes)
    var = ((c - mean) ** 2).mean(axis=axes)
    rstd = 1.0 / np.sqrt(var + EPS)
    xhat = (c - mean) * rstd
    return gamma * xhat + beta, (mean, rstd)


def bn_bwd(dy, c, stats, gamma):
    """Backward of training-mode batch normalisation."""
    mean, rstd = stats
    axes = tuple(range(c.ndim - 1))
    m = int(np.prod([c.shape[a] for a in axes]))
    xhat = (c - mean) * rstd
    dbeta = dy.sum(axis=axes)
    dgamma = (dy * xhat).sum(axis=axes)
    dx = (gamma * rstd / m) * (m * dy - dbeta - xhat * dgamma)
    return dx, dgamma, dbeta


def maxpool_fwd(x, k=3, s=2, p=1):
    N, H, Wd, C = x.shape
    Ho = (H + 2 * p - k) // s + 1
    Wo = (Wd + 2 * p - k) // s + 1
    xp = np.pad(x, ((0, 0), (p, p), (p, p), (0, 0)), constant_values=-np.inf)
    out = np.full((N, Ho, Wo, C), -np.inf, dtype=x.dtype)
    arg = np.zeros((N, Ho, Wo, C), dtype=np.int64)
    for kh in range(k):
        for kw in range(k):
            v = xp[:, kh:kh + s * (Ho - 1) + 1:s, kw:kw + s * (Wo - 1) + 1:s, :]
            better = v > out          # strict: the first maximum in row-major order wins
            out = np.where(better, v, out)
            arg = np.where(better, kh * k + kw, arg)
    return out, arg


def maxpool_bwd(dy, arg, x_shape, k=3, s=2, p=1):
    N, H, Wd, C = x_shape
    _, Ho, Wo, _ = dy.shape
    dxp = np.zeros((N, H + 2 * p, Wd + 2 * p, C), dtype=dy.dtype)
    for kh in range(k):
        for kw in range(k):
            sel = np.where(arg == kh * k + kw, dy, 0)
            dxp[:, kh:kh + s * (Ho - 1) + 1:s, kw:kw + s * (Wo - 1) + 1:s, :] += sel
    return dxp[:, p:p + H, p:p + Wd, :]


def softmax_ce(logits, labels, scale):
    """Sum over rows of -log softmax(logits)[label], times ``scale``; and its gradient."""
    m = logits.max(axis=1, keepdims=True)
    e = np.exp(logits - m)
    ssum = e.sum(axis=1, keepdims=True)
    p = e / ssum
    rows = np.arange(logits.shape[0])
    nll = (np.log(ssum[:, 0]) + m[:, 0]) - logits[rows, labels]
    loss = nll.sum() * scale
    d = p.copy()
    d[rows, labels] -= 1
    return loss, d * scale, p


def sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


# --------------------------------------------------------------------------
# units: fwd(x, P, ext) -> (y, saved, loss_part); bwd(g, x, y, saved, P, ext, need_dx)
#        -> (dx, {param_name: grad})
# P maps the unit's local parameter names to arrays; ext carries external
# per-unit inputs (the LSTM step's x_t and labels).
# --------------------------------------------------------------------------

class MLPBlock:
    """y = x + relu(x W + b)."""
    kind = "mlp"

    def __init__(self, prec=F64):
        self.prec = prec

    def fwd(self, x, P, ext=None):
        z = x @ P["W"] + P["b"]
        y = x + relu(z)
        return y, {"z": z}, 0.0

    def bwd(self, g, x, y, saved, P, ext=None, need_dx=True):
        dr = g * (saved["z"] > 0)
        grads = {"W": x.T @ dr, "b": dr.sum(axis=0)}
        dx = g + dr @ P["W"].T if need_dx else None
        return dx, grads


class Stem3:
    """CIFAR stem: relu(bn(conv3x3(x)))."""
    kind = "stem3"

    def __init__(self, prec=F64):
        self.prec = prec

    def fwd(self, x, P, ext=None):
        c = conv2d(x, P["W"], 1, 1)
        b, st = bn_fwd(c, P["gamma"], P["beta"])
        return relu(b), {"c": c, "st": st}, 0.0

    def bwd(self, g, x, y, saved, P, ext=None, need_dx=True):
        d = g * (y > 0)
        dc, dgam, dbet = bn_bwd(d, saved["c"], saved["st"], P["gamma"])
        grads = {"W": conv2d_wgrad(dc, x, P["W"].shape, 1, 1), "gamma": dgam, "beta": dbet}
        dx = conv2d_dgrad(dc, P["W"], x.shape, 1, 1) if need_dx else None
        return dx, grads


def shortcut_a(x, stride, cout):
    """Option-A shortcut: subsample by the stride, then append zero channels."""
    xs = x[:, ::stride, ::stride, :] if stride > 1 else x
    cin = x.shape[3]
    if cout == cin:
        return xs
    pad = np.zeros(xs.shape[:3] + (cout - cin,), dtype=x.dtype)
    return np.concatenate([xs, pad], axis=3)


def shortcut_a_bwd(d, x_shape, stride):
    cin = x_shape[3]
    dx = np.zeros(x_shape, dtype=d.dtype)
    if stride > 1:
        dx[:, ::stride, ::stride, :] = d[:, :, :, :cin]
    else:
        dx[...] = d[:, :, :, :cin]
    return dx


class BasicBlock:
    """y = relu(bn2(conv3x3(relu(bn1(conv3x3(x, stride))))) + shortcut(x))."""
    kind = "basic"

    def __init__(self, stride, cin, cout, prec=F64):
        self.stride, self.cin, self.cout, self.prec = stride, cin, cout, prec

    def fwd(self, x, P, ext=None):
        c1 = conv2d(x, P["W1"], self.stride, 1)
        b1, st1 = bn_fwd(c1, P["gamma1"], P["beta1"])
        r1 = relu(b1)
        c2 = conv2d(r1, P["W2"], 1, 1)
        b2, st2 = bn_fwd(c2, P["gamma2"], P["beta2"])
        y = relu(b2 + shortcut_a(x, self.stride, self.cout))
        return y, {"c1": c1, "st1": st1, "r1": r1, "c2": c2, "st2": st2}, 0.0

    def bwd(self, g, x, y, saved, P, ext=None, need_dx=True):
        ds = g * (y > 0)
        dc2, dgam2, dbet2 = bn_bwd(ds, saved["c2"], saved["st2"], P["gamma2"])
        dW2 = conv2d_wgrad(dc2, saved["r1"], P["W2"].shape, 1, 1)
        dr1 = conv2d_dgrad(dc2, P["W2"], saved["r1"].shape, 1, 1)
        db1 = dr1 * (saved["r1"] > 0)
        dc1, dgam1, dbet1 = bn_bwd(db1, saved["c1"], saved["st1"], P["gamma1"])
        dW1 = conv2d_wgrad(dc1, x, P["W1"].shape, self.stride, 1)
        grads = {"W1": dW1, "gamma1": dgam1, "beta1": dbet1,
                 "W2": dW2, "gamma2": dgam2, "beta2": dbet2}
        dx = None
        if need_dx:
            dx = conv2d_dgrad(dc1, P["W1"], x.shape, self.stride, 1) + \
                shortcut_a_bwd(ds, x.shape, self.stride)
        return dx, grads


class Stem7:
    """ImageNet stem: maxpool3x3/2(relu(bn(conv7x7/2 pad 3(x))))."""
    kind = "stem7"

    def __init__(self, prec=F64):
        self.prec = prec

    def fwd(self, x, P, ext=None):
        pr = self.prec
        c = pr.st(conv2d(pr.st(x), pr.st(P["W"]), 2, 3))
        b, st = bn_fwd(c, P["gamma"], P["beta"])
        r = pr.st(relu(b))
        y, arg = maxpool_fwd(r)
        return y, {"c": c, "st": st, "r": r, "arg": arg}, 0.0

    def bwd(self, g, x, y, saved, P, ext=None, need_dx=True):
        pr = self.prec
        dr = maxpool_bwd(g, saved["arg"], saved["r"].shape)
        d = dr * (saved["r"] > 0)
        dc, dgam, dbet = bn_bwd(d, saved["c"], saved["st"], P["gamma"])
        dc = pr.st(dc)
        grads = {"W": conv2d_wgrad(dc, pr.st(x), P["W"].shape, 2, 3), "gamma": dgam, "beta": dbet}
        dx = conv2d_dgrad(dc, pr.st(P["W"]), x.shape, 2, 3) if need_dx else None
        return dx, grads


class Bottleneck:
    """y = relu(bn3(conv1x1(relu(bn2(conv3x3_s(relu(bn1(conv1x1(x)))))))) + sc(x)),
    sc = bn_p(conv1x1_s(x)) for a projection block, else x."""
    kind = "bottleneck"

    def __init__(self, stride, cin, width, cout, proj, prec=F64):
        self.stride, self.cin, self.width, self.cout, self.proj = stride, cin, width, cout, proj
        self.prec = prec

    def fwd(self, x, P, ext=None):
        pr, s = self.prec, self.stride
        c1 = pr.st(conv2d(x, pr.st(P["W1"]), 1, 0))
        b1, st1 = bn_fwd(c1, P["gamma1"], P["beta1"])
        r1 = pr.st(relu(b1))
        c2 = pr.st(conv2d(r1, pr.st(P["W2"]), s, 1))
        b2, st2 = bn_fwd(c2, P["gamma2"], P["beta2"])
        r2 = pr.st(relu(b2))
        c3 = pr.st(conv2d(r2, pr.st(P["W3"]), 1, 0))
        b3, st3 = bn_fwd(c3, P["gamma3"], P["beta3"])
        saved = {"c1": c1, "st1": st1, "r1": r1, "c2": c2, "st2": st2, "r2": r2,
                 "c3": c3, "st3": st3}
        if self.proj:
            cp = pr.st(conv2d(x, pr.st(P["Wp"]), s, 0))
            bp, stp = bn_fwd(cp, P["gammap"], P["betap"])
            saved.update(cp=cp, stp=stp)
            sc = bp
        else:
            sc = x
        y = pr.st(relu(b3 + sc))
        return y, saved, 0.0

    def bwd(self, g, x, y, saved, P, ext=None, need_dx=True):
        pr, s = self.prec, self.stride
        ds = g * (y > 0)
        dc3, dgam3, dbet3 = bn_bwd(ds, saved["c3"], saved["st3"], P["gamma3"])
        dc3 = pr.st(dc3)
        dW3 = conv2d_wgrad(dc3, saved["r2"], P["W3"].shape, 1, 0)
        dr2 = conv2d_dgrad(dc3, pr.st(P["W3"]), saved["r2"].shape, 1, 0)
        dc2, dgam2, dbet2 = bn_bwd(dr2 * (saved["r2"] > 0), saved["c2"], saved["st2"], P["gamma2"])
        dc2 = pr.st(dc2)
        dW2 = conv2d_wgrad(dc2, saved["r1"], P["W2"].shape, s, 1)
        dr1 = conv2d_dgrad(dc2, pr.st(P["W2"]), saved["r1"].shape, s, 1)
        dc1, dgam1, dbet1 = bn_bwd(dr1 * (saved["r1"] > 0), saved["c1"], saved["st1"], P["gamma1"])
        dc1 = pr.st(dc1)
        dW1 = conv2d_wgrad(dc1, x, P["W1"].shape, 1, 0)
        grads = {"W1": dW1, "gamma1": dgam1, "beta1": dbet1, "W2": dW2, "gamma2": dgam2,
                 "beta2": dbet2, "W3": dW3, "gamma3": dgam3, "beta3": dbet3}
        dx_sc = ds
        if self.proj:
            dcp, dgamp, dbetp = bn_bwd(ds, saved["cp"], saved["stp"], P["gammap"])
            dcp = pr.st(dcp)
            grads.update(Wp=conv2d_wgrad(dcp, x, P["Wp"].shape, s, 0), gammap=dgamp, betap=dbetp)
            dx_sc = conv2d_dgrad(dcp, pr.st(P["Wp"]), x.shape, s, 0) if need_dx else None
        dx = None
        if need_dx:
            dx = conv2d_dgrad(dc1, pr.st(P["W1"]), x.shape, 1, 0) + dx_sc
        return dx, grads


class LSTMStep:
    """One time step with its softmax head.

    State in: (h_{t-1}, c_{t-1}); external: x_t [B,E], labels_t [B].
    z = x_t W_x + h_{t-1} W_h + b; gates i,f,g,o; c_t = f c_{t-1} + i g;
    h_t = o tanh(c_t); logits = h_t W_o + b_o; loss part = scale * sum_b CE.
    """
    kind = "lstm"

    def __init__(self, hidden, scale, prec=F64):
        self.H, self.scale, self.prec = hidden, scale, prec

    def fwd(self, state, P, ext):
        pr, H = self.prec, self.H
        h0, c0 = state
        x_t, lab = ext
        z = pr.st(x_t) @ pr.st(P["W_x"]) + h0 @ pr.st(P["W_h"]) + P["b"]
        i = sigmoid(z[:, :H])
        f = sigmoid(z[:, H:2 * H])
        gg = np.tanh(z[:, 2 * H:3 * H])
        o = sigmoid(z[:, 3 * H:])
        c = f * c0 + i * gg
        h = pr.st(o * np.tanh(c))
        logits = h @ pr.st(P["W_o"]) + P["b_o"]
        loss, dlog, p = softmax_ce(logits, lab, self.scale)
        return (h, c), {"i": i, "f": f, "g": gg, "o": o, "dlog": dlog}, loss

    def bwd(self, g, state, out, saved, P, ext, need_dx=True):
        pr, H = self.prec, self.H
        h0, c0 = state
        h, c = out
        dh, dc = g
        x_t, lab = ext
        dlog = pr.st(saved["dlog"])
        grads = {"W_o": h.T @ dlog, "b_o": saved["dlog"].sum(axis=0)}
        dh = dh + dlog @ pr.st(P["W_o"]).T
        i, f, gg, o = saved["i"], saved["f"], saved["g"], saved["o"]
        tc = np.tanh(c)
        do = dh * tc
        dct = dc + dh * o * (1 - tc * tc)
        di = dct * gg
        dg = dct * i
        df = dct * c0
        dz = np.concatenate([di * i * (1 - i), df * f * (1 - f), dg * (1 - gg * gg),
                             do * o * (1 - o)], axis=1)
        dzr = pr.st(dz)
        grads.update(W_x=pr.st(x_t).T @ dzr, W_h=h0.T @ dzr, b=dz.sum(axis=0))
        dh0 = dzr @ pr.st(P["W_h"]).T
        dc0 = dct * f
        return (dh0, dc0), grads


# --------------------------------------------------------------------------
# chain heads: fwd(x, P, target) -> (loss, g, saved)
# --------------------------------------------------------------------------

def mse_head(x, target):
    """L = mean over all elements of (x - t)^2; dL/dx = 2 (x - t) / count."""
    d = x - target
    cnt = d.size
    return (d * d).sum() / cnt, 2.0 * d / cnt


def pool_fc_ce_head(x, W, b, labels, prec=F64):
    """Global average pool, FC, softmax cross-entropy (mean over the batch)."""
    N, H, Wd, C = x.shape
    pooled = x.mean(axis=(1, 2))
    logits = pooled @ W + b
    loss, dlog, _ = softmax_ce(logits, labels, 1.0 / N)
    grads = {"W": pooled.T @ dlog, "b": dlog.sum(axis=0)}
    dpooled = dlog @ W.T
    g = np.broadcast_to(dpooled[:, None, None, :] / (H * Wd), x.shape).copy()
    return loss, g, grads
