"""GPU parity of the single bf16 operators of the bottleneck ResNet units
(section 5.2's deep residual network, the conv-BN-activation pipeline of
section 4.2) at the real channel widths, through the C ABI's operator calls.

Both sides receive exactly the same inputs: values drawn on the host, rounded
to bf16 by the oracle's rounding (so the upload to bf16 is exact) and given to
the GPU operator and to the float64 oracle.  With identical inputs the only
differences left are the GPU's fp32 accumulation order and, for bf16 outputs,
the rounding decision of values whose fp32 sum lies within that accumulation
error of a bf16 rounding midpoint.  Bars, per output:

* fp32 outputs (data and weight gradients, batch-norm sums and statistics):
  max |gpu - oracle| / max |oracle| <= 1e-4 (the fp32 bar);
* bf16 outputs (convolution outputs, batch-norm applies and backward, max
  pool): every element within one bf16 spacing of the exact value (one of the
  two bf16 neighbours of it) plus 1e-5 of the tensor's max-abs (the fp32
  accumulation error of values near zero), and at most 1% of the elements
  rounded differently from the exact value's nearest bf16;
* max pool and im2col: exact.

Shapes: the 7x7 stride-2 stem with its max pool at 224 x 224, the 1x1, 3x3
and projection convolutions of stages 1-4 (64 ... 2048 channels, strides 1
and 2), split-K weight gradients, every epilogue the units use (BF16STATS,
BNBWD, ADDMASK, ADD), ragged pixel counts and a narrow-channel case.
"""
import numpy as np
import pytest

from oracle import units as U

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _K():
    from paper_1604_06174_amd import ckpt as K
    return K


DEV = "cuda:0"


def bf(a):
    return U.bf16_round(np.asarray(a, np.float32)).astype(np.float32)


def dbf(a):  # exact: the values are bf16 already
    return torch.from_numpy(np.ascontiguousarray(bf(a))).to(DEV).to(torch.bfloat16)


def df(a):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, np.float32))).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.float().cpu().numpy().astype(np.float64)


def spacing(v):
    """bf16 spacing at |v| (8 significant bits): 2^(floor(log2 |v|) - 7)."""
    a = np.abs(np.asarray(v, np.float64))
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, np.exp2(e - 7), 0.0)


def check_f32(name, g, o, tol=1e-4):
    g = np.asarray(g, np.float64).reshape(-1)
    o = np.asarray(o, np.float64).reshape(-1)
    err = float(np.max(np.abs(g - o)) / max(np.max(np.abs(o)), 1e-30))
    print(f"    {name}: fp32 max rel {err:.2e}", flush=True)
    assert err <= tol, (name, err)


def check_bf16(name, g, o):
    g = np.asarray(g, np.float64).reshape(-1)
    o = np.asarray(o, np.float64).reshape(-1)
    tol = spacing(o) + 1e-5 * np.max(np.abs(o))
    bad = np.abs(g - o) > tol
    nearest = bf(o).astype(np.float64)
    frac = float(np.mean(g != nearest))
    err = float(np.max(np.abs(g - o)) / max(np.max(np.abs(o)), 1e-30))
    print(f"    {name}: bf16 max rel {err:.2e}, {int(bad.sum())} beyond one spacing, "
          f"{frac:.1e} rounded differently", flush=True)
    assert not bad.any(), (name, int(bad.sum()), np.flatnonzero(bad)[:8])
    assert frac <= 1e-2, (name, frac)


def act(rng, shape):
    """A post-ReLU activation: half zeros, the rest |N(0, 1)|."""
    return bf(np.maximum(rng.standard_normal(shape), 0))


def he(rng, co, r, ci):
    return bf(rng.normal(0.0, np.sqrt(2.0 / (r * r * ci)), (co, r, r, ci)))


def stats_of(c):
    """Batch-norm mean and 1/std (biased variance, eps 1e-5) over all but the
    channel axis, rounded to f32 as the GPU keeps them."""
    _, (mean, rstd) = U.bn_fwd(np.asarray(c, np.float64), 1.0, 0.0)
    return np.concatenate([mean, rstd]).astype(np.float32)


def finalize_fwd(K, stats, nb, j, m):
    st = torch.empty(2 * j, dtype=torch.float32, device=DEV)
    K.op_bn_finalize(False, stats, nb, j, m, st)
    return host(st)


def finalize_bwd(K, part, nb, j, m):
    sums = torch.empty(2 * j, dtype=torch.float32, device=DEV)
    dg = torch.empty(j, dtype=torch.float32, device=DEV)
    db = torch.empty(j, dtype=torch.float32, device=DEV)
    K.op_bn_finalize(True, part, nb, j, m, sums, dg, db)
    return host(sums), host(dg), host(db)


# --------------------------------------------------------------------------
# convolutions (implicit GEMM) and their statistics epilogue
# --------------------------------------------------------------------------
CONV = {
    # name: (n, h, ci, co, r, s)
    "s1_3x3_w64": (2, 56, 64, 64, 3, 1),
    "s2_3x3_w128_stride2": (2, 56, 128, 128, 3, 2),
    "s3_3x3_w256_stride2": (2, 28, 256, 256, 3, 2),
    "s4_3x3_w512": (2, 7, 512, 512, 3, 1),
    "proj_1x1_256to512_stride2": (2, 56, 256, 512, 1, 2),
    "proj_1x1_1024to2048_stride2": (2, 14, 1024, 2048, 1, 2),
    "narrow_3x3_8to16_odd": (3, 13, 8, 16, 3, 1),
}


def _geo(K, n, h, ci, co, r, s):
    p = r // 2
    ho = (h + 2 * p - r) // s + 1
    return K.conv_geo(n, h, h, ci, ho, ho, co, r, s, p), ho, p


@pytest.mark.parametrize("case", list(CONV))
def test_conv_fwd_stats(case):
    K = _K()
    n, h, ci, co, r, s = CONV[case]
    print(f"[op conv fwd] {case}", flush=True)
    rng = np.random.default_rng(11)
    geo, ho, p = _geo(K, n, h, ci, co, r, s)
    x, w = act(rng, (n, h, h, ci)), he(rng, co, r, ci)
    m = n * ho * ho
    rb, _ = K.op_gemm_bf16_blocks(m, co)
    y = torch.empty((n, ho, ho, co), dtype=torch.bfloat16, device=DEV)
    stats = torch.empty(rb * 2 * co, dtype=torch.float64, device=DEV)
    K.op_conv_bf16_fwd(geo, dbf(x), dbf(w), y, stats)
    st = finalize_fwd(K, stats, rb, co, m)
    ref = U.conv2d(x.astype(np.float64), w.astype(np.float64), s, p)
    check_bf16("y", host(y), ref)
    check_f32("mean|rstd", st, stats_of(bf(ref)))


@pytest.mark.parametrize("case", list(CONV))
@pytest.mark.parametrize("epi", ["store", "add", "bnbwd"])
def test_conv_dgrad(case, epi):
    K = _K()
    n, h, ci, co, r, s = CONV[case]
    print(f"[op conv dgrad] {case} epilogue {epi}", flush=True)
    rng = np.random.default_rng(12)
    geo, ho, p = _geo(K, n, h, ci, co, r, s)
    dy = bf(rng.standard_normal((n, ho, ho, co)) * 0.1)
    w = he(rng, co, r, ci)
    dx = torch.empty((n, h, h, ci), dtype=torch.float32, device=DEV)
    prod = U.conv2d_dgrad(dy.astype(np.float64), w.astype(np.float64), (n, h, h, ci), s, p)
    if epi == "store":
        K.op_conv_bf16_dgrad(geo, dbf(dy), dbf(w), dx, K.EPI_STORE)
        check_f32("dx", host(dx), prod)
    elif epi == "add":
        d = rng.standard_normal((n, h, h, ci)).astype(np.float32) * 0.05
        dx.copy_(df(d))  # D aliases C, as the projection's data gradient uses it
        K.op_conv_bf16_dgrad(geo, dbf(dy), dbf(w), dx, K.EPI_ADD, d=dx)
        check_f32("dx + d", host(dx), prod + d)
    else:
        cv = bf(rng.standard_normal((n, h, h, ci)))        # the batch norm's input
        st = stats_of(cv)
        mask = act(rng, (n, h, h, ci))                      # its ReLU output
        m = n * h * h
        rb, _ = K.op_gemm_bf16_blocks(m, ci)
        part = torch.empty(rb * 2 * ci, dtype=torch.float64, device=DEV)
        K.op_conv_bf16_dgrad(geo, dbf(dy), dbf(w), dx, K.EPI_BNBWD, mask=dbf(mask), cv=dbf(cv),
                             bst=df(st), stats=part)
        ds = prod * (mask > 0)
        check_f32("ds", host(dx), ds)
        sums, dg, db = finalize_bwd(K, part, rb, ci, m)
        xh = (cv.astype(np.float64) - st[:ci]) * st[ci:]
        ref_db = ds.reshape(-1, ci).sum(0)
        ref_dg = (ds * xh).reshape(-1, ci).sum(0)
        check_f32("sum ds", db, ref_db)
        check_f32("sum ds xhat", dg, ref_dg)
        check_f32("means", sums, np.concatenate([ref_db, ref_dg]) / m)


@pytest.mark.parametrize("case", list(CONV))
@pytest.mark.parametrize("splits", [1, 4])
def test_conv_wgrad(case, splits):
    K = _K()
    n, h, ci, co, r, s = CONV[case]
    print(f"[op conv wgrad] {case} splits {splits}", flush=True)
    rng = np.random.default_rng(13)
    geo, ho, p = _geo(K, n, h, ci, co, r, s)
    x = act(rng, (n, h, h, ci))
    dy = bf(rng.standard_normal((n, ho, ho, co)) * 0.1)
    dw = torch.empty((co, r, r, ci), dtype=torch.float32, device=DEV)
    part = torch.empty(max(splits, 1) * co * r * r * ci, dtype=torch.float32, device=DEV)
    K.op_conv_bf16_wgrad(geo, dbf(x), dbf(dy), part, splits, dw)
    ref = U.conv2d_wgrad(dy.astype(np.float64), x.astype(np.float64), (co, r, r, ci), s, p)
    check_f32("dw", host(dw), ref)


# --------------------------------------------------------------------------
# dense products: the 1x1 convolutions of stride 1
# --------------------------------------------------------------------------
DENSE = {
    # name: (pixels m, ci, co)
    "s1_1x1_64to256": (2 * 56 * 56, 64, 256),
    "s1_1x1_256to64": (2 * 56 * 56, 256, 64),
    "s3_1x1_1024to256": (2 * 14 * 14, 1024, 256),
    "s4_1x1_512to2048_ragged": (2 * 7 * 7, 512, 2048),
    "narrow_1x1_16to8_ragged": (3 * 13 * 13, 16, 8),
}


@pytest.mark.parametrize("case", list(DENSE))
def test_gemm_1x1_fwd_stats(case):
    K = _K()
    m, ci, co = DENSE[case]
    print(f"[op 1x1 fwd] {case}", flush=True)
    rng = np.random.default_rng(21)
    x = act(rng, (m, ci))
    w = he(rng, co, 1, ci).reshape(co, ci)
    rb, _ = K.op_gemm_bf16_blocks(m, co)
    y = torch.empty((m, co), dtype=torch.bfloat16, device=DEV)
    stats = torch.empty(rb * 2 * co, dtype=torch.float64, device=DEV)
    K.op_gemm_bf16(m, co, ci, dbf(x), ci, True, dbf(w), ci, True, None, co, K.EPI_BF16STATS,
                   cb=y, stats=stats)
    ref = x.astype(np.float64) @ w.astype(np.float64).T
    check_bf16("y", host(y), ref)
    check_f32("mean|rstd", finalize_fwd(K, stats, rb, co, m), stats_of(bf(ref)))


@pytest.mark.parametrize("case", list(DENSE))
@pytest.mark.parametrize("epi", ["store", "add", "addmask", "bnbwd"])
def test_gemm_1x1_dgrad(case, epi):
    """dx [m, ci] = dc [m, co] (bf16, k contiguous) times W [co, ci] (bf16)."""
    K = _K()
    m, ci, co = DENSE[case]
    print(f"[op 1x1 dgrad] {case} epilogue {epi}", flush=True)
    rng = np.random.default_rng(22)
    dc = bf(rng.standard_normal((m, co)) * 0.1)
    w = he(rng, co, 1, ci).reshape(co, ci)
    prod = dc.astype(np.float64) @ w.astype(np.float64)
    out = torch.empty((m, ci), dtype=torch.float32, device=DEV)
    if epi == "store":
        K.op_gemm_bf16(m, ci, co, dbf(dc), co, True, dbf(w), ci, False, out, ci, K.EPI_STORE)
        check_f32("dx", host(out), prod)
    elif epi == "add":
        d = rng.standard_normal((m, ci)).astype(np.float32) * 0.05
        out.copy_(df(d))
        K.op_gemm_bf16(m, ci, co, dbf(dc), co, True, dbf(w), ci, False, out, ci, K.EPI_ADD, d=out,
                       ldd=ci)
        check_f32("dx + d", host(out), prod + d)
    elif epi == "addmask":
        d = rng.standard_normal((m, ci)).astype(np.float32) * 0.05
        mask = act(rng, (m, ci))
        K.op_gemm_bf16(m, ci, co, dbf(dc), co, True, dbf(w), ci, False, out, ci, K.EPI_ADDMASK,
                       d=df(d), ldd=ci, mask=dbf(mask))
        check_f32("dx + [mask > 0] d", host(out), prod + d * (mask > 0))
    else:
        cv = bf(rng.standard_normal((m, ci)))
        st = stats_of(cv)
        mask = act(rng, (m, ci))
        rb, _ = K.op_gemm_bf16_blocks(m, ci)
        part = torch.empty(rb * 2 * ci, dtype=torch.float64, device=DEV)
        K.op_gemm_bf16(m, ci, co, dbf(dc), co, True, dbf(w), ci, False, out, ci, K.EPI_BNBWD,
                       mask=dbf(mask), cv=dbf(cv), bst=df(st), stats=part)
        ds = prod * (mask > 0)
        check_f32("ds", host(out), ds)
        sums, dg, db = finalize_bwd(K, part, rb, ci, m)
        xh = (cv.astype(np.float64) - st[:ci]) * st[ci:]
        check_f32("sum ds", db, ds.sum(0))
        check_f32("sum ds xhat", dg, (ds * xh).sum(0))


@pytest.mark.parametrize("case", list(DENSE))
@pytest.mark.parametrize("splits", [1, 5])
def test_gemm_1x1_wgrad(case, splits):
    """dW [co, ci] = dc^T x: both operands k-major ([pixels, channels])."""
    K = _K()
    m, ci, co = DENSE[case]
    print(f"[op 1x1 wgrad] {case} splits {splits}", flush=True)
    rng = np.random.default_rng(23)
    dc = bf(rng.standard_normal((m, co)) * 0.1)
    x = act(rng, (m, ci))
    dw = torch.empty((co, ci), dtype=torch.float32, device=DEV)
    if splits == 1:
        K.op_gemm_bf16(co, ci, m, dbf(dc), co, False, dbf(x), ci, False, dw, ci, K.EPI_STORE)
    else:
        part = torch.empty(splits * co * ci, dtype=torch.float32, device=DEV)
        K.op_gemm_bf16(co, ci, m, dbf(dc), co, False, dbf(x), ci, False, part, ci, K.EPI_STORE,
                       splits=splits)
        K.op_sum_partials(part, splits, co * ci, dw)
    check_f32("dW", host(dw), dc.astype(np.float64).T @ x.astype(np.float64))


# --------------------------------------------------------------------------
# the stem: 7x7 / 2 convolution through im2col + GEMM, max pool 3x3 / 2
# --------------------------------------------------------------------------
def test_stem_im2col_conv_maxpool():
    K = _K()
    print("[op stem] 2 x 224 x 224 x 3 -> 112 x 112 x 64 -> max pool 56 x 56", flush=True)
    rng = np.random.default_rng(31)
    n, h, c0 = 2, 224, 64
    ho = (h + 6 - 7) // 2 + 1
    x = bf(rng.random((n, h, h, 3)))
    w = he(rng, c0, 7, 3)
    m = n * ho * ho
    col = torch.empty((m, 147), dtype=torch.bfloat16, device=DEV)
    K.op_im2col7(n, h, h, ho, ho, dbf(x), col)
    # the network's form: rows padded to 160 (zero past 147), the product
    # over K = 160 with the weights padded the same way
    colp = torch.full((m, 160), float("nan"), dtype=torch.bfloat16, device=DEV)
    K.op_im2col7(n, h, h, ho, ho, dbf(x), colp, kp=160)
    assert torch.equal(colp[:, :147], col)
    assert bool((colp[:, 147:] == 0).all())
    # the patch matrix times the flattened weights is the convolution
    rb, _ = K.op_gemm_bf16_blocks(m, c0)
    cv = torch.empty((m, c0), dtype=torch.bfloat16, device=DEV)
    stats = torch.empty(rb * 2 * c0, dtype=torch.float64, device=DEV)
    K.op_gemm_bf16(m, c0, 147, col, 147, True, dbf(w.reshape(c0, 147)), 147, True, None, c0,
                   K.EPI_BF16STATS, cb=cv, stats=stats)
    ref = U.conv2d(x.astype(np.float64), w.astype(np.float64), 2, 3)
    check_bf16("stem conv", host(cv).reshape(ref.shape), ref)
    wp = np.zeros((c0, 160), np.float32)
    wp[:, :147] = w.reshape(c0, 147)
    cvp = torch.empty((m, c0), dtype=torch.bfloat16, device=DEV)
    K.op_gemm_bf16(m, c0, 160, colp, 160, True, dbf(wp), 160, True, None, c0,
                   K.EPI_BF16STATS, cb=cvp, stats=stats)
    check_bf16("stem conv, padded rows", host(cvp).reshape(ref.shape), ref)
    # the pool of a post-ReLU tensor, forward and backward, exact
    r = act(rng, (n, ho, ho, c0))
    pooled = (ho + 2 - 3) // 2 + 1
    y = torch.empty((n, pooled, pooled, c0), dtype=torch.bfloat16, device=DEV)
    rd = dbf(r)
    K.op_maxpool(False, n, ho, ho, c0, pooled, pooled, rd, y)
    yr, arg = U.maxpool_fwd(r.astype(np.float64))
    assert np.array_equal(host(y), yr)
    g = rng.standard_normal((n, pooled, pooled, c0)).astype(np.float32)
    dr = torch.empty((n, ho, ho, c0), dtype=torch.float32, device=DEV)
    K.op_maxpool(True, n, ho, ho, c0, pooled, pooled, rd, dr, g=df(g), y=y)
    check_f32("max pool gradient", host(dr), U.maxpool_bwd(g.astype(np.float64), arg, r.shape), 1e-6)
    # the two-pass form (the network's): the same bits
    dr2 = torch.empty_like(dr)
    ws = torch.empty(n * pooled * pooled * c0, dtype=torch.uint8, device=DEV)
    K.op_maxpool(True, n, ho, ho, c0, pooled, pooled, rd, dr2, g=df(g), y=y, arg=ws)
    assert torch.equal(dr2, dr)
    # the stem's weight gradient: patches^T dc, split over the pixels
    dc = bf(rng.standard_normal((m, c0)) * 0.1)
    part = torch.empty(8 * c0 * 147, dtype=torch.float32, device=DEV)
    dw = torch.empty((c0, 147), dtype=torch.float32, device=DEV)
    K.op_gemm_bf16(c0, 147, m, dbf(dc), c0, False, col, 147, False, part, 147, K.EPI_STORE, splits=8)
    K.op_sum_partials(part, 8, c0 * 147, dw)
    ref_dw = U.conv2d_wgrad(dc.reshape(n, ho, ho, c0).astype(np.float64), x.astype(np.float64),
                            (c0, 7, 7, 3), 2, 3)
    check_f32("stem dW", host(dw), ref_dw.reshape(c0, 147))


# --------------------------------------------------------------------------
# batch norm (bf16 tensors, f64 sums): apply with each shortcut, backward
# --------------------------------------------------------------------------
BN = {"w64_56": (2 * 56 * 56, 64), "w256_28": (2 * 28 * 28, 256), "w2048_7_ragged": (3 * 7 * 7, 2048),
      "w8_odd": (3 * 13 * 13, 8)}


def _bn_params(rng, j):
    return (rng.uniform(0.5, 1.5, j).astype(np.float32), rng.normal(0, 0.3, j).astype(np.float32))


@pytest.mark.parametrize("case", list(BN))
@pytest.mark.parametrize("res", ["none", "id", "bn"])
def test_bnb_apply(case, res):
    K = _K()
    p, j = BN[case]
    print(f"[op bn apply] {case} shortcut {res}", flush=True)
    rng = np.random.default_rng(41)
    c = bf(rng.standard_normal((p, j)) * 2 + 0.5)
    st = stats_of(c)
    gam, bet = _bn_params(rng, j)
    x = bf(rng.standard_normal((p, j)))
    y = torch.empty((p, j), dtype=torch.bfloat16, device=DEV)
    pre = gam * ((c.astype(np.float64) - st[:j]) * st[j:]) + bet
    if res == "none":
        K.op_bnb_apply(K.BNB_RES_NONE, p, j, dbf(c), df(st), df(gam), df(bet), y=y)
    elif res == "id":
        K.op_bnb_apply(K.BNB_RES_ID, p, j, dbf(c), df(st), df(gam), df(bet), x=dbf(x), y=y)
        pre = pre + x
    else:
        stp = stats_of(x)
        gp, bp = _bn_params(rng, j)
        K.op_bnb_apply(K.BNB_RES_BN, p, j, dbf(c), df(st), df(gam), df(bet), x=dbf(x), stp=df(stp),
                       gp=df(gp), bp=df(bp), y=y)
        pre = pre + gp * ((x.astype(np.float64) - stp[:j]) * stp[j:]) + bp
    check_bf16("y", host(y), np.maximum(pre, 0))


@pytest.mark.parametrize("case", list(BN))
@pytest.mark.parametrize("masked", [True, False])
def test_bnb_backward(case, masked):
    K = _K()
    p, j = BN[case]
    print(f"[op bn backward] {case} masked {masked}", flush=True)
    rng = np.random.default_rng(42)
    c = bf(rng.standard_normal((p, j)) * 2 + 0.5)
    st = stats_of(c)
    gam, _ = _bn_params(rng, j)
    g = rng.standard_normal((p, j)).astype(np.float32)
    ym = act(rng, (p, j))
    nb = K.op_bnb_partial_blocks(p, j)
    part = torch.empty(nb * 2 * j, dtype=torch.float64, device=DEV)
    sums = torch.empty(2 * j, dtype=torch.float32, device=DEV)
    dg = torch.empty(j, dtype=torch.float32, device=DEV)
    db = torch.empty(j, dtype=torch.float32, device=DEV)
    d = torch.empty((p, j), dtype=torch.bfloat16, device=DEV)
    K.op_bnb_backward(p, j, df(g), dbf(ym) if masked else None, dbf(c), df(st), df(gam), part, sums,
                      dg, db, d)
    ds = g.astype(np.float64) * ((ym > 0) if masked else 1.0)
    xh = (c.astype(np.float64) - st[:j]) * st[j:]
    rdb, rdg = ds.sum(0), (ds * xh).sum(0)
    check_f32("dbeta", host(db), rdb)
    check_f32("dgamma", host(dg), rdg)
    ref = gam * st[j:] * (ds - rdb / p - xh * (rdg / p))
    check_bf16("dc", host(d), ref)
    # the element pass alone, from the same sums
    d2 = torch.empty((p, j), dtype=torch.bfloat16, device=DEV)
    K.op_bnb_backward_apply(p, j, df(g), dbf(ym) if masked else None, dbf(c), df(st), df(gam), sums, d2)
    assert torch.equal(d, d2)


def test_operator_arguments_are_validated():
    K = _K()
    x = torch.zeros(64, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(K.CkptError) as e:
        K.op_conv_bf16_fwd(K.conv_geo(1, 4, 4, 12, 4, 4, 16, 3, 1, 1), x, x, x, x)  # 12 channels
    assert e.value.code == K.E_UNSUPPORTED
    with pytest.raises(K.CkptError) as e:
        K.op_conv_bf16_fwd(K.conv_geo(1, 4, 4, 16, 3, 3, 16, 3, 1, 1), x, x, x, x)  # wrong ho
    assert e.value.code == K.E_UNSUPPORTED
    with pytest.raises(K.CkptError) as e:
        K.op_gemm_bf16(8, 8, 8, x, 8, True, x, 8, True, x, 8, K.EPI_ADD, splits=2)
    assert e.value.code == K.E_INVALID
    with pytest.raises(K.CkptError) as e:
        K.op_bnb_apply(K.BNB_RES_ID, 8, 8, x, x, x, x, y=x)  # identity shortcut without x
    assert e.value.code == K.E_INVALID
