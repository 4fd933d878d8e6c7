"""GPU parity of every per-layer entry point against the oracle, through the
C ABI (paper_1912_12675_amd.psw), on seeded inputs that span several tiles
and ragged tails.  Tolerances: the oracle is float64; the GPU accumulates in
float32, so the worst error relative to the largest reference magnitude is
held to 2e-5 (fp32).  In bf16 mode both sides round the same float32 operands
to bfloat16, so the same bound applies."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

TOL = 2e-5


@pytest.fixture(scope="module")
def P():
    from paper_1912_12675_amd import psw
    psw.lib()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return psw


def dev(a, dtype=torch.float32):
    return torch.as_tensor(np.ascontiguousarray(a)).to(dtype).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.double().cpu().numpy()


def assert_close(gpu, ref, tol=TOL, what=""):
    g = host(gpu) if isinstance(gpu, torch.Tensor) else np.asarray(gpu)
    r = np.asarray(ref, dtype=np.float64)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    scale = max(np.abs(r).max(), 1e-30)
    err = np.abs(g - r).max() / scale
    assert err <= tol, f"{what}: max err {err:.3e} (scale {scale:.3e})"


def f32(rng, shape, scale=1.0):
    return (rng.standard_normal(shape) * scale).astype(np.float32)


CONV = [
    # N, C, H, W, K, R, stride, pad
    (2, 16, 32, 32, 16, 3, 1, 1),
    (2, 16, 32, 32, 32, 3, 2, 1),
    (2, 32, 16, 16, 64, 3, 2, 1),
    (2, 64, 8, 8, 64, 3, 1, 1),
    (3, 3, 32, 32, 16, 3, 1, 1),
    (3, 5, 13, 11, 7, 3, 1, 1),
    (2, 6, 14, 14, 16, 5, 1, 0),
    (2, 1, 28, 28, 6, 5, 1, 2),
    (2, 3, 9, 9, 20, 5, 2, 2),
    (1, 33, 7, 9, 70, 3, 1, 1),
    (5, 3, 6, 6, 4, 1, 1, 0),
    (1, 64, 4, 4, 130, 3, 1, 1),
    # shapes of the direct 3x3 kernel: ResNet groups 1-3, the stride-2
    # transitions, VGG layers with several input-channel chunks and
    # several output-channel blocks
    (3, 32, 16, 16, 32, 3, 1, 1),
    (2, 64, 32, 32, 64, 3, 1, 1),
    (2, 128, 16, 16, 128, 3, 1, 1),
    (2, 256, 8, 8, 256, 3, 1, 1),
    (3, 16, 16, 16, 64, 3, 2, 1),
    (2, 48, 16, 16, 32, 3, 2, 1),
    # the ResNet group-2 and group-3 weight-gradient tilings need 2 and 4
    # images per workgroup
    (4, 32, 16, 16, 32, 3, 1, 1),
    (8, 64, 8, 8, 64, 3, 1, 1),
]


@pytest.mark.parametrize("case", CONV, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
def test_conv_parity(P, oracle, case, bf16):
    N, C, H, W, K, R, st, pad = case
    print(f"conv {case} bf16={bf16}", flush=True)
    rng = np.random.default_rng(abs(hash(case)) % 2**32)
    x, w, b = f32(rng, (N, C, H, W)), f32(rng, (K, C, R, R), 0.3), f32(rng, (K,))
    Pq = (H + 2 * pad - R) // st + 1
    Qq = (W + 2 * pad - R) // st + 1
    dy = f32(rng, (N, K, Pq, Qq))
    xg, wg, bg, dyg = dev(x), dev(w), dev(b), dev(dy)
    # forward, with and without bias + ReLU
    y = torch.empty((N, K, Pq, Qq), device="cuda")
    P.psw_conv_fwd(xg, wg, y, st, pad, bf16=bf16)
    ref = oracle.conv_fwd(x, w, None, st, pad, bf16=bf16)
    assert_close(y, ref, what="fwd")
    P.psw_conv_fwd(xg, wg, y, st, pad, bias=bg, relu=True, bf16=bf16)
    assert_close(y, np.maximum(oracle.conv_fwd(x, w, b, st, pad, bf16=bf16), 0), what="fwd+bias+relu")
    # backward data, overwrite and accumulate
    dx = torch.full((N, C, H, W), 7.0, device="cuda")
    P.psw_conv_bwd_data(x.shape, wg, dyg, dx, st, pad, bf16=bf16)
    refdx = oracle.conv_bwd_data(x.shape, w, dy, st, pad, bf16=bf16)
    assert_close(dx, refdx, what="bwd_data")
    base = f32(rng, (N, C, H, W))
    dx = dev(base)
    P.psw_conv_bwd_data(x.shape, wg, dyg, dx, st, pad, accumulate=True, bf16=bf16)
    assert_close(dx, refdx + base, what="bwd_data accumulate")
    # backward weight (+ bias)
    dw = torch.full((K, C, R, R), 7.0, device="cuda")
    db = torch.full((K,), 7.0, device="cuda")
    P.psw_conv_bwd_weight(xg, dyg, dw, st, pad, dbias=db, bf16=bf16)
    rdw, rdb = oracle.conv_bwd_weight(x, w.shape, dy, st, pad, bias=True, bf16=bf16)
    assert_close(dw, rdw, what="bwd_weight")
    assert_close(db, rdb, what="bwd_bias")


@pytest.mark.parametrize("shape,res_kind,relu", [
    ((2, 16, 32, 32), "identity", True),
    ((3, 32, 16, 16), "optionA", True),
    ((5, 7, 3, 5), None, False),
    ((4, 64, 8, 8), "optionA", False),
    ((2, 10, 9, 9), None, True),
])
def test_bn_parity(P, oracle, shape, res_kind, relu):
    print(f"bn {shape} {res_kind} relu={relu}", flush=True)
    rng = np.random.default_rng(sum(shape))
    N, C, H, W = shape
    y = f32(rng, shape, 2.0) + 0.5
    g = rng.uniform(0.5, 1.5, C).astype(np.float32)
    be = f32(rng, (C,))
    res = None
    if res_kind == "identity":
        res = f32(rng, shape)
    elif res_kind == "optionA":
        res = f32(rng, (N, C // 2, 2 * H, 2 * W))
    rm, rv = np.zeros(C), np.ones(C)
    z_ref, mean_ref, inv_ref = oracle.bn_fwd(y, g, be, res=res, relu=relu, run_mean=rm, run_var=rv)
    yg = dev(y)
    z = torch.empty(shape, device="cuda")
    sm, si = torch.empty(C, device="cuda"), torch.empty(C, device="cuda")
    rmg, rvg = torch.zeros(C, device="cuda"), torch.ones(C, device="cuda")
    P.psw_bn_relu_fwd(yg, dev(g), dev(be), z, sm, si, res=None if res is None else dev(res), relu=relu,
                      run_mean=rmg, run_var=rvg)
    assert_close(z, z_ref, what="z")
    assert_close(sm, mean_ref, what="mean")
    assert_close(si, inv_ref, what="invstd")
    assert_close(rmg, rm, what="run_mean")
    assert_close(rvg, rv, what="run_var")
    dz = f32(rng, shape)
    dy_ref, dg_ref, db_ref, dres_ref = oracle.bn_bwd(dz, z_ref, y, g, mean_ref, inv_ref, relu=relu,
                                                     res_shape=None if res is None else res.shape)
    # backward from the GPU's own forward outputs (z, mean, invstd)
    dy = torch.empty(shape, device="cuda")
    dgam, dbet = torch.empty(C, device="cuda"), torch.empty(C, device="cuda")
    dres = None if res is None else torch.full(res.shape, 3.0, device="cuda")
    P.psw_bn_relu_bwd(dev(dz), z, yg, dev(g), sm, si, dy, dgam, dbet, dres=dres, relu=relu)
    assert_close(dy, dy_ref, 5e-5, what="dy")
    assert_close(dgam, dg_ref, what="dgamma")
    assert_close(dbet, db_ref, what="dbeta")
    if res is not None:
        assert_close(dres, dres_ref, what="dres")
        base = f32(rng, res.shape)
        dres2 = dev(base)
        P.psw_bn_relu_bwd(dev(dz), z, yg, dev(g), sm, si, dy, dgam, dbet, dres=dres2, relu=relu, res_accumulate=True)
        assert_close(dres2, dres_ref + base, what="dres accumulate")


@pytest.mark.parametrize("shape", [(2, 3, 8, 8), (2, 5, 7, 9), (3, 64, 32, 32)])
def test_maxpool_parity(P, oracle, shape):
    rng = np.random.default_rng(sum(shape))
    x = f32(rng, shape)
    y_ref, am_ref = oracle.maxpool_fwd(x, 2, 2)
    N, C, H, W = shape
    y = torch.empty(y_ref.shape, device="cuda")
    am = torch.empty(y_ref.shape, dtype=torch.int32, device="cuda")
    xg = dev(x)
    P.psw_pool_fwd(P.PSW_POOL_MAX, xg, y, 2, 2, argmax=am)
    assert_close(y, y_ref, 0.0, what="y")
    torch.cuda.synchronize()
    np.testing.assert_array_equal(am.cpu().numpy(), am_ref)
    dy = f32(rng, y_ref.shape)
    dx = torch.full(shape, 5.0, device="cuda")
    P.psw_pool_bwd(P.PSW_POOL_MAX, shape, dev(dy), dx, 2, 2, argmax=am)
    assert_close(dx, oracle.maxpool_bwd(shape, 2, 2, dy, am_ref), 0.0, what="dx")
    # ties: all-equal windows route to the first element
    z = torch.zeros(shape, device="cuda")
    P.psw_pool_fwd(P.PSW_POOL_MAX, z, y, 2, 2, argmax=am)
    _, am0 = oracle.maxpool_fwd(np.zeros(shape), 2, 2)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(am.cpu().numpy(), am0)


@pytest.mark.parametrize("shape", [(3, 64, 8, 8), (2, 5, 7, 3)])
def test_gavgpool_parity(P, oracle, shape):
    rng = np.random.default_rng(sum(shape))
    x = f32(rng, shape)
    y = torch.empty(shape[:2], device="cuda")
    P.psw_pool_fwd(P.PSW_POOL_GAVG, dev(x), y)
    assert_close(y, oracle.gavgpool_fwd(x), what="y")
    dy = f32(rng, shape[:2])
    dx = torch.empty(shape, device="cuda")
    P.psw_pool_bwd(P.PSW_POOL_GAVG, shape, dev(dy), dx)
    assert_close(dx, oracle.gavgpool_bwd(shape, dy), what="dx")
    base = f32(rng, shape)
    dx = dev(base)
    P.psw_pool_bwd(P.PSW_POOL_GAVG, shape, dev(dy), dx, accumulate=True)
    assert_close(dx, oracle.gavgpool_bwd(shape, dy) + base, what="dx acc")


@pytest.mark.parametrize("n,fin,fout,relu", [(5, 37, 13, False), (128, 64, 10, False), (3, 400, 120, True),
                                             (70, 300, 130, True), (4, 2048, 96, False),
                                             (256, 100, 16, True), (64, 4096, 64, False)])
@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
def test_fc_parity(P, oracle, n, fin, fout, relu, bf16):
    rng = np.random.default_rng(n * 1000 + fin + fout)
    x, w, b = f32(rng, (n, fin)), f32(rng, (fout, fin), 0.1), f32(rng, (fout,))
    y = torch.empty((n, fout), device="cuda")
    P.psw_fc_fwd(dev(x), dev(w), y, b=dev(b), relu=relu, bf16=bf16)
    ref = oracle.fc_fwd(x, w, b, bf16=bf16)
    if relu:
        ref = np.maximum(ref, 0)
    assert_close(y, ref, what="fc fwd")
    dy = f32(rng, (n, fout))
    dx, dw, db = torch.empty((n, fin), device="cuda"), torch.empty((fout, fin), device="cuda"), \
        torch.empty(fout, device="cuda")
    P.psw_fc_bwd(dev(x), dev(w), dev(dy), dw, dx=dx, db=db, bf16=bf16)
    rdx, rdw, rdb = oracle.fc_bwd(x, w, dy, bf16=bf16)
    assert_close(dx, rdx, what="fc dx")
    assert_close(dw, rdw, what="fc dw")
    assert_close(db, rdb, what="fc db")
    base = f32(rng, (n, fin))
    dx2 = dev(base)
    P.psw_fc_bwd(dev(x), dev(w), dev(dy), dw, dx=dx2, dx_accumulate=True, bf16=bf16)
    assert_close(dx2, rdx + base, what="fc dx acc")


@pytest.mark.parametrize("n,p,offset", [(5, 0.5, 0), (1 << 20, 0.3, 0), (1000003, 0.5, 1), (4097, 0.9, 3)])
def test_dropout_parity(P, oracle, n, p, offset):
    """Keep decisions bit-exact against the oracle's (integer comparisons of
    the same Philox words); kept values within fp32 rounding; forward and
    accumulating backward; ragged counts and misaligned (scalar) views."""
    from paper_1912_12675_amd import synth
    k = synth.dropout_threshold(p)
    rng = np.random.default_rng(n + offset)
    x = f32(rng, (n,))
    seed, op, t = 0x0123_4567_89AB_CDEF, 11, (1 << 32) + 17
    xb = torch.zeros(n + offset, device="cuda")
    xb[offset:] = dev(x)
    yb = torch.full((n + offset,), 7.0, device="cuda")
    P.psw_dropout(xb[offset:], yb[offset:], k, seed, op, t)
    ref = oracle.dropout_fwd(x, k, seed, op, t)
    y = yb[offset:].cpu().numpy()
    np.testing.assert_array_equal(y == 0, ref == 0)
    np.testing.assert_allclose(y, ref, rtol=2e-7, atol=0)
    assert yb[:offset].eq(7.0).all()
    base = f32(rng, (n,))
    gb = torch.zeros(n + offset, device="cuda")
    gb[offset:] = dev(base)
    P.psw_dropout(xb[offset:], gb[offset:], k, seed, op, t, accumulate=True)
    np.testing.assert_allclose(gb[offset:].cpu().numpy(), base + oracle.dropout_bwd(x, k, seed, op, t), rtol=1e-6,
                               atol=1e-6)


def test_dropout_rejects_bad_arguments(P):
    x = torch.zeros(8, device="cuda")
    for kw in (dict(p24=0), dict(p24=1 << 24)):
        with pytest.raises(P.PswError):
            P.psw_dropout(x, x, kw["p24"], 1, 0, 0)
    with pytest.raises(P.PswError):
        P.psw_dropout(x, x, 100, 1, 0, -1)
    P.psw_dropout(x[:0], x[:0], 100, 1, 0, 0)  # empty: nothing to do


def test_relu_mask(P):
    rng = np.random.default_rng(1)
    z = np.maximum(f32(rng, (1000,)), 0)
    g = f32(rng, (1000,))
    gg = dev(g)
    P.psw_relu_mask(dev(z), gg)
    assert_close(gg, np.where(z > 0, g, 0.0), 0.0)


@pytest.mark.parametrize("n,classes", [(9, 10), (128, 10), (300, 7)])
def test_softmax_xent_parity(P, oracle, n, classes):
    rng = np.random.default_rng(n + classes)
    z = f32(rng, (n, classes), 3.0)
    lab = rng.integers(0, classes, n).astype(np.int32)
    loss = torch.empty(1, device="cuda")
    dz = torch.empty((n, classes), device="cuda")
    P.psw_softmax_xent(dev(z), dev(lab, torch.int32), loss, dz)
    rl, rdz = oracle.softmax_xent(z, lab)
    assert_close(loss, [rl], what="loss")
    assert_close(dz, rdz, what="dz")


@pytest.mark.parametrize("count,nesterov,wd,inplace", [(1000, False, 0.0, False), (4099, True, 5e-4, True),
                                                       (1, False, 1e-4, True)])
def test_sgd_parity(P, oracle, count, nesterov, wd, inplace):
    rng = np.random.default_rng(count)
    w, v, g = f32(rng, (count,)), f32(rng, (count,)), f32(rng, (count,))
    wg, vg, gg = dev(w), dev(v), dev(g)
    out = wg if inplace else torch.empty(count, device="cuda")
    P.psw_sgd_momentum_step(wg, out, vg, gg, 0.05, 0.9, wd, nesterov)
    rw, rv = oracle.sgd(w, v, g, 0.05, 0.9, wd, nesterov)
    assert_close(out, rw, 1e-6, what="w")
    assert_close(vg, rv, 1e-6, what="v")
