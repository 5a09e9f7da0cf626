"""GPU parity of the HIP path against the CPU oracle (through the C ABI).

int32 accumulators must match bit-exactly; fp32 outputs within 1e-5 relative
(y_ref = 0 requires y = 0).  Quantized activations and their scales must match
bit-exactly (both sides decide in fp32).
"""
import ctypes
import sys

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

RTOL = 1e-5
# host threads of the oracle in the full-size checks (the CPU share of one GPU)
ORACLE_THREADS = 16


def _sh():
    import paper_2601_07892_amd as sh
    return sh


def _say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def dev():
    d = torch.device("cuda:0")
    torch.cuda.set_device(d)
    return d


def _y_ok(y, y_ref):
    y = np.asarray(y, np.float64)
    bad = np.abs(y - y_ref) > RTOL * np.abs(y_ref)
    return not bad.any()


def _run(dev, t, q, sx, sw, kernel, m, with_acc=True, packed=None):
    sh = _sh()
    n, k = t.shape
    w = torch.from_numpy(packed if packed is not None else sh.sherry_pack(t)).to(dev)
    qd = torch.from_numpy(np.ascontiguousarray(q)).to(dev)
    sxd = torch.from_numpy(np.ascontiguousarray(sx)).to(dev)
    y = torch.full((m, n), float("nan"), dtype=torch.float32, device=dev)
    acc = torch.full((m, n), -7, dtype=torch.int32, device=dev) if with_acc else None
    sh.sherry_gemm_ex(w, qd, sxd, sw, y, acc, m, n, k, kernel)
    torch.cuda.synchronize()
    return y.cpu().numpy(), (acc.cpu().numpy() if with_acc else None)


# ---------------------------------------------------------------- quantizer

@pytest.mark.parametrize("m,k,outl", [(1, 4, 0.0), (3, 1000, 0.0), (7, 2048, 0.01),
                                      (64, 8192, 0.01), (2048, 3072, 0.01), (5, 14336, 0.01),
                                      (3, 16388, 0.0), (2, 40000, 0.01)])
def test_quantize_bit_exact(dev, m, k, outl):
    sh = _sh()
    _say("quantize", m, k, outl)
    x = synth.activations(m, k, 31, "q", outlier_frac=outl)
    if m >= 3:
        x[1] = 0.0           # all-zero token
        x[2, :4] = [0.5, 1.5, 2.5, -127.0]  # ties after scaling by absmax 127
        x[2, 4:] = 0.0
    xd = torch.from_numpy(x).to(dev)
    q = torch.empty((m, k), dtype=torch.int8, device=dev)
    sx = torch.empty(m, dtype=torch.float32, device=dev)
    sh.sherry_quantize_act(xd, q, sx)
    torch.cuda.synchronize()
    q_ref, sx_ref = oracle.quantize_act(x)
    assert np.array_equal(sx.cpu().numpy(), sx_ref)
    assert np.array_equal(q.cpu().numpy(), q_ref)


def _near_tie_rows(k, seed):
    """Rows whose values sit on, or within a few ulps of, the rounding
    boundaries (j + 1/2) * s of their own scale s = absmax / 127, for several
    absmax values (s exact, s inexact, s denormal-range)."""
    rng = np.random.default_rng(seed)
    rows = []
    for amax in (127.0, 1.0, 3.0e-3, 1.7e-36, 2.5e30, 0.7):
        s = np.float32(np.float32(amax) / np.float32(127.0))
        j = rng.integers(-127, 127, k).astype(np.float32)
        x = ((j + np.float32(0.5)) * s).astype(np.float32)
        steps = rng.integers(-3, 4, k)
        x = np.array([np.float32(v) if d == 0 else
                      np.nextafter(v, np.float32(np.inf) if d > 0 else np.float32(-np.inf),
                                   dtype=np.float32) for v, d in zip(x, steps)], np.float32)
        for d in range(2):  # some values two and three ulps away
            sel = rng.random(k) < 0.2
            x[sel] = np.nextafter(x[sel], np.float32(np.inf), dtype=np.float32)
        x[0] = np.float32(amax)
        x = np.clip(x, -np.float32(amax), np.float32(amax))
        rows.append(x)
    return np.stack(rows).astype(np.float32)


@pytest.mark.parametrize("k", [256, 4096])
def test_quantize_near_ties(dev, k):
    # values on and next to the half-integer boundaries of x / s: the kernels
    # round through a reciprocal and fall back to the division near them
    sh = _sh()
    x = _near_tie_rows(k, 36 + k)
    m = x.shape[0]
    xd = torch.from_numpy(x).to(dev)
    q = torch.empty((m, k), dtype=torch.int8, device=dev)
    sx = torch.empty(m, dtype=torch.float32, device=dev)
    sh.sherry_quantize_act(xd, q, sx)
    torch.cuda.synchronize()
    q_ref, sx_ref = oracle.quantize_act(x)
    assert np.array_equal(sx.cpu().numpy(), sx_ref)
    assert np.array_equal(q.cpu().numpy(), q_ref)
    # the fused kernel quantizes the same rows on chip: one-hot T reads q back
    n = 64
    t = np.tile(np.array([0, 1, 1, 1], np.int8), (n, k // 4))
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    for r in range(m):
        a = torch.empty(n, dtype=torch.int32, device=dev)
        y = torch.empty(n, dtype=torch.float32, device=dev)
        s1 = torch.empty(1, dtype=torch.float32, device=dev)
        sh.sherry_gemv_f32(w, xd[r].contiguous(), s1, 1.0, y, a, n, k)
        torch.cuda.synchronize()
        assert s1.item() == sx_ref[r]
        assert np.array_equal(a.cpu().numpy(), oracle.gemm_i32(q_ref[r:r + 1], t)[0])


# ------------------------------------------------------- decode kernel (M<=4)

GEMV_SHAPES = [(1, 4), (64, 128), (65, 132), (1, 124), (130, 1028), (257, 2048),
               (512, 2048), (300, 3072), (64, 8192 + 4)]


@pytest.mark.parametrize("n,k", GEMV_SHAPES)
@pytest.mark.parametrize("m", [1, 2, 3, 4])
def test_gemv_kernel_parity(dev, m, n, k):
    sh = _sh()
    _say("gemv", m, n, k)
    t = synth.ternary_34(n, k, 32, "gv", n, k)
    q = synth.int8_any(m, k, 32, "gv", m, k)
    sx = np.abs(synth.activations(1, m, 32, "gvs", m)[0]).astype(np.float32) + 0.01
    sw = synth.weight_scale(32, "gv", n, k)
    y, acc = _run(dev, t, q, sx, sw, sh.SHERRY_KERNEL_GEMV, m)
    acc_ref = oracle.gemm_i32(q, t, threads=4)
    assert np.array_equal(acc, acc_ref)
    assert _y_ok(y, oracle.epilogue(acc_ref, sx, sw))


# ---------------------------------------------------------- MFMA kernel

MFMA_CASES = [(5, 64, 128), (16, 65, 132), (32, 256, 1024), (33, 300, 1032), (64, 512, 2048),
              (100, 257, 516), (256, 512, 2048), (300, 700, 3072), (512, 1024, 1536),
              (1, 128, 256), (4, 64, 128)]


@pytest.mark.parametrize("m,n,k", MFMA_CASES)
def test_mfma_kernel_parity(dev, m, n, k):
    sh = _sh()
    _say("mfma", m, n, k)
    t = synth.ternary_34(n, k, 33, "mf", n, k)
    q = synth.int8_any(m, k, 33, "mf", m, k)
    sx = np.abs(synth.activations(1, m, 33, "mfs", m)[0]).astype(np.float32) + 0.01
    sw = synth.weight_scale(33, "mf", n, k)
    y, acc = _run(dev, t, q, sx, sw, sh.SHERRY_KERNEL_MFMA, m)
    acc_ref = oracle.gemm_i32(q, t, threads=8)
    assert np.array_equal(acc, acc_ref)
    assert _y_ok(y, oracle.epilogue(acc_ref, sx, sw))


def test_mfma_large_tile_config(dev):
    # M, N large enough that the 256x256 tile configuration is chosen
    sh = _sh()
    m, n, k = 2048, 8192, 640
    _say("mfma-large", m, n, k)
    t = synth.ternary_34(n, k, 34, "ml")
    q = synth.int8_any(m, k, 34, "ml")
    sx = np.full(m, 0.5, np.float32)
    y, acc = _run(dev, t, q, sx, 0.25, sh.SHERRY_KERNEL_MFMA, m)
    assert np.array_equal(acc, oracle.gemm_i32(q, t, threads=ORACLE_THREADS))
    # exact scale products: y = acc / 8 exactly
    assert np.array_equal(y.astype(np.float64), acc.astype(np.float64) * 0.125)


@pytest.mark.parametrize("kernel", ["MFMA", "SKINNY"])
@pytest.mark.parametrize("m,n,k", [(64, 256, 512), (300, 512, 1032), (2048, 1024, 640)])
def test_epilogue_unaligned_outputs(dev, kernel, m, n, k):
    # y and acc 4 bytes past a 16-byte boundary (n a multiple of 4): the MFMA
    # kernels' 16-byte row stores must fall back to 4-byte stores
    sh = _sh()
    _say("unaligned epilogue", kernel, m, n, k)
    t = synth.ternary_34(n, k, 37, "ua", n, k)
    q = synth.int8_any(m, k, 37, "uaq", m, k)
    sx = np.abs(synth.activations(1, m, 37, "uas", m)[0]).astype(np.float32) + 0.01
    sw = _channel_scales(n, 37)
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    yb = torch.full((m * n + 4,), float("nan"), dtype=torch.float32, device=dev)
    ab = torch.full((m * n + 4,), -7, dtype=torch.int32, device=dev)
    y, acc = yb[1:1 + m * n], ab[1:1 + m * n]
    assert y.data_ptr() % 16 == 4 and acc.data_ptr() % 16 == 4
    sh.sherry_gemm_channel(w, torch.from_numpy(q).to(dev), torch.from_numpy(sx).to(dev),
                           torch.from_numpy(sw).to(dev), y, acc, m, n, k,
                           getattr(sh, "SHERRY_KERNEL_" + kernel))
    torch.cuda.synchronize()
    acc_ref = oracle.gemm_i32(q, t, threads=8)
    assert np.array_equal(acc.cpu().numpy().reshape(m, n), acc_ref)
    assert _y_ok(y.cpu().numpy().reshape(m, n), oracle.epilogue_rows(acc_ref, sx, sw))
    # the guard words on both sides are untouched
    assert np.isnan(yb[0].item()) and np.isnan(yb[-3:].cpu().numpy()).all()
    assert ab[0].item() == -7 and (ab[-3:].cpu().numpy() == -7).all()


# ------------------------------------------- activation-table kernel (M = 1)

ALUT_CASES = [(1, 4), (64, 128), (65, 132), (300, 1032), (2048, 2048), (512, 8192),
              (3072, 8188), (100, 260)]


@pytest.mark.parametrize("n,k", ALUT_CASES)
@pytest.mark.parametrize("channel", [False, True])
def test_activation_table_kernel_parity(dev, n, k, channel):
    sh = _sh()
    _say("alut", n, k, channel)
    t = synth.ternary_34(n, k, 39, "al", n, k)
    q = synth.int8_any(1, k, 39, "alq", k)
    q[0, :min(k, 8)] = [-128, -128, -128, -128, 127, 127, 127, 127][:min(k, 8)]  # extreme entries
    sx = np.array([0.037], np.float32)
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    y = torch.full((n,), float("nan"), dtype=torch.float32, device=dev)
    acc = torch.full((n,), -7, dtype=torch.int32, device=dev)
    qd, sxd = torch.from_numpy(q).to(dev), torch.from_numpy(sx).to(dev)
    if channel:
        sw = _channel_scales(n, 39)
        sh.sherry_gemm_channel(w, qd, sxd, torch.from_numpy(sw).to(dev), y, acc, 1, n, k,
                               sh.SHERRY_KERNEL_ALUT)
    else:
        sw = synth.weight_scale(39, "al", n, k)
        sh.sherry_gemm_ex(w, qd, sxd, sw, y, acc, 1, n, k, sh.SHERRY_KERNEL_ALUT)
    torch.cuda.synchronize()
    acc_ref = oracle.gemm_i32(q, t, threads=8)
    assert np.array_equal(acc.cpu().numpy(), acc_ref[0])
    assert _y_ok(y.cpu().numpy(), _epi(acc_ref, sx, sw)[0])


def test_activation_table_matches_weight_table_kernel(dev):
    # bit-identical y and acc to the weight-table GEMV on a LLaMA-3.2-3B down
    # projection shape
    sh = _sh()
    n, k = 3072, 8192
    _say("alut vs gemv", n, k)
    t = synth.ternary_34(n, k, 41, "av")
    q = synth.int8_any(1, k, 41, "avq")
    sx = np.array([0.02], np.float32)
    ya, aa = _run(dev, t, q, sx, 0.03, sh.SHERRY_KERNEL_ALUT, 1)
    yg, ag = _run(dev, t, q, sx, 0.03, sh.SHERRY_KERNEL_GEMV, 1)
    assert np.array_equal(aa, ag) and np.array_equal(ya, yg)


@pytest.mark.parametrize("m,kernel", [(1, "GEMV"), (4, "GEMV"), (5, "SKINNY"), (40, "SKINNY"),
                                      (64, "MFMA")])
def test_longest_k(dev, m, kernel):
    # k = SHERRY_MAX_K with the largest sums the bound allows: x = -128 against
    # rows of +1 (code 0) reach 128 * 3K/4 = 16,773,120 < 2^24, still exact in
    # fp32; other rows are random
    sh = _sh()
    n, k = 70, sh.SHERRY_MAX_K
    _say("longest k", m, kernel)
    t = synth.ternary_34(n, k, 45, "lk")
    t[0] = np.tile(np.array([0, 1, 1, 1], np.int8), k // 4)
    t[1] = -t[0]
    q = synth.int8_any(m, k, 45, "lkq")
    q[0] = -128
    sx = np.full(m, 0.5, np.float32)
    y, acc = _run(dev, t, q, sx, 0.25, getattr(sh, "SHERRY_KERNEL_" + kernel), m)
    acc_ref = oracle.gemm_i32(q, t, threads=8)
    assert acc_ref[0, 0] == -128 * 3 * (k // 4) and acc_ref[0, 1] == 128 * 3 * (k // 4)
    assert np.array_equal(acc, acc_ref)
    # exact scales: y = acc / 8 exactly
    assert np.array_equal(y.astype(np.float64), acc.astype(np.float64) * 0.125)


# The MFMA tile configuration follows from (m, n): m <= 32 -> 32x256; else
# the cheapest of 256x256, 128x256, 128x128 by rounds of 256 workgroups x
# tile area.  These are the M = 2048 prefill shapes of LLaMA-3.2-3B (the
# launch configurations the benchmark times), checked on every output:
# q/o and down -> 128x256, k/v -> 128x128, gate/up -> 256x256.
PREFILL_3B = [("q", 3072, 3072), ("k", 1024, 3072), ("gate", 8192, 3072), ("down", 3072, 8192)]


@pytest.mark.parametrize("kernel", ["MFMA", "SKINNY"])
@pytest.mark.parametrize("name,n,k", PREFILL_3B)
def test_prefill_shapes_full(dev, name, n, k, kernel):
    # both MFMA paths (LDS-tiled and register-decoded) at M = 2048, every
    # int32 accumulator and every fp32 output against the oracle
    sh = _sh()
    m = 2048
    _say("prefill", kernel, name, m, n, k)
    t = synth.ternary_34(n, k, 35, "pf", name)
    x = synth.activations(m, k, 35, "pfx", name, outlier_frac=0.01)
    q, sx = oracle.quantize_act(x)
    sw = synth.weight_scale(35, "pfs", name)
    y, acc = _run(dev, t, q, sx, sw, getattr(sh, "SHERRY_KERNEL_" + kernel), m)
    acc_ref = oracle.gemm_i32(q, t, threads=ORACLE_THREADS)
    assert np.array_equal(acc, acc_ref)
    assert _y_ok(y, oracle.epilogue(acc_ref, sx, sw))


# ------------------------------------------------------ end-to-end + dispatch

@pytest.mark.parametrize("m,n,k", [(1, 2048, 2048), (4, 1024, 3072), (16, 1024, 3072),
                                   (64, 1024, 4096)])
def test_end_to_end_auto(dev, m, n, k):
    sh = _sh()
    _say("e2e", m, n, k)
    t = synth.ternary_34(n, k, 35, "e2e", n, k)
    x = synth.activations(m, k, 35, "e2e", m, k, outlier_frac=0.01)
    sw = synth.weight_scale(35, "e2e")
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    xd = torch.from_numpy(x).to(dev)
    q = torch.empty((m, k), dtype=torch.int8, device=dev)
    sx = torch.empty(m, dtype=torch.float32, device=dev)
    y = torch.empty((m, n), dtype=torch.float32, device=dev)
    acc = torch.empty((m, n), dtype=torch.int32, device=dev)
    sh.sherry_quantize_act(xd, q, sx)
    sh.sherry_gemm(w, q, sx, sw, y, acc, m, n, k)
    torch.cuda.synchronize()
    q_ref, sx_ref, acc_ref, y_ref = oracle.linear(x, t, sw, threads=8)
    assert np.array_equal(q.cpu().numpy(), q_ref)
    assert np.array_equal(acc.cpu().numpy(), acc_ref)
    assert _y_ok(y.cpu().numpy(), y_ref)


def test_kernels_agree_bitwise(dev):
    sh = _sh()
    n, k = 320, 1280
    t = synth.ternary_34(n, k, 36, "agree")
    for m in (1, 2, 3, 4):
        q = synth.int8_any(m, k, 36, "agree", m)
        sx = np.full(m, 0.1, np.float32)
        y1, a1 = _run(dev, t, q, sx, 0.03, sh.SHERRY_KERNEL_GEMV, m)
        y2, a2 = _run(dev, t, q, sx, 0.03, sh.SHERRY_KERNEL_MFMA, m)
        assert np.array_equal(a1, a2) and np.array_equal(y1, y2)


# ---------------------------------------------------------- closed forms

def test_one_hot_and_all_ones(dev):
    sh = _sh()
    n, k = 200, 384
    t = synth.ternary_34(n, k, 37, "oh")
    for kk in (0, 1, 127, 128, 383):
        e = np.zeros((1, k), np.int8)
        e[0, kk] = 1
        _, acc = _run(dev, t, e, np.ones(1, np.float32), 1.0, sh.SHERRY_KERNEL_GEMV, 1)
        assert np.array_equal(acc[0], t[:, kk].astype(np.int32))
    ones = np.ones((1, k), np.int8)
    _, acc = _run(dev, t, ones, np.ones(1, np.float32), 1.0, sh.SHERRY_KERNEL_GEMV, 1)
    assert np.array_equal(acc[0], t.astype(np.int32).sum(1))


def test_identity_reads_back_t(dev):
    # X = identity (M = K): acc = T^T, every weight read back through the MFMA path
    sh = _sh()
    n, k = 192, 256
    t = synth.ternary_34(n, k, 38, "id")
    eye = np.eye(k, dtype=np.int8)
    _, acc = _run(dev, t, eye, np.ones(k, np.float32), 1.0, sh.SHERRY_KERNEL_MFMA, k)
    assert np.array_equal(acc, t.T.astype(np.int32))


def test_mirror_negates(dev):
    # flipping every sign bit (code ^ 0x1C) is T -> -T: the product negates
    sh = _sh()
    n, k = 128, 512
    t = synth.ternary_34(n, k, 39, "mir")
    q = synth.int8_any(2, k, 39, "mir")
    _, a1 = _run(dev, t, q, np.ones(2, np.float32), 1.0, sh.SHERRY_KERNEL_GEMV, 2)
    _, a2 = _run(dev, (-t).astype(np.int8), q, np.ones(2, np.float32), 1.0,
                 sh.SHERRY_KERNEL_GEMV, 2)
    assert np.array_equal(a1, -a2)


def test_extreme_activations(dev):
    sh = _sh()
    n, k = 64, 8192
    t = synth.ternary_34(n, k, 40, "ext")
    for val in (-128, 127):
        q = np.full((1, k), val, np.int8)
        for kern in (sh.SHERRY_KERNEL_GEMV, sh.SHERRY_KERNEL_MFMA):
            _, acc = _run(dev, t, q, np.ones(1, np.float32), 1.0, kern, 1)
            assert np.array_equal(acc[0], val * t.astype(np.int32).sum(1))


def test_zero_scale_and_no_acc(dev):
    sh = _sh()
    n, k = 96, 256
    t = synth.ternary_34(n, k, 41, "zs")
    q = synth.int8_any(1, k, 41, "zs")
    y, _ = _run(dev, t, q, np.zeros(1, np.float32), 0.02, sh.SHERRY_KERNEL_GEMV, 1,
                with_acc=False)
    assert np.all(y == 0)


def test_guard_bands_and_determinism(dev):
    sh = _sh()
    n, k, m = 100, 260, 3
    t = synth.ternary_34(n, k, 42, "gb")
    q = synth.int8_any(m, k, 42, "gb")
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    qd = torch.from_numpy(q).to(dev)
    sx = torch.ones(m, dtype=torch.float32, device=dev)
    pad = 256
    for kern in (sh.SHERRY_KERNEL_GEMV, sh.SHERRY_KERNEL_MFMA):
        ybuf = torch.full((m * n + 2 * pad,), 12345.0, dtype=torch.float32, device=dev)
        abuf = torch.full((m * n + 2 * pad,), 777, dtype=torch.int32, device=dev)
        y = ybuf[pad:pad + m * n]
        a = abuf[pad:pad + m * n]
        outs = []
        for _ in range(3):
            sh.sherry_gemm_ex(w, qd, sx, 1.0, y, a, m, n, k, kern)
            torch.cuda.synchronize()
            outs.append(a.cpu().numpy().copy())
        yb, ab = ybuf.cpu().numpy(), abuf.cpu().numpy()
        assert np.all(yb[:pad] == 12345.0) and np.all(yb[pad + m * n:] == 12345.0)
        assert np.all(ab[:pad] == 777) and np.all(ab[pad + m * n:] == 777)
        assert all(np.array_equal(outs[0], o) for o in outs[1:])
        assert np.array_equal(outs[0].reshape(m, n), oracle.gemm_i32(q, t))


# ---------------------------------------------------------- batched decode

def _epi(acc, sx, sw):
    """Oracle epilogue for a per-tensor (float) or per-channel (array) scale."""
    if np.ndim(sw):
        return oracle.epilogue_rows(acc, sx, sw)
    return oracle.epilogue(acc, sx, sw)


def _desc_scale(d, dev, keep, n, seed, i, channel, k=None):
    """Per-tensor scale, or (channel and even i) a per-channel vector in
    d.w_scales, or (channel == "mixed", i % 3 == 1) per-group scales in
    d.w_group_scales; returns what the oracle epilogue takes (a float, a
    vector, or ("groups", matrix))."""
    if channel and i % 2 == 0:
        sw = _channel_scales(n, seed * 1000 + i)
        swd = torch.from_numpy(sw).to(dev)
        keep.append(swd)
        d.w_scales = swd.data_ptr()
        d.w_scale = float("nan")  # unused
        return sw
    if channel == "mixed" and i % 3 == 1:
        gs = _group_scales(n, k, seed * 1000 + i)
        gsd = torch.from_numpy(gs).to(dev)
        keep.append(gsd)
        d.w_group_scales = gsd.data_ptr()
        d.w_scale = float("nan")
        return ("groups", gs)
    return None


def _batched(dev, shapes, seed, want_acc=True, channel=False):
    sh = _sh()
    descs = (sh.sherry_gemv_desc * len(shapes))()
    keep, refs = [], []
    for i, (n, k) in enumerate(shapes):
        t = synth.ternary_34(n, k, seed, "b", i)
        q = synth.int8_any(1, k, seed, "b", i)
        sx = np.array([0.01 * (i + 1)], np.float32)
        sw = synth.weight_scale(seed, "b", i)
        w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
        qd = torch.from_numpy(q).to(dev)
        sxd = torch.from_numpy(sx).to(dev)
        y = torch.full((n,), float("nan"), dtype=torch.float32, device=dev)
        a = torch.full((n,), -9, dtype=torch.int32, device=dev) if want_acc else None
        keep += [w, qd, sxd, y, a]
        d = descs[i]
        d.w, d.x, d.x_scale, d.y = w.data_ptr(), qd.data_ptr(), sxd.data_ptr(), y.data_ptr()
        d.acc = a.data_ptr() if want_acc else None
        d.n, d.k, d.w_scale = n, k, sw
        swc = _desc_scale(d, dev, keep, n, seed, i, channel, k)
        sw = sw if swc is None else swc
        refs.append((t, q, sx, sw, y, a))
    total = sh.sherry_gemv_batched_prepare(descs)
    ddev = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
    sh.sherry_gemv_batched(ddev, len(shapes), total)
    torch.cuda.synchronize()
    return refs


def test_batched_gemv_parity(dev):
    _say("batched small")
    shapes = [(64, 128), (65, 132), (2048, 2048), (512, 2048), (300, 8192), (1, 4), (70, 1032)]
    for t, q, sx, sw, y, a in _batched(dev, shapes, 43):
        acc_ref = oracle.gemm_i32(q, t, threads=8)
        assert np.array_equal(a.cpu().numpy(), acc_ref[0])
        assert _y_ok(y.cpu().numpy(), oracle.epilogue(acc_ref, sx, sw)[0])


def test_batched_gemv_channel_scales(dev):
    # per-channel scales in half of the descriptors of one grouped launch
    _say("batched channel scales")
    shapes = [(64, 128), (65, 132), (2048, 2048), (512, 2048), (300, 8192), (1, 4), (70, 1032)]
    for t, q, sx, sw, y, a in _batched(dev, shapes, 47, channel=True):
        acc_ref = oracle.gemm_i32(q, t, threads=8)
        assert np.array_equal(a.cpu().numpy(), acc_ref[0])
        assert _y_ok(y.cpu().numpy(), _epi(acc_ref, sx, sw)[0])


def _check_mixed(q, t, sx, sw, y, a):
    if isinstance(sw, tuple):
        y_ref, mag, acc_ref = oracle.product_groups(q, t, sx, sw[1], threads=8)
        assert np.array_equal(a, acc_ref[0])
        assert _group_ok(y, y_ref[0], mag[0], t.shape[1])
    else:
        acc_ref = oracle.gemm_i32(q, t, threads=8)
        assert np.array_equal(a, acc_ref[0])
        assert _y_ok(y, _epi(acc_ref, sx, sw)[0])


def test_batched_gemv_mixed_scales(dev):
    # per-tensor, per-channel and per-group descriptors in one grouped launch
    _say("batched mixed scales")
    shapes = [(64, 128), (65, 132), (2048, 2048), (512, 2048), (300, 8192), (1, 4), (70, 1032),
              (130, 3076)]
    for t, q, sx, sw, y, a in _batched(dev, shapes, 48, channel="mixed"):
        _check_mixed(q, t, sx, sw, y.cpu().numpy(), a.cpu().numpy())


def test_batched_split_paths(dev):
    # K chosen so that the tiles are split over 1, 2 and 4 waves, with uneven
    # and partial last containers
    _say("batched split paths")
    shapes = [(3072, 3072), (1024, 3072), (130, 3076), (200, 6140), (64, 6148), (100, 8196),
              (65, 14336), (3, 4)]
    for t, q, sx, sw, y, a in _batched(dev, shapes, 46):
        acc_ref = oracle.gemm_i32(q, t, threads=8)
        assert np.array_equal(a.cpu().numpy(), acc_ref[0])
        assert _y_ok(y.cpu().numpy(), oracle.epilogue(acc_ref, sx, sw)[0])


def test_batched_decode_step_llama_1b(dev):
    # one decode step of LLaMA-3.2-1B linear layers (16 layers x 7 shapes), in
    # the grouped launch the benchmark times; every output of all 112 products
    _say("batched llama-1b step")
    spec = synth.LLAMA_1B
    shapes = [(lin.n, lin.k) for _, lin in synth.model_linears(spec)]
    refs = _batched(dev, shapes, 44)
    assert len(refs) == 112
    for t, q, sx, sw, y, a in refs:
        acc_ref = oracle.gemm_i32(q, t, threads=ORACLE_THREADS)
        assert np.array_equal(a.cpu().numpy(), acc_ref[0])
        assert _y_ok(y.cpu().numpy(), oracle.epilogue(acc_ref, sx, sw)[0])


# ---------------------------------------------------------- 2-bit reference

@pytest.mark.parametrize("n,k", [(64, 64), (65, 68), (300, 2048), (128, 4100)])
def test_gemv2_parity(dev, n, k):
    sh = _sh()
    t = synth.ternary_any(n, k, 45, "g2", n, k)
    q = synth.int8_any(1, k, 45, "g2", n, k)
    w2 = torch.from_numpy(sh.sherry_pack2(t)).to(dev)
    qd = torch.from_numpy(q).to(dev)
    sx = torch.full((1,), 0.5, dtype=torch.float32, device=dev)
    y = torch.empty(n, dtype=torch.float32, device=dev)
    a = torch.empty(n, dtype=torch.int32, device=dev)
    sh.sherry_gemv2(w2, qd, sx, 0.25, y, a, n, k)
    torch.cuda.synchronize()
    acc_ref = oracle.gemm_i32(q, t)[0]
    assert np.array_equal(a.cpu().numpy(), acc_ref)
    assert np.array_equal(y.cpu().numpy().astype(np.float64), acc_ref * 0.125)


def test_stream_read_checksum(dev):
    sh = _sh()
    # the slice a workgroup reads: the smallest power of two past which a
    # second workgroup is needed
    slice_bytes = next(1 << i for i in range(10, 31) if sh.sherry_stream_read_groups((1 << i) + 1) == 2)
    nbytes = 3 * slice_bytes + 4096
    src = torch.randint(0, 2**31 - 1, (nbytes // 4,), dtype=torch.int32, device=dev)
    groups = sh.sherry_stream_read_groups(nbytes)
    sink = torch.empty(groups, dtype=torch.int32, device=dev)
    sh.sherry_stream_read(src, nbytes, sink)
    torch.cuda.synchronize()
    h = src.cpu().numpy().view(np.uint32)
    per = slice_bytes // 4
    assert groups == 4
    ref = [np.bitwise_xor.reduce(h[g * per:(g + 1) * per]) for g in range(groups)]
    assert np.array_equal(sink.cpu().numpy().view(np.uint32), np.array(ref, np.uint32))


# ------------------------------------------ fused quantization + M = 1 product

def _fused_ref(x, t, sw):
    q, sx = oracle.quantize_act(x)
    acc = oracle.gemm_i32(q, t, threads=8)
    return sx, acc, oracle.epilogue(acc, sx, sw)


@pytest.mark.parametrize("n,k,outl", [(64, 128, 0.0), (65, 132, 0.01), (2048, 2048, 0.01),
                                      (300, 8192, 0.01), (1, 4, 0.0), (70, 1032, 0.0),
                                      (130, 14336, 0.01), (64, 32768, 0.01), (3, 32764, 0.0)])
def test_fused_gemv_parity(dev, n, k, outl):
    sh = _sh()
    _say("fused", n, k, outl)
    t = synth.ternary_34(n, k, 47, "fu", n, k)
    x = synth.activations(1, k, 47, "fux", n, k, outlier_frac=outl)
    sw = synth.weight_scale(47, "fus", n, k)
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    xd = torch.from_numpy(x).to(dev)
    sxd = torch.full((1,), float("nan"), dtype=torch.float32, device=dev)
    y = torch.full((n,), float("nan"), dtype=torch.float32, device=dev)
    a = torch.full((n,), -7, dtype=torch.int32, device=dev)
    sh.sherry_gemv_f32(w, xd, sxd, sw, y, a, n, k)
    torch.cuda.synchronize()
    sx_ref, acc_ref, y_ref = _fused_ref(x, t, sw)
    assert sxd.cpu().numpy()[0] == sx_ref[0]
    assert np.array_equal(a.cpu().numpy(), acc_ref[0])
    assert _y_ok(y.cpu().numpy(), y_ref[0])
    # bit-identical to quantize + product as two calls
    q2 = torch.empty(k, dtype=torch.int8, device=dev)
    s2 = torch.empty(1, dtype=torch.float32, device=dev)
    y2 = torch.empty(n, dtype=torch.float32, device=dev)
    sh.sherry_quantize_act(xd.view(1, k), q2.view(1, k), s2)
    sh.sherry_gemv(w, q2, s2, sw, y2, None, n, k)
    torch.cuda.synchronize()
    assert np.array_equal(y2.cpu().numpy().view(np.uint32), y.cpu().numpy().view(np.uint32))


def test_fused_gemv_zero_row_and_no_outputs(dev):
    sh = _sh()
    n, k = 200, 640
    t = synth.ternary_34(n, k, 48, "fz")
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    xd = torch.zeros(k, dtype=torch.float32, device=dev)
    sxd = torch.full((1,), 5.0, dtype=torch.float32, device=dev)
    y = torch.full((n,), float("nan"), dtype=torch.float32, device=dev)
    a = torch.full((n,), -7, dtype=torch.int32, device=dev)
    sh.sherry_gemv_f32(w, xd, sxd, 0.5, y, a, n, k)
    torch.cuda.synchronize()
    assert sxd.item() == 0.0
    assert not a.any().item() and not y.any().item()
    # x_scale and acc are optional
    x = synth.activations(1, k, 48, "fzx")
    xd = torch.from_numpy(x).to(dev)
    sh.sherry_gemv_f32(w, xd, None, 0.5, y, None, n, k)
    torch.cuda.synchronize()
    _, _, y_ref = _fused_ref(x, t, 0.5)
    assert _y_ok(y.cpu().numpy(), y_ref[0])


def _fused_batched(dev, shapes, seed, with_scale=True, channel=False, il=False):
    # il: lane-interleaved weights (sherry_pack_il) on sherry_gemv_f32_il_batched
    sh = _sh()
    descs = (sh.sherry_gemv_f32_desc * len(shapes))()
    keep, hold = [], []
    for i, (n, k) in enumerate(shapes):
        t = synth.ternary_34(n, k, seed, "fb", i)
        x = synth.activations(1, k, seed, "fbx", i, outlier_frac=0.01)
        sw = synth.weight_scale(seed, "fbs", i)
        w = torch.from_numpy(sh.sherry_pack_il(t) if il else sh.sherry_pack(t)).to(dev)
        xd = torch.from_numpy(x).to(dev)
        sxd = torch.full((1,), float("nan"), dtype=torch.float32, device=dev)
        y = torch.full((n,), float("nan"), dtype=torch.float32, device=dev)
        a = torch.full((n,), -7, dtype=torch.int32, device=dev)
        d = descs[i]
        d.w, d.x, d.y, d.acc = w.data_ptr(), xd.data_ptr(), y.data_ptr(), a.data_ptr()
        d.x_scale = sxd.data_ptr() if with_scale else None
        d.n, d.k, d.w_scale = n, k, sw
        swc = _desc_scale(d, dev, hold, n, seed, i, channel, k)
        keep.append((t, x, sw if swc is None else swc, w, xd, sxd, y, a))
    if il:
        total = sh.sherry_gemv_f32_il_batched_prepare(descs)
        dd = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
        sh.sherry_gemv_f32_il_batched(dd, len(shapes), total)
    else:
        total = sh.sherry_gemv_f32_batched_prepare(descs)
        dd = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
        sh.sherry_gemv_f32_batched(dd, len(shapes), total)
    torch.cuda.synchronize()
    return keep


@pytest.mark.parametrize("il", [False, True])
def test_fused_batched_parity(dev, il):
    _say("fused batched", "il" if il else "tiled")
    # rows of 17-32 units run unsplit in one wave (3072: 24 units; 4000: a
    # ragged 32nd unit), 2176 (17 units) is the shortest such row
    shapes = [(64, 128), (65, 132), (2048, 2048), (512, 2048), (300, 8192), (1, 4), (70, 1032),
              (100, 8196), (65, 14336), (3, 32768), (96, 3072), (33, 4000), (130, 2176),
              (64, 4224)]
    for t, x, sw, w, xd, sxd, y, a in _fused_batched(dev, shapes, 49, il=il):
        sx_ref, acc_ref, y_ref = _fused_ref(x, t, sw)
        assert sxd.cpu().numpy()[0] == sx_ref[0]
        assert np.array_equal(a.cpu().numpy(), acc_ref[0])
        assert _y_ok(y.cpu().numpy(), y_ref[0])


@pytest.mark.parametrize("il", [False, True])
def test_fused_batched_channel_scales(dev, il):
    _say("fused batched channel scales", "il" if il else "tiled")
    shapes = [(64, 128), (65, 132), (2048, 2048), (300, 8192), (1, 4), (100, 8196)]
    for t, x, sw, w, xd, sxd, y, a in _fused_batched(dev, shapes, 51, channel=True, il=il):
        q, sx = oracle.quantize_act(x)
        assert sxd.cpu().numpy()[0] == sx[0]
        acc_ref = oracle.gemm_i32(q, t, threads=8)
        assert np.array_equal(a.cpu().numpy(), acc_ref[0])
        assert _y_ok(y.cpu().numpy(), _epi(acc_ref, sx, sw)[0])


def test_fused_batched_mixed_scales(dev):
    _say("fused batched mixed scales")
    # per-group descriptors (i % 3 == 1) on rows of 24, 17, 33 and a ragged 32
    # units: unsplit rows of the grouped fused kernel and the first split
    shapes = [(64, 128), (96, 3072), (2048, 2048), (300, 8192), (130, 2176), (1, 4),
              (100, 8196), (64, 4224), (70, 260), (65, 132), (33, 4000)]
    for t, x, sw, w, xd, sxd, y, a in _fused_batched(dev, shapes, 52, channel="mixed"):
        q, sx = oracle.quantize_act(x)
        assert sxd.cpu().numpy()[0] == sx[0]
        _check_mixed(q, t, sx, sw, y.cpu().numpy(), a.cpu().numpy())


def test_fused_batched_layouts_agree(dev):
    # tiled and lane-interleaved weights of the same matrices: the same bits
    # (int32 sums are exact; the epilogue is the same arithmetic)
    _say("fused batched tiled vs il")
    shapes = [(64, 128), (65, 132), (2048, 2048), (300, 8192), (1, 4), (70, 1032), (3, 32768),
              (130, 2176), (64, 4224)] + [(64 + 37 * (i % 5), 4 * (1 + (i * 97) % 700))
                                          for i in range(60)]
    a = _fused_batched(dev, shapes, 53, channel="mixed_no_groups")
    b = _fused_batched(dev, shapes, 53, channel="mixed_no_groups", il=True)
    for ka, kb in zip(a, b):
        assert np.array_equal(ka[6].cpu().numpy().view(np.uint32), kb[6].cpu().numpy().view(np.uint32))
        assert np.array_equal(ka[7].cpu().numpy(), kb[7].cpu().numpy())
        assert ka[5].cpu().numpy()[0] == kb[5].cpu().numpy()[0]


@pytest.mark.parametrize("il", [False, True])
def test_fused_batched_decode_step_llama_1b(dev, il):
    # the benchmark's decode step: 112 products of LLaMA-3.2-1B, one fused
    # launch; every int32 accumulator and fp32 output against the oracle
    _say("fused batched llama-1b step", "il" if il else "tiled")
    shapes = [(lin.n, lin.k) for _, lin in synth.model_linears(synth.LLAMA_1B)]
    keep = _fused_batched(dev, shapes, 50, with_scale=False, il=il)
    assert len(keep) == 112
    for t, x, sw, w, xd, sxd, y, a in keep:
        q, sx = oracle.quantize_act(x)
        acc_ref = oracle.gemm_i32(q, t, threads=ORACLE_THREADS)
        assert np.array_equal(a.cpu().numpy(), acc_ref[0])
        assert _y_ok(y.cpu().numpy(), oracle.epilogue(acc_ref, sx, sw)[0])


# ------------------------------------- register-decoded MFMA (small M first)

# A lone launch splits K over S = 1, 2, 4 or 8 waves per tile (more splits
# for fewer tiles, at most half the containers): these cover every S for 32-
# and 64-token staging, splits that end early or own no container, and the
# LDS reduction of the partial sums.  Above 64 tokens the launch stages
# 64-token blocks along a second grid dimension: ragged last blocks, a single
# block, and many blocks.
SKINNY_CASES = [(5, 64, 128), (16, 65, 132), (32, 300, 1032), (33, 130, 2048), (64, 512, 1024),
                (1, 64, 128), (4, 257, 3076), (17, 1000, 2056), (64, 70, 4), (48, 3072, 8192),
                (40, 100, 384), (20, 200, 896), (9, 16384, 256),
                (65, 64, 128), (128, 130, 1032), (129, 520, 2052), (300, 64, 388),
                (700, 1100, 1536), (2048, 96, 256), (257, 4096, 1024)]


@pytest.mark.parametrize("m,n,k", SKINNY_CASES)
def test_skinny_kernel_parity(dev, m, n, k):
    # ragged n (partial 64-row tiles and 8-tile workgroups), ragged k (partial
    # containers, k % 16 != 0 rows, chunk boundaries), 1..64 tokens
    sh = _sh()
    _say("skinny", m, n, k)
    t = synth.ternary_34(n, k, 51, "sk", n, k)
    q = synth.int8_any(m, k, 51, "sk", m, k)
    sx = np.abs(synth.activations(1, m, 51, "sks", m)[0]).astype(np.float32) + 0.01
    sw = synth.weight_scale(51, "sk", n, k)
    y, acc = _run(dev, t, q, sx, sw, sh.SHERRY_KERNEL_SKINNY, m)
    acc_ref = oracle.gemm_i32(q, t, threads=8)
    assert np.array_equal(acc, acc_ref)
    assert _y_ok(y, oracle.epilogue(acc_ref, sx, sw))


def test_skinny_extreme_values(dev):
    # all activations -128 or 127 and all-ones / all-minus patterns: the
    # largest |acc| the kernel can meet at this K
    sh = _sh()
    m, n, k = 40, 128, 4096
    q = np.where(synth.int8_any(m, k, 52, "ext") >= 0, 127, -128).astype(np.int8)
    t = synth.ternary_34(n, k, 52, "ext")
    y, acc = _run(dev, t, q, np.ones(m, np.float32), 1.0, sh.SHERRY_KERNEL_SKINNY, m)
    assert np.array_equal(acc, oracle.gemm_i32(q, t, threads=8))


def _skinny_batched(dev, cases, seed, channel=False):
    sh = _sh()
    descs = (sh.sherry_gemm_desc * len(cases))()
    keep, hold = [], []
    for i, (m, n, k) in enumerate(cases):
        t = synth.ternary_34(n, k, seed, "sb", i)
        q = synth.int8_any(m, k, seed, "sbq", i)
        sx = np.abs(synth.activations(1, m, seed, "sbs", i)[0]).astype(np.float32) + 0.01
        sw = synth.weight_scale(seed, "sbw", i)
        w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
        qd = torch.from_numpy(q).to(dev)
        sxd = torch.from_numpy(sx).to(dev)
        y = torch.full((m, n), float("nan"), dtype=torch.float32, device=dev)
        a = torch.full((m, n), -7, dtype=torch.int32, device=dev)
        d = descs[i]
        d.w, d.x, d.x_scale, d.y, d.acc = (w.data_ptr(), qd.data_ptr(), sxd.data_ptr(),
                                           y.data_ptr(), a.data_ptr())
        d.n, d.k, d.m, d.w_scale = n, k, m, sw
        swc = _desc_scale(d, dev, hold, n, seed, i, channel)
        keep.append((t, q, sx, sw if swc is None else swc, w, qd, sxd, y, a))
    total, max_m = sh.sherry_gemm_batched_prepare(descs)
    dd = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
    sh.sherry_gemm_batched(dd, len(cases), total, max_m)
    torch.cuda.synchronize()
    return keep, max_m


def test_skinny_batched_channel_scales(dev):
    _say("skinny batched channel scales")
    cases = [(5, 64, 128), (16, 65, 132), (1, 600, 2048), (32, 512, 3072), (64, 300, 2052)]
    keep, _ = _skinny_batched(dev, cases, 55, channel=True)
    for t, q, sx, sw, w, qd, sxd, y, a in keep:
        acc_ref = oracle.gemm_i32(q, t, threads=8)
        assert np.array_equal(a.cpu().numpy(), acc_ref)
        assert _y_ok(y.cpu().numpy(), _epi(acc_ref, sx, sw))


@pytest.mark.parametrize("big", [False, True])
def test_skinny_batched_parity(dev, big):
    _say("skinny batched", big)
    cases = [(5, 64, 128), (16, 65, 132), (1, 600, 2048), (32, 512, 3072), (8, 130, 1032)]
    if big:
        cases += [(64, 300, 2052), (40, 64, 4)]
    keep, max_m = _skinny_batched(dev, cases, 53)
    assert max_m == max(c[0] for c in cases)
    for t, q, sx, sw, w, qd, sxd, y, a in keep:
        acc_ref = oracle.gemm_i32(q, t, threads=8)
        assert np.array_equal(a.cpu().numpy(), acc_ref)
        assert _y_ok(y.cpu().numpy(), oracle.epilogue(acc_ref, sx, sw))


def test_skinny_batched_any_m(dev):
    # products longer than one token block (several 64-token blocks, ragged
    # last block) grouped with short ones in one launch
    _say("skinny batched any m")
    cases = [(65, 64, 128), (300, 520, 2052), (5, 130, 1032), (129, 257, 388), (200, 64, 4)]
    keep, max_m = _skinny_batched(dev, cases, 57, channel=True)
    assert max_m == 300
    for t, q, sx, sw, w, qd, sxd, y, a in keep:
        acc_ref = oracle.gemm_i32(q, t, threads=8)
        assert np.array_equal(a.cpu().numpy(), acc_ref)
        assert _y_ok(y.cpu().numpy(), _epi(acc_ref, sx, sw))


def test_skinny_batched_group_scales(dev):
    # per-group descriptors (K split in two, 32-token blocks, no int32 totals)
    # grouped with per-tensor and per-channel ones in one launch
    sh = _sh()
    _say("skinny batched group scales")
    cases = [(5, 64, 128), (100, 257, 3076), (16, 600, 2048), (33, 130, 1028), (1, 70, 132),
             (64, 512, 8192)]
    descs = (sh.sherry_gemm_desc * len(cases))()
    keep = []
    for i, (m, n, k) in enumerate(cases):
        t = synth.ternary_34(n, k, 61, "sg", i)
        q = synth.int8_any(m, k, 61, "sgq", i)
        sx = np.abs(synth.activations(1, m, 61, "sgs", i)[0]).astype(np.float32) + 0.01
        w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
        qd, sxd = torch.from_numpy(q).to(dev), torch.from_numpy(sx).to(dev)
        y = torch.full((m, n), float("nan"), dtype=torch.float32, device=dev)
        a = torch.full((m, n), -7, dtype=torch.int32, device=dev)
        d = descs[i]
        d.w, d.x, d.x_scale, d.y = w.data_ptr(), qd.data_ptr(), sxd.data_ptr(), y.data_ptr()
        d.n, d.k, d.m, d.w_scale = n, k, m, 0.03
        extra = None
        if i % 3 == 1 or i == 5:
            gs = torch.from_numpy(_group_scales(n, k, 61 + i)).to(dev)
            d.w_group_scales, d.acc, extra = gs.data_ptr(), None, ("groups", gs)
        elif i % 3 == 2:
            sw = torch.from_numpy(_channel_scales(n, 61 + i)).to(dev)
            d.w_scales, d.acc, extra = sw.data_ptr(), a.data_ptr(), ("rows", sw)
        else:
            d.acc = a.data_ptr()
        keep.append((t, q, sx, w, qd, sxd, y, a, extra))
    total, max_m = sh.sherry_gemm_batched_prepare(descs)
    assert max_m == 32 | sh.SHERRY_LAUNCH_GROUPS
    dd = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
    sh.sherry_gemm_batched(dd, len(cases), total, max_m)
    torch.cuda.synchronize()
    for t, q, sx, w, qd, sxd, y, a, extra in keep:
        k = t.shape[1]
        if extra and extra[0] == "groups":
            y_ref, mag, _ = oracle.product_groups(q, t, sx, extra[1].cpu().numpy(), threads=8)
            assert _group_ok(y.cpu().numpy(), y_ref, mag, k)
            assert (a.cpu().numpy() == -7).all()  # no totals requested, none written
        else:
            acc_ref = oracle.gemm_i32(q, t, threads=8)
            assert np.array_equal(a.cpu().numpy(), acc_ref)
            sw = extra[1].cpu().numpy() if extra else 0.03
            assert _y_ok(y.cpu().numpy(), _epi(acc_ref, sx, sw))


@pytest.mark.parametrize("spec_name,m", [("LLAMA_3B", 16), ("STRESS_8B", 64), ("LLAMA_3B", 2048)])
def test_skinny_batched_model_step_full(dev, spec_name, m):
    # every linear of one layer of the model at M tokens in one grouped
    # launch (the configurations the benchmark times), every output
    _say("skinny step", spec_name, m)
    spec = getattr(synth, spec_name)
    blk = synth.llama_block(spec["hidden"], spec["kv"], spec["inter"])
    keep, _ = _skinny_batched(dev, [(m, lin.n, lin.k) for lin in blk], 54)
    for t, q, sx, sw, w, qd, sxd, y, a in keep:
        acc_ref = oracle.gemm_i32(q, t, threads=ORACLE_THREADS)
        assert np.array_equal(a.cpu().numpy(), acc_ref)
        assert _y_ok(y.cpu().numpy(), oracle.epilogue(acc_ref, sx, sw))


# ------------------------------------- per-channel scales (Eq. 5 per row)

def _channel_scales(n, seed):
    rng = np.random.default_rng(seed)
    return (rng.random(n) * 0.05 + 0.001).astype(np.float32)


# every kernel (GEMV up to 4 tokens, register-decoded, LDS-tiled) with ragged
# n and k: int32 acc as the per-tensor path, y scaled per output channel
CHANNEL_CASES = [(1, 70, 132, "GEMV"), (4, 600, 2048, "GEMV"), (9, 130, 1028, "SKINNY"),
                 (100, 257, 388, "SKINNY"), (33, 300, 1032, "MFMA"), (300, 520, 2052, "MFMA"),
                 (40, 258, 1028, "MFMA"), (130, 1027, 640, "MFMA")]


@pytest.mark.parametrize("m,n,k,kernel", CHANNEL_CASES)
def test_gemm_channel_parity(dev, m, n, k, kernel):
    sh = _sh()
    _say("channel", kernel, m, n, k)
    t = synth.ternary_34(n, k, 61, "ch", n, k)
    q = synth.int8_any(m, k, 61, "chq", m, k)
    sx = np.abs(synth.activations(1, m, 61, "chs", m)[0]).astype(np.float32) + 0.01
    sw = _channel_scales(n, 61)
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    y = torch.full((m, n), float("nan"), dtype=torch.float32, device=dev)
    acc = torch.full((m, n), -7, dtype=torch.int32, device=dev)
    sh.sherry_gemm_channel(w, torch.from_numpy(q).to(dev), torch.from_numpy(sx).to(dev),
                           torch.from_numpy(sw).to(dev), y, acc, m, n, k,
                           getattr(sh, "SHERRY_KERNEL_" + kernel))
    torch.cuda.synchronize()
    acc_ref = oracle.gemm_i32(q, t, threads=8)
    assert np.array_equal(acc.cpu().numpy(), acc_ref)
    assert _y_ok(y.cpu().numpy(), oracle.epilogue_rows(acc_ref, sx, sw))


@pytest.mark.parametrize("n,k", [(70, 132), (3072, 8192)])
def test_gemv_f32_channel_parity(dev, n, k):
    sh = _sh()
    _say("f32 channel", n, k)
    t = synth.ternary_34(n, k, 62, "fch", n, k)
    x = synth.activations(1, k, 62, "fchx", n, k, outlier_frac=0.01)
    sw = _channel_scales(n, 62)
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    xs = torch.empty(1, dtype=torch.float32, device=dev)
    y = torch.full((1, n), float("nan"), dtype=torch.float32, device=dev)
    acc = torch.full((1, n), -7, dtype=torch.int32, device=dev)
    sh.sherry_gemv_f32_channel(w, torch.from_numpy(x[0]).to(dev), xs, torch.from_numpy(sw).to(dev),
                               y, acc, n, k)
    torch.cuda.synchronize()
    q, sx = oracle.quantize_act(x)
    assert np.array_equal(xs.cpu().numpy(), sx)
    acc_ref = oracle.gemm_i32(q, t, threads=8)
    assert np.array_equal(acc.cpu().numpy(), acc_ref)
    assert _y_ok(y.cpu().numpy(), oracle.epilogue_rows(acc_ref, sx, sw))


# --------------------------------- Sparse-AbsMean ternarize + pack (Eq. 4-5)

def _weights_with_ties(n, k, seed):
    w = synth.dense_weights(n, k, seed, "tp", n, k)
    rng = np.random.default_rng(seed)
    nb = k // 4
    for _ in range(max(1, n * nb // 50)):
        row, b = rng.integers(0, n), rng.integers(0, nb)
        kind = rng.integers(0, 4)
        blk = w[row, 4 * b:4 * b + 4]
        if kind == 0:      # tie for the smallest magnitude
            blk[:] = [0.5, -0.25, 0.25, -0.5]
        elif kind == 1:    # zeros, also among the kept weights
            blk[:] = [0.0, 0.0, -0.0, 0.3]
        elif kind == 2:    # all equal magnitudes
            blk[:] = [-0.1, 0.1, -0.1, 0.1]
        else:              # negative zero kept as +1
            blk[:] = [-0.0, 1.0, -2.0, 3.0]
    return w


def _ulp_close(a, b):
    a = np.asarray(a, np.float32)
    b = np.asarray(b, np.float32)
    return bool(np.all(np.abs(a.astype(np.float64) - b.astype(np.float64)) <=
                       np.spacing(np.maximum(np.abs(a), np.abs(b)))))


@pytest.mark.parametrize("n,k", [(1, 4), (63, 128), (64, 132), (70, 1028), (130, 260),
                                 (1031, 516), (4097, 256), (512, 4096), (8192, 3072)])
def test_ternarize_pack_parity(dev, n, k):
    # packed bytes identical to packing the oracle's ternary matrix (padding
    # included); per-channel alpha within one fp32 unit of the oracle's fp64
    # mean (the summation order differs)
    sh = _sh()
    _say("ternarize_pack", n, k)
    w = _weights_with_ties(n, k, 63)
    t_ref, alpha_ref = oracle.ternarize_rows(w)
    packed_ref = oracle.pack(t_ref)
    wd = torch.from_numpy(w).to(dev)
    packed = torch.full((sh.sherry_packed_bytes(n, k),), 0xA5, dtype=torch.uint8, device=dev)
    alpha = torch.full((n,), float("nan"), dtype=torch.float32, device=dev)
    sh.sherry_ternarize_pack(wd, n, k, packed, alpha)
    torch.cuda.synchronize()
    assert np.array_equal(packed.cpu().numpy(), packed_ref)
    assert _ulp_close(alpha.cpu().numpy(), alpha_ref.astype(np.float32))


def test_ternarize_pack_then_channel_product(dev):
    # fp32 weights -> GPU ternarize+pack -> per-channel product with the GPU
    # alpha, against the oracle chain (ternarize_rows, quantize_act, gemm,
    # epilogue_rows with the same alpha)
    sh = _sh()
    m, n, k = 16, 3072, 3072
    _say("ternarize -> channel product", m, n, k)
    w = synth.dense_weights(n, k, 64, "tpc")
    x = synth.activations(m, k, 64, "tpcx", outlier_frac=0.01)
    packed = torch.empty((sh.sherry_packed_bytes(n, k),), dtype=torch.uint8, device=dev)
    alpha = torch.empty((n,), dtype=torch.float32, device=dev)
    sh.sherry_ternarize_pack(torch.from_numpy(w).to(dev), n, k, packed, alpha)
    q, sx = oracle.quantize_act(x)
    y = torch.empty((m, n), dtype=torch.float32, device=dev)
    acc = torch.empty((m, n), dtype=torch.int32, device=dev)
    sh.sherry_gemm_channel(packed, torch.from_numpy(q).to(dev), torch.from_numpy(sx).to(dev),
                           alpha, y, acc, m, n, k)
    torch.cuda.synchronize()
    t_ref, _ = oracle.ternarize_rows(w)
    acc_ref = oracle.gemm_i32(q, t_ref, threads=8)
    assert np.array_equal(acc.cpu().numpy(), acc_ref)
    assert _y_ok(y.cpu().numpy(), oracle.epilogue_rows(acc_ref, sx, alpha.cpu().numpy()))


# ------------------------------------ per-group scales (group 128 along K)

def _group_scales(n, k, seed):
    rng = np.random.default_rng(seed)
    return (rng.random((n, (k + 127) // 128)) * 0.05 + 0.001).astype(np.float32)


def _group_ok(y, y_ref, mag, k):
    # fp32 summation in any order: |y - y_ref| <= (G + 4) * 2^-24 * mag
    bound = ((k + 127) // 128 + 4) * 2.0 ** -24 * mag + 1e-30
    return bool(np.all(np.abs(np.asarray(y, np.float64) - y_ref) <= bound))


# GEMV (m <= 4), the register-decoded kernel (32-token blocks, K split in
# 2, 4 or 8) and the LDS-tiled kernel (128 x 128 tiles), with ragged n, a
# partial last group, and the int32 totals
GROUP_CASES = [(1, 70, 132, "GEMV"), (4, 600, 2048, "GEMV"), (3, 300, 8196, "GEMV"),
               (5, 64, 128, "SKINNY"), (33, 130, 1028, "SKINNY"), (100, 257, 3076, "SKINNY"),
               (17, 3072, 8192, "SKINNY"), (5, 64, 128, "MFMA"), (33, 130, 1028, "MFMA"),
               (300, 520, 2052, "MFMA"), (256, 1024, 3072, "MFMA"), (130, 200, 8196, "MFMA")]


@pytest.mark.parametrize("m,n,k,kernel", GROUP_CASES)
def test_gemm_group_parity(dev, m, n, k, kernel):
    sh = _sh()
    _say("group", kernel, m, n, k)
    t = synth.ternary_34(n, k, 71, "gr", n, k)
    q = synth.int8_any(m, k, 71, "grq", m, k)
    sx = np.abs(synth.activations(1, m, 71, "grs", m)[0]).astype(np.float32) + 0.01
    gs = _group_scales(n, k, 71)
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    y = torch.full((m, n), float("nan"), dtype=torch.float32, device=dev)
    acc = torch.full((m, n), -7, dtype=torch.int32, device=dev)
    sh.sherry_gemm_group(w, torch.from_numpy(q).to(dev), torch.from_numpy(sx).to(dev),
                         torch.from_numpy(gs).to(dev), y, acc, m, n, k,
                         getattr(sh, "SHERRY_KERNEL_" + kernel))
    torch.cuda.synchronize()
    y_ref, mag, acc_ref = oracle.product_groups(q, t, sx, gs, threads=8)
    assert np.array_equal(acc.cpu().numpy(), acc_ref)
    assert _group_ok(y.cpu().numpy(), y_ref, mag, k)


def test_gemm_group_without_acc(dev):
    sh = _sh()
    m, n, k = 40, 200, 1024
    _say("group no acc", m, n, k)
    t = synth.ternary_34(n, k, 72, "gra")
    q = synth.int8_any(m, k, 72, "graq")
    sx = np.full(m, 0.02, np.float32)
    gs = _group_scales(n, k, 72)
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    y = torch.full((m, n), float("nan"), dtype=torch.float32, device=dev)
    sh.sherry_gemm_group(w, torch.from_numpy(q).to(dev), torch.from_numpy(sx).to(dev),
                         torch.from_numpy(gs).to(dev), y, None, m, n, k)
    torch.cuda.synchronize()
    y_ref, mag, _ = oracle.product_groups(q, t, sx, gs, threads=8)
    assert _group_ok(y.cpu().numpy(), y_ref, mag, k)


@pytest.mark.parametrize("n,k", [(70, 132), (2048, 8192)])
def test_gemv_f32_group_parity(dev, n, k):
    sh = _sh()
    _say("f32 group", n, k)
    t = synth.ternary_34(n, k, 73, "fgr", n, k)
    x = synth.activations(1, k, 73, "fgrx", n, k, outlier_frac=0.01)
    gs = _group_scales(n, k, 73)
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    xs = torch.empty(1, dtype=torch.float32, device=dev)
    y = torch.full((1, n), float("nan"), dtype=torch.float32, device=dev)
    acc = torch.full((1, n), -7, dtype=torch.int32, device=dev)
    sh.sherry_gemv_f32_group(w, torch.from_numpy(x[0]).to(dev), xs, torch.from_numpy(gs).to(dev),
                             y, acc, n, k)
    torch.cuda.synchronize()
    q, sx = oracle.quantize_act(x)
    assert np.array_equal(xs.cpu().numpy(), sx)
    y_ref, mag, acc_ref = oracle.product_groups(q, t, sx, gs, threads=8)
    assert np.array_equal(acc.cpu().numpy(), acc_ref)
    assert _group_ok(y.cpu().numpy(), y_ref, mag, k)


def test_graph_replay_matches_eager(dev):
    # the kernels launched from a captured HIP graph, replayed several times
    # with eager work and synchronisation in between: every replay must give
    # the eager results (fused grouped decode, register-decoded and LDS-tiled
    # products, quantization)
    sh = _sh()
    _say("graph replay")
    shapes = [(512, 2048), (2048, 2048), (300, 8192)]
    fd = _fused_batched(dev, shapes, 71)  # eager run, outputs checked elsewhere
    descs = (sh.sherry_gemv_f32_desc * len(shapes))()
    for i, (t, x, sw, w, xd, sxd, y, a) in enumerate(fd):
        d = descs[i]
        d.w, d.x, d.x_scale, d.y, d.acc = (w.data_ptr(), xd.data_ptr(), sxd.data_ptr(),
                                           y.data_ptr(), a.data_ptr())
        d.n, d.k, d.w_scale = t.shape[0], t.shape[1], sw
    total = sh.sherry_gemv_f32_batched_prepare(descs)
    ddev = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
    m, n, k = 96, 520, 2052
    tt = synth.ternary_34(n, k, 72, "gr")
    wq = torch.from_numpy(sh.sherry_pack(tt)).to(dev)
    xf = torch.from_numpy(synth.activations(m, k, 72, "grx")).to(dev)
    qd = torch.empty((m, k), dtype=torch.int8, device=dev)
    sxd2 = torch.empty(m, dtype=torch.float32, device=dev)
    y1 = torch.empty((m, n), dtype=torch.float32, device=dev)
    y2 = torch.empty((m, n), dtype=torch.float32, device=dev)

    def work():
        sh.sherry_gemv_f32_batched(ddev, len(shapes), total)
        sh.sherry_quantize_act(xf, qd, sxd2)
        sh.sherry_gemm_ex(wq, qd, sxd2, 0.02, y1, None, m, n, k, sh.SHERRY_KERNEL_SKINNY)
        sh.sherry_gemm_ex(wq, qd, sxd2, 0.02, y2, None, m, n, k, sh.SHERRY_KERNEL_MFMA)

    work()
    torch.cuda.synchronize()
    ref = [v.clone() for v in [e[6] for e in fd] + [e[7] for e in fd] + [e[5] for e in fd]
           + [qd, sxd2, y1, y2]]
    outs = [e[6] for e in fd] + [e[7] for e in fd] + [e[5] for e in fd] + [qd, sxd2, y1, y2]
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            work()
    torch.cuda.synchronize()
    for rep in range(3):
        for o in outs:  # eager work between replays: poison every output
            if o.dtype.is_floating_point:
                o.fill_(float("nan"))
            else:
                o.fill_(-3)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for o, r in zip(outs, ref):
            assert torch.equal(o, r), rep
