"""GPU parity of the comparison layouts (2-bit and 1.67-bit, Sec. 2.3) against
the CPU oracle, through the C ABI: the int32 accumulators bit-exact, the fp32
outputs within 1e-5 relative (here bit-exact: the scales are powers of two).
The oracle multiplies the unpacked ternary matrix; it never reads either
layout."""
import sys

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

ORACLE_THREADS = 16
RTOL = 1e-5


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


LAYOUTS = {
    # name: (host packer, single product, grouped prepare, grouped launch, oracle unpack)
    "2bit": ("sherry_pack2", "sherry_gemv2", "sherry_gemv2_batched_prepare",
             "sherry_gemv2_batched", oracle.unpack2),
    "1.67bit": ("sherry_pack3", "sherry_gemv3", "sherry_gemv3_batched_prepare",
                "sherry_gemv3_batched", oracle.unpack3),
}


def _check(acc, y, t, q, sx, sw):
    acc_ref = oracle.gemm_i32(q, t, threads=ORACLE_THREADS)[0]
    assert np.array_equal(acc, acc_ref)
    y_ref = oracle.epilogue(acc_ref[None, :], np.array([sx], np.float32), sw)[0]
    assert not (np.abs(y.astype(np.float64) - y_ref) > RTOL * np.abs(y_ref)).any()


@pytest.mark.parametrize("layout", list(LAYOUTS))
@pytest.mark.parametrize("n,k", [(1, 4), (64, 64), (64, 96), (65, 68), (63, 100), (130, 1028),
                                 (300, 2048), (128, 4100), (257, 3072), (70, 14336)])
def test_single_product_parity(dev, layout, n, k):
    sh = _sh()
    pack, call = getattr(sh, LAYOUTS[layout][0]), getattr(sh, LAYOUTS[layout][1])
    _say(layout, "single", n, k)
    t = synth.ternary_any(n, k, 61, "cmp", layout, n, k)
    q = synth.int8_any(1, k, 61, "cmpx", layout, n, k)
    p = pack(t)
    # the host packer writes what the oracle reads back
    assert np.array_equal(LAYOUTS[layout][4](p, n, k), t)
    w = torch.from_numpy(p).to(dev)
    sx = torch.full((1,), 0.5, dtype=torch.float32, device=dev)
    y = torch.full((n,), float("nan"), dtype=torch.float32, device=dev)
    a = torch.full((n,), -7, dtype=torch.int32, device=dev)
    call(w, torch.from_numpy(q).to(dev), sx, 0.25, y, a, n, k)
    torch.cuda.synchronize()
    _check(a.cpu().numpy(), y.cpu().numpy(), t, q, 0.5, 0.25)


@pytest.mark.parametrize("layout", list(LAYOUTS))
def test_extreme_activations(dev, layout):
    # every activation -128 or 127, weights all +1 / all -1 / 3:4: the
    # 2-bit product's sum correction and the 1.67-bit activation slicing at
    # their extremes
    sh = _sh()
    pack, call = getattr(sh, LAYOUTS[layout][0]), getattr(sh, LAYOUTS[layout][1])
    n, k = 192, 2052
    t = np.ones((n, k), np.int8)
    t[64:128] = -1
    t[128:] = synth.ternary_34(64, k, 62, "ext")
    for fill in (-128, 127):
        _say(layout, "extreme", fill)
        q = np.full((1, k), fill, np.int8)
        q[0, 5::7] = -fill if fill != -128 else 127
        w = torch.from_numpy(pack(t)).to(dev)
        sx = torch.full((1,), 1.0, dtype=torch.float32, device=dev)
        y = torch.empty(n, dtype=torch.float32, device=dev)
        a = torch.empty(n, dtype=torch.int32, device=dev)
        call(w, torch.from_numpy(q).to(dev), sx, 1.0, y, a, n, k)
        torch.cuda.synchronize()
        _check(a.cpu().numpy(), y.cpu().numpy(), t, q, 1.0, 1.0)


def _grouped(dev, layout, shapes, seed, tag):
    sh = _sh()
    pack = getattr(sh, LAYOUTS[layout][0])
    prep, run = getattr(sh, LAYOUTS[layout][2]), getattr(sh, LAYOUTS[layout][3])
    descs = (sh.sherry_gemv_desc * len(shapes))()
    keep, cases = [], []
    for i, (n, k) in enumerate(shapes):
        t = synth.ternary_34(n, k, seed, tag, i) if i % 2 else synth.ternary_any(n, k, seed, tag, i)
        q = synth.int8_any(1, k, seed, tag + "x", i)
        sx, sw = 2.0 ** -(i % 5), 2.0 ** -(1 + i % 3)
        w = torch.from_numpy(pack(t)).to(dev)
        qd = torch.from_numpy(q).to(dev)
        sxd = torch.full((1,), sx, dtype=torch.float32, device=dev)
        y = torch.full((n,), float("nan"), dtype=torch.float32, device=dev)
        a = torch.full((n,), -7, dtype=torch.int32, device=dev)
        keep += [w, qd, sxd, y, a]
        d = descs[i]
        d.w, d.x, d.x_scale, d.y, d.acc = (w.data_ptr(), qd.data_ptr(), sxd.data_ptr(),
                                           y.data_ptr(), a.data_ptr())
        d.n, d.k, d.w_scale = n, k, sw
        cases.append((t, q, sx, sw, y, a))
    total = prep(descs)
    dd = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
    run(dd, len(shapes), total)
    torch.cuda.synchronize()
    for (t, q, sx, sw, y, a) in cases:
        _check(a.cpu().numpy(), y.cpu().numpy(), t, q, sx, sw)


@pytest.mark.parametrize("layout", list(LAYOUTS))
def test_grouped_ragged_parity(dev, layout):
    # 70 products (two ballot rounds of the descriptor search), ragged n and k
    shapes = [(64 + 37 * (i % 5), 4 * (1 + (i * 97) % 700)) for i in range(70)]
    _say(layout, "grouped ragged", len(shapes))
    _grouped(dev, layout, shapes, 63, "cmpg" + layout)


@pytest.mark.parametrize("layout", list(LAYOUTS))
def test_grouped_8b_layer_full_size(dev, layout):
    # one layer of the 8B-scale stress model (hidden 4096, intermediate
    # 14336, kv 1024) in one grouped launch, every output checked
    blk = synth.llama_block(synth.STRESS_8B["hidden"], synth.STRESS_8B["kv"],
                            synth.STRESS_8B["inter"])
    shapes = [(lin.n, lin.k) for lin in blk]
    _say(layout, "grouped 8b layer", shapes)
    _grouped(dev, layout, shapes, 64, "cmp8b" + layout)
