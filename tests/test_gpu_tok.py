"""GPU parity of the small-M matrix-core kernels against the CPU oracle: the
GEMV for up to four tokens (SHERRY_KERNEL_GEMV_TOK: activations staged in
LDS, one int8 MFMA per 4-code chunk), single and grouped launches, with
per-tensor, per-channel and per-group scales, and the 16-token window kernel
of grouped launches: int32 accumulators bit-exact, fp32 outputs within 1e-5
relative (per-group scales: within the fp32-sum bound of sherry_gemm_group)."""
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


def _y_ok(y, y_ref):
    y = np.asarray(y, np.float64)
    return not (np.abs(y - y_ref) > RTOL * np.abs(y_ref)).any()


def _epi(acc, sx, sw):
    return oracle.epilogue_rows(acc, sx, sw) if np.ndim(sw) else oracle.epilogue(acc, sx, sw)


def _scales(m, seed, tag):
    return (np.abs(synth.activations(1, m, seed, tag)[0]) + 0.01).astype(np.float32)


# ragged n and k, several row tiles and K splits, and the longest k each m
# can stage (m * ceil(k/128) * 128 <= 32768)
CASES = [(1, 64, 128), (2, 65, 132), (3, 130, 1028), (4, 300, 2048), (4, 257, 3076),
         (1, 70, 32768), (2, 129, 16380), (3, 64, 10880), (4, 600, 8192), (4, 3072, 8192)]


@pytest.mark.parametrize("m,n,k", CASES)
@pytest.mark.parametrize("channel", [False, True])
def test_tok_kernel_parity(dev, m, n, k, channel):
    sh = _sh()
    _say("tok", m, n, k, channel)
    t = synth.ternary_34(n, k, 71, "tok", m, n, k)
    q = synth.int8_any(m, k, 71, "tokq", m, n, k)
    sx = _scales(m, 71, "toks%d" % m)
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    qd, sxd = torch.from_numpy(q).to(dev), torch.from_numpy(sx).to(dev)
    y = torch.full((m, n), float("nan"), dtype=torch.float32, device=dev)
    a = torch.full((m, n), -7, dtype=torch.int32, device=dev)
    if channel:
        sw = (np.random.default_rng(n + k).random(n) * 0.05 + 0.001).astype(np.float32)
        swd = torch.from_numpy(sw).to(dev)
        sh.sherry_gemm_channel(w, qd, sxd, swd, y, a, m, n, k, sh.SHERRY_KERNEL_GEMV_TOK)
    else:
        sw = 0.0173
        sh.sherry_gemm_ex(w, qd, sxd, sw, y, a, m, n, k, sh.SHERRY_KERNEL_GEMV_TOK)
    torch.cuda.synchronize()
    acc_ref = oracle.gemm_i32(q, t, threads=ORACLE_THREADS)
    assert np.array_equal(a.cpu().numpy(), acc_ref)
    assert _y_ok(y.cpu().numpy(), _epi(acc_ref, sx, sw))


def test_tok_kernel_extremes_and_agreement(dev):
    # activations at -128 / 127, all-(+1) and all-(-1) rows next to 3:4 rows;
    # the same product on the v_dot4 GEMV gives the same bits
    sh = _sh()
    m, n, k = 4, 192, 4096
    q = np.where(synth.int8_any(m, k, 72, "ext") >= 0, 127, -128).astype(np.int8)
    t = synth.ternary_34(n, k, 72, "ext")
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    qd = torch.from_numpy(q).to(dev)
    sxd = torch.ones(m, dtype=torch.float32, device=dev)
    outs = []
    for kern in (sh.SHERRY_KERNEL_GEMV_TOK, sh.SHERRY_KERNEL_GEMV):
        y = torch.empty((m, n), dtype=torch.float32, device=dev)
        a = torch.empty((m, n), dtype=torch.int32, device=dev)
        sh.sherry_gemm_ex(w, qd, sxd, 1.0, y, a, m, n, k, kern)
        torch.cuda.synchronize()
        outs.append((y.cpu().numpy(), a.cpu().numpy()))
    assert np.array_equal(outs[0][1], oracle.gemm_i32(q, t, threads=ORACLE_THREADS))
    assert np.array_equal(outs[0][0].view(np.uint32), outs[1][0].view(np.uint32))
    assert np.array_equal(outs[0][1], outs[1][1])


def test_tok_kernel_rejects_what_it_cannot_stage(dev):
    sh = _sh()
    L = sh.lib
    w = torch.zeros(sh.sherry_packed_bytes(64, 8320), dtype=torch.uint8, device=dev)
    x = torch.zeros((5, 8320), dtype=torch.int8, device=dev)
    sx = torch.ones(5, dtype=torch.float32, device=dev)
    y = torch.empty((5, 64), dtype=torch.float32, device=dev)
    for m, k in ((4, 8320), (5, 128), (3, 11008), (1, 32896)):
        assert L.sherry_gemm_ex(w.data_ptr(), x.data_ptr(), sx.data_ptr(), 1.0, y.data_ptr(),
                                None, m, 64, k, sh.SHERRY_KERNEL_GEMV_TOK, None) == \
            sh.SHERRY_E_SHAPE


def _group_scales(n, k, seed):
    rng = np.random.default_rng(seed)
    return (rng.random((n, (k + 127) // 128)) * 0.05 + 0.001).astype(np.float32)


def _group_ok(y, y_ref, mag, k):
    # fp32 summation in any order: |y - y_ref| <= (G + 4) * 2^-24 * mag
    bound = ((k + 127) // 128 + 4) * 2.0 ** -24 * mag + 1e-30
    return bool(np.all(np.abs(np.asarray(y, np.float64) - y_ref) <= bound))


# per-group scales on the token kernel: ragged n, a partial last group, K
# split over several waves, the longest k each m can stage
GROUP_TOK_CASES = [(1, 70, 132), (2, 65, 1028), (3, 130, 3076), (4, 600, 2048), (4, 3072, 8192),
                   (1, 64, 32768), (2, 257, 16380)]


@pytest.mark.parametrize("m,n,k", GROUP_TOK_CASES)
def test_tok_kernel_group_scales(dev, m, n, k):
    sh = _sh()
    _say("tok group", m, n, k)
    t = synth.ternary_34(n, k, 81, "tgr", n, k)
    q = synth.int8_any(m, k, 81, "tgrq", m, k)
    sx = _scales(m, 81, "tgrs%d" % m)
    gs = _group_scales(n, k, 81 + n)
    w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    y = torch.full((m, n), float("nan"), dtype=torch.float32, device=dev)
    acc = torch.full((m, n), -7, dtype=torch.int32, device=dev)
    sh.sherry_gemm_group(w, torch.from_numpy(q).to(dev), torch.from_numpy(sx).to(dev),
                         torch.from_numpy(gs).to(dev), y, acc, m, n, k, sh.SHERRY_KERNEL_GEMV_TOK)
    torch.cuda.synchronize()
    y_ref, mag, acc_ref = oracle.product_groups(q, t, sx, gs, threads=ORACLE_THREADS)
    assert np.array_equal(acc.cpu().numpy(), acc_ref)
    assert _group_ok(y.cpu().numpy(), y_ref, mag, k)


def test_tok_kernel_group_scales_rejects_long_rows(dev):
    sh = _sh()
    w = torch.zeros(sh.sherry_packed_bytes(64, 8320), dtype=torch.uint8, device=dev)
    x = torch.zeros((4, 8320), dtype=torch.int8, device=dev)
    sx = torch.ones(4, dtype=torch.float32, device=dev)
    gs = torch.ones((64, 65), dtype=torch.float32, device=dev)
    y = torch.empty((4, 64), dtype=torch.float32, device=dev)
    assert sh.lib.sherry_gemm_group(w.data_ptr(), x.data_ptr(), sx.data_ptr(), gs.data_ptr(),
                                    y.data_ptr(), None, 4, 64, 8320, sh.SHERRY_KERNEL_GEMV_TOK,
                                    None) == sh.SHERRY_E_SHAPE


def _grouped(dev, cases, seed, channel=False, groups=False, il=False, outs=None):
    # il: lane-interleaved weights on sherry_gemm_il_batched; outs: a list that
    # receives each product's (y, acc) as host arrays
    sh = _sh()
    descs = (sh.sherry_gemm_desc * len(cases))()
    keep = []
    for i, (m, n, k) in enumerate(cases):
        t = synth.ternary_34(n, k, seed, "tg", i)
        q = synth.int8_any(m, k, seed, "tgq", i)
        sx = _scales(m, seed, "tgs%d" % i)
        w = torch.from_numpy(sh.sherry_pack_il(t) if il else sh.sherry_pack(t)).to(dev)
        qd, sxd = torch.from_numpy(q).to(dev), torch.from_numpy(sx).to(dev)
        y = torch.full((m, n), float("nan"), dtype=torch.float32, device=dev)
        a = torch.full((m, n), -7, dtype=torch.int32, device=dev)
        d = descs[i]
        d.w, d.x, d.x_scale, d.y = w.data_ptr(), qd.data_ptr(), sxd.data_ptr(), y.data_ptr()
        d.acc = a.data_ptr() if i % 4 != 3 else None
        d.n, d.k, d.m, d.w_scale = n, k, m, synth.weight_scale(seed, "tgw", i)
        sw, hold = d.w_scale, None
        if channel and i % 2 == 0:
            sw = (np.random.default_rng(seed + i).random(n) * 0.05 + 0.001).astype(np.float32)
            hold = torch.from_numpy(sw).to(dev)
            d.w_scales = hold.data_ptr()
        elif groups and i % 3 != 2:
            # per-group scales (no int32 totals with them)
            sw = ("groups", _group_scales(n, k, seed + i))
            hold = torch.from_numpy(sw[1]).to(dev)
            d.w_group_scales, d.acc = hold.data_ptr(), None
        keep.append((t, q, sx, sw, d.acc is not None, w, qd, sxd, y, a, hold))
    if il:
        total, max_m = sh.sherry_gemm_il_batched_prepare(descs)
        dd = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
        sh.sherry_gemm_il_batched(dd, len(cases), total, max_m)
    else:
        total, max_m = sh.sherry_gemm_batched_prepare(descs)
        dd = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
        sh.sherry_gemm_batched(dd, len(cases), total, max_m)
    torch.cuda.synchronize()
    if outs is not None:
        outs.extend((y.cpu().numpy(), a.cpu().numpy()) for *_, y, a, hold in keep)
    for t, q, sx, sw, has_acc, w, qd, sxd, y, a, hold in keep:
        if isinstance(sw, tuple):
            y_ref, mag, _ = oracle.product_groups(q, t, sx, sw[1], threads=ORACLE_THREADS)
            assert (a.cpu().numpy() == -7).all()
            assert _group_ok(y.cpu().numpy(), y_ref, mag, t.shape[1])
            continue
        acc_ref = oracle.gemm_i32(q, t, threads=ORACLE_THREADS)
        if has_acc:
            assert np.array_equal(a.cpu().numpy(), acc_ref)
        else:
            assert (a.cpu().numpy() == -7).all()
        assert _y_ok(y.cpu().numpy(), _epi(acc_ref, sx, sw))
    return max_m


@pytest.mark.parametrize("il", [False, True])
@pytest.mark.parametrize("channel", [False, True])
def test_tok_batched_parity(dev, channel, il):
    # 70 products of 1-4 tokens (two ballot rounds of the descriptor search)
    _say("tok batched", channel, "il" if il else "tiled")
    cases = [(1 + i % 4, 64 + 37 * (i % 5), 4 * (1 + (i * 97) % 700)) for i in range(70)]
    assert _grouped(dev, cases, 73, channel, il=il) == 4


def test_tok_batched_group_scales(dev):
    # 70 products of 1-4 tokens, two in three with per-group scales, the
    # rest per-channel or per-tensor: all on the token kernel
    _say("tok batched groups")
    cases = [(1 + i % 4, 64 + 37 * (i % 5), 4 * (1 + (i * 97) % 700)) for i in range(70)]
    assert _grouped(dev, cases, 82, channel=False, groups=True) == 4 | _sh().SHERRY_LAUNCH_GROUPS


def test_tok_batched_group_scales_model_step_full(dev):
    # one LLaMA-3.2-3B layer at 4 tokens with per-group scales, every output
    _say("tok batched groups 3b layer")
    spec = synth.LLAMA_3B
    blk = synth.llama_block(spec["hidden"], spec["kv"], spec["inter"])
    assert _grouped(dev, [(4, lin.n, lin.k) for lin in blk], 83, groups=True) == \
        4 | _sh().SHERRY_LAUNCH_GROUPS


@pytest.mark.parametrize("il", [False, True])
@pytest.mark.parametrize("m", [2, 4])
def test_tok_batched_model_step_full(dev, m, il):
    # one LLaMA-3.2-3B layer at M tokens in one grouped launch, every output
    _say("tok batched 3b layer", m, "il" if il else "tiled")
    spec = synth.LLAMA_3B
    blk = synth.llama_block(spec["hidden"], spec["kv"], spec["inter"])
    assert _grouped(dev, [(m, lin.n, lin.k) for lin in blk], 74, il=il) == m


@pytest.mark.parametrize("il", [False, True])
def test_small_m_too_long_goes_to_window_kernel(dev, il):
    # m <= 4 but one product cannot stage its activations: every product
    # runs on the 16-token window kernel (launch value 5)
    _say("small m, long k", "il" if il else "tiled")
    cases = [(4, 64, 8320), (2, 130, 1028), (1, 65, 132)]
    assert _grouped(dev, cases, 75, il=il) == 5


# 5-16 tokens: the window kernel (16 token rows staged per 1024-value window
# of K, one 32x32x32 MFMA per 4-code chunk for 64 rows), with ragged n and k
# (k % 16 != 0: the last piece of a row is read word by word), partial
# windows, several windows, per-channel scales and products without acc
WINDOW_CASES = [(5, 64, 128), (16, 65, 132), (9, 600, 2048), (16, 257, 3076), (12, 130, 1028),
                (16, 3072, 8192), (7, 70, 4), (16, 1024, 3072), (6, 520, 14340)]


@pytest.mark.parametrize("il", [False, True])
@pytest.mark.parametrize("channel", [False, True])
def test_window_kernel_grouped_parity(dev, channel, il):
    _say("window kernel", channel, "il" if il else "tiled")
    assert _grouped(dev, WINDOW_CASES, 76, channel, il=il) == 16


@pytest.mark.parametrize("il", [False, True])
def test_window_kernel_many_products(dev, il):
    # 70 products of 5-16 tokens (two ballot rounds of the descriptor search)
    _say("window kernel, 70 products", "il" if il else "tiled")
    cases = [(5 + i % 12, 64 + 37 * (i % 5), 4 * (1 + (i * 97) % 700)) for i in range(70)]
    assert _grouped(dev, cases, 77, il=il) == 16


@pytest.mark.parametrize("il", [False, True])
@pytest.mark.parametrize("m", [8, 16])
def test_window_kernel_model_step_full(dev, m, il):
    # one LLaMA-3.2-3B layer at M tokens in one grouped launch, every output
    _say("window kernel 3b layer", m, "il" if il else "tiled")
    spec = synth.LLAMA_3B
    blk = synth.llama_block(spec["hidden"], spec["kv"], spec["inter"])
    assert _grouped(dev, [(m, lin.n, lin.k) for lin in blk], 78, il=il) == m


def test_window_kernel_group_scales(dev):
    # 5-16 tokens, per-group scales on every other product (k % 512 == 0),
    # per-channel or per-tensor on the rest: one window-kernel launch
    _say("window kernel groups")
    cases = [(5, 64, 512), (16, 65, 1024), (9, 600, 2048), (16, 257, 3072), (12, 130, 4096),
             (16, 3072, 8192), (7, 70, 1536), (6, 520, 14336)]
    G = _sh().SHERRY_LAUNCH_GROUPS
    assert _grouped(dev, cases, 84, groups=True) == 16 | G


def test_window_kernel_group_scales_model_step_full(dev):
    # one LLaMA-3.2-3B layer at 16 tokens with per-group scales, every output
    _say("window kernel groups 3b layer")
    spec = synth.LLAMA_3B
    blk = synth.llama_block(spec["hidden"], spec["kv"], spec["inter"])
    assert _grouped(dev, [(16, lin.n, lin.k) for lin in blk], 85, groups=True) == \
        16 | _sh().SHERRY_LAUNCH_GROUPS


def test_window_kernel_group_scales_need_whole_chunks(dev):
    # a per-group product with k % 512 != 0 sends the launch to the
    # register-decoded kernel (launch value 17 with the flag)
    _say("window kernel groups, ragged k")
    cases = [(8, 64, 1028), (5, 130, 512)]
    assert _grouped(dev, cases, 86, groups=True) == 17 | _sh().SHERRY_LAUNCH_GROUPS


@pytest.mark.parametrize("il", [False, True])
@pytest.mark.parametrize("m,k", [(16, 4096), (4, 8192)])
def test_window_kernel_extremes(dev, m, k, il):
    # activations at -128 / 127 for every token, k = 4096 (4 windows) at 16
    # tokens and the longest k four tokens can stage (token kernels); row 0
    # follows token 0's signs (three of every four weights), row 1 their
    # opposite: the largest sums the activations allow
    _say("extremes", m, k, "il" if il else "tiled")
    sh = _sh()
    n = 192
    q = np.where(synth.int8_any(m, k, 79, "wext") >= 0, 127, -128).astype(np.int8)
    t = synth.ternary_34(n, k, 79, "wext")
    sg = np.where(q[0] >= 0, 1, -1).astype(np.int8).reshape(-1, 4)
    aligned = sg.copy()
    aligned[:, 0] = 0
    t[0] = aligned.reshape(-1)
    t[1] = -aligned.reshape(-1)
    w = torch.from_numpy(sh.sherry_pack_il(t) if il else sh.sherry_pack(t)).to(dev)
    qd = torch.from_numpy(q).to(dev)
    sxd = torch.ones(m, dtype=torch.float32, device=dev)
    y = torch.empty((m, n), dtype=torch.float32, device=dev)
    a = torch.empty((m, n), dtype=torch.int32, device=dev)
    descs = (sh.sherry_gemm_desc * 1)()
    d = descs[0]
    d.w, d.x, d.x_scale, d.y, d.acc = w.data_ptr(), qd.data_ptr(), sxd.data_ptr(), y.data_ptr(), a.data_ptr()
    d.n, d.k, d.m, d.w_scale = n, k, m, 1.0
    prep = sh.sherry_gemm_il_batched_prepare if il else sh.sherry_gemm_batched_prepare
    launch = sh.sherry_gemm_il_batched if il else sh.sherry_gemm_batched
    total, max_m = prep(descs)
    assert max_m == m
    launch(torch.from_numpy(sh.descs_to_bytes(descs)).to(dev), 1, total, max_m)
    torch.cuda.synchronize()
    acc_ref = oracle.gemm_i32(q, t, threads=ORACLE_THREADS)
    assert acc_ref[0, 0] == np.abs(q[0].astype(np.int64)).reshape(-1, 4)[:, 1:].sum()
    assert np.array_equal(a.cpu().numpy(), acc_ref)


@pytest.mark.parametrize("mmax", [4, 16])
def test_grouped_layouts_agree(dev, mmax):
    # the same grouped products on tiled and on lane-interleaved weights:
    # the same bits, y and int32 accumulators
    _say("grouped tiled vs il", mmax)
    cases = [(1 + i % mmax, 64 + 37 * (i % 5), 4 * (1 + (i * 97) % 700)) for i in range(40)]
    a, b = [], []
    _grouped(dev, cases, 87, channel=True, outs=a)
    _grouped(dev, cases, 87, channel=True, il=True, outs=b)
    for (ya, aa), (yb, ab) in zip(a, b):
        assert np.array_equal(ya.view(np.uint32), yb.view(np.uint32))
        assert np.array_equal(aa, ab)


@pytest.mark.parametrize("n,k", [(1, 4), (64, 128), (65, 132), (300, 3076), (2048, 8192)])
def test_interleave_on_device_matches_host(dev, n, k):
    # the device converter writes what the host interleaved packer writes;
    # from GPU-ternarized weights too
    sh = _sh()
    _say("interleave", n, k)
    t = synth.ternary_34(n, k, 88, "ilv", n, k)
    tiled = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    il = torch.full_like(tiled, 0xA5)
    sh.sherry_interleave(tiled, il, n, k)
    torch.cuda.synchronize()
    assert np.array_equal(il.cpu().numpy(), sh.sherry_pack_il(t))


def test_interleave_after_gpu_ternarize(dev):
    sh = _sh()
    n, k = 300, 3076
    w = torch.from_numpy(synth.dense_weights(n, k, 89, "tpil")).to(dev)
    packed = torch.empty(sh.sherry_packed_bytes(n, k), dtype=torch.uint8, device=dev)
    alpha = torch.empty(n, dtype=torch.float32, device=dev)
    sh.sherry_ternarize_pack(w, n, k, packed, alpha)
    il = torch.empty_like(packed)
    sh.sherry_interleave(packed, il, n, k)
    torch.cuda.synchronize()
    t = sh.sherry_unpack(packed.cpu().numpy(), n, k)
    assert np.array_equal(il.cpu().numpy(), sh.sherry_pack_il(t))
    assert np.array_equal(sh.sherry_unpack_il(il.cpu().numpy(), n, k), t)
