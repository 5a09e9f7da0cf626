"""Host-side tests of the C ABI: exports, validation, packing parity.

No GPU needed: every device call here fails host validation before anything
is enqueued (fake pointers are never dereferenced).
"""
import ctypes
import json
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
import paper_2601_07892_amd as sh
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sherry.h")
GOLDEN = os.path.join(ROOT, "tests", "golden")
L = sh.lib
FAKE = 0x10000  # 64 KiB-aligned, never dereferenced
FAKE_MIS = FAKE + 2


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(sherry_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert len(names) >= 17
    out = subprocess.run(["nm", "-D", "--defined-only", sh.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (sherry_\w+)", out))
    for n in names:
        assert n in exported, n
        assert hasattr(L, n), n
    assert set(names) == set(sh.EXPORTS)


def test_status_strings_and_version():
    for st in range(7):
        assert sh._status_str(st)
    assert "gfx950" in sh.sherry_version()


def test_packed_bytes():
    assert sh.sherry_packed_bytes(2048, 2048) == 2048 * 2048 * 5 // 32
    assert sh.sherry_packed_bytes(1, 4) == 64 * 128 * 5 // 32
    assert sh.sherry_packed_bytes(0, 4) == 0
    assert sh.sherry_packed_bytes(4, 6) == 0
    assert sh.sherry_packed_bytes(4, sh.SHERRY_MAX_K + 4) == 0
    for n, k in [(1, 4), (70, 1032), (2048, 8192)]:
        assert sh.sherry_packed_bytes(n, k) == oracle.packed_bytes(n, k)
        assert sh.sherry_packed2_bytes(n, k) == oracle.packed2_bytes(n, k)


# ------------------------------------------------------------- packing parity

@pytest.mark.parametrize("n,k", [(1, 4), (1, 8), (3, 124), (63, 128), (64, 132), (65, 516),
                                 (130, 1032), (257, 2048), (64, 4100)])
def test_pack_matches_oracle(n, k):
    t = synth.ternary_34(n, k, 21, "pk")
    p = sh.sherry_pack(t)
    assert np.array_equal(p, oracle.pack(t))
    assert np.array_equal(sh.sherry_unpack(p, n, k), t)
    assert np.array_equal(oracle.unpack(p, n, k), t)
    t2 = synth.ternary_any(n, k, 21, "pk2")
    p2 = sh.sherry_pack2(t2)
    assert np.array_equal(p2, oracle.pack2(t2))
    assert np.array_equal(oracle.unpack2(p2, n, k), t2)


@pytest.mark.parametrize("n,k", [(1, 1), (1, 3), (2, 4), (63, 95), (64, 96), (65, 97),
                                 (130, 1028), (257, 2048), (64, 3072), (3, 14336)])
def test_pack3_matches_oracle(n, k):
    t = synth.ternary_any(n, k, 25, "pk3")
    assert sh.sherry_packed3_bytes(n, k) == oracle.packed3_bytes(n, k)
    p3 = sh.sherry_pack3(t)
    assert np.array_equal(p3, oracle.pack3(t))
    assert np.array_equal(sh.sherry_unpack3(p3, n, k), t)
    # 3:4 matrices are ternary too (the 8B-scale comparison packs the same T)
    t34 = synth.ternary_34(n, (k + 3) // 4 * 4, 25, "pk3s")
    assert np.array_equal(sh.sherry_pack3(t34), oracle.pack3(t34))


def test_pack3_rejects_values_codes_and_buffers():
    t = synth.ternary_any(3, 10, 26, "bad3")
    t[2, 4] = -2
    bad = ctypes.c_int64(-1)
    out = np.zeros(sh.sherry_packed3_bytes(3, 10), np.uint8)
    assert L.sherry_pack3(t.ctypes.data, 3, 10, out.ctypes.data, out.nbytes,
                          ctypes.byref(bad)) == sh.SHERRY_E_INVALID
    assert bad.value == 24
    t[2, 4] = 1
    assert L.sherry_pack3(t.ctypes.data, 3, 10, out.ctypes.data, out.nbytes - 1,
                          None) == sh.SHERRY_E_BUFSIZE
    assert L.sherry_pack3(t.ctypes.data, 0, 10, out.ctypes.data, out.nbytes,
                          None) == sh.SHERRY_E_SHAPE
    p = sh.sherry_pack3(t)
    for code in range(27, 32):  # unused codes, written into row 1's code 0
        q = p.copy()
        q[16] = (q[16] & 0xE0) | code
        with pytest.raises(sh.SherryError):
            sh.sherry_unpack3(q, 3, 10)
    assert sh.sherry_packed3_bytes(1, sh.SHERRY_MAX_K + 1) == 0


@pytest.mark.parametrize("idx", [0, 1, 2])
def test_pack_hand_derived_fixtures(idx):
    with open(os.path.join(GOLDEN, "packed_fixtures.json")) as f:
        fx = json.load(f)["five_bit"][idx]
    g = oracle.code_table()
    t = np.tile(np.array([0, 1, 1, 1], np.int8), (fx["n"], fx["k"] // 4))
    for row, blk, code in fx["blocks"]:
        t[row, 4 * blk:4 * blk + 4] = g[code]
    p = sh.sherry_pack(t)
    assert p.size == fx["total_bytes"]
    nz = {int(i): int(p[i]) for i in np.nonzero(p)[0]}
    assert nz == {int(a): b for a, b in fx["nonzero"].items()}


@pytest.mark.parametrize("idx", [0, 1])
def test_pack_il_hand_derived_fixtures(idx):
    with open(os.path.join(GOLDEN, "packed_fixtures.json")) as f:
        fx = json.load(f)["lane_interleaved"][idx]
    g = oracle.code_table()
    t = np.tile(np.array([0, 1, 1, 1], np.int8), (fx["n"], fx["k"] // 4))
    for row, blk, code in fx["blocks"]:
        t[row, 4 * blk:4 * blk + 4] = g[code]
    p = sh.sherry_pack_il(t)
    assert p.size == fx["total_bytes"]
    nz = {int(i): int(p[i]) for i in np.nonzero(p)[0]}
    assert nz == {int(a): b for a, b in fx["nonzero"].items()}


@pytest.mark.parametrize("n,k", [(1, 4), (64, 128), (65, 132), (130, 1028), (300, 3076),
                                 (2100, 2048)])
def test_pack_il_matches_oracle(n, k):
    t = synth.ternary_34(n, k, 23, "il", n, k)
    p = sh.sherry_pack_il(t)
    assert np.array_equal(p, oracle.pack_il(t))
    assert np.array_equal(sh.sherry_unpack_il(p, n, k), t)
    assert np.array_equal(oracle.unpack_il(p, n, k), t)


def test_pack_il_errors():
    t = synth.ternary_34(5, 64, 24, "ile")
    t[3, 20:24] = [1, 1, 0, 0]
    with pytest.raises(sh.SherryError) as e:
        sh.sherry_pack_il(t)
    assert e.value.status == sh.SHERRY_E_NOT_3_4 and e.value.bad_block == 3 * 16 + 5
    L = sh.lib
    good = synth.ternary_34(5, 64, 24, "ilg")
    out = np.zeros(sh.sherry_packed_bytes(5, 64), np.uint8)
    assert L.sherry_pack_il(good.ctypes.data, 5, 64, out.ctypes.data, out.nbytes - 1,
                            None) == sh.SHERRY_E_BUFSIZE
    assert L.sherry_pack_il(good.ctypes.data, 5, 66, out.ctypes.data, out.nbytes,
                            None) == sh.SHERRY_E_SHAPE
    t_out = np.zeros((5, 64), np.int8)
    assert L.sherry_unpack_il(out.ctypes.data, out.nbytes - 1, 5, 64,
                              t_out.ctypes.data) == sh.SHERRY_E_BUFSIZE
    assert L.sherry_unpack_il(None, out.nbytes, 5, 64, t_out.ctypes.data) == sh.SHERRY_E_INVALID


def test_il_fused_prepare_rejects_group_scales():
    descs = (sh.sherry_gemv_f32_desc * 2)()
    for d in descs:
        d.w, d.x, d.y = FAKE, FAKE, FAKE
        d.n, d.k, d.w_scale = 64, 128, 1.0
    assert sh.sherry_gemv_f32_il_batched_prepare(descs) == sh.sherry_gemv_f32_batched_prepare(descs)
    descs[1].w_group_scales = FAKE
    with pytest.raises(sh.SherryError):
        sh.sherry_gemv_f32_il_batched_prepare(descs)
    L = sh.lib
    assert L.sherry_gemv_f32_il_batched(None, 1, 1, None) == sh.SHERRY_E_INVALID
    assert L.sherry_gemv_f32_il_batched(FAKE + 4, 1, 1, None) == sh.SHERRY_E_ALIGN


def test_grouped_prepare_numbers_blocks_longest_rows_first():
    # one LLaMA-3.2-3B layer in model order and reversed, on the three
    # grouped kernels: each product's range [block_begin, block_begin +
    # block_count) is the same in both orders, the ranges tile the launch, and
    # the products with the longest rows (k = 8192) come first
    spec = synth.LLAMA_3B
    blk = synth.llama_block(spec["hidden"], spec["kv"], spec["inter"])
    for m, prepare in ((4, sh.sherry_gemm_batched_prepare), (16, sh.sherry_gemm_batched_prepare),
                       (64, sh.sherry_gemm_batched_prepare), (4, sh.sherry_gemm_il_batched_prepare),
                       (16, sh.sherry_gemm_il_batched_prepare)):
        got = []
        for order in (list(range(len(blk))), list(reversed(range(len(blk))))):
            descs = (sh.sherry_gemm_desc * len(blk))()
            for j, i in enumerate(order):
                d = descs[j]
                d.w, d.x, d.x_scale, d.y = FAKE, FAKE, FAKE, FAKE
                d.n, d.k, d.m, d.w_scale = blk[i].n, blk[i].k, m, 0.02
            total, _ = prepare(descs)
            r = {i: (descs[j].block_begin, descs[j].block_count) for j, i in enumerate(order)}
            spans = sorted(r.values())
            assert spans[0][0] == 0 and all(a[0] + a[1] == b[0] for a, b in zip(spans, spans[1:]))
            assert spans[-1][0] + spans[-1][1] == total
            assert all(c >= 1 for _, c in spans)
            longest = max(lin.k for lin in blk)
            first = [i for i in r if blk[i].k == longest]
            assert sorted(r[i][0] for i in first) == [b for b, _ in spans[:len(first)]]
            got.append((r, total))
        assert got[0][0].keys() == got[1][0].keys() and got[0][1] == got[1][1]
        assert all(got[0][0][i][1] == got[1][0][i][1] for i in got[0][0])


def test_il_grouped_prepare_without_launch():
    def prep(cases, group=False):
        descs = (sh.sherry_gemm_desc * len(cases))()
        for i, (m, n, k) in enumerate(cases):
            d = descs[i]
            d.w, d.x, d.x_scale, d.y = FAKE, FAKE, FAKE, FAKE
            d.n, d.k, d.m, d.w_scale = n, k, m, 0.02
            if group and i == 0:
                d.w_group_scales = FAKE
        total, max_m = sh.sherry_gemm_il_batched_prepare(descs)
        return [d.block_begin for d in descs], total, max_m
    # the same block counts and launch values as the tiled grouped launches
    # (blocks numbered longest rows first: the k = 8192 product's 24, then the
    # k = 3072 ones in array order)
    assert prep([(4, 3072, 3072), (2, 1024, 3072), (1, 3072, 8192)]) == ([24, 36, 0], 40, 4)
    assert prep([(4, 3072, 8320), (1, 64, 128)]) == ([0, 12], 13, 5)
    assert prep([(16, 3072, 8192), (9, 1024, 3072)]) == ([0, 12], 16, 16)
    with pytest.raises(sh.SherryError) as e:
        prep([(17, 64, 128)])
    assert e.value.status == sh.SHERRY_E_SHAPE
    with pytest.raises(sh.SherryError) as e:
        prep([(2, 64, 128)], group=True)
    assert e.value.status == sh.SHERRY_E_INVALID
    L = sh.lib
    assert L.sherry_gemm_il_batched(None, 1, 1, 4, None) == sh.SHERRY_E_INVALID
    assert L.sherry_gemm_il_batched(FAKE, 1, 1, 17, None) == sh.SHERRY_E_SHAPE
    assert L.sherry_gemm_il_batched(FAKE, 1, 1, 0, None) == sh.SHERRY_E_SHAPE
    assert L.sherry_gemm_il_batched(FAKE + 4, 1, 1, 16, None) == sh.SHERRY_E_ALIGN


def test_interleave_validation_without_launch():
    L = sh.lib
    assert L.sherry_interleave(None, FAKE, 64, 128, None) == sh.SHERRY_E_INVALID
    assert L.sherry_interleave(FAKE, FAKE, 64, 128, None) == sh.SHERRY_E_INVALID
    assert L.sherry_interleave(FAKE, FAKE + 4096, 64, 130, None) == sh.SHERRY_E_SHAPE
    assert L.sherry_interleave(FAKE + 4, FAKE + 4096, 64, 128, None) == sh.SHERRY_E_ALIGN


def test_pack_large_multithreaded():
    n, k = 4096, 2048  # many row tiles -> several host threads
    t = synth.ternary_34(n, k, 22, "big")
    p = sh.sherry_pack(t)
    assert np.array_equal(sh.sherry_unpack(p, n, k), t)
    # spot-check against the oracle on a slice of row tiles
    sub = t[128:256]
    assert np.array_equal(sh.sherry_pack(sub), oracle.pack(sub))


@pytest.mark.parametrize("zeros", [0, 2, 3, 4])
def test_pack_rejects_non_34(zeros):
    n, k = 700, 256
    t = synth.ternary_34(n, k, 23, "rej")
    blk = np.array([0] * zeros + [1] * (4 - zeros), np.int8)
    t[650, 8:12] = blk
    t[300, 100:104] = blk
    with pytest.raises(sh.SherryError) as e:
        sh.sherry_pack(t)
    assert e.value.status == sh.SHERRY_E_NOT_3_4
    assert e.value.bad_block == 300 * (k // 4) + 25 == oracle.pack_bad_block(t)


def test_pack_rejects_bad_values_and_buffers():
    t = synth.ternary_34(2, 8, 24, "val")
    t[1, 4:8] = [0, 1, 2, 1]
    with pytest.raises(sh.SherryError) as e:
        sh.sherry_pack(t)
    assert e.value.bad_block == 3
    t = synth.ternary_34(2, 8, 24, "buf")
    small = np.zeros(sh.sherry_packed_bytes(2, 8) - 1, np.uint8)
    assert L.sherry_pack(t.ctypes.data, 2, 8, small.ctypes.data, small.nbytes, None) == \
        sh.SHERRY_E_BUFSIZE
    assert L.sherry_pack(None, 2, 8, small.ctypes.data, small.nbytes, None) == sh.SHERRY_E_INVALID
    assert L.sherry_pack(t.ctypes.data, 2, 6, small.ctypes.data, small.nbytes, None) == \
        sh.SHERRY_E_SHAPE
    t2 = np.zeros((1, 8), np.int8)
    t2[0, 3] = 5
    bad = ctypes.c_int64(-1)
    out = np.zeros(sh.sherry_packed2_bytes(1, 8), np.uint8)
    assert L.sherry_pack2(t2.ctypes.data, 1, 8, out.ctypes.data, out.nbytes,
                          ctypes.byref(bad)) == sh.SHERRY_E_INVALID
    assert bad.value == 3


# -------------------------------------------------- validation of device calls

def test_gemm_validation_without_launch():
    g = L.sherry_gemm_ex
    # null pointers
    assert g(None, FAKE, FAKE, 1.0, FAKE, None, 1, 64, 128, 0, None) == sh.SHERRY_E_INVALID
    assert g(FAKE, FAKE, FAKE, 1.0, None, None, 1, 64, 128, 0, None) == sh.SHERRY_E_INVALID
    # shapes
    for m, n, k in [(0, 64, 128), (1, 0, 128), (1, 64, 0), (1, 64, 130),
                    (1, 64, sh.SHERRY_MAX_K + 4)]:
        assert g(FAKE, FAKE, FAKE, 1.0, FAKE, None, m, n, k, 0, None) == sh.SHERRY_E_SHAPE
    # GEMV kernel is limited to m <= 4
    assert g(FAKE, FAKE, FAKE, 1.0, FAKE, None, 5, 64, 128, sh.SHERRY_KERNEL_GEMV,
             None) == sh.SHERRY_E_SHAPE
    # alignment: packed weights 16 B, activations 16 B for the MFMA kernel
    assert g(FAKE_MIS, FAKE, FAKE, 1.0, FAKE, None, 1, 64, 128, 0, None) == sh.SHERRY_E_ALIGN
    assert g(FAKE, FAKE + 4, FAKE, 1.0, FAKE, None, 64, 64, 128, sh.SHERRY_KERNEL_MFMA,
             None) == sh.SHERRY_E_ALIGN
    assert g(FAKE, FAKE, FAKE, 1.0, FAKE, FAKE_MIS, 64, 64, 128, sh.SHERRY_KERNEL_MFMA,
             None) == sh.SHERRY_E_ALIGN
    assert g(FAKE, FAKE, FAKE, 1.0, FAKE, None, 8, 64, 128, 7, None) == sh.SHERRY_E_INVALID
    assert L.sherry_gemv(FAKE, FAKE + 1, FAKE, 1.0, FAKE, None, 64, 128, None) == \
        sh.SHERRY_E_ALIGN
    assert L.sherry_quantize_act(FAKE + 4, 1, 128, FAKE, FAKE, None) == sh.SHERRY_E_ALIGN
    assert L.sherry_quantize_act(FAKE, 1, 126, FAKE, FAKE, None) == sh.SHERRY_E_SHAPE
    assert L.sherry_quantize_act(None, 1, 128, FAKE, FAKE, None) == sh.SHERRY_E_INVALID
    assert L.sherry_gemv2(FAKE, FAKE, FAKE, 1.0, FAKE, None, 64, 126, None) == sh.SHERRY_E_SHAPE
    assert L.sherry_gemv3(FAKE, FAKE, FAKE, 1.0, FAKE, None, 64, 126, None) == sh.SHERRY_E_SHAPE
    assert L.sherry_gemv3(FAKE_MIS, FAKE, FAKE, 1.0, FAKE, None, 64, 128, None) == \
        sh.SHERRY_E_ALIGN
    assert L.sherry_gemv3(None, FAKE, FAKE, 1.0, FAKE, None, 64, 128, None) == sh.SHERRY_E_INVALID
    assert L.sherry_stream_read(FAKE, 100, FAKE, None) == sh.SHERRY_E_SHAPE
    assert L.sherry_stream_read(FAKE + 8, 128, FAKE, None) == sh.SHERRY_E_ALIGN


def test_kernel_choice_by_m():
    for m in (1, 2, 3, 4):
        assert sh.sherry_gemm_kernel_for(m, 2048, 2048) == sh.SHERRY_KERNEL_GEMV
    for m in (5, 16, 32, 64, 65, 512):
        assert sh.sherry_gemm_kernel_for(m, 2048, 2048) == sh.SHERRY_KERNEL_SKINNY
    # up to 8192 tokens every product is register-decoded
    for m in (513, 2048, 8192):
        for n, k in ((2048, 2048), (8192, 2048), (2048, 8192), (3072, 3072), (14336, 4096)):
            assert sh.sherry_gemm_kernel_for(m, n, k) == sh.SHERRY_KERNEL_SKINNY
    # longer products: the LDS-tiled kernel for k <= 2048 and k <= n
    for m in (8193, 16384):
        assert sh.sherry_gemm_kernel_for(m, 2048, 2048) == sh.SHERRY_KERNEL_MFMA
        assert sh.sherry_gemm_kernel_for(m, 8192, 2048) == sh.SHERRY_KERNEL_MFMA
        assert sh.sherry_gemm_kernel_for(m, 2048, 8192) == sh.SHERRY_KERNEL_SKINNY
        assert sh.sherry_gemm_kernel_for(m, 3072, 3072) == sh.SHERRY_KERNEL_SKINNY
    assert sh.sherry_gemm_kernel_for(0, 2048, 2048) == -sh.SHERRY_E_SHAPE


def test_batched_prepare():
    shapes = [(2048, 2048), (512, 2048), (8192, 2048), (2048, 8192), (70, 132)]
    descs = (sh.sherry_gemv_desc * len(shapes))()
    for i, (n, k) in enumerate(shapes):
        descs[i].w = FAKE
        descs[i].x = FAKE
        descs[i].x_scale = FAKE
        descs[i].y = FAKE
        descs[i].acc = None
        descs[i].n = n
        descs[i].k = k
        descs[i].w_scale = 0.02
    total = sh.sherry_gemv_batched_prepare(descs)
    begins = [d.block_begin for d in descs]
    # 8-wave workgroups; a 64-row tile with C containers is split over the
    # smallest power of two S <= 8 with C/S <= 16 waves, 8/S tiles per block:
    # (32 tiles, S=1) 4, (8, S=1) 1, (128, S=1) 16, (32, S=4) 16, (2, S=1) 1
    assert begins == [0, 4, 5, 21, 37]
    assert total == 38
    assert ctypes.sizeof(sh.sherry_gemv_desc) == 72
    descs[3].k = 6
    with pytest.raises(sh.SherryError):
        sh.sherry_gemv_batched_prepare(descs)
    descs[3].k = 8192
    descs[1].w = FAKE + 8
    with pytest.raises(sh.SherryError):
        sh.sherry_gemv_batched_prepare(descs)
    assert L.sherry_gemv_batched(None, 1, 1, None) == sh.SHERRY_E_INVALID
    assert L.sherry_gemv_batched(FAKE + 4, 1, 1, None) == sh.SHERRY_E_ALIGN


def test_gemm_batched_prepare_picks_the_token_gemv():
    def prep(cases, group=False):
        descs = (sh.sherry_gemm_desc * len(cases))()
        for i, (m, n, k) in enumerate(cases):
            d = descs[i]
            d.w, d.x, d.x_scale, d.y = FAKE, FAKE, FAKE, FAKE
            d.n, d.k, d.m, d.w_scale = n, k, m, 0.02
            if group and i == 0:
                d.w_group_scales = FAKE
        total, max_m = sh.sherry_gemm_batched_prepare(descs)
        return [d.block_begin for d in descs], total, max_m
    # up to 4 tokens, activations fit 32 KB of LDS: the matrix-core GEMV
    # (the int8 GEMV's work split, 8-wave blocks, at most 16 units per wave:
    # 48 tiles x S=2 / 8, 16 x 2 / 8, 48 x 4 / 8)
    # (blocks numbered longest rows first: the k = 8192 product's 24, then the
    # k = 3072 ones in array order)
    assert prep([(4, 3072, 3072), (2, 1024, 3072), (1, 3072, 8192)]) == ([24, 36, 0], 40, 4)
    assert prep([(1, 64, 128)]) == ([0], 1, 1)
    # too long for the staging, or 5-16 tokens: the 16-token window kernel
    # (launch value 5-16; four 64-row tiles per workgroup, whole K)
    assert prep([(4, 3072, 8320), (1, 64, 128)]) == ([0, 12], 13, 5)
    assert prep([(5, 64, 128)]) == ([0], 1, 5)
    assert prep([(16, 3072, 8192), (9, 1024, 3072)]) == ([0, 12], 16, 16)
    # per-group scales up to 4 tokens stay on the token GEMV; with more
    # tokens, or more than 16 tokens, the register-decoded kernel (launch
    # value at least 17)
    G = sh.SHERRY_LAUNCH_GROUPS  # set in the launch value with per-group scales
    assert prep([(2, 64, 128), (1, 64, 128)], group=True)[2] == 2 | G
    assert prep([(5, 64, 128), (1, 64, 128)], group=True)[2] == 17 | G
    assert prep([(4, 3072, 8320)], group=True)[2] == 17 | G
    # the window kernel takes per-group scales of whole 512-value chunks
    assert prep([(16, 3072, 8192), (9, 1024, 3072)], group=True) == ([0, 12], 16, 16 | G)
    assert prep([(5, 64, 512), (1, 64, 128)], group=True)[2] == 5 | G
    assert prep([(17, 64, 128)])[2] == 17


def test_comparison_batched_prepare():
    # (n, k) -> workgroups: units of 64 (2-bit) or 96 (1.67-bit) weights per
    # row, at most 20 / 16 units per wave, 8 waves per workgroup
    shapes = [(4096, 4096), (1024, 4096), (14336, 4096), (4096, 14336), (70, 100)]
    for prep, run, exp in (
            (sh.sherry_gemv2_batched_prepare, L.sherry_gemv2_batched,
             # C = 64, 64, 64, 224, 2 -> S = 4, 4, 4, 8, 1
             ([0, 32, 40, 152, 216], 217)),
            (sh.sherry_gemv3_batched_prepare, L.sherry_gemv3_batched,
             # C = 43, 43, 43, 150, 2 -> S = 4, 4, 4, 8, 1
             ([0, 32, 40, 152, 216], 217))):
        descs = (sh.sherry_gemv_desc * len(shapes))()
        for i, (n, k) in enumerate(shapes):
            descs[i].w, descs[i].x, descs[i].x_scale, descs[i].y = FAKE, FAKE, FAKE, FAKE
            descs[i].n, descs[i].k, descs[i].w_scale = n, k, 0.02
        total = prep(descs)
        assert [d.block_begin for d in descs] == exp[0] and total == exp[1]
        descs[2].w_scales = FAKE  # one scale per tensor only
        with pytest.raises(sh.SherryError):
            prep(descs)
        descs[2].w_scales = None
        descs[4].k = 102
        with pytest.raises(sh.SherryError):
            prep(descs)
        assert run(None, 1, 1, None) == sh.SHERRY_E_INVALID
        assert run(FAKE + 4, 1, 1, None) == sh.SHERRY_E_ALIGN


def test_fused_validation_without_launch():
    f = L.sherry_gemv_f32
    assert f(None, FAKE, FAKE, 1.0, FAKE, None, 64, 128, None) == sh.SHERRY_E_INVALID
    assert f(FAKE, None, FAKE, 1.0, FAKE, None, 64, 128, None) == sh.SHERRY_E_INVALID
    assert f(FAKE, FAKE, FAKE, 1.0, None, None, 64, 128, None) == sh.SHERRY_E_INVALID
    # k beyond the on-chip row, not a multiple of 4, zero n
    assert f(FAKE, FAKE, FAKE, 1.0, FAKE, None, 64, sh.SHERRY_FUSED_MAX_K + 4, None) == \
        sh.SHERRY_E_SHAPE
    assert f(FAKE, FAKE, FAKE, 1.0, FAKE, None, 64, 130, None) == sh.SHERRY_E_SHAPE
    assert f(FAKE, FAKE, FAKE, 1.0, FAKE, None, 0, 128, None) == sh.SHERRY_E_SHAPE
    # fp32 activations need 16-byte alignment; scale and acc 4
    assert f(FAKE, FAKE + 4, FAKE, 1.0, FAKE, None, 64, 128, None) == sh.SHERRY_E_ALIGN
    assert f(FAKE, FAKE, FAKE + 2, 1.0, FAKE, None, 64, 128, None) == sh.SHERRY_E_ALIGN
    assert f(FAKE, FAKE, FAKE, 1.0, FAKE, FAKE + 2, 64, 128, None) == sh.SHERRY_E_ALIGN
    shapes = [(2048, 2048), (8192, 2048), (2048, 8192), (3072, 3072)]
    descs = (sh.sherry_gemv_f32_desc * len(shapes))()
    for i, (n, k) in enumerate(shapes):
        descs[i].w, descs[i].x, descs[i].x_scale, descs[i].y = FAKE, FAKE, None, FAKE
        descs[i].n, descs[i].k, descs[i].w_scale = n, k, 0.02
    total = sh.sherry_gemv_f32_batched_prepare(descs)
    # fused workgroups are longer: C/S <= 16 containers per wave, and a row
    # of up to 32 containers is not split (k = 3072: 24 containers, S = 1)
    assert [d.block_begin for d in descs] == [0, 4, 20, 36] and total == 42
    assert ctypes.sizeof(sh.sherry_gemv_f32_desc) == 72
    descs[3].k = 40000
    with pytest.raises(sh.SherryError):
        sh.sherry_gemv_f32_batched_prepare(descs)
    assert L.sherry_gemv_f32_batched(None, 1, 1, None) == sh.SHERRY_E_INVALID
    assert L.sherry_gemv_f32_batched(FAKE + 4, 1, 1, None) == sh.SHERRY_E_ALIGN


def test_skinny_validation_without_launch():
    g = L.sherry_gemm_ex
    assert g(FAKE, FAKE, FAKE, 1.0, FAKE, None, 0, 64, 128, sh.SHERRY_KERNEL_SKINNY,
             None) == sh.SHERRY_E_SHAPE
    assert g(FAKE, FAKE + 4, FAKE, 1.0, FAKE, None, 16, 64, 128, sh.SHERRY_KERNEL_SKINNY,
             None) == sh.SHERRY_E_ALIGN
    cases = [(16, 2048, 2048), (64, 8192, 2048), (1, 70, 132)]
    descs = (sh.sherry_gemm_desc * len(cases))()
    for i, (m, n, k) in enumerate(cases):
        d = descs[i]
        d.w, d.x, d.x_scale, d.y, d.acc = FAKE, FAKE, FAKE, FAKE, None
        d.m, d.n, d.k, d.w_scale = m, n, k, 0.02
    total, max_m = sh.sherry_gemm_batched_prepare(descs)
    # one workgroup per 8 row tiles: 32 tiles -> 4, 128 -> 16, 2 -> 1
    assert [d.block_begin for d in descs] == [0, 4, 20] and total == 21 and max_m == 64
    assert ctypes.sizeof(sh.sherry_gemm_desc) == 80
    # longer products run in 64-token blocks: 65 tokens -> 2 blocks of 16
    descs[1].m = 65
    total, max_m = sh.sherry_gemm_batched_prepare(descs)
    assert [d.block_begin for d in descs] == [0, 4, 36] and total == 37 and max_m == 65
    # 2048 tokens -> 32 token blocks of each product's tile groups
    descs[0].m = 2048
    total, max_m = sh.sherry_gemm_batched_prepare(descs)
    assert [d.block_begin for d in descs] == [0, 128, 160] and total == 161
    # every m <= 32: 32-token blocks
    for d, m in zip(descs, (32, 20, 1)):
        d.m = m
    total, max_m = sh.sherry_gemm_batched_prepare(descs)
    assert [d.block_begin for d in descs] == [0, 4, 20] and total == 21 and max_m == 32
    descs[0].m = 33
    total, max_m = sh.sherry_gemm_batched_prepare(descs)
    assert total == 21 and max_m == 33
    descs[1].m = 64
    descs[2].x = FAKE + 4
    with pytest.raises(sh.SherryError):
        sh.sherry_gemm_batched_prepare(descs)
    assert L.sherry_gemm_batched(FAKE, 1, 1, sh.SHERRY_MAX_M + 1, None) == sh.SHERRY_E_SHAPE
    assert L.sherry_gemm_batched(FAKE, 1, 1, 0, None) == sh.SHERRY_E_SHAPE
    assert L.sherry_gemm_batched(FAKE + 4, 1, 1, 16, None) == sh.SHERRY_E_ALIGN
    assert L.sherry_gemm_batched(None, 1, 1, 16, None) == sh.SHERRY_E_INVALID
    # the value under the per-group flag is checked as without it
    G = sh.SHERRY_LAUNCH_GROUPS
    assert L.sherry_gemm_batched(FAKE, 1, 1, 0 | G, None) == sh.SHERRY_E_SHAPE
    assert L.sherry_gemm_batched(FAKE, 1, 1, (sh.SHERRY_MAX_M + 1) | G, None) == sh.SHERRY_E_SHAPE
    assert L.sherry_gemm_batched(FAKE + 4, 1, 1, 16 | G, None) == sh.SHERRY_E_ALIGN
    assert L.sherry_gemm_batched(FAKE + 4, 1, 1, 4 | G, None) == sh.SHERRY_E_ALIGN


def test_channel_and_ternarize_validation_without_launch():
    # per-channel products need a scale vector; ternarize-pack checks shape,
    # buffer size and alignment before anything is enqueued
    g = L.sherry_gemm_channel
    assert g(FAKE, FAKE, FAKE, None, FAKE, None, 16, 64, 128, sh.SHERRY_KERNEL_SKINNY,
             None) == sh.SHERRY_E_INVALID
    assert g(FAKE, FAKE, FAKE, FAKE + 2, FAKE, None, 16, 64, 128, sh.SHERRY_KERNEL_SKINNY,
             None) == sh.SHERRY_E_ALIGN
    assert g(FAKE, FAKE, FAKE, FAKE, FAKE, None, 5, 64, 128, sh.SHERRY_KERNEL_GEMV,
             None) == sh.SHERRY_E_SHAPE
    assert g(FAKE, FAKE, FAKE, FAKE, FAKE, None, 1, 64, 130, sh.SHERRY_KERNEL_AUTO,
             None) == sh.SHERRY_E_SHAPE
    f = L.sherry_gemv_f32_channel
    assert f(FAKE, FAKE, FAKE, None, FAKE, None, 64, 128, None) == sh.SHERRY_E_INVALID
    assert f(FAKE, FAKE, FAKE, FAKE + 1, FAKE, None, 64, 128, None) == sh.SHERRY_E_ALIGN
    t = L.sherry_ternarize_pack
    need = sh.sherry_packed_bytes(70, 132)
    assert t(None, 70, 132, FAKE, need, None, None) == sh.SHERRY_E_INVALID
    assert t(FAKE, 70, 130, FAKE, need, None, None) == sh.SHERRY_E_SHAPE
    assert t(FAKE, 70, 132, FAKE, need - 1, None, None) == sh.SHERRY_E_BUFSIZE
    assert t(FAKE + 4, 70, 132, FAKE, need, None, None) == sh.SHERRY_E_ALIGN
    assert t(FAKE, 70, 132, FAKE, need, FAKE + 2, None) == sh.SHERRY_E_ALIGN


def test_group_validation_without_launch():
    g = L.sherry_gemm_group
    assert g(FAKE, FAKE, FAKE, None, FAKE, None, 1, 64, 128, sh.SHERRY_KERNEL_AUTO,
             None) == sh.SHERRY_E_INVALID
    assert g(FAKE, FAKE, FAKE, FAKE + 2, FAKE, None, 1, 64, 128, sh.SHERRY_KERNEL_AUTO,
             None) == sh.SHERRY_E_ALIGN
    assert g(FAKE, FAKE + 4, FAKE, FAKE, FAKE, None, 16, 64, 128, sh.SHERRY_KERNEL_MFMA,
             None) == sh.SHERRY_E_ALIGN
    assert g(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE + 2, 16, 64, 128, sh.SHERRY_KERNEL_MFMA,
             None) == sh.SHERRY_E_ALIGN
    assert g(FAKE, FAKE, FAKE, FAKE, FAKE, None, 1, 64, 128, sh.SHERRY_KERNEL_ALUT,
             None) == sh.SHERRY_E_INVALID
    assert g(FAKE, FAKE, FAKE, FAKE, FAKE, None, 5, 64, 128, sh.SHERRY_KERNEL_GEMV,
             None) == sh.SHERRY_E_SHAPE
    f = L.sherry_gemv_f32_group
    assert f(FAKE, FAKE, FAKE, None, FAKE, None, 64, 128, None) == sh.SHERRY_E_INVALID
    assert f(FAKE, FAKE, FAKE, FAKE + 1, FAKE, None, 64, 128, None) == sh.SHERRY_E_ALIGN


def test_batched_scale_fields_validation():
    # a descriptor takes per-channel or per-group scales, not both
    for cls, prep in ((sh.sherry_gemv_desc, L.sherry_gemv_batched_prepare),
                      (sh.sherry_gemv_f32_desc, L.sherry_gemv_f32_batched_prepare)):
        descs = (cls * 1)()
        d = descs[0]
        d.w, d.x, d.x_scale, d.y = FAKE, FAKE, FAKE, FAKE
        d.n, d.k, d.w_scale = 64, 128, 1.0
        total = ctypes.c_int64(0)
        d.w_scales, d.w_group_scales = FAKE, FAKE
        assert prep(descs, 1, ctypes.byref(total)) == sh.SHERRY_E_INVALID
        d.w_scales, d.w_group_scales = None, FAKE + 2
        assert prep(descs, 1, ctypes.byref(total)) == sh.SHERRY_E_ALIGN
        d.w_group_scales = FAKE
        assert prep(descs, 1, ctypes.byref(total)) == sh.SHERRY_OK and total.value >= 1


def test_activation_table_kernel_validation_without_launch():
    g = L.sherry_gemm_ex
    K = sh.SHERRY_KERNEL_ALUT
    # one token only, k up to SHERRY_ALUT_MAX_K, never the automatic choice
    assert g(FAKE, FAKE, FAKE, 1.0, FAKE, None, 2, 64, 128, K, None) == sh.SHERRY_E_SHAPE
    assert g(FAKE, FAKE, FAKE, 1.0, FAKE, None, 1, 64, sh.SHERRY_ALUT_MAX_K + 4, K,
             None) == sh.SHERRY_E_SHAPE
    assert g(FAKE, FAKE + 2, FAKE, 1.0, FAKE, None, 1, 64, 128, K, None) == sh.SHERRY_E_ALIGN
    assert g(FAKE, FAKE, FAKE, 1.0, FAKE, FAKE + 2, 1, 64, 128, K, None) == sh.SHERRY_E_ALIGN
    assert g(FAKE, FAKE, FAKE, 1.0, FAKE, None, 1, 64, 128, 6, None) == sh.SHERRY_E_INVALID
    # the matrix-core GEMV stages at most 32 KB of activations, 4 tokens
    T = sh.SHERRY_KERNEL_GEMV_TOK
    for m, k in ((5, 128), (4, 8320), (3, 10996), (1, 32900)):
        assert g(FAKE, FAKE, FAKE, 1.0, FAKE, None, m, 64, k, T, None) == sh.SHERRY_E_SHAPE
    assert g(FAKE, FAKE + 2, FAKE, 1.0, FAKE, None, 1, 64, 128, T, None) == sh.SHERRY_E_ALIGN
    for m in (1, 4, 16, 2048):
        assert sh.sherry_gemm_kernel_for(m, 2048, 2048) != K
    # per-group scales have no activation-table variant
    assert L.sherry_gemm_group(FAKE, FAKE, FAKE, FAKE, FAKE, None, 1, 64, 128, K,
                               None) == sh.SHERRY_E_INVALID


def test_grouped_per_group_scales_validation():
    cases = [(16, 2048, 2048), (100, 8192, 2048), (1, 70, 132)]
    descs = (sh.sherry_gemm_desc * len(cases))()
    for i, (m, n, k) in enumerate(cases):
        d = descs[i]
        d.w, d.x, d.x_scale, d.y, d.acc = FAKE, FAKE, FAKE, FAKE, None
        d.m, d.n, d.k, d.w_scale = m, n, k, 0.02
    descs[1].w_group_scales = FAKE
    total, max_m = sh.sherry_gemm_batched_prepare(descs)
    # a descriptor with per-group scales makes the launch run 32-token blocks
    # and splits its tiles' K in two (4 tiles per workgroup):
    # 32 tiles -> 4 x 1 block; 128 tiles -> 32 x 4 token blocks; 2 tiles -> 1
    assert max_m == 32 | sh.SHERRY_LAUNCH_GROUPS
    assert [d.block_begin for d in descs] == [0, 4, 132] and total == 133
    descs[1].acc = FAKE  # no int32 totals with per-group scales
    with pytest.raises(sh.SherryError):
        sh.sherry_gemm_batched_prepare(descs)
    descs[1].acc = None
    descs[1].w_scales = FAKE  # per-channel and per-group exclude each other
    with pytest.raises(sh.SherryError):
        sh.sherry_gemm_batched_prepare(descs)
    descs[1].w_scales = None
    descs[1].w_group_scales = FAKE + 2
    with pytest.raises(sh.SherryError):
        sh.sherry_gemm_batched_prepare(descs)


def test_import_fails_loudly_without_the_library(tmp_path):
    # no CPU fallback: a copy of the package without libsherry.so refuses to
    # import
    import shutil
    import subprocess
    import sys
    pkg = os.path.dirname(sh.__file__)
    dst = tmp_path / "paper_2601_07892_amd"
    shutil.copytree(pkg, dst, ignore=shutil.ignore_patterns("*.so", "__pycache__", "csrc"))
    r = subprocess.run([sys.executable, "-c", "import paper_2601_07892_amd"], cwd=tmp_path,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "not built" in r.stderr
