"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these re-types the oracle's own formula: each compares it with a
hand-derived fixture, a count or identity the paper states, a library routine
(numpy), or brute force on tiny inputs.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
SYM = {"+": 1, "-": -1, "0": 0}


def _golden_table():
    rows = {}
    with open(os.path.join(GOLDEN, "code_table.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            c, w = line.split()
            rows[int(c)] = [SYM[ch] for ch in w]
    return rows


# ---------------------------------------------------------------- code table

def test_code_table_matches_hand_derived_table():
    g = _golden_table()
    assert sorted(g) == list(range(32))
    t = oracle.code_table()
    for c in range(32):
        assert list(t[c]) == g[c], c


def test_exactly_32_of_81_ternary_tuples_are_codes():
    # Sec. 3.1 point 3: C(4,3) * 2^3 = 32 states saturate 5 bits
    accepted = 0
    codes = set()
    for w in itertools.product((-1, 0, 1), repeat=4):
        c = oracle.encode_block(w)
        if c >= 0:
            accepted += 1
            codes.add(c)
            assert list(oracle.decode_code(c)) == list(w)
            assert sum(1 for v in w if v == 0) == 1
        else:
            assert sum(1 for v in w if v == 0) != 1
    assert accepted == 32
    assert codes == set(range(32))


def test_mirror_pairs():
    # Appendix C: with one shared sign bit, 3:4 has 16 patterns -> code and
    # its mirror differ only in the sign bits and negate each other.
    pairs = set()
    for c in range(32):
        m = c ^ 0b11100
        assert list(oracle.decode_code(m)) == list(-oracle.decode_code(c))
        pairs.add(frozenset((c, m)))
    assert len(pairs) == 16


def test_sign_bit_and_four_index_bits():
    # Sec. 3.1 / Appendix A reading: one sign bit and a 4-bit index.  With the
    # third sign bit s2 as the sign, every code is +-(a code with s2 clear):
    # decode(c) = (-1)^s2 * decode((c & 15) ^ (12 if s2 else 0)), and the 16
    # codes with s2 clear are 16 distinct patterns (the activation-table
    # kernel's 16 entries per block of 4 activations).
    canon = {tuple(oracle.decode_code(i)) for i in range(16)}
    assert len(canon) == 16
    for c in range(32):
        s2 = c >> 4
        idx = (c & 15) ^ (12 if s2 else 0)
        assert idx < 16
        want = -oracle.decode_code(idx) if s2 else oracle.decode_code(idx)
        assert list(oracle.decode_code(c)) == list(want)


def test_low_two_bits_are_zero_position():
    for c in range(32):
        w = oracle.decode_code(c)
        assert w[c & 3] == 0


# ------------------------------------------------------------ packed layout

def _fixture_t(fx):
    n, k = fx["n"], fx["k"]
    t = np.tile(np.array([0, 1, 1, 1], np.int8), (n, k // 4))
    g = _golden_table()
    for row, blk, code in fx["blocks"]:
        t[row, 4 * blk:4 * blk + 4] = g[code]
    return t


@pytest.mark.parametrize("idx", [0, 1, 2])
def test_pack_hand_derived_bytes(idx):
    with open(os.path.join(GOLDEN, "packed_fixtures.json")) as f:
        fx = json.load(f)["five_bit"][idx]
    t = _fixture_t(fx)
    p = oracle.pack(t)
    assert p.size == fx["total_bytes"] == oracle.packed_bytes(fx["n"], fx["k"])
    nz = {int(i): int(p[i]) for i in np.nonzero(p)[0]}
    assert nz == {int(a): b for a, b in fx["nonzero"].items()}
    assert np.array_equal(oracle.unpack(p, fx["n"], fx["k"]), t)


@pytest.mark.parametrize("idx", [0, 1])
def test_pack_il_hand_derived_bytes(idx):
    with open(os.path.join(GOLDEN, "packed_fixtures.json")) as f:
        fx = json.load(f)["lane_interleaved"][idx]
    t = _fixture_t(fx)
    p = oracle.pack_il(t)
    assert p.size == fx["total_bytes"] == oracle.packed_bytes(fx["n"], fx["k"])
    nz = {int(i): int(p[i]) for i in np.nonzero(p)[0]}
    assert nz == {int(a): b for a, b in fx["nonzero"].items()}
    assert np.array_equal(oracle.unpack_il(p, fx["n"], fx["k"]), t)


@pytest.mark.parametrize("n,k", [(1, 4), (64, 128), (65, 132), (130, 1028), (200, 260)])
def test_pack_il_round_trip_and_same_codes(n, k):
    # the interleaved layout is a per-unit permutation of the tiled one: the
    # same bytes size, every unit holding the same multiset of 5-bit codes,
    # and the matrix read back exactly
    t = synth.ternary_34(n, k, 8, "il", n, k)
    a, b = oracle.pack(t), oracle.pack_il(t)
    assert a.size == b.size
    assert np.array_equal(oracle.unpack_il(b, n, k), t)

    def unit_codes(p):
        bits = np.unpackbits(p.reshape(-1, 1280), axis=1, bitorder="little")
        head = bits[:, :1024 * 8].reshape(-1, 64, 128)
        tail = bits[:, 1024 * 8:].reshape(-1, 64, 32)
        stream = np.concatenate([head, tail], axis=2).reshape(-1, 64, 32, 5)
        codes = (stream * (1 << np.arange(5))).sum(-1)
        return np.sort(codes.reshape(codes.shape[0], -1), axis=1)
    assert np.array_equal(unit_codes(a), unit_codes(b))
    if n > 1:
        assert not np.array_equal(a, b)


def test_pack_il_rejects_non_34():
    t = np.zeros((3, 8), np.int8)
    t.reshape(3, 2, 4)[:, :, 1:] = 1
    t[2, 4:8] = [1, 1, 1, 1]
    with pytest.raises(oracle.OracleError):
        oracle.pack_il(t)


@pytest.mark.parametrize("idx", [0, 1])
def test_pack2_hand_derived_bytes(idx):
    with open(os.path.join(GOLDEN, "packed_fixtures.json")) as f:
        fx = json.load(f)["two_bit"][idx]
    t = np.zeros((fx["n"], fx["k"]), np.int8)
    for row, kk, w in fx["weights"]:
        t[row, kk] = w
    p = oracle.pack2(t)
    assert p.size == fx["total_bytes"]
    exp = np.full(fx["total_bytes"], fx["fill"], np.uint8)
    for a, b in fx["bytes"].items():
        exp[int(a)] = b
    assert np.array_equal(p, exp)
    assert np.array_equal(oracle.unpack2(p, fx["n"], fx["k"]), t)


def test_packed_sizes_are_1p25_bits():
    # 5 bits per 4 weights (Sec. 3.1); exact for multiples of 64 x 512
    for n, k in [(2048, 2048), (512, 2048), (8192, 2048), (2048, 8192),
                 (3072, 3072), (1024, 3072), (14336, 4096)]:
        assert oracle.packed_bytes(n, k) * 32 == 5 * n * k
        assert oracle.packed2_bytes(n, k) * 4 == n * k
    assert oracle.packed_bytes(0, 4) == 0
    assert oracle.packed_bytes(4, 6) == 0


@pytest.mark.parametrize("k", [4, 8, 12, 124, 128, 132, 516, 2048])
@pytest.mark.parametrize("n", [1, 63, 65])
def test_pack_round_trip(n, k):
    t = synth.ternary_34(n, k, 1, "rt")
    p = oracle.pack(t)
    assert np.array_equal(oracle.unpack(p, n, k), t)
    # 3:4 invariant of Eq. 3: every row keeps exactly 3K/4 non-zeros
    assert np.all(np.abs(oracle.unpack(p, n, k)).sum(axis=1) == 3 * k // 4)
    t2 = synth.ternary_any(n, k, 1, "rt2")
    assert np.array_equal(oracle.unpack2(oracle.pack2(t2), n, k), t2)


@pytest.mark.parametrize("zeros", [0, 2, 3, 4])
def test_pack_rejects_non_34_blocks(zeros):
    t = synth.ternary_34(3, 64, 2, "bad")
    blk = np.array([0] * zeros + [1] * (4 - zeros), np.int8)
    t[2, 20:24] = blk
    assert oracle.pack_bad_block(t) == 2 * 16 + 5
    t[1, 4:8] = blk
    assert oracle.pack_bad_block(t) == 1 * 16 + 1


def test_pack_rejects_out_of_set_values():
    t = synth.ternary_34(1, 8, 3, "oos")
    t[0, 5] = 2 if t[0, 5] != 0 else t[0, 5]
    t[0, 4:8] = [0, 2, 1, 1]
    assert oracle.pack_bad_block(t) == 1


# ---------------------------------------------------------------- product

def _brute(x, t):
    m, k = x.shape
    n = t.shape[0]
    out = [[0] * n for _ in range(m)]
    for i in range(m):
        for j in range(n):
            s = 0
            for kk in range(k):
                s += int(x[i, kk]) * int(t[j, kk])
            out[i][j] = s
    return np.array(out, dtype=np.int64)


@pytest.mark.parametrize("m,n,k", [(1, 1, 4), (2, 3, 8), (3, 5, 12)])
def test_gemm_brute_force_tiny(m, n, k):
    x = synth.int8_any(m, k, 4, "bf")
    t = synth.ternary_34(n, k, 4, "bf")
    assert np.array_equal(oracle.gemm_i32(x, t).astype(np.int64), _brute(x, t))


def test_gemm_all_code_pairs():
    # K=8 and 1024 rows: every ordered pair of the 32 codes appears once
    g = oracle.code_table()
    t = np.concatenate([np.concatenate([g[a], g[b]])[None]
                        for a in range(32) for b in range(32)]).astype(np.int8)
    x = synth.int8_any(3, 8, 5, "pairs")
    assert np.array_equal(oracle.gemm_i32(x, t).astype(np.int64), _brute(x, t))


@pytest.mark.parametrize("m,n,k", [(1, 257, 2048), (7, 130, 516), (16, 64, 1028)])
def test_gemm_matches_numpy(m, n, k):
    x = synth.int8_any(m, k, 6, "np")
    t = synth.ternary_34(n, k, 6, "np")
    ref = x.astype(np.int64) @ t.astype(np.int64).T
    assert np.array_equal(oracle.gemm_i32(x, t), ref)
    assert np.array_equal(oracle.gemm_i32(x, t, threads=4), ref)
    for i, j in [(0, 0), (m - 1, n - 1), (m // 2, n // 3)]:
        assert oracle.dot_i32(x[i], t[j]) == ref[i, j]


def test_gemm_closed_forms():
    n, k = 40, 64
    t = synth.ternary_34(n, k, 7, "cf")
    # one-hot activation reads back one column of T
    for kk in (0, 13, 63):
        e = np.zeros((1, k), np.int8)
        e[0, kk] = 1
        assert np.array_equal(oracle.gemm_i32(e, t)[0], t[:, kk].astype(np.int32))
    # all-ones activation gives the row sums
    ones = np.ones((1, k), np.int8)
    assert np.array_equal(oracle.gemm_i32(ones, t)[0], t.astype(np.int32).sum(1))
    # extreme magnitudes: |acc| <= 128 * 3K/4
    xm = np.full((1, k), -128, np.int8)
    assert np.all(np.abs(oracle.gemm_i32(xm, t)) <= 128 * 3 * k // 4)


# ------------------------------------------------------ activation quant

def test_quantize_hand_derived():
    x = np.array([
        [127.0, -63.5, 0.5, 1.5, 2.5, -127.0, 0.0, 3.49],
        [254.0, 1.0, 3.0, -254.0, 5.0, -1.0, 0.0, 0.0],
        [0.0] * 8,
    ], np.float32)
    q, sx = oracle.quantize_act(x)
    # row 0: absmax 127 -> sx 1; ties go to even (-63.5 -> -64, 0.5 -> 0,
    # 1.5 -> 2, 2.5 -> 2)
    assert sx[0] == 1.0
    assert list(q[0]) == [127, -64, 0, 2, 2, -127, 0, 3]
    # row 1: absmax 254 -> sx 2; 1/2 -> 0, 3/2 -> 2, 5/2 -> 2, -1/2 -> -0
    assert sx[1] == 2.0
    assert list(q[1]) == [127, 0, 2, -127, 2, 0, 0, 0]
    # all-zero row: scale 0, codes 0
    assert sx[2] == 0.0 and not q[2].any()


def _rne_f32(fr):
    """The float32 nearest to the rational fr, ties to the even significand,
    found exactly by comparing the three float32 neighbours as fractions."""
    from fractions import Fraction
    f = np.float32(float(fr))
    best = None
    for c in (np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))):
        odd = int(np.float32(c).view(np.uint32)) & 1
        key = (abs(Fraction(float(c)) - fr), odd)
        if best is None or key < best[0]:
            best = (key, np.float32(c))
    return best[1]


def _rne_int(fr):
    """Round a rational to the nearest integer, ties to even (exact)."""
    from fractions import Fraction
    fl = fr.numerator // fr.denominator
    rest = fr - fl
    return fl + 1 if rest > Fraction(1, 2) or (rest == Fraction(1, 2) and fl % 2) else fl


def _q_division(x, s):
    # the reading: the IEEE fp32 quotient x / s, then to the nearest integer
    from fractions import Fraction
    return _rne_int(Fraction(float(_rne_f32(Fraction(float(x)) / Fraction(float(s))))))


def _q_reciprocal(x, s):
    # a plausible wrong oracle: fp32 reciprocal of s, then an fp32 product
    from fractions import Fraction
    r = _rne_f32(1 / Fraction(float(s)))
    return _rne_int(Fraction(float(_rne_f32(Fraction(float(x)) * Fraction(float(r))))))


def test_quantize_ieee_division_at_inexact_scales():
    # The reading of the quantizer takes the IEEE fp32 quotient x / s.  At a
    # scale that is not a power of two, x * (1/s) rounds differently for some
    # x; every expected code here is derived with exact rational arithmetic
    # (the fp32 scale absmax/127 and the fp32 quotient both rounded exactly),
    # independently of the oracle.  absmax 3, x = -2.7992127: s = 3/127
    # rounded, x/s rounds to -118.5000... -> -119, x*(1/s) to -118.
    from fractions import Fraction
    x = np.array([[3.0, -2.7992127]], np.float32)
    q, sx = oracle.quantize_act(x)
    assert sx[0] == _rne_f32(Fraction(3) / 127)
    assert list(q[0]) == [127, -119]
    assert _q_reciprocal(np.float32(-2.7992127), sx[0]) == -118  # the pin discriminates
    # rows at four inexact scales: absmax first, then values one or two ulps
    # around half-integer multiples of the scale, where the two readings split
    rng = np.random.default_rng(20260107)
    found = 0
    for amax in (3.0, 0.7, 11.3, 1e-3):
        s = _rne_f32(Fraction(float(np.float32(amax))) / 127)
        cands = []
        for _ in range(400):
            h = int(rng.integers(-126, 126)) + 0.5
            v = np.float32(float(s) * h)
            for _ in range(int(rng.integers(0, 3))):
                v = np.nextafter(v, np.float32(np.inf) if rng.random() < 0.5 else np.float32(-np.inf))
            cands.append(v)
        row = np.array([np.float32(amax)] + cands, np.float32)[None, :]
        q, sx = oracle.quantize_act(row)
        assert sx[0] == s
        want = [127] + [max(-127, min(127, _q_division(v, s))) for v in cands]
        assert list(q[0].astype(int)) == want
        found += sum(_q_division(v, s) != _q_reciprocal(v, s) for v in cands)
    assert found >= 10  # the rows do separate the division from the reciprocal


def test_quantize_properties():
    x = synth.activations(9, 1000, 8, "qp", outlier_frac=0.01)
    q, sx = oracle.quantize_act(x)
    assert q.dtype == np.int8 and np.all(np.abs(q.astype(int)) <= 127)
    for r in range(9):
        amax = np.max(np.abs(x[r]))
        assert sx[r] == np.float32(amax) / np.float32(127.0)
        i = int(np.argmax(np.abs(x[r])))
        assert abs(int(q[r, i])) == 127
        # dequantization error is at most half a step (plus fp32 slack)
        err = np.abs(q[r].astype(np.float64) * sx[r] - x[r])
        assert np.all(err <= 0.5 * sx[r] * (1 + 1e-6))
    # exact multiples j * sx map back to j
    s = np.float32(0.25)
    j = np.arange(-127, 128, dtype=np.float32)
    q2, sx2 = oracle.quantize_act((j * s)[None, :])
    assert sx2[0] == s and np.array_equal(q2[0].astype(np.float32), j)


# ---------------------------------------------------------------- epilogue

def test_epilogue_exact_products():
    acc = np.array([[0, 1, -3, 1 << 20], [7, -7, 5, -(1 << 22)]], np.int32)
    sx = np.array([0.5, 0.125], np.float32)
    y = oracle.epilogue(acc, sx, 0.25)
    assert np.array_equal(y, acc * np.array([[0.125], [0.03125]]))


def test_linear_path_matches_float_reference():
    x = synth.activations(3, 256, 9, "lin")
    t = synth.ternary_34(50, 256, 9, "lin")
    sw = synth.weight_scale(9, "lin")
    q, sx, acc, y = oracle.linear(x, t, sw)
    ref = (q.astype(np.float64) @ t.astype(np.float64).T) * sx[:, None].astype(np.float64) * sw
    assert np.allclose(y, ref, rtol=1e-12, atol=0)
    # and the quantized product approximates the fp32 product X T^T sw
    full = x.astype(np.float64) @ t.astype(np.float64).T * sw
    assert np.max(np.abs(y - full)) < 0.05 * np.max(np.abs(full))


# --------------------------------------------------------------- ternarizer

def test_ternarizer_is_optimal_per_block():
    # Appendix D: for any alpha > 0 the best 3:4 block maximises sum W*T,
    # i.e. drop the smallest |W| and keep signs.  Check by brute force over
    # all 32 patterns.
    w = synth.dense_weights(6, 64, 10, "tern")
    t, alpha = oracle.ternarize(w)
    g = oracle.code_table().astype(np.float64)
    for row in range(6):
        for b in range(16):
            wb = w[row, 4 * b:4 * b + 4].astype(np.float64)
            best = np.max(g @ wb)
            assert np.isclose(float(t[row, 4 * b:4 * b + 4].astype(np.float64) @ wb), best)
            for a in (alpha, 0.3, 2.0):
                errs = ((wb[None, :] - a * g) ** 2).sum(1)
                tb = t[row, 4 * b:4 * b + 4].astype(np.float64)
                assert ((wb - a * tb) ** 2).sum() <= errs.min() + 1e-12
    # every block keeps exactly one zero
    assert np.all((t.reshape(6, 16, 4) == 0).sum(-1) == 1)


def test_ternarizer_alpha_is_least_squares():
    # Eq. 5: alpha* = mean |W| over kept weights = <W,T>/<T,T>
    w = synth.dense_weights(8, 128, 11, "alpha")
    t, alpha = oracle.ternarize(w)
    tt = t.astype(np.float64).ravel()
    sol = np.linalg.lstsq(tt[:, None], w.astype(np.float64).ravel(), rcond=None)[0][0]
    assert np.isclose(alpha, sol, rtol=1e-12)


def test_ternarizer_rows_alpha_is_per_channel_least_squares():
    # Eq. 5 per output channel: alpha_j = <W_j, T_j> / <T_j, T_j>, i.e. the
    # least-squares scale of row j given its 3:4 pattern; the pattern is the
    # per-tensor ternarizer's, and with equal kept counts per row the
    # per-tensor alpha is the mean of the per-row ones.
    w = synth.dense_weights(7, 96, 12, "alpha_rows")
    w[3] *= 25.0  # rows of very different magnitude
    t, alpha = oracle.ternarize_rows(w)
    t0, alpha0 = oracle.ternarize(w)
    assert np.array_equal(t, t0)
    for j in range(7):
        tj = t[j].astype(np.float64)
        sol = np.linalg.lstsq(tj[:, None], w[j].astype(np.float64), rcond=None)[0][0]
        assert np.isclose(alpha[j], sol, rtol=1e-12)
    assert np.isclose(alpha.mean(), alpha0, rtol=1e-12)
    assert alpha[3] > 10 * np.delete(alpha, 3).max()


def test_epilogue_rows_is_dequantized_product():
    # [T alpha]_ij = T_ij alpha_j (footnote to Eq. 2): the per-channel result
    # equals the product of the dequantized operands, (q * sx) @ (T * sw)^T,
    # computed in the other order; with one sw for every channel it is the
    # per-tensor epilogue.
    rng = np.random.default_rng(13)
    q = rng.integers(-127, 128, (5, 64)).astype(np.int8)
    t = synth.ternary_34(9, 64, 13, "epr")
    sx = (rng.random(5) + 0.01).astype(np.float32)
    sw = (rng.random(9) * 0.05 + 0.001).astype(np.float32)
    acc = oracle.gemm_i32(q, t)
    y = oracle.epilogue_rows(acc, sx, sw)
    ref = (q.astype(np.float64) * sx.astype(np.float64)[:, None]) @ \
        (t.astype(np.float64) * sw.astype(np.float64)[:, None]).T
    assert np.allclose(y, ref, rtol=1e-12, atol=0)
    y1 = oracle.epilogue_rows(acc, sx, np.full(9, sw[0], np.float32))
    assert np.array_equal(y1, oracle.epilogue(acc, sx, float(sw[0])))


def test_product_groups_pins():
    # per-group scales (group 128 along K): (1) equal scales across a row's
    # groups give the per-channel product; (2) the dequantized operands
    # multiplied in the other order give the same y; (3) a scale in one group
    # only isolates that K slice (catches an off-by-one in the grouping)
    rng = np.random.default_rng(21)
    m, n, k = 3, 7, 300  # three groups, the last one partial (44 values)
    q = rng.integers(-127, 128, (m, k)).astype(np.int8)
    t = synth.ternary_34(n, k, 21, "grp")
    sx = (rng.random(m) + 0.01).astype(np.float32)
    s = (rng.random((n, 3)) * 0.05 + 0.001).astype(np.float32)
    y, mag, acc = oracle.product_groups(q, t, sx, s)
    assert np.array_equal(acc, oracle.gemm_i32(q, t))
    ch = np.repeat(s[:, :1], 3, axis=1)
    y1, _, _ = oracle.product_groups(q, t, sx, ch)
    assert np.allclose(y1, oracle.epilogue_rows(oracle.gemm_i32(q, t), sx, s[:, 0]),
                       rtol=1e-12, atol=0)
    s_exp = np.repeat(s.astype(np.float64), 128, axis=1)[:, :k]
    ref = (q.astype(np.float64) * sx.astype(np.float64)[:, None]) @ \
        (t.astype(np.float64) * s_exp).T
    assert np.allclose(y, ref, rtol=1e-12, atol=0)
    assert np.all(mag >= np.abs(y) * (1 - 1e-12))
    one = np.zeros_like(s)
    one[:, 2] = 1.0
    y2, _, _ = oracle.product_groups(q, t, np.ones(m, np.float32), one)
    assert np.array_equal(y2, oracle.gemm_i32(q[:, 256:], t[:, 256:]).astype(np.float64))


def test_ternarizer_ties_and_zeros():
    w = np.array([[0.5, -0.5, 0.5, -0.5, 0.0, 0.0, 1.0, -2.0]], np.float32)
    t, _ = oracle.ternarize(w)
    # ties for the smallest |W| go to the lowest position; a kept zero is +1
    assert list(t[0]) == [0, -1, 1, -1, 0, 1, 1, -1]


# ------------------------------------------------ 1.67-bit comparison layout

def _golden_table3():
    rows = {}
    with open(os.path.join(GOLDEN, "code3_table.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            c, w = line.split()
            rows[int(c)] = [SYM[ch] for ch in w]
    return rows


def test_code3_table_matches_hand_written_table():
    g = _golden_table3()
    assert sorted(g) == list(range(27))
    t, used = oracle.code3_table()
    # three weights in five bits: 3^3 = 27 of the 32 codes (Sec. 2.3)
    assert used == 27 == 3 ** 3 and 2 ** 5 - used == 5
    for c in range(27):
        assert list(t[c]) == g[c], c
    # every ternary triple has exactly one code, and it decodes back
    seen = set()
    for w in itertools.product((-1, 0, 1), repeat=3):
        c = oracle.encode3(w)
        assert 0 <= c < 27 and c not in seen
        seen.add(c)
        assert tuple(int(v) for v in t[c]) == w
    assert oracle.encode3((2, 0, 0)) == -1 and oracle.encode3((0, 0, -2)) == -1


def test_code3_mirror():
    # negating a block maps code c to 26 - c (the digits t+1 become 2 - (t+1))
    t, _ = oracle.code3_table()
    for c in range(27):
        assert np.array_equal(t[26 - c], -t[c])


def _zero_row3():
    fx = json.load(open(os.path.join(GOLDEN, "packed_fixtures.json")))["about_code3"]
    head = bytes.fromhex(fx.split("head ")[1].split(",")[0].replace(" ", ""))
    tail = bytes.fromhex(fx.split("tail ")[1].split(" (")[0].replace(" ", ""))
    assert len(head) == 16 and len(tail) == 4
    return head, tail


@pytest.mark.parametrize("idx", [0, 1, 2, 3])
def test_pack3_hand_derived_bytes(idx):
    with open(os.path.join(GOLDEN, "packed_fixtures.json")) as f:
        fx = json.load(f)["code3"][idx]
    t = np.zeros((fx["n"], fx["k"]), np.int8)
    for row, kk, w in fx["weights"]:
        t[row, kk] = w
    p = oracle.pack3(t)
    assert p.size == fx["total_bytes"] == oracle.packed3_bytes(fx["n"], fx["k"])
    head, tail = _zero_row3()
    exp = np.zeros(fx["total_bytes"], np.uint8)
    for unit in range(0, fx["total_bytes"], 1280):
        for i in range(64):
            exp[unit + 16 * i:unit + 16 * i + 16] = np.frombuffer(head, np.uint8)
            exp[unit + 1024 + 4 * i:unit + 1024 + 4 * i + 4] = np.frombuffer(tail, np.uint8)
    for a, b in fx["bytes"].items():
        exp[int(a)] = b
    assert np.array_equal(p, exp)
    assert np.array_equal(oracle.unpack3(p, fx["n"], fx["k"]), t)


def test_packed3_sizes_are_5_bits_per_3_weights():
    # 5/3 bits per weight once rows and K fill whole units (64 x 96)
    for n, k in [(64, 96), (3072, 3072), (1024, 3072), (4096, 14400), (128, 192)]:
        assert oracle.packed3_bytes(n, k) * 24 == 5 * n * k
    # padding: K = 2048 rounds up to 2112 (22 units of 96)
    assert oracle.packed3_bytes(2048, 2048) == 2048 * 22 * 20
    assert oracle.packed3_bytes(0, 3) == 0 and oracle.packed3_bytes(3, 0) == 0


@pytest.mark.parametrize("k", [1, 2, 3, 4, 95, 96, 97, 100, 191, 2048])
@pytest.mark.parametrize("n", [1, 63, 65])
def test_pack3_round_trip(n, k):
    t = synth.ternary_any(n, k, 3, "rt3")
    assert np.array_equal(oracle.unpack3(oracle.pack3(t), n, k), t)


def test_pack3_rejects_values_and_unpack3_rejects_unused_codes():
    t = synth.ternary_any(2, 10, 4, "bad3")
    t[1, 7] = 2
    with pytest.raises(oracle.OracleError, match="at 17"):
        oracle.pack3(t)
    t[1, 7] = 0
    p = oracle.pack3(t)
    # code 0 of row 1 sits in stream bits 0..4 of bytes 16..; write each
    # unused code (27..31) there
    for bad in range(27, 32):
        q = p.copy()
        q[16] = (q[16] & 0xE0) | bad
        with pytest.raises(oracle.OracleError):
            oracle.unpack3(q, 2, 10)
    # a valid code in the same place decodes
    q = p.copy()
    q[16] = (q[16] & 0xE0) | 26
    assert list(oracle.unpack3(q, 2, 10)[1, :3]) == [1, 1, 1]
