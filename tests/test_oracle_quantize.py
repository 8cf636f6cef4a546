"""Pins for the oracle's quantiser and packer (Sec. 2, Eq. 3-5), all on the CPU.

Nothing here re-types the oracle's formulas: the discretisation is pinned by hand-worked
values and by the properties that single out Eq. (3) (monotone, sign-preserving, magnitude
2 exactly beyond |W| = 1); the scale by least squares (numpy's lstsq), by a numerical
minimiser of the directly evaluated error ||W - alpha W~||^2 (scipy), and by closed-form
special cases; the packer by a bf16 decoding rule that is applied to whole words.
"""
import numpy as np
import pytest
import scipy.optimize

import oracle
import synth

F32 = np.float32


def _codes(vals):
    return oracle.quantize(np.array([vals], dtype=F32)).codes[0]


# ---------------------------------------------------------------------------------------
# Eq. (3): hand-worked values, including every boundary the cases name
# ---------------------------------------------------------------------------------------
def test_discretise_worked_boundaries():
    tiny = np.nextafter(F32(0), F32(1))          # smallest positive denormal
    below_m1 = np.nextafter(F32(-1), F32(-2))     # just below -1
    above_p1 = np.nextafter(F32(1), F32(2))       # just above +1
    above_m1 = np.nextafter(F32(-1), F32(0))
    below_p1 = np.nextafter(F32(1), F32(0))
    fmax = np.finfo(F32).max
    vals = [-fmax, -2.0, below_m1, -1.0, above_m1, -0.5, -tiny, -0.0, 0.0, tiny, 0.5,
            below_p1, 1.0, above_p1, 2.0, fmax]
    # -2 if W < -1; -1 if -1 <= W <= 0; 1 if 0 < W <= 1; 2 if W > 1 (both zeros are "<= 0").
    expect = [-2, -2, -2, -1, -1, -1, -1, -1, -1, 1, 1, 1, 1, 2, 2, 2]
    assert _codes(vals).tolist() == expect


def test_worked_example_two_magnitudes():
    # W = [0.5, -0.5, 3, -3]: codes [1, -1, 2, -2]; B1 = {0.5, -0.5}, B2 = {3, -3};
    # sum_B1 |W| = 1, sum_B2 |W| = 6, alpha = (1 + 2*6) / (2 + 4*2) = 13/10.
    q = oracle.quantize(np.array([[0.5, -0.5, 3.0, -3.0]], F32))
    assert q.codes[0].tolist() == [1, -1, 2, -2]
    assert (q.b1_size[0], q.b2_size[0]) == (2, 2)
    assert q.b1_sum[0] == 1.0 and q.b2_sum[0] == 6.0
    assert q.alpha64[0] == pytest.approx(1.3, abs=1e-15)
    # J(alpha) = 2*(0.5-1.3)^2 + 2*(3-2.6)^2 = 1.28 + 0.32 = 1.6
    W = np.array([0.5, -0.5, 3.0, -3.0])
    assert np.sum((W - q.alpha64[0] * q.codes[0]) ** 2) == pytest.approx(1.6, abs=1e-12)


def test_worked_example_boundaries_in_sets():
    # W = [-1, 0, 1, 1.5, -2]: codes [-1, -1, 1, 2, -2]; B1 = {-1, 0, 1} (sum 2),
    # B2 = {1.5, -2} (sum 3.5); alpha = (2 + 7) / (3 + 8) = 9/11.
    q = oracle.quantize(np.array([[-1.0, 0.0, 1.0, 1.5, -2.0]], F32))
    assert q.codes[0].tolist() == [-1, -1, 1, 2, -2]
    assert (q.b1_size[0], q.b2_size[0]) == (3, 2)
    assert q.alpha64[0] == pytest.approx(9.0 / 11.0, abs=1e-15)


# ---------------------------------------------------------------------------------------
# Eq. (3): the properties that characterise the rule, over wide random inputs
# ---------------------------------------------------------------------------------------
def _wide_weights(n, seed_name):
    a = synth.normal(0, seed_name + "a", (n,), 1.5)
    b = synth.normal(0, seed_name + "b", (n,), 0.05)
    edge = np.array([-1, 0, 1], F32)[synth.rng(0, seed_name + "c").integers(0, 3, n)]
    nudge = synth.rng(0, seed_name + "d").integers(-2, 3, n)
    c = edge.copy()
    for i in range(n):  # walk a few ulps either side of -1, 0 and 1
        for _ in range(abs(int(nudge[i]))):
            c[i] = np.nextafter(c[i], F32(np.sign(nudge[i]) * 3))
    return np.concatenate([a, b, c]).astype(F32)


def test_discretise_characterisation():
    w = _wide_weights(4000, "char")
    codes = oracle.quantize(w[None, :]).codes[0].astype(np.int64)
    assert set(np.unique(codes)) <= {-2, -1, 1, 2}
    # positive exactly for W > 0; magnitude 2 exactly for |W| > 1
    assert np.array_equal(codes > 0, w > 0)
    assert np.array_equal(np.abs(codes) == 2, np.abs(w) > 1)
    # monotone non-decreasing in W
    order = np.argsort(w, kind="stable")
    assert np.all(np.diff(codes[order]) >= 0)


def test_nonfinite_rejected():
    for bad in (np.inf, -np.inf, np.nan):
        with pytest.raises(oracle.OracleError):
            oracle.quantize(np.array([[0.3, bad]], F32))


# ---------------------------------------------------------------------------------------
# Eq. (4)-(5): the scale
# ---------------------------------------------------------------------------------------
@pytest.mark.parametrize("std", [0.05, 0.7, 1.0, 3.0])
def test_alpha_is_least_squares_fit(std):
    K, n = 7, 301
    w = synth.normal(0, "lsq%g" % std, (K, n), std)
    q = oracle.quantize(w)
    for k in range(K):
        A = q.codes[k].astype(np.float64)[:, None]
        sol, *_ = np.linalg.lstsq(A, w[k].astype(np.float64), rcond=None)
        assert q.alpha64[k] == pytest.approx(sol[0], rel=1e-12)
        # a numerical minimiser of the error evaluated directly (not through Eq. 4)
        J = lambda a: float(np.sum((w[k].astype(np.float64) - a * q.codes[k]) ** 2))
        res = scipy.optimize.minimize_scalar(J, bracket=(0.0, 10.0 * std), tol=1e-12)
        assert q.alpha64[k] == pytest.approx(res.x, rel=1e-6)
        assert J(q.alpha64[k]) <= J(q.alpha64[k] * 1.001) and J(q.alpha64[k]) <= J(q.alpha64[k] * 0.999)


def test_alpha_special_cases():
    g = synth.rng(0, "special")
    small = g.uniform(-1, 1, size=(3, 97)).astype(F32)   # all |W| <= 1: alpha = mean |W|
    q = oracle.quantize(small)
    assert np.allclose(q.alpha64, np.abs(small.astype(np.float64)).mean(axis=1), rtol=1e-14)
    big = (np.sign(g.uniform(-1, 1, size=(3, 97))) * g.uniform(1.01, 5, size=(3, 97))).astype(F32)
    q = oracle.quantize(big)                              # all |W| > 1: alpha = mean |W| / 2
    assert np.allclose(q.alpha64, np.abs(big.astype(np.float64)).mean(axis=1) / 2, rtol=1e-14)
    const = np.full((1, 50), 0.375, F32)                  # W = c * 1, 0 < c <= 1: alpha = c
    assert oracle.quantize(const).alpha64[0] == 0.375
    zero = np.zeros((1, 10), F32)                         # all-zero filter: alpha = 0, codes -1
    qz = oracle.quantize(zero)
    assert qz.alpha64[0] == 0.0 and qz.codes[0].tolist() == [-1] * 10


def test_eq4_expansion_and_set_sizes():
    K, n = 5, 513
    w = synth.normal(0, "eq4", (K, n), 1.0)
    q = oracle.quantize(w)
    w64 = w.astype(np.float64)
    assert np.array_equal(q.b2_size, (np.abs(w) > 1).sum(axis=1))
    assert np.array_equal(q.b1_size + q.b2_size, np.full(K, n))
    for k in range(K):
        C = np.sum(w64[k] ** 2)
        for a in (0.1, q.alpha64[k], 2.5):
            direct = np.sum((w64[k] - a * q.codes[k]) ** 2)
            expanded = (q.b1_size[k] + 4 * q.b2_size[k]) * a * a \
                - 2 * (q.b1_sum[k] + 2 * q.b2_sum[k]) * a + C
            assert direct == pytest.approx(expanded, rel=1e-10, abs=1e-9)


def test_alpha_fp32_is_single_rounding():
    w = synth.normal(0, "a32", (64, 200), 0.8)
    q = oracle.quantize(w)
    assert np.array_equal(q.alpha, q.alpha64.astype(np.float32))


# ---------------------------------------------------------------------------------------
# Packed layout: round trip, and the word-level bf16 decoding rule the format is built for
# ---------------------------------------------------------------------------------------
BF16_OF_CODE = {1: 0x3F80, 2: 0x4000, -1: 0xBF80, -2: 0xC000}


@pytest.mark.parametrize("K,n", [(1, 1), (3, 25), (32, 25), (64, 64), (65, 129), (10, 512), (130, 800)])
def test_pack_roundtrip_and_bf16_rule(K, n):
    g = synth.rng(0, "pack%d_%d" % (K, n))
    codes = np.array([-2, -1, 1, 2], np.int8)[g.integers(0, 4, size=(K, n))]
    words = oracle.pack(codes)
    KB, NB = (K + 63) // 64, (n + 63) // 64
    assert words.size == KB * NB * 64 * 4
    assert np.array_equal(oracle.unpack(words, K, n), codes)
    # Decode whole words: pair j of a word is ((word >> j) & 0x01010101) << 7 plus
    # 0x3F803F80, whose low half is the bf16 of element 2j and high half of element 2j+1.
    blk = words.reshape(KB, NB, 64, 4)
    for j in range(8):
        t = ((blk >> np.uint32(j)) & np.uint32(0x01010101)) << np.uint32(7)
        pair = t + np.uint32(0x3F803F80)
        lo = (pair & np.uint32(0xFFFF)).astype(np.uint16)
        hi = (pair >> np.uint32(16)).astype(np.uint16)
        for kb in range(KB):
            for kk in range(64):
                k = kb * 64 + kk
                for nb in range(NB):
                    for wi in range(4):
                        for e, half in ((2 * j, lo), (2 * j + 1, hi)):
                            i = nb * 64 + wi * 16 + e
                            if k < K and i < n:
                                assert half[kb, nb, kk, wi] == BF16_OF_CODE[int(codes[k, i])]
                            else:  # padding decodes as +1 with all bits zero
                                assert half[kb, nb, kk, wi] == 0x3F80
    # padding words of padding filters are entirely zero
    for kb in range(KB):
        for kk in range(64):
            if kb * 64 + kk >= K:
                assert not blk[kb, :, kk, :].any()


def test_pack_rejects_bad_codes():
    with pytest.raises(oracle.OracleError):
        oracle.pack(np.array([[0, 1]], np.int8))


# ---------------------------------------------------------------------------------------
# Discretisation variants (Sec. 2 chooses the deterministic rule for simplicity)
# ---------------------------------------------------------------------------------------
def test_variant_threshold_one_is_eq3():
    w = synth.normal(0, "var_eq3", (40, 300), 1.0)
    a, b = oracle.quantize(w), oracle.quantize_variant(w, 1.0)
    assert np.array_equal(a.codes, b.codes)
    assert np.array_equal(a.b2_size, b.b2_size)
    assert np.max(np.abs(a.alpha64 - b.alpha64) / a.alpha64) < 1e-14


def test_variant_threshold_hand_values():
    # t = 0.5: -2 below -0.5, -1 on [-0.5, 0], 1 on (0, 0.5], 2 above 0.5
    w = np.array([[-0.75, -0.5, -0.25, 0.0, 0.25, 0.5, 0.75]], np.float32)
    q = oracle.quantize_variant(w, 0.5)
    assert q.codes[0].tolist() == [-2, -1, -1, -1, 1, 1, 2]
    # alpha = sum W c / sum c^2 = (1.5 + 0.5 + 0.25 + 0 + 0.25 + 0.5 + 1.5) / (4 + 1 + 1 + 1 + 1 + 1 + 4)
    assert q.alpha64[0] == pytest.approx(4.5 / 13, rel=1e-15)


def test_variant_alpha_is_the_least_squares_scale():
    # whatever the codes, alpha minimises ||W - alpha c||^2: the numpy least-squares fit
    w = synth.normal(0, "var_ls", (12, 257), 0.8)
    u = synth.uniform(0, "var_ls_u", (12, 257))
    for q in (oracle.quantize_variant(w, 0.3), oracle.quantize_variant(w, 1.0, u)):
        for k in range(12):
            c = q.codes[k].astype(np.float64)[:, None]
            fit = np.linalg.lstsq(c, w[k].astype(np.float64), rcond=None)[0][0]
            assert q.alpha64[k] == pytest.approx(fit, rel=1e-12)


def test_stochastic_hand_values():
    w = np.array([[1.5, 1.5, -1.25, -1.25, 0.0, 0.0, 0.5, 0.5, 3.0, -7.0]], np.float32)
    u = np.array([[0.49, 0.51, 0.24, 0.26, 0.49, 0.5, 0.74, 0.76, 0.999, 0.999]], np.float32)
    q = oracle.quantize_variant(w, 1.0, u)
    # 1.5 -> 2 with probability 0.5; -1.25 -> -2 with probability 0.25; 0 -> 1 with
    # probability 0.5; 0.5 -> 1 with probability 0.75; beyond +-2 always +-2
    assert q.codes[0].tolist() == [2, 1, -2, -1, 1, -1, 1, -1, 2, -2]


def test_stochastic_rounding_is_unbiased():
    # E[code] = clamp(W, -2, 2): averaged over 40000 draws per weight, within 5 standard errors
    vals = np.array([-2.5, -1.75, -1.0, -0.6, -0.0, 0.3, 0.99, 1.01, 1.5, 1.9, 2.0], np.float32)
    draws = 40000
    w = np.repeat(vals[None, :], draws, axis=0).T.copy()
    u = np.minimum(synth.uniform(0, "var_unbiased", w.shape), np.float32(1 - 2 ** -24))  # [0, 1)
    q = oracle.quantize_variant(w, 1.0, u)
    mean = q.codes.astype(np.float64).mean(axis=1)
    target = np.clip(vals.astype(np.float64), -2, 2)
    se = np.maximum(q.codes.astype(np.float64).std(axis=1), 1e-3) / np.sqrt(draws)
    assert np.all(np.abs(mean - target) <= 5 * se + 1e-12), (mean, target)
    # only the two levels around each weight ever occur
    for row, v in zip(q.codes, vals):
        lo, hi = {True: (-2, -1), False: (-1, 1)}[bool(v < -1)] if v <= 1 else (1, 2)
        assert set(np.unique(row)).issubset({lo, hi})


def test_codes_of_bits_follow_eq3():
    # the bit-pattern form used by the exhaustive GPU check: hand values at the boundaries
    # (just below / at / above +1 and -1, both zeros, denormals, infinities, NaN marker)
    pats = {0x3F7FFFFF: 1, 0x3F800000: 1, 0x3F800001: 2, 0xBF7FFFFF: -1, 0xBF800000: -1, 0xBF800001: -2,
            0x00000000: -1, 0x80000000: -1, 0x00000001: 1, 0x80000001: -1, 0x7F800000: 2, 0xFF800000: -2,
            0x7FC00000: 0, 0xFFC00001: 0, 0x7F7FFFFF: 2, 0xFF7FFFFF: -2}
    for b, want in pats.items():
        assert int(oracle.codes_of_bits(b, 1)[0]) == want, hex(b)
    # and it agrees with the quantiser's codes on every finite value of a strided sweep
    start, count = 0x3E000000, 1 << 20
    got = oracle.codes_of_bits(start, count)
    w = (np.arange(start, start + count, dtype=np.uint64).astype(np.uint32)).view(np.float32).reshape(256, -1)
    assert np.all(np.isfinite(w))
    assert np.array_equal(got.reshape(256, -1), oracle.quantize(w).codes)
