"""Pins of the fp64 oracle against facts that do not come from the oracle.

Each pin targets a plausible mistake: wrong bit order or packing axis (numpy's
packbits, worked words), wrong sign decode (round trips, closed forms), a
dropped or mis-scaled delta term or a transposed operand (exact brute force,
one-hot rows, distributivity), wrong tenant routing (tenant invariants).
"""
import os

import numpy as np
import pytest

import oracle
from oracle import brute
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "pack_words.txt")


def numpy_pack(plus: np.ndarray) -> np.ndarray:
    """Library packer: numpy.packbits little-endian bit order, bytes -> '<u4'."""
    rows, K = plus.shape
    return np.packbits(plus.astype(np.uint8), axis=-1, bitorder="little").view("<u4").reshape(rows, K // 32)


def numpy_signs(packed: np.ndarray, K: int) -> np.ndarray:
    """Library decode: numpy.unpackbits little-endian -> +1/-1."""
    bits = np.unpackbits(np.ascontiguousarray(packed).view(np.uint8), axis=-1,
                         bitorder="little")[..., :K]
    return bits.astype(np.float64) * 2.0 - 1.0


def bf16(bits):
    return wl.bf16_bits_to_f32(bits).astype(np.float64)


# ---------------------------------------------------------------- pack / unpack

def _parse_positions(spec, K):
    if spec == "all":
        return list(range(K))
    if spec == "none":
        return []
    if spec == "even":
        return list(range(0, K, 2))
    if spec == "odd":
        return list(range(1, K, 2))
    out = []
    for part in spec.split(","):
        if "-" in part:
            a, b = part.split("-")
            out.extend(range(int(a), int(b) + 1))
        else:
            out.append(int(part))
    return out


def _golden_cases():
    cases = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, K, pos, words = [c.strip() for c in line.split("|")]
            cases.append((name, int(K), pos, [int(w, 16) for w in words.split()]))
    return cases


@pytest.mark.parametrize("case", _golden_cases(), ids=lambda c: c[0])
@pytest.mark.parametrize("dtype", ["f32", "i8", "bf16"])
def test_pack_worked_words(case, dtype):
    name, K, spec, words = case
    plus = np.zeros(K, dtype=bool)
    plus[_parse_positions(spec, K)] = True
    s = np.where(plus, 1.0, -1.0).astype(np.float32)[None]
    if dtype == "i8":
        s = s.astype(np.int8)
    elif dtype == "bf16":
        s = wl.f32_to_bf16_bits(s)
    got = oracle.pack(s)
    assert [int(w) for w in got[0]] == words


@pytest.mark.parametrize("rows,K", [(1, 32), (7, 96), (33, 256), (64, 4096)])
def test_pack_equals_numpy_packbits(rows, K):
    rng = np.random.default_rng(rows * 1000 + K)
    plus = rng.random((rows, K)) < 0.5
    ref = numpy_pack(plus)
    f = np.where(plus, 1.0, -1.0).astype(np.float32)
    np.testing.assert_array_equal(oracle.pack(f), ref)
    np.testing.assert_array_equal(oracle.pack(f.astype(np.int8)), ref)
    np.testing.assert_array_equal(oracle.pack(wl.f32_to_bf16_bits(f)), ref)


def test_pack_special_values():
    # bit = complement of the sign bit, whatever the magnitude
    f = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, -np.nan, 1e-45, -1e-45,
                  3.5, -3.5, 1e38, -1e38] + [1.0] * 20, dtype=np.float32)
    signbit = np.signbit(f)
    ref = numpy_pack(~signbit[None])
    np.testing.assert_array_equal(oracle.pack(f[None]), ref)
    i8 = np.arange(-128, 128, dtype=np.int16).astype(np.int8).reshape(8, 32)
    np.testing.assert_array_equal(oracle.pack(i8), numpy_pack(i8 >= 0))
    bits = np.arange(0, 65536, 2048, dtype=np.uint16)[None]  # 32 patterns
    np.testing.assert_array_equal(oracle.pack(bits), numpy_pack((bits >> 15) == 0))


def test_roundtrips():
    rng = np.random.default_rng(5)
    words = wl.uniform_words(rng, (17, 8))
    signs = oracle.unpack(words, 256)
    np.testing.assert_array_equal(signs, numpy_signs(words, 256))
    np.testing.assert_array_equal(oracle.pack(signs.astype(np.float32)), words)
    s = wl.random_signs_i8(rng, (9, 64))
    np.testing.assert_array_equal(oracle.unpack(oracle.pack(s), 64), s.astype(np.float64))


def test_pack_rejects_ragged_k():
    with pytest.raises(ValueError):
        oracle.pack(np.ones((2, 48), dtype=np.float32))


# --------------------------------------------------------------------- matmul

def _exact_vs_oracle(p: wl.Problem, rel=1e-15):
    packed = p.packed if p.packed is not None else np.stack([oracle.pack(s) for s in p.signs])
    exact = brute.matmul_exact(p.x.tolist(), p.w.tolist(), packed.tolist(), p.alpha.tolist(),
                               None if p.tenant_ids is None else p.tenant_ids.tolist())
    got = oracle.matmul(p.x, p.w, packed, p.alpha, p.tenant_ids)
    for m in range(p.M):
        for n in range(p.N):
            e = exact[m][n]
            if e is None:
                assert np.isnan(got[m, n])
                continue
            err = abs(float(e - type(e)(got[m, n])))
            scale = max(abs(float(e)), 1e-300)
            # the fp64 sum of K products has error <= ~K*eps*sum|terms|; bound it by
            # the row's absolute sum to stay meaningful under cancellation
            absum = sum(abs(bf16(p.x[m, k])) * (abs(bf16(p.w[n, k])) + abs(float(p.alpha[0 if p.tenant_ids is None else p.tenant_ids[m]])))
                        for k in range(p.K))
            assert err <= rel * scale + 4 * p.K * 2.0 ** -53 * absum, (m, n, err, float(e))


def test_brute_force_2x32x4():
    p = wl.make_problem(2, 4, 32, 1, seed=11, y_dtype="f32")
    _exact_vs_oracle(p)


@pytest.mark.parametrize("M,N,K,T", [(1, 1, 32, 1), (3, 5, 64, 2), (4, 3, 96, 3)])
def test_brute_force_random_tiny(M, N, K, T):
    p = wl.make_problem(M, N, K, T, seed=M * 100 + N * 10 + K, multi_tenant=T > 1)
    _exact_vs_oracle(p)


def test_brute_force_tiny_int8_signs():
    p = wl.make_problem(2, 6, 64, 1, seed=3, signs_as_int8=True)
    _exact_vs_oracle(p)


def test_brute_force_self_pins():
    # the brute force's own bf16 decode and sign extraction against numpy
    rng = np.random.default_rng(1)
    bits = wl.normal_bf16(rng, (64,), 3.0)
    for b in bits:
        assert float(brute.bf16_bits_to_fraction(int(b))) == float(wl.bf16_bits_to_f32(np.array([b]))[0])
    words = wl.uniform_words(rng, (2,))
    ref = numpy_signs(words[None], 64)[0]
    assert [brute.sign_from_words(words, k) for k in range(64)] == ref.tolist()


def test_distributivity():
    # x (W + a S)^T computed by numpy in fp64 with numpy's own sign decode
    p = wl.make_problem(5, 37, 128, 1, seed=7)
    S = numpy_signs(p.packed[0], p.K)
    fused = bf16(p.x) @ (bf16(p.w) + np.float64(p.alpha[0]) * S).T
    got = oracle.matmul(p.x, p.w, p.packed, p.alpha)
    np.testing.assert_allclose(got, fused, rtol=1e-12, atol=1e-12 * np.abs(fused).max())


def test_alpha_zero_is_plain_gemm():
    p = wl.make_problem(6, 33, 256, 1, seed=8)
    a0 = np.zeros(1, dtype=np.float32)
    got = oracle.matmul(p.x, p.w, p.packed, a0)
    ref = bf16(p.x) @ bf16(p.w).T
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13 * np.abs(ref).max())


def test_sign_flip_negates_delta_exactly():
    p = wl.make_problem(3, 9, 160, 1, seed=9)
    b1, d1, _ = oracle.matmul_parts(p.x, p.w, p.packed, p.alpha)
    b2, d2, _ = oracle.matmul_parts(p.x, p.w, ~p.packed, p.alpha)
    assert np.array_equal(d2, -d1)
    assert np.array_equal(b1, b2)


def test_closed_form_ones_row():
    # x = 1, W = 0:  y[n] = alpha * (2 popcount(S[n]) - K), exactly
    rng = np.random.default_rng(10)
    K, N = 224, 19
    words = wl.uniform_words(rng, (1, N, K // 32))
    x = np.full((2, K), 0x3F80, dtype=np.uint16)         # bf16 1.0
    w = np.zeros((N, K), dtype=np.uint16)
    for a in (1.0, 2.0 ** -10, 7.25e-4):
        alpha = np.array([a], dtype=np.float32)
        y = oracle.matmul(x, w, words, alpha)
        pc = np.array([sum(int(v).bit_count() for v in words[0, n]) for n in range(N)])
        ref = np.float64(alpha[0]) * (2 * pc - K)
        assert np.array_equal(y[0], ref) and np.array_equal(y[1], ref)


def test_one_hot_rows_pick_weights_and_signs():
    # x = e_k:  y[n] = W[n, k] + alpha * s[n, k] for every k (all bit positions, word edges)
    p = wl.make_problem(1, 11, 96, 1, seed=12)
    S = numpy_signs(p.packed[0], p.K)
    x = np.zeros((p.K, p.K), dtype=np.uint16)
    x[np.arange(p.K), np.arange(p.K)] = 0x3F80
    y = oracle.matmul(x, p.w, p.packed, p.alpha)           # [K, N]
    ref = bf16(p.w).T + np.float64(p.alpha[0]) * S.T
    assert np.array_equal(y, ref)


def test_tenant_routing_invariants():
    rng = np.random.default_rng(13)
    M, N, K, T = 12, 7, 64, 4
    p = wl.make_problem(M, N, K, T, seed=14, multi_tenant=True)
    y = oracle.matmul(p.x, p.w, p.packed, p.alpha, p.tenant_ids)
    # each row equals the single-tenant result of its own tenant
    for m in range(M):
        t = p.tenant_ids[m]
        ys = oracle.matmul(p.x[m:m + 1], p.w, p.packed[t], p.alpha[t:t + 1])
        assert np.array_equal(y[m], ys[0])
    # permuting rows together with their tenant ids permutes the output
    perm = rng.permutation(M)
    yp = oracle.matmul(p.x[perm], p.w, p.packed, p.alpha, p.tenant_ids[perm])
    assert np.array_equal(yp, y[perm])
    # identical tenants == one tenant
    same = np.repeat(p.packed[:1], T, axis=0)
    a_same = np.repeat(p.alpha[:1], T)
    y1 = oracle.matmul(p.x, p.w, same, a_same, p.tenant_ids)
    y0 = oracle.matmul(p.x, p.w, p.packed[:1], p.alpha[:1])
    assert np.array_equal(y1, y0)
    # out-of-range tenant ids give NaN rows, other rows unaffected
    bad = p.tenant_ids.copy()
    bad[3], bad[5] = -1, T
    yb = oracle.matmul(p.x, p.w, p.packed, p.alpha, bad)
    assert np.all(np.isnan(yb[[3, 5]]))
    keep = [m for m in range(M) if m not in (3, 5)]
    assert np.array_equal(yb[keep], y[keep])


def test_sampled_columns_match_full():
    p = wl.make_problem(4, 50, 64, 2, seed=15, multi_tenant=True)
    full = oracle.matmul(p.x, p.w, p.packed, p.alpha, p.tenant_ids)
    idx = np.array([49, 0, 17, 17, 3])
    part = oracle.matmul(p.x, p.w, p.packed, p.alpha, p.tenant_ids, n_idx=idx)
    assert np.array_equal(part, full[:, idx])


def test_empty_shapes():
    x = np.zeros((0, 64), dtype=np.uint16)
    w = np.zeros((5, 64), dtype=np.uint16)
    y = oracle.matmul(x, w, np.zeros((1, 5, 2), np.uint32), np.ones(1, np.float32))
    assert y.shape == (0, 5)
    # K = 0: every sum is empty, so y = 0
    y = oracle.matmul(np.zeros((2, 0), np.uint16), np.zeros((3, 0), np.uint16),
                      np.zeros((1, 3, 0), np.uint32), np.ones(1, np.float32))
    assert np.array_equal(y, np.zeros((2, 3)))


# ---------------------------------------------------------------- compress

def _fraction_bf16(bits):
    from fractions import Fraction
    return Fraction(float(wl.bf16_bits_to_f32(np.array([bits], np.uint16))[0]))


def test_compress_bits_equal_numpy_signbit():
    # library routine: numpy's fp64 difference, np.signbit and packbits
    rng = np.random.default_rng(30)
    for rows, K in ((3, 32), (17, 96), (64, 1024)):
        base = wl.normal_bf16(rng, (rows, K), 0.02)
        fine = wl.normal_bf16(rng, (rows, K), 0.02)
        fine[:, ::7] = base[:, ::7]  # equal entries: delta = +0 -> +1
        packed, _, _ = oracle.compress(fine, base)
        d = bf16(fine) - bf16(base)
        np.testing.assert_array_equal(packed, numpy_pack(~np.signbit(d)))


def test_compress_sums_exact_brute_force():
    # exact rational sums of |fine - base| (bf16 values are dyadic rationals)
    from fractions import Fraction
    rng = np.random.default_rng(31)
    rows, K = 3, 64
    base = wl.normal_bf16(rng, (rows, K), 1.0)
    fine = wl.normal_bf16(rng, (rows, K), 1e-3)  # very different magnitudes
    _, row_abs, alpha = oracle.compress(fine, base)
    exact = [sum((abs(_fraction_bf16(fine[r, k]) - _fraction_bf16(base[r, k])) for k in range(K)),
                 Fraction(0)) for r in range(rows)]
    for r in range(rows):
        assert abs(Fraction(row_abs[r]) - exact[r]) <= exact[r] * Fraction(1, 10 ** 14)
    mean = sum(exact, Fraction(0)) / (rows * K)
    assert abs(Fraction(alpha) - mean) <= mean * Fraction(1, 10 ** 14)


def test_compress_closed_form_scaled_signs():
    # base = 0, fine = c * s with c = 2^-7 (exact in bf16): signs come back, alpha = c
    rng = np.random.default_rng(32)
    rows, K = 9, 160
    s = np.where(rng.random((rows, K)) < 0.5, 1.0, -1.0).astype(np.float32)
    c = 2.0 ** -7
    fine = wl.f32_to_bf16_bits(s * np.float32(c))
    base = np.zeros((rows, K), np.uint16)
    packed, row_abs, alpha = oracle.compress(fine, base)
    np.testing.assert_array_equal(packed, numpy_pack(s > 0))
    assert alpha == c
    assert np.all(row_abs == K * c)


def test_compress_least_squares_scale():
    # alpha minimises ||delta - a*s||^2 for the returned signs: the derivative
    # sum s (delta - alpha s) vanishes and nearby scales do worse
    rng = np.random.default_rng(33)
    rows, K = 40, 512
    base = wl.normal_bf16(rng, (rows, K), 0.02)
    fine = wl.f32_to_bf16_bits(bf16(base).astype(np.float32)
                               + rng.standard_normal((rows, K)).astype(np.float32) * 1e-3)
    packed, _, alpha = oracle.compress(fine, base)
    d = bf16(fine) - bf16(base)
    s = numpy_signs(packed, K)

    def obj(a):
        return float(np.sum((d - a * s) ** 2))
    grad = float(np.sum(s * (d - alpha * s)))
    assert abs(grad) <= 1e-9 * float(np.sum(np.abs(d)))
    assert obj(alpha) < obj(alpha * (1 + 1e-3)) and obj(alpha) < obj(alpha * (1 - 1e-3))


def test_compress_worked_rows_and_signed_zeros():
    # hand-derived words: bit i of word 0 <-> k = i; +1 where fine - base >= +0
    K = 32
    half, quarter = 0x3F00, 0x3E80          # 0.5, 0.25 in bf16
    one, one5, two = 0x3F80, 0x3FC0, 0x4000  # 1.0, 1.5, 2.0
    base = np.full((4, K), half, np.uint16)
    fine = base.copy()
    # row 0: +0.25 at even k, -0.25 at odd k  -> 0x55555555, |delta| = 0.25 each
    fine[0, 0::2] = 0x3F40                   # 0.75
    fine[0, 1::2] = quarter
    # row 1: equal -> delta = +0 everywhere -> 0xFFFFFFFF, sum 0
    # row 2: 1.0 - 1.5 = -0.5 everywhere except k = 31 where 2.0 - 1.5 = +0.5 -> 0x80000000
    base[2] = one5
    fine[2] = one
    fine[2, 31] = two
    # row 3: signed zeros: (-0) - (+0) = -0 -> 0 at k=0; (+0) - (-0) = +0 -> 1 at k=1;
    #        (-0) - (-0) = +0 -> 1 at k=2; the rest equal -> 1
    base[3, 0], fine[3, 0] = 0x0000, 0x8000
    base[3, 1], fine[3, 1] = 0x8000, 0x0000
    base[3, 2], fine[3, 2] = 0x8000, 0x8000
    packed, row_abs, alpha = oracle.compress(fine, base)
    assert [int(w) for w in packed[:, 0]] == [0x55555555, 0xFFFFFFFF, 0x80000000, 0xFFFFFFFE]
    assert list(row_abs) == [8.0, 0.0, 16.0, 0.0]
    assert alpha == 24.0 / (4 * K)


# ---------------------------------------------------------------- fp16 inputs

def test_f16_decode_every_finite_pattern():
    # one-hot x picks W[n][0]; alpha = 0, so y[n] is the exact value of the
    # fp16 pattern, compared with numpy's float16 -> float64 conversion
    pats = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    finite = pats[((pats >> 10) & 0x1F) != 0x1F]
    N, K = finite.size, 32
    w = np.zeros((N, K), np.uint16)
    w[:, 0] = finite
    x = np.zeros((1, K), np.uint16)
    x[0, 0] = 0x3C00  # 1.0
    packed = np.zeros((1, N, 1), np.uint32)
    y = oracle.matmul(x, w, packed, np.zeros(1, np.float32), dtype="f16")[0]
    ref = finite.view(np.float16).astype(np.float64)
    assert np.array_equal(y, ref)


def test_brute_force_f16_decoder_matches_numpy():
    pats = np.arange(0, 1 << 16, 7, dtype=np.uint32).astype(np.uint16)
    pats = pats[((pats >> 10) & 0x1F) != 0x1F]
    from fractions import Fraction
    for h in pats:
        assert brute.f16_bits_to_fraction(int(h)) == Fraction(float(np.uint16(h).view(np.float16)))


@pytest.mark.parametrize("M,N,K,T", [(2, 3, 32, 1), (3, 2, 64, 2)])
def test_brute_force_f16(M, N, K, T):
    rng = np.random.default_rng(M * 10 + K)
    p = wl.make_problem(M, N, K, T, seed=M + N + K, multi_tenant=T > 1, dtype="f16", y_dtype="f32")
    exact = brute.matmul_exact(p.x, p.w, p.packed, p.alpha, p.tenant_ids, dtype="f16")
    y = oracle.matmul(p.x, p.w, p.packed, p.alpha, p.tenant_ids, dtype="f16")
    for m in range(M):
        for n in range(N):
            e = float(exact[m][n])
            assert abs(y[m, n] - e) <= 1e-15 * max(1.0, abs(e)), (m, n)


def test_f16_compress_bits_equal_numpy_signbit():
    rng = np.random.default_rng(34)
    base = wl.normal_f16(rng, (20, 256), 0.02)
    fine = wl.normal_f16(rng, (20, 256), 0.02)
    fine[:, ::5] = base[:, ::5]
    packed, row_abs, _ = oracle.compress(fine, base, dtype="f16")
    d = base.view(np.float16).astype(np.float64)
    d = fine.view(np.float16).astype(np.float64) - d
    np.testing.assert_array_equal(packed, numpy_pack(~np.signbit(d)))
