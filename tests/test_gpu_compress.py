"""Parity of the HIP delta compression (packed signs of W_fine - W_base and
their least-squares scale) with the fp64 oracle."""
import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_util import dev_bf16, host_words, log, torch

pytestmark = pytest.mark.gpu


def run(fine, base, with_alpha=True):
    import paper_2609_36800_amd as bd
    t = torch()
    packed, alpha, row_abs = bd.compress(dev_bf16(fine), dev_bf16(base), with_alpha=with_alpha)
    t.cuda.synchronize()
    a = None if alpha is None else float(alpha.cpu().numpy()[0])
    return host_words(packed), a, row_abs.cpu().numpy().astype(np.float64)


def sum_bound(K):
    # fp32 sums of nonnegative terms: a lane adds 8 elements of every fourth
    # 512-element chunk in sequence, then six butterfly levels and three
    # additions of the wave sums; each |delta| is rounded at most once
    per_lane = 8 * -(-K // 2048)
    return (per_lane + 6 + 3 + 1) * 2.0 ** -24


@pytest.mark.parametrize("rows,K", [(1, 32), (3, 96), (17, 2080), (64, 4096), (130, 11008),
                                    (5, 512), (7, 2048 + 512)])
def test_compress_parity(rows, K):
    rng = np.random.default_rng(rows * 131 + K)
    base = wl.normal_bf16(rng, (rows, K), 0.02)
    fine = wl.f32_to_bf16_bits(wl.bf16_bits_to_f32(base)
                               + rng.standard_normal((rows, K)).astype(np.float32) * 5e-4)
    fine[:, ::13] = base[:, ::13]  # some zero deltas
    log(f"compress rows={rows} K={K}")
    packed, alpha, row_abs = run(fine, base)
    p_ref, r_ref, a_ref = oracle.compress(fine, base)
    np.testing.assert_array_equal(packed, p_ref)
    rel = np.abs(row_abs - r_ref) / np.maximum(r_ref, 1e-300)
    assert rel.max() <= sum_bound(K), rel.max()
    assert abs(alpha - a_ref) <= a_ref * (sum_bound(K) + 2.0 ** -24)


def test_compress_llama_shape_and_scale_quality():
    rows, K = 11008, 4096
    rng = np.random.default_rng(7)
    base = wl.normal_bf16(rng, (rows, K), 0.02)
    fine = wl.f32_to_bf16_bits(wl.bf16_bits_to_f32(base)
                               + rng.standard_normal((rows, K)).astype(np.float32) * 1e-3)
    log("compress 11008x4096")
    packed, alpha, row_abs = run(fine, base)
    p_ref, r_ref, a_ref = oracle.compress(fine, base)
    np.testing.assert_array_equal(packed, p_ref)
    assert np.max(np.abs(row_abs - r_ref) / r_ref) <= sum_bound(K)
    assert abs(alpha - a_ref) <= a_ref * (sum_bound(K) + 2.0 ** -24)
    # the least-squares scale does better than no delta at all
    d = wl.bf16_bits_to_f32(fine).astype(np.float64) - wl.bf16_bits_to_f32(base)
    s = oracle.unpack(packed[:64], K)
    assert np.linalg.norm(d[:64] - alpha * s) < np.linalg.norm(d[:64])


def test_compress_closed_form_and_special_values():
    rows, K = 6, 4096
    rng = np.random.default_rng(8)
    s = np.where(rng.random((rows, K)) < 0.5, 1.0, -1.0).astype(np.float32)
    c = 2.0 ** -7
    fine = wl.f32_to_bf16_bits(s * np.float32(c))
    base = np.zeros((rows, K), np.uint16)
    log("compress closed form")
    packed, alpha, row_abs = run(fine, base)
    np.testing.assert_array_equal(packed, oracle.pack(s))
    assert alpha == c and np.all(row_abs == K * c)
    # equal weights: every delta is +0 -> all bits set, zero scale
    packed, alpha, row_abs = run(base, base)
    assert np.all(packed == 0xFFFFFFFF) and alpha == 0.0 and np.all(row_abs == 0)
    # signed zeros: (-0)-(+0) = -0 -> 0; (+0)-(-0) = +0 -> 1; (-0)-(-0) = +0 -> 1
    f = np.zeros((1, 32), np.uint16)
    b = np.zeros((1, 32), np.uint16)
    f[0, 0], b[0, 0] = 0x8000, 0x0000
    f[0, 1], b[0, 1] = 0x0000, 0x8000
    f[0, 2], b[0, 2] = 0x8000, 0x8000
    packed, _, _ = run(f, b)
    assert int(packed[0, 0]) == 0xFFFFFFFE


def test_compress_without_alpha_and_deterministic():
    rows, K = 300, 1024
    rng = np.random.default_rng(9)
    base = wl.normal_bf16(rng, (rows, K), 0.02)
    fine = wl.normal_bf16(rng, (rows, K), 0.02)
    log("compress determinism / no alpha")
    p1, a1, r1 = run(fine, base)
    p2, a2, r2 = run(fine, base, with_alpha=False)
    assert a2 is None
    np.testing.assert_array_equal(p1, p2)
    np.testing.assert_array_equal(r1, r2)
    p3, a3, r3 = run(fine, base)
    assert a1 == a3
    np.testing.assert_array_equal(r1, r3)
