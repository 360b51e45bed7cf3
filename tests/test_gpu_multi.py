"""Parity of the tenant-slot batched kernel (multi_kernel) with the fp64 oracle.

The dispatcher sends it batched requests with K a multiple of 128 that the
gathered-fragment kernel does not take: up to 16 rows (up to 7 rows, or more
than 8 tenants, above 4096 features), K not a multiple of 256 at most 4096
features, or more than 16 distinct tenants.
The cases cover every (row fragments, staged slots) configuration (1 to 4
fragments of 16 rows; 4, 8 or 16 slots), K from one 128-k tile up to a few
dozen, more than 4096 features, several passes over the tenants, out-of-range
ids and the exact ones/zero-weight form.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_util import host_out, log, run_matmul
from tolerance import check

pytestmark = pytest.mark.gpu

SKINNY = 1

CASES = [  # M, N, K, T: (row fragments MB, staged slots P)
    (1, 80, 384, 3),        # MB 1, P 4
    (8, 70, 640, 7),        # MB 1, P 8
    (16, 50, 1152, 16),     # MB 1, P 16, K = 9 tiles
    (32, 60, 640, 16),      # MB 2, P 16 (K not a multiple of 256)
    (24, 4112, 384, 20),    # MB 2, more than 4096 features and 16 tenants
    (12, 4112, 640, 9),     # MB 1, more than 4096 features, 9 tenants
    (7, 4160, 384, 3),      # MB 1, more than 4096 features, 7 rows
    (20, 40, 128, 2),       # MB 2, P 4, one tile
    (40, 50, 896, 8),       # MB 3, P 8
    (48, 30, 128, 5),       # MB 3, P 8, one tile
    (44, 36, 384, 3),       # MB 3, P 4
    (64, 40, 384, 8),       # MB 4, P 8
    (60, 40, 640, 3),       # MB 4, P 4
    (64, 30, 512, 40),      # MB 4, more than 16 tenants: passes of 8 slots
    (30, 24, 1408, 28),     # MB 2, passes of 16 slots, K = 11 tiles
]


@pytest.mark.parametrize("M,N,K,T", CASES)
@pytest.mark.parametrize("yd", ["f32", "bf16"])
def test_multi_kernel_shapes(M, N, K, T, yd):
    p = wl.make_problem(M, N, K, T, seed=M * 7 + N + K + T, multi_tenant=True, y_dtype=yd)
    log(f"multi M={M} N={N} K={K} T={T} {yd} tenants present {len(np.unique(p.tenant_ids))}")
    y = host_out(run_matmul(p, path=SKINNY))
    relf, _ = check(y, oracle.matmul(p.x, p.w, p.packed, p.alpha, p.tenant_ids),
                    p.x, p.w, p.alpha, p.tenant_ids)
    if yd == "f32":
        assert relf < 1e-5, relf


@pytest.mark.parametrize("M,K", [(12, 640), (32, 384), (56, 896)])
def test_multi_kernel_invalid_ids_are_nan_rows(M, K):
    N, T = 40, 6
    p = wl.make_problem(M, N, K, T, seed=M + K, multi_tenant=True, y_dtype="f32")
    tid = p.tenant_ids.copy()
    tid[[0, M // 2, M - 1]] = [-1, T, 1 << 30]
    p.tenant_ids = tid
    log(f"multi invalid ids M={M} K={K}")
    y = host_out(run_matmul(p, path=SKINNY))
    bad = (tid < 0) | (tid >= T)
    assert np.all(np.isnan(y[bad]))
    ref = oracle.matmul(p.x, p.w, p.packed, p.alpha, np.where(bad, 0, tid))
    relf, _ = check(y[~bad], ref[~bad], p.x[~bad], p.w, p.alpha, tid[~bad])
    assert relf < 1e-5, relf


def test_multi_kernel_ones_zero_weight_exact():
    # x = 1, W = 0: y[m, n] = alpha_t * (2 popcount(S_t[n]) - K) exactly, per tenant
    rng = np.random.default_rng(12)
    M, N, K, T = 24, 40, 640, 11
    packed = wl.uniform_words(rng, (T, N, K // 32))
    alpha = (0.5 * (1 + np.arange(T))).astype(np.float32)
    tid = (np.arange(M) % T).astype(np.int32)
    p = wl.Problem("ones", np.full((M, K), 0x3F80, np.uint16), np.zeros((N, K), np.uint16),
                   alpha, packed=packed, tenant_ids=tid, y_dtype="f32")
    log("multi ones/zero-weight exact")
    y = host_out(run_matmul(p, path=SKINNY))
    pc = np.array([[sum(int(v).bit_count() for v in packed[t, n]) for n in range(N)] for t in range(T)])
    ref = alpha[tid][:, None].astype(np.float64) * (2 * pc[tid] - K)
    assert np.array_equal(y, ref)
