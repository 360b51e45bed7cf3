"""Parity of the wide batched decode kernel (48 or 64 features per workgroup,
whole-line copies) with the fp64 oracle.

Batched requests of 17 to 64 rows over at most 16 distinct tenants, K a
multiple of 128, take it when its feature groups fill the CUs: 48 features
per group for 161 to 256 groups (N from about 7.7k to 12.3k), 64 features for
193 to 256 groups (N to 16k, at most 8 tenants).  Cases cover both feature
widths, both x-row forms (32 and 64), both sign-slot counts, a K whose last
512-k sign super-tile is partial or that is shorter than one super-tile, the
shortest K (four 64-k tiles), ragged N, fragment layouts up to three fragments
per wave, absent tenants, out-of-range ids, fp16, both output types and
bitwise repeatability.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_util import host_out, log, run_matmul, torch
from tolerance import check

pytestmark = pytest.mark.gpu

SKINNY = 1

CASES = [  # M, N, K, T: form
    (32, 11008, 4096, 16),   # 48 features, 32 x rows, 16 sign slots (multi-tenant decode shape)
    (64, 11008, 4096, 8),    # 48 features, 64 x rows, 8 slots (LLaMA gate/up shape)
    (64, 11008, 1152, 8),    # last super-tile partial
    (20, 10000, 640, 16),    # ragged N (last group 16 features), 16 slots
    (64, 9300, 512, 3),      # one super-tile
    (36, 8600, 384, 4),      # 180 groups, K shorter than a super-tile
    (17, 7777, 256, 2),      # 163 groups, K of four tiles
    (48, 12288, 768, 12),    # 256 groups, 64 x rows, 16 slots
    (64, 11008, 512, 16),    # 64 rows over 16 tenants: up to 19 fragments
    (24, 14336, 512, 8),     # 64 features (224 groups)
    (40, 16384, 384, 6),     # 64 features (256 groups), 64 x rows
]


def oracle_y(p, tid=None):
    tid = p.tenant_ids if tid is None else tid
    return oracle.matmul(p.x, p.w, p.packed, p.alpha, tid, dtype=p.dtype)


@pytest.mark.parametrize("M,N,K,T", CASES)
@pytest.mark.parametrize("yd", ["f32", "bf16"])
def test_wide_parity(M, N, K, T, yd):
    p = wl.make_problem(M, N, K, T, seed=3 * M + N + K + T, multi_tenant=True, y_dtype=yd)
    log(f"wide M={M} N={N} K={K} T={T} {yd} tenants present {len(np.unique(p.tenant_ids))}")
    y = host_out(run_matmul(p, path=SKINNY))
    relf, _ = check(y, oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)
    if yd == "f32":
        assert relf < 1e-5, relf


@pytest.mark.parametrize("M,N,K,T,counts", [
    (32, 11008, 512, 16, [1] * 15 + [17]),        # 17 fragments: three on wave 0
    (32, 11008, 512, 16, [2] * 16),               # 16 fragments of 2 rows
    (64, 11008, 384, 16, [1] * 15 + [49]),        # 19 fragments
    (64, 11008, 512, 8, [64] + [0] * 7),          # one tenant, four fragments
    (48, 9300, 1024, 8, [0, 0, 17, 31, 0, 0, 0, 0]),   # two tenants present, slots compacted
    (64, 11008, 640, 8, [0, 9, 0, 40, 0, 15, 0, 0]),   # three present
])
def test_wide_fragment_layouts(M, N, K, T, counts):
    T = len(counts)
    p = wl.make_problem(M, N, K, T, seed=M + N + len(counts), multi_tenant=True, y_dtype="f32")
    ids = np.repeat(np.arange(T), counts).astype(np.int32)
    assert ids.size == M
    p.tenant_ids = np.random.default_rng(sum(counts[:3])).permutation(ids)
    log(f"wide fragments M={M} N={N} K={K} T={T} counts={counts}")
    y = host_out(run_matmul(p, path=SKINNY))
    relf, _ = check(y, oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)
    assert relf < 1e-5, relf


@pytest.mark.parametrize("M,N,K,T", [(40, 11008, 512, 6), (24, 14336, 384, 8)])
def test_wide_invalid_ids_are_nan_rows(M, N, K, T):
    p = wl.make_problem(M, N, K, T, seed=N + 31, multi_tenant=True, y_dtype="f32")
    tid = p.tenant_ids.copy()
    tid[[0, 7, M - 1]] = [-1, T, 1 << 30]
    p.tenant_ids = tid
    log(f"wide invalid ids M={M} N={N} K={K}")
    y = host_out(run_matmul(p, path=SKINNY))
    bad = (tid < 0) | (tid >= T)
    assert np.all(np.isnan(y[bad]))
    ref = oracle_y(p, np.where(bad, 0, tid))
    relf, _ = check(y[~bad], ref[~bad], p.x[~bad], p.w, p.alpha, tid[~bad])
    assert relf < 1e-5, relf


@pytest.mark.parametrize("M,N,K,T", [(64, 11008, 1024, 8), (32, 11008, 1024, 16), (40, 16384, 384, 6)])
def test_wide_f16(M, N, K, T):
    p = wl.make_problem(M, N, K, T, seed=M + 77, multi_tenant=True, y_dtype="half", dtype="f16")
    log(f"wide f16 M={M} N={N} K={K} T={T}")
    y = host_out(run_matmul(p, path=SKINNY))
    check(y, oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids, dtype="f16")


@pytest.mark.parametrize("M,N,K,T", [(64, 11008, 1152, 8), (32, 11008, 1024, 16)])
def test_wide_repeatable(M, N, K, T):
    # same inputs, three calls: bitwise identical
    t = torch()
    p = wl.make_problem(M, N, K, T, seed=M + 5, multi_tenant=True, y_dtype="f32")
    log(f"wide repeat M={M} N={N} K={K} T={T}")
    ys = [run_matmul(p, path=SKINNY) for _ in range(3)]
    for y in ys[1:]:
        assert t.equal(y, ys[0])
