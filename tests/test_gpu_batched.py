"""Parity of the batched decode-shaped kernels with the fp64 oracle.

Batched requests with at most 16 distinct tenants take the kernel that
gathers each tenant's rows into 16-row fragments (one sign decode per tenant
and k-block): at most 4096 features, 17 to 64 rows and K a multiple of 256
(8-wave workgroups, one per CU); above 4096 features, 17 to 64 rows, or 8 to
16 rows over at most 8 tenants, K a multiple of 128 (4-wave workgroups, two or
three per CU; 33 to 64 rows over more than 8 tenants keep 8 waves).  Other
requests take the tenant-slot kernel.  Cases cover the 32-row and 64-row forms
of both workgroup sizes and both tenant-slot configurations of each (up to 8
and up to 16 tenants), tenant ids
used directly as sign slots (at most that many tenants) and compacted (more),
a K that ends inside a 1024-k sign super-tile, more row fragments than one pass
holds, out-of-range ids, the exact decode-isolating forms, fp16 and run-to-run
determinism.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_util import dev_half, dev_f32, dev_i32, dev_words, host_out, log, run_matmul, torch
from tolerance import check

pytestmark = pytest.mark.gpu

SKINNY = 1


def oracle_y(p, tid=None):
    tid = p.tenant_ids if tid is None else tid
    return oracle.matmul(p.x, p.w, p.packed, p.alpha, tid)


CASES = [  # M, N, K, T
    (1, 80, 256, 3), (16, 40, 512, 16), (32, 100, 768, 16),
    (33, 17, 2304, 9), (40, 70, 768, 11), (48, 20, 256, 5), (56, 50, 1024, 16),
    (64, 64, 512, 8), (64, 40, 512, 16), (64, 96, 4096, 8), (64, 30, 11008, 8),
    (36, 40, 11008, 4), (64, 33, 1280, 12), (64, 20, 512, 64),
    (17, 60, 1024, 12), (24, 50, 2304, 5), (32, 70, 4096, 8), (32, 40, 512, 40),
    (20, 4096, 512, 10), (20, 4112, 512, 10),
    # above 4096 features: 4-wave workgroups, 128-k tiles
    (64, 4200, 640, 8), (40, 4112, 1152, 3), (33, 4128, 128, 8), (48, 4160, 512, 16),
    (32, 4112, 640, 8), (24, 4200, 896, 16), (17, 4128, 128, 12), (32, 4144, 384, 40),
    (16, 4112, 768, 8), (8, 4112, 384, 5), (12, 4112, 512, 12), (64, 4112, 384, 12),
]


@pytest.mark.parametrize("M,N,K,T", CASES)
@pytest.mark.parametrize("yd", ["f32", "bf16"])
def test_batched_ragged(M, N, K, T, yd):
    p = wl.make_problem(M, N, K, T, seed=M * 5 + N + K + T, multi_tenant=True, y_dtype=yd)
    log(f"batched M={M} N={N} K={K} T={T} {yd} tenants present {len(np.unique(p.tenant_ids))}")
    y = host_out(run_matmul(p, path=SKINNY))
    relf, _ = check(y, oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)
    if yd == "f32":
        assert relf < 1e-5, relf


@pytest.mark.parametrize("M,T,counts", [
    (64, 16, [1] * 15 + [49]),          # 15 + 4 = 19 fragments: two passes of 12
    (64, 16, [4] * 16),                 # 16 fragments of 4 rows
    (48, 16, [17, 31] + [0] * 14),      # tenants split over two fragments
    (64, 8, [64] + [0] * 7),            # one tenant, four fragments
    (32, 16, [1] * 15 + [17]),          # 15 + 2 = 17 fragments: two passes of 16
    (32, 16, [2] * 16),                 # 16 fragments of 2 rows
    (32, 8, [32] + [0] * 7),            # one tenant, two fragments
    (16, 8, [2] * 8),                   # 8 fragments of 2 rows
    (16, 8, [16] + [0] * 7),            # one tenant, one fragment
])
@pytest.mark.parametrize("N,K", [(60, 1024), (4112, 768)])
def test_batched_fragment_layouts(M, T, counts, N, K):
    p = wl.make_problem(M, N, K, T, seed=M + T + len(counts), multi_tenant=True, y_dtype="f32")
    ids = np.repeat(np.arange(T), counts).astype(np.int32)
    p.tenant_ids = np.random.default_rng(sum(counts[:3])).permutation(ids)
    log(f"batched fragments M={M} N={N} K={K} T={T} counts={counts}")
    y = host_out(run_matmul(p, path=SKINNY))
    relf, _ = check(y, oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)
    assert relf < 1e-5, relf


def test_batched_invalid_ids_are_nan_rows():
    M, N, K, T = 40, 50, 512, 6
    p = wl.make_problem(M, N, K, T, seed=31, multi_tenant=True, y_dtype="f32")
    tid = p.tenant_ids.copy()
    tid[[0, 7, 39]] = [-1, T, 1 << 30]
    p.tenant_ids = tid
    log("batched invalid ids")
    y = host_out(run_matmul(p, path=SKINNY))
    bad = (tid < 0) | (tid >= T)
    assert np.all(np.isnan(y[bad]))
    ref = oracle_y(p, np.where(bad, 0, tid))
    relf, _ = check(y[~bad], ref[~bad], p.x[~bad], p.w, p.alpha, tid[~bad])
    assert relf < 1e-5, relf


@pytest.mark.parametrize("a", [1.0, 2.0 ** -10])
def test_batched_ones_zero_weight_exact(a):
    # x = 1, W = 0: y[m, n] = alpha_t * (2 popcount(S_t[n]) - K) exactly, per tenant
    rng = np.random.default_rng(8)
    M, N, K, T = 40, 48, 2048, 5
    packed = wl.uniform_words(rng, (T, N, K // 32))
    alpha = (a * (1 + np.arange(T))).astype(np.float32)
    tid = (np.arange(M) % T).astype(np.int32)
    p = wl.Problem("ones", np.full((M, K), 0x3F80, np.uint16), np.zeros((N, K), np.uint16),
                   alpha, packed=packed, tenant_ids=tid, y_dtype="f32")
    log(f"batched ones/zero-weight exact alpha={a}")
    y = host_out(run_matmul(p, path=SKINNY))
    pc = np.array([[sum(int(v).bit_count() for v in packed[t, n]) for n in range(N)] for t in range(T)])
    ref = alpha[tid][:, None].astype(np.float64) * (2 * pc[tid] - K)
    assert np.array_equal(y, ref)


def test_batched_one_hot_rows_every_bit_position():
    # x = e_k (row k), tenants alternating: y[k, n] = W[n, k] + alpha_t * s_t[n, k]
    K, N, T = 256, 40, 3
    base = wl.make_problem(1, N, K, T, seed=9, multi_tenant=True)
    rows = np.arange(64)
    for k0 in (0, 64, 128, 192):
        x = np.zeros((64, K), np.uint16)
        x[rows, k0 + rows] = 0x3F80
        tid = (rows % T).astype(np.int32)
        p = wl.Problem("onehot", x, base.w, base.alpha, packed=base.packed, tenant_ids=tid, y_dtype="f32")
        log(f"batched one-hot rows k0={k0}")
        y = host_out(run_matmul(p, path=SKINNY))
        ref = oracle.matmul(x, p.w, p.packed, p.alpha, tid)
        np.testing.assert_allclose(y, ref, rtol=2.0 ** -23, atol=0)


@pytest.mark.parametrize("M,N", [(64, 300), (64, 4400), (32, 4400)])
def test_batched_deterministic(M, N):
    p = wl.make_problem(M, N, 4096, 8, seed=33, multi_tenant=True, y_dtype="bf16")
    log(f"batched determinism M={M} N={N}")
    y1 = run_matmul(p, path=SKINNY).view(torch().int16).cpu().numpy()
    y2 = run_matmul(p, path=SKINNY).view(torch().int16).cpu().numpy()
    assert np.array_equal(y1, y2)


def test_batched_f16():
    import paper_2609_36800_amd as bd
    t = torch()
    p = wl.make_problem(48, 90, 1536, 7, seed=34, multi_tenant=True, y_dtype="f32", dtype="f16")
    log("batched f16")
    y = bd.matmul(dev_half(p.x, "f16"), dev_half(p.w, "f16"), dev_words(p.packed), dev_f32(p.alpha),
                  tenant_ids=dev_i32(p.tenant_ids), out_dtype=t.float32, path=SKINNY)
    t.cuda.synchronize()
    y = host_out(y)
    ref = oracle.matmul(p.x, p.w, p.packed, p.alpha, p.tenant_ids, dtype="f16")
    relf, _ = check(y, ref, p.x, p.w, p.alpha, p.tenant_ids, dtype="f16")
    assert relf < 1e-5, relf


@pytest.mark.parametrize("M,K", [(40, 512), (8, 256), (300, 128)])
def test_validation_mode_rejects_out_of_range_ids(M, K, monkeypatch):
    # BITDELTA_VALIDATE=1: the ids are read back before any launch; an id outside
    # [0, T) returns the tenant status and leaves the output untouched
    import paper_2609_36800_amd as bd
    t = torch()
    N, T = 48, 5
    p = wl.make_problem(M, N, K, T, seed=M + K + 3, multi_tenant=True, y_dtype="f32")
    tid = p.tenant_ids.copy()
    tid[M // 2] = T
    args = (dev_half(p.x, "bf16"), dev_half(p.w, "bf16"), dev_words(p.packed), dev_f32(p.alpha))
    monkeypatch.setenv("BITDELTA_VALIDATE", "1")
    log(f"validation mode M={M} K={K}")
    y = t.full((M, N), 7.0, dtype=t.float32, device="cuda")
    with pytest.raises(bd.BitDeltaError) as e:
        bd.matmul(*args, tenant_ids=dev_i32(tid), out=y)
    assert e.value.status == -8
    t.cuda.synchronize()
    assert bool((y == 7.0).all())
    # valid ids in validation mode: the same result as without it
    y1 = bd.matmul(*args, tenant_ids=dev_i32(p.tenant_ids), out_dtype=t.float32)
    monkeypatch.setenv("BITDELTA_VALIDATE", "0")
    y0 = bd.matmul(*args, tenant_ids=dev_i32(p.tenant_ids), out_dtype=t.float32)
    t.cuda.synchronize()
    assert t.equal(y0, y1)
    relf, _ = check(host_out(y1), oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)
    if M <= 64:     # decode-shaped paths never round the effective weight
        assert relf < 1e-5, relf
