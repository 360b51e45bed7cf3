"""fp16 inputs (the paper's own BitDelta precision): parity of every kernel path
with the fp64 oracle, decode-isolating exact cases, the fused path's rounding
rule, pack / unpack / compress of fp16 data."""
import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_util import dev_half, dev_words, host_out, host_words, log, run_matmul, torch
from tolerance import check

pytestmark = pytest.mark.gpu

SKINNY, PREFILL = 1, 2


def ref(p, rows=None, cols=None):
    x = p.x if rows is None else p.x[rows]
    tid = p.tenant_ids if (p.tenant_ids is None or rows is None) else p.tenant_ids[rows]
    return oracle.matmul(x, p.w, p.packed, p.alpha, tid, n_idx=cols, dtype="f16")


def f16_check(y, p, rows=None, cols=None, tid=None):
    r = ref(p, rows, cols)
    t = p.tenant_ids if tid is None else tid
    return check(y, r, p.x, p.w, p.alpha, t, rows=rows, dtype="f16")


@pytest.mark.parametrize("M", [1, 4, 16])
def test_f16_decode_shapes(M):
    p = wl.decode(M, seed=3, dtype="f16")
    log(f"f16 decode M={M}")
    f16_check(host_out(run_matmul(p)), p)


@pytest.mark.parametrize("M,N,K,T,yd", [(1, 33, 96, 1, "f32"), (16, 300, 4000, 1, "half"),
                                        (40, 200, 1024, 1, "f32"), (64, 130, 544, 1, "half"),
                                        (32, 1000, 4096, 16, "half"), (50, 70, 160, 5, "f32"),
                                        (64, 256, 256, 64, "f32"), (20, 99, 2048, 3, "half")])
def test_f16_skinny_paths(M, N, K, T, yd):
    p = wl.make_problem(M, N, K, T, seed=M + N + K + T, multi_tenant=T > 1, dtype="f16",
                        y_dtype=yd)
    log(f"f16 skinny M={M} N={N} K={K} T={T} y={p.y_dtype}")
    y = host_out(run_matmul(p, path=SKINNY))
    relf, _ = f16_check(y, p)
    if p.y_dtype == "f32":
        assert relf < 1e-5, relf


@pytest.mark.parametrize("M,N,K,yd", [(65, 17, 32, "f32"), (300, 520, 544, "half"),
                                      (513, 1000, 128, "half"), (257, 255, 64, "f32"),
                                      (1000, 300, 4096, "half"), (129, 513, 1088, "f32")])
def test_f16_prefill(M, N, K, yd):
    p = wl.make_problem(M, N, K, 1, seed=M + 2 * N + K, dtype="f16", y_dtype=yd)
    log(f"f16 prefill M={M} N={N} K={K} y={p.y_dtype}")
    f16_check(host_out(run_matmul(p, path=PREFILL)), p)


@pytest.mark.parametrize("M,N,K,T,yd", [(300, 520, 576, 8, "half"), (513, 1000, 128, 17, "f32"),
                                        (700, 70, 640, 40, "half")])
def test_f16_grouped_prefill(M, N, K, T, yd):
    p = wl.make_problem(M, N, K, T, seed=M + N + K + T, multi_tenant=True, dtype="f16",
                        y_dtype=yd)
    log(f"f16 grouped prefill M={M} N={N} K={K} T={T} y={p.y_dtype}")
    f16_check(host_out(run_matmul(p, path=PREFILL)), p)


def test_f16_prefill_workload_sampled():
    p = wl.prefill(seed=1, dtype="f16")
    log(f"f16 prefill workload: {p.name}")
    y = run_matmul(p)
    rng = np.random.default_rng(5)
    rows = np.unique(np.concatenate([rng.choice(p.M, 200, replace=False), [0, 255, 256, p.M - 1]]))
    cols = np.unique(np.concatenate([rng.choice(p.N, 200, replace=False), [0, 255, 256, p.N - 1]]))
    yh = host_out(y[torch().from_numpy(rows).cuda()][:, torch().from_numpy(cols).cuda()])
    f16_check(yh, p, rows=rows, cols=cols)


@pytest.mark.parametrize("path", [SKINNY, PREFILL])
@pytest.mark.parametrize("a", [1.0, 2.0 ** -10])
def test_f16_ones_row_zero_weight_exact(path, a):
    # x = 1, W = 0: y[n] = alpha (2 popcount(S[n]) - K) exactly; alpha is exact in
    # fp16, so the fused weight fp16(0 + fp16(+-alpha)) is +-alpha itself
    rng = np.random.default_rng(4)
    M, N, K = (8 if path == SKINNY else 70), 300, 4096
    p = wl.Problem("ones", np.full((M, K), 0x3C00, np.uint16), np.zeros((N, K), np.uint16),
                   np.array([a], np.float32), packed=wl.uniform_words(rng, (1, N, K // 32)),
                   y_dtype="f32", dtype="f16")
    log(f"f16 ones/zero-weight exact path={path} alpha={a}")
    y = host_out(run_matmul(p, path=path))
    pc = np.array([sum(int(v).bit_count() for v in p.packed[0, n]) for n in range(N)])
    assert np.array_equal(y, np.broadcast_to(a * (2 * pc - K).astype(np.float64), y.shape))


def test_f16_one_hot_rows_decode_path():
    # x = e_k: y = W[n, k] + alpha s[n, k], one fp32 rounding on the decode path
    K, N = 96, 40
    base = wl.make_problem(1, N, K, 1, seed=6, dtype="f16")
    x = np.zeros((K, K), np.uint16)
    x[np.arange(K), np.arange(K)] = 0x3C00
    p = wl.Problem("onehot", x, base.w, base.alpha, packed=base.packed, y_dtype="f32", dtype="f16")
    log("f16 one-hot rows")
    y = host_out(run_matmul(p, path=SKINNY))
    np.testing.assert_allclose(y, ref(p), rtol=2.0 ** -23, atol=0)


@pytest.mark.parametrize("K", [96, 128, 4096])
def test_f16_fused_weight_rounding_exact(K):
    # x = e_k on the fused path: y[k, n] = fp16_rne(W[n, k] + fp16_rne(s alpha)),
    # the sum exact in fp64 and rounded once by numpy's float64 -> float16
    N = 300
    base = wl.make_problem(1, N, K, 1, seed=K + 2, dtype="f16")
    rows = np.unique(np.concatenate([np.arange(0, K, max(1, K // 160)), [K - 1]]))
    x = np.zeros((len(rows), K), np.uint16)
    x[np.arange(len(rows)), rows] = 0x3C00
    p = wl.Problem("onehot-exact", x, base.w, base.alpha, packed=base.packed, y_dtype="f32",
                   dtype="f16")
    log(f"f16 fused-weight rounding K={K}")
    y = host_out(run_matmul(p, path=PREFILL))
    s = oracle.unpack(p.packed[0], K)[:, rows].T
    w = p.w[:, rows].T.view(np.float16).astype(np.float64)
    a = np.float64(np.float16(p.alpha[0]))
    eff = (w + np.where(s > 0, a, -a)).astype(np.float16).astype(np.float64)
    assert np.array_equal(y, eff)


def test_f16_grouped_equals_single_tenant_runs():
    M, N, K, T = 700, 264, 192, 5
    p = wl.make_problem(M, N, K, T, seed=40, multi_tenant=True, dtype="f16", y_dtype="half")
    log("f16 grouped == per-tenant single runs")
    t = torch()
    y = run_matmul(p, path=PREFILL)
    for ten in np.unique(p.tenant_ids):
        rows = np.nonzero(p.tenant_ids == ten)[0]
        q = wl.Problem("one", p.x[rows], p.w, p.alpha[ten:ten + 1], packed=p.packed[ten:ten + 1],
                       y_dtype="f16", dtype="f16")
        ys = run_matmul(q, path=PREFILL)
        assert t.equal(y[t.from_numpy(rows).cuda()].view(t.int16), ys.view(t.int16)), ten


def test_f16_deterministic():
    t = torch()
    for M in (16, 600):
        p = wl.make_problem(M, 1000, 1024, 1, seed=41, dtype="f16", y_dtype="half")
        log(f"f16 determinism M={M}")
        assert t.equal(run_matmul(p).view(t.int16), run_matmul(p).view(t.int16))


def test_f16_invalid_tenant_rows_nan():
    M, N, K, T = 300, 100, 256, 4
    p = wl.make_problem(M, N, K, T, seed=42, multi_tenant=True, dtype="f16", y_dtype="half")
    p.tenant_ids[[0, 150, 299]] = [-1, T, 99]
    log("f16 invalid ids")
    for path in (SKINNY, PREFILL):
        y = host_out(run_matmul(p, path=path))
        assert np.all(np.isnan(y[[0, 150, 299]]))
        keep = np.setdiff1d(np.arange(M), [0, 150, 299])
        assert np.all(np.isfinite(y[keep]))


def test_f16_pack_unpack():
    import paper_2609_36800_amd as bd
    t = torch()
    log("f16 pack / unpack")
    rng = np.random.default_rng(43)
    s = wl.random_signs_i8(rng, (37, 4096)).astype(np.float16).view(np.uint16)
    s[0, :8] = [0x0000, 0x8000, 0x7C00, 0xFC00, 0x7E00, 0xFE00, 0x0001, 0x8001]
    got = host_words(bd.pack(dev_half(s, "f16")))
    np.testing.assert_array_equal(got, oracle.pack(s))
    words = wl.uniform_words(rng, (7, 160 // 32))
    out = bd.unpack(dev_words(words), 160, t.float16)
    np.testing.assert_array_equal(out.float().cpu().numpy().astype(np.float64),
                                  oracle.unpack(words, 160))
    np.testing.assert_array_equal(host_words(bd.pack(out)), words)


@pytest.mark.parametrize("rows,K", [(3, 96), (64, 4096), (130, 11008)])
def test_f16_compress(rows, K):
    import paper_2609_36800_amd as bd
    t = torch()
    rng = np.random.default_rng(rows + K)
    base = wl.normal_f16(rng, (rows, K), 0.02)
    fine = (base.view(np.float16).astype(np.float32)
            + rng.standard_normal((rows, K)).astype(np.float32) * 5e-4).astype(np.float16).view(np.uint16)
    fine[:, ::11] = base[:, ::11]
    log(f"f16 compress rows={rows} K={K}")
    packed, alpha, row_abs = bd.compress(dev_half(fine, "f16"), dev_half(base, "f16"))
    t.cuda.synchronize()
    p_ref, r_ref, a_ref = oracle.compress(fine, base, dtype="f16")
    np.testing.assert_array_equal(host_words(packed), p_ref)
    bound = (8 * -(-K // 2048) + 10) * 2.0 ** -24
    r = row_abs.cpu().numpy().astype(np.float64)
    assert np.max(np.abs(r - r_ref) / r_ref) <= bound
    assert abs(float(alpha.cpu()[0]) - a_ref) <= a_ref * (bound + 2.0 ** -24)
