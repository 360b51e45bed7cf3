"""Parity of the HIP binary-delta matmul with the fp64 oracle.

Every test prints its case before the first GPU call.  Full-size workloads are
checked on every output where the oracle finishes in seconds, else on sampled
rows and columns that include tile edges and the ragged tail.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_util import dev_bf16, dev_f32, dev_i32, dev_words, host_out, host_words, log, run_matmul, torch
from tolerance import check

pytestmark = pytest.mark.gpu

SKINNY, PREFILL = 1, 2


def oracle_y(p, rows=None, cols=None, packed=None):
    x = p.x if rows is None else p.x[rows]
    tid = p.tenant_ids if (p.tenant_ids is None or rows is None) else p.tenant_ids[rows]
    return oracle.matmul(x, p.w, p.packed if packed is None else packed, p.alpha, tid, n_idx=cols)


def sample_cols(N, count, rng, tile=256):
    edge = {0, N - 1}
    for b in range(tile, N, tile):
        edge.update({b - 1, b})
    edge = sorted(e for e in edge if 0 <= e < N)
    rest = rng.choice(N, size=min(count, N), replace=False)
    return np.unique(np.concatenate([np.array(edge, dtype=np.int64), rest.astype(np.int64)]))


# ------------------------------------------------------------------ workloads

def test_tiny_workload_both_paths():
    import paper_2609_36800_amd as bd
    p = wl.tiny(seed=0)
    log(f"tiny workload: {p.name}")
    t = torch()
    # signs are drawn as int8 and packed on the device; bit-exact with the oracle packer
    packed_dev = bd.pack(t.from_numpy(p.signs[0]).cuda())
    packed = host_words(packed_dev)[None]
    np.testing.assert_array_equal(packed[0], oracle.pack(p.signs[0]))
    ref = oracle.matmul(p.x, p.w, packed, p.alpha)
    for path in (SKINNY, PREFILL):
        y = host_out(run_matmul(p, packed=packed, path=path))
        relf, _ = check(y, ref, p.x, p.w, p.alpha)
        if path == SKINNY:
            assert relf < 1e-5, relf


@pytest.mark.parametrize("M", [1, 16])
def test_decode_workload(M):
    p = wl.decode(M, seed=0)
    log(f"decode workload: {p.name}")
    y = host_out(run_matmul(p))
    ref = oracle_y(p)
    check(y, ref, p.x, p.w, p.alpha)


def test_multi_tenant_decode_workload():
    p = wl.mt_decode(seed=0)
    log(f"multi-tenant decode workload: {p.name}, tenants present {len(np.unique(p.tenant_ids))}")
    y = host_out(run_matmul(p))
    ref = oracle_y(p)
    check(y, ref, p.x, p.w, p.alpha, p.tenant_ids)


def test_prefill_workload_full():
    # every one of the 4096 x 4096 outputs against the fp64 oracle (about 275
    # GFLOP of fp64 work on the host: seconds with OpenMP)
    p = wl.prefill(seed=0)
    log(f"prefill workload (full output): {p.name}")
    y = host_out(run_matmul(p))
    check(y, oracle_y(p), p.x, p.w, p.alpha)


def test_llama_sweep_layer0_full():
    # one whole matrix of each type (q, k, v, o, gate, up, down): every output
    shared = wl.llama_shared_inputs(seed=0)
    for idx in range(len(wl.LLAMA_MATRICES)):
        p = wl.llama_matrix(0, idx, shared=shared)
        log(f"llama sweep (full output): {p.name}")
        y = host_out(run_matmul(p))
        check(y, oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)


@pytest.mark.parametrize("layer", list(range(32)))
def test_llama_sweep_layer_sampled(layer):
    # every matrix of the 32-layer sweep, each checked on its own
    shared = wl.llama_shared_inputs(seed=0)
    rng = np.random.default_rng(layer)
    for idx in range(len(wl.LLAMA_MATRICES)):
        p = wl.llama_matrix(layer, idx, shared=shared)
        log(f"llama sweep: {p.name}")
        y = run_matmul(p)
        cols = sample_cols(p.N, 192, rng)
        yh = host_out(y[:, cols])
        ref = oracle_y(p, cols=cols)
        check(yh, ref, p.x, p.w, p.alpha, p.tenant_ids)


# --------------------------------------------------------- ragged shapes, paths

@pytest.mark.parametrize("M,N,K", [(1, 1, 32), (3, 17, 96), (15, 300, 288), (16, 33, 4096),
                                   (17, 129, 160), (33, 16, 64), (63, 47, 1024), (64, 300, 544)])
@pytest.mark.parametrize("yd", ["f32", "bf16"])
def test_skinny_single_ragged(M, N, K, yd):
    p = wl.make_problem(M, N, K, 1, seed=M * 7 + N + K, y_dtype=yd)
    log(f"skinny single M={M} N={N} K={K} {yd}")
    y = host_out(run_matmul(p, path=SKINNY))
    relf, _ = check(y, oracle_y(p), p.x, p.w, p.alpha)
    if yd == "f32":
        assert relf < 1e-5, relf


@pytest.mark.parametrize("M,N,K,T", [(1, 16, 64, 3), (5, 17, 96, 2), (17, 100, 256, 16),
                                     (32, 300, 1024, 16), (64, 33, 160, 8), (64, 65, 64, 64),
                                     (40, 48, 4096, 1), (100, 50, 128, 5)])
@pytest.mark.parametrize("yd", ["f32", "bf16"])
def test_skinny_multi_ragged(M, N, K, T, yd):
    p = wl.make_problem(M, N, K, T, seed=M + N * 3 + K + T, multi_tenant=True, y_dtype=yd)
    log(f"skinny multi M={M} N={N} K={K} T={T} {yd}")
    y = host_out(run_matmul(p))
    relf, _ = check(y, oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)
    if yd == "f32":
        assert relf < 1e-5, relf


# K a multiple of 64 selects the streaming kernel, other K the general one
@pytest.mark.parametrize("M,N,K", [(65, 17, 32), (300, 520, 544), (513, 1000, 96),
                                   (4, 256, 64), (256, 256, 256), (1000, 300, 4096),
                                   (300, 520, 576), (513, 1000, 128), (257, 255, 64),
                                   (1, 300, 192), (600, 70, 640), (129, 513, 1088)])
@pytest.mark.parametrize("yd", ["f32", "bf16"])
def test_prefill_ragged(M, N, K, yd):
    p = wl.make_problem(M, N, K, 1, seed=M + N + K * 5, y_dtype=yd)
    log(f"prefill M={M} N={N} K={K} {yd}")
    y = host_out(run_matmul(p, path=PREFILL))
    check(y, oracle_y(p), p.x, p.w, p.alpha)


# more distinct tenants than one pass of the batched kernel holds (16 slots up
# to 32 rows, 8 above): later passes re-stream x and signs and skip the base
@pytest.mark.parametrize("M,N,K,T", [(32, 150, 384, 32), (48, 200, 512, 40), (64, 130, 256, 64),
                                     (20, 70, 1024, 20), (33, 16, 128, 33)])
def test_multi_tenant_several_passes(M, N, K, T):
    p = wl.make_problem(M, N, K, T, seed=M * 3 + T, multi_tenant=True, y_dtype="f32")
    p.tenant_ids = np.random.default_rng(M + T).permutation(np.arange(M) % T).astype(np.int32)
    log(f"multi-tenant passes M={M} N={N} K={K} T={T} distinct={len(np.unique(p.tenant_ids))}")
    y = host_out(run_matmul(p))
    relf, _ = check(y, oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)
    assert relf < 1e-5, relf


def test_skinny_forced_above_64_rows():
    p = wl.make_problem(150, 70, 256, 1, seed=3, y_dtype="f32")
    log("skinny forced M=150")
    y = host_out(run_matmul(p, path=SKINNY))
    relf, _ = check(y, oracle_y(p), p.x, p.w, p.alpha)
    assert relf < 1e-5


# ------------------------------------------------------ decode-isolating checks

@pytest.mark.parametrize("path", [SKINNY, PREFILL])
@pytest.mark.parametrize("a", [1.0, 2.0 ** -10])
def test_ones_row_zero_weight_exact(path, a):
    # x = 1, W = 0:  y[n] = alpha * (2 popcount(S[n]) - K), exactly
    rng = np.random.default_rng(4)
    M, N, K = (8 if path == SKINNY else 70), 300, 4096
    p = wl.Problem("ones", np.full((M, K), 0x3F80, np.uint16), np.zeros((N, K), np.uint16),
                   np.array([a], np.float32), packed=wl.uniform_words(rng, (1, N, K // 32)),
                   y_dtype="f32")
    log(f"ones/zero-weight exact path={path} alpha={a}")
    y = host_out(run_matmul(p, path=path))
    pc = np.array([sum(int(v).bit_count() for v in p.packed[0, n]) for n in range(N)])
    ref = a * (2 * pc - K).astype(np.float64)
    assert np.array_equal(y, np.broadcast_to(ref, y.shape))


@pytest.mark.parametrize("path", [SKINNY, PREFILL])
def test_one_hot_rows_every_bit_position(path):
    # x = e_k:  y[k, n] = W[n, k] + alpha * s[n, k]; covers all 32 bit positions and word edges
    K, N = 96, 40
    base = wl.make_problem(1, N, K, 1, seed=6)
    rows = np.arange(K)       # skinny serves these 96 rows in launches of 64
    x = np.zeros((len(rows), K), np.uint16)
    x[np.arange(len(rows)), rows] = 0x3F80
    p = wl.Problem("onehot", x, base.w, base.alpha, packed=base.packed, y_dtype="f32")
    log(f"one-hot rows path={path}")
    y = host_out(run_matmul(p, path=path))
    ref = oracle.matmul(x, p.w, p.packed, p.alpha)
    if path == SKINNY:
        # one fp32 rounding of W + alpha*s
        np.testing.assert_allclose(y, ref, rtol=2.0 ** -23, atol=0)
    else:
        # the fused path rounds W + alpha*s to bf16 first
        np.testing.assert_allclose(y, ref, rtol=2.0 ** -8, atol=0)


@pytest.mark.parametrize("K", [96, 128, 4096])
def test_prefill_effective_weight_rounding_exact(K):
    # x = e_k: y[k, n] is the fused path's effective weight itself, which is
    # bf16_rne(fp32(W + s*alpha)); checked bit for bit on rows spanning the K tiles
    N = 300
    base = wl.make_problem(1, N, K, 1, seed=K + 1)
    rows = np.unique(np.concatenate([np.arange(0, K, max(1, K // 160)), [K - 1]]))
    x = np.zeros((len(rows), K), np.uint16)
    x[np.arange(len(rows)), rows] = 0x3F80
    p = wl.Problem("onehot-exact", x, base.w, base.alpha, packed=base.packed, y_dtype="f32")
    log(f"effective-weight rounding K={K}")
    y = host_out(run_matmul(p, path=PREFILL))
    s = oracle.unpack(p.packed[0], K)[:, rows].T  # [rows, N] of +-1
    wv = wl.bf16_bits_to_f32(p.w[:, rows].T)
    a = np.float32(p.alpha[0])
    eff = (wv + np.where(s > 0, a, -a).astype(np.float32)).astype(np.float32)
    ref = wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(eff))
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("path", [SKINNY, PREFILL])
def test_sign_only_random_x(path):
    # W = 0: only the delta term remains, so an error in it is first-order
    M = 16 if path == SKINNY else 128
    p = wl.make_problem(M, 200, 1024, 1, seed=9, y_dtype="f32")
    p.w = np.zeros_like(p.w)
    log(f"sign-only path={path}")
    y = host_out(run_matmul(p, path=path))
    ref = oracle_y(p)
    rel = np.linalg.norm(y - ref) / np.linalg.norm(ref)
    # the fused path carries bf16(+-alpha) as its weight: one bf16 rounding of alpha
    assert rel < (1e-5 if path == SKINNY else 2.0 ** -8), rel


@pytest.mark.parametrize("a", [0.0, -3e-4, 0.25, 100.0])
def test_alpha_values(a):
    for M, path in ((16, SKINNY), (96, PREFILL)):
        p = wl.make_problem(M, 130, 256, 1, seed=10, y_dtype="f32")
        p.alpha = np.array([a], np.float32)
        log(f"alpha={a} M={M} path={path}")
        y = host_out(run_matmul(p, path=path))
        check(y, oracle_y(p), p.x, p.w, p.alpha)


def test_k_zero_writes_zeros():
    import paper_2609_36800_amd as bd
    t = torch()
    for M, path in ((5, SKINNY), (80, PREFILL)):
        log(f"K=0 M={M} path={path}")
        x = t.empty((M, 0), dtype=t.bfloat16, device="cuda")
        w = t.empty((7, 0), dtype=t.bfloat16, device="cuda")
        pk = t.empty((1, 7, 0), dtype=t.int32, device="cuda")
        a = t.ones(1, dtype=t.float32, device="cuda")
        y = t.full((M, 7), 5.0, dtype=t.float32, device="cuda")
        bd.matmul(x, w, pk, a, out=y, path=path)
        t.cuda.synchronize()
        assert t.count_nonzero(y).item() == 0


def test_empty_rows_leave_output_untouched():
    import paper_2609_36800_amd as bd
    t = torch()
    log("M=0 / N=0 no-op")
    x = t.zeros((0, 64), dtype=t.bfloat16, device="cuda")
    w = t.zeros((8, 64), dtype=t.bfloat16, device="cuda")
    pk = t.zeros((1, 8, 2), dtype=t.int32, device="cuda")
    a = t.ones(1, dtype=t.float32, device="cuda")
    y = bd.matmul(x, w, pk, a)
    t.cuda.synchronize()
    assert y.shape == (0, 8)


@pytest.mark.parametrize("path", [SKINNY, PREFILL])
@pytest.mark.parametrize("x_std", [1e30, 1e-30])
def test_extreme_magnitudes(path, x_std):
    # x near the top (or far down) of the bf16 range, sums still inside fp32
    M = 8 if path == SKINNY else 72
    p = wl.make_problem(M, 64, 128, 1, seed=11, y_dtype="f32", x_std=x_std)
    log(f"extreme magnitudes x_std={x_std} path={path}")
    y = host_out(run_matmul(p, path=path))
    check(y, oracle_y(p), p.x, p.w, p.alpha)


@pytest.mark.parametrize("path", [SKINNY, PREFILL])
def test_overflow_to_inf(path):
    # x near the top of the bf16 range against same-signed weights: every
    # product has the row's sign, the exact sums exceed the fp32 range, and the
    # outputs must be infinities of that sign; other rows stay finite
    M = 8 if path == SKINNY else 80
    N, K = 48, 256
    p = wl.make_problem(M, N, K, 1, seed=17, y_dtype="f32")
    big = wl.f32_to_bf16_bits(np.float32(3.0e38))
    x = p.x.copy()
    x[0, :] = big
    x[1, :] = big ^ 0x8000
    w = p.w.copy()
    w[:16, :] = 0x3F80          # +1
    w[16:32, :] = 0xBF80        # -1
    # signs agree with the weights, so the separate base and sign sums of the
    # decode path overflow with the same sign (no inf - inf)
    pk = p.packed.copy()
    pk[0, :16, :] = 0xFFFFFFFF
    pk[0, 16:32, :] = 0
    p.x, p.w, p.packed = x, w, pk
    p.alpha = np.array([1e-3], np.float32)
    log(f"overflow to inf path={path}")
    y = host_out(run_matmul(p, path=path))
    assert np.all(y[0, :16] == np.inf) and np.all(y[0, 16:32] == -np.inf)
    assert np.all(y[1, :16] == -np.inf) and np.all(y[1, 16:32] == np.inf)
    assert np.all(np.isfinite(y[2:]))
    ref = oracle_y(p, rows=np.arange(2, M))
    check(y[2:], ref, p.x, p.w, p.alpha, rows=np.arange(2, M))


def test_cancellation_rows():
    # rows with paired +v / -v entries cancel the base sum; the delta must survive
    p = wl.make_problem(4, 96, 256, 1, seed=12, y_dtype="f32")
    x = p.x.copy()
    x[:, 128:] = x[:, :128] ^ 0x8000
    p.x = x
    w = p.w.copy()
    w[:, 128:] = w[:, :128]
    p.w = w
    log("cancellation rows")
    for path in (SKINNY, PREFILL):
        y = host_out(run_matmul(p, path=path))
        ref = oracle_y(p)
        scale = np.abs(wl.bf16_bits_to_f32(p.x).astype(np.float64)).sum(axis=1)[:, None]
        err = np.abs(y - ref) / (scale * (p.alpha[0] + 0.1))
        assert err.max() < (1e-6 if path == SKINNY else 1e-2), err.max()


# ------------------------------------------------------ determinism and tenants

@pytest.mark.parametrize("case", ["decode16", "mt", "prefill"])
def test_bitwise_deterministic(case):
    p = {"decode16": lambda: wl.make_problem(16, 4096, 4096, 1, seed=13),
         "mt": lambda: wl.make_problem(32, 2000, 4096, 16, seed=13, multi_tenant=True),
         "prefill": lambda: wl.make_problem(512, 512, 1024, 1, seed=13)}[case]()
    log(f"determinism {case}")
    t = torch()
    y1 = run_matmul(p)
    y2 = run_matmul(p)
    assert t.equal(y1.view(t.int16), y2.view(t.int16))


def test_tenant_invariants():
    rng = np.random.default_rng(14)
    M, N, K, T = 48, 200, 512, 6
    p = wl.make_problem(M, N, K, T, seed=15, multi_tenant=True, y_dtype="f32")
    log("tenant invariants")
    y = host_out(run_matmul(p))
    # permuting rows with their ids permutes the output
    perm = rng.permutation(M)
    q = wl.Problem("perm", p.x[perm], p.w, p.alpha, packed=p.packed, tenant_ids=p.tenant_ids[perm],
                   y_dtype="f32")
    np.testing.assert_allclose(host_out(run_matmul(q)), y[perm], rtol=1e-6, atol=1e-6)
    # identical tenants == the single-tenant form
    same = wl.Problem("same", p.x, p.w, np.repeat(p.alpha[:1], T), packed=np.repeat(p.packed[:1], T, 0),
                      tenant_ids=p.tenant_ids, y_dtype="f32")
    single = wl.Problem("single", p.x, p.w, p.alpha[:1], packed=p.packed[:1], y_dtype="f32")
    np.testing.assert_allclose(host_out(run_matmul(same)), host_out(run_matmul(single)),
                               rtol=1e-6, atol=1e-6)
    # out-of-range ids -> NaN rows, the others unchanged
    bad = p.tenant_ids.copy()
    bad[[0, 7, 47]] = [-1, T, 1 << 30]
    r = wl.Problem("bad", p.x, p.w, p.alpha, packed=p.packed, tenant_ids=bad, y_dtype="f32")
    yb = host_out(run_matmul(r))
    assert np.all(np.isnan(yb[[0, 7, 47]]))
    keep = np.setdiff1d(np.arange(M), [0, 7, 47])
    np.testing.assert_array_equal(yb[keep], y[keep])


def test_all_rows_one_tenant_matches_single_path():
    p = wl.make_problem(20, 77, 256, 4, seed=16, multi_tenant=True, y_dtype="f32")
    p.tenant_ids = np.full(20, 2, np.int32)
    log("all rows on tenant 2")
    y = host_out(run_matmul(p))
    s = wl.Problem("t2", p.x, p.w, p.alpha[2:3], packed=p.packed[2:3], y_dtype="f32")
    np.testing.assert_allclose(y, host_out(run_matmul(s)), rtol=1e-6, atol=1e-6)


# ------------------------------------------- batched form: grouped fused GEMM

def _grouped(p, yd=None):
    return host_out(run_matmul(p, path=PREFILL, y_dtype=yd))


@pytest.mark.parametrize("M,N,K,T", [(65, 300, 128, 3), (300, 520, 576, 8), (513, 1000, 128, 17),
                                     (1000, 257, 256, 2), (257, 255, 64, 5), (700, 70, 640, 40),
                                     (2048, 300, 128, 1), (600, 513, 1088, 300)])
@pytest.mark.parametrize("yd", ["f32", "bf16"])
def test_grouped_prefill_ragged(M, N, K, T, yd):
    p = wl.make_problem(M, N, K, T, seed=M + 3 * N + K + T, multi_tenant=True, y_dtype=yd)
    log(f"grouped prefill M={M} N={N} K={K} T={T} {yd} present={len(np.unique(p.tenant_ids))}")
    y = _grouped(p)
    check(y, oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)


@pytest.mark.parametrize("ids", ["prompts", "sorted", "one-of-eight", "big-tenant"])
def test_grouped_prefill_equals_single_tenant_runs(ids):
    # every row of tenant t gets exactly what the single-tenant fused kernel
    # gives for that row with (alpha_t, S_t): same arithmetic, bit for bit
    M, N, K, T = 900, 520, 256, 8
    p = wl.make_problem(M, N, K, T, seed=21, multi_tenant=True, y_dtype="bf16")
    rng = np.random.default_rng(22)
    if ids == "prompts":
        p.tenant_ids = wl.prompt_tenant_ids(rng, M, T, 6)
    elif ids == "sorted":
        p.tenant_ids = np.sort(p.tenant_ids)
    elif ids == "one-of-eight":
        p.tenant_ids = np.full(M, 5, np.int32)
    else:
        p.tenant_ids = np.where(rng.random(M) < 0.9, 2, rng.integers(0, T, M)).astype(np.int32)
    log(f"grouped == per-tenant single runs, ids={ids}")
    y = run_matmul(p, path=PREFILL)
    t = torch()
    for ten in np.unique(p.tenant_ids):
        rows = np.nonzero(p.tenant_ids == ten)[0]
        q = wl.Problem("one", p.x[rows], p.w, p.alpha[ten:ten + 1], packed=p.packed[ten:ten + 1],
                       y_dtype="bf16")
        ys = run_matmul(q, path=PREFILL)
        assert t.equal(y[t.from_numpy(rows).cuda()].view(t.int16), ys.view(t.int16)), ten


def test_grouped_prefill_invalid_ids_nan_rows():
    M, N, K, T = 400, 300, 192, 4
    p = wl.make_problem(M, N, K, T, seed=23, multi_tenant=True, y_dtype="f32")
    log("grouped prefill invalid ids")
    y = _grouped(p)
    bad = p.tenant_ids.copy()
    idx = [0, 1, 255, 256, 399]
    bad[idx] = [-1, T, 1 << 30, -(1 << 31), T + 7]
    r = wl.Problem("bad", p.x, p.w, p.alpha, packed=p.packed, tenant_ids=bad, y_dtype="f32")
    yb = _grouped(r)
    assert np.all(np.isnan(yb[idx]))
    keep = np.setdiff1d(np.arange(M), idx)
    np.testing.assert_array_equal(yb[keep], y[keep])
    # every id invalid: all rows NaN
    r.tenant_ids = np.full(M, -3, np.int32)
    assert np.all(np.isnan(_grouped(r)))


@pytest.mark.parametrize("T", [1, 3])
def test_grouped_prefill_effective_weight_exact(T):
    # one-hot rows spread over the tenants: y[row, n] = bf16_rne(W[n,k] + s_t[n,k] alpha_t)
    K, N = 384, 264
    base = wl.make_problem(1, N, K, T, seed=24)
    cols = np.arange(K)
    rows = np.concatenate([cols] * 2)  # 768 rows: several tiles per tenant
    x = np.zeros((len(rows), K), np.uint16)
    x[np.arange(len(rows)), rows] = 0x3F80
    tid = np.random.default_rng(25).integers(0, T, len(rows)).astype(np.int32)
    p = wl.Problem("onehot-grouped", x, base.w, base.alpha, packed=base.packed, tenant_ids=tid,
                   y_dtype="f32")
    log(f"grouped effective-weight rounding T={T}")
    y = _grouped(p)
    ref = np.empty_like(y)
    wv = wl.bf16_bits_to_f32(p.w)
    for ten in range(T):
        s = oracle.unpack(p.packed[ten], K)  # [N, K]
        a = np.float32(p.alpha[ten])
        eff = (wv + np.where(s > 0, a, -a).astype(np.float32)).astype(np.float32)
        effb = wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(eff))  # [N, K]
        sel = np.nonzero(tid == ten)[0]
        ref[sel] = effb[:, rows[sel]].T
    assert np.array_equal(y, ref)


def _prompt_problem(M, N, K, T, yd, seed, prompts, dtype="bf16"):
    p = wl.make_problem(M, N, K, T, seed=seed, multi_tenant=True, y_dtype=yd, dtype=dtype)
    p.tenant_ids = wl.prompt_tenant_ids(np.random.default_rng(seed + 1), M, T, prompts)
    tiles = sum(-(-int(c) // 256) for c in np.bincount(p.tenant_ids)) * -(-N // 256)
    return p, tiles


# More output tiles than CUs: the first 256 tiles run whole, the leftover ones
# are split along K over the otherwise idle CUs and a second launch adds the
# chunks' partial sums in chunk order.
@pytest.mark.parametrize("M,N,K,T,yd", [(16640, 1024, 256, 5, "bf16"), (16640, 1024, 256, 5, "f32"),
                                        (8320, 2048, 512, 3, "bf16"), (4096, 4096, 1024, 8, "bf16")])
def test_grouped_prefill_split_tiles(M, N, K, T, yd):
    p, tiles = _prompt_problem(M, N, K, T, yd, seed=M + N + K, prompts=12)
    assert tiles > 256, tiles
    log(f"grouped prefill with split tiles M={M} N={N} K={K} T={T} {yd} tiles={tiles}")
    t = torch()
    y1 = run_matmul(p, path=PREFILL)
    y2 = run_matmul(p, path=PREFILL)
    assert t.equal(y1.view(t.int16), y2.view(t.int16)), "split result differs between calls"
    check(host_out(y1), oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)


def test_grouped_prefill_split_fp16():
    p, tiles = _prompt_problem(8320, 2048, 512, 3, "half", seed=77, prompts=10, dtype="f16")
    assert tiles > 256, tiles
    log(f"grouped prefill with split tiles, fp16, tiles={tiles}")
    y = host_out(run_matmul(p, path=PREFILL))
    ref = oracle.matmul(p.x, p.w, p.packed, p.alpha, p.tenant_ids, dtype="f16")
    check(y, ref, p.x, p.w, p.alpha, p.tenant_ids, dtype="f16")


def test_grouped_prefill_split_then_one_round():
    # on one stream: a call that splits, then calls whose tile upper bound
    # allows a split but whose actual tiles fit one round (the second launch
    # must then leave y alone), then the split call again
    p, tiles = _prompt_problem(4096, 4096, 512, 8, "bf16", seed=31, prompts=16)
    assert tiles > 256, tiles
    q = wl.make_problem(4096, 4096, 512, 200, seed=32, multi_tenant=True, y_dtype="bf16")
    q.tenant_ids = np.repeat(np.array([7, 150], np.int32), 2048)    # 16 row tiles: one round
    log(f"grouped prefill: split ({tiles} tiles), one round (256 tiles), split again")
    t = torch()
    a1 = run_matmul(p, path=PREFILL)
    b = run_matmul(q, path=PREFILL)
    a2 = run_matmul(p, path=PREFILL)
    assert t.equal(a1.view(t.int16), a2.view(t.int16))
    check(host_out(a1), oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)
    rows = np.concatenate([np.arange(0, 4096, 61), [2047, 2048, 4095]])
    check(host_out(b[t.from_numpy(rows).cuda()]), oracle_y(q, rows=rows), q.x, q.w, q.alpha,
          q.tenant_ids[rows], rows=rows)


def test_grouped_prefill_tenant_limit():
    import paper_2609_36800_amd as bd
    M, N, K = 300, 64, 128
    p = wl.make_problem(M, N, K, 2048, seed=26, multi_tenant=True, y_dtype="f32")
    log("grouped prefill T=2048 (limit)")
    check(_grouped(p), oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)
    assert bd.matmul_path(M, N, K, 2048, True) == PREFILL
    assert bd.matmul_path(M, N, K, 2049, True) == SKINNY


def test_grouped_prefill_one_row_per_tenant():
    # 2048 tenants of one row each: every tenant's only tile is a 1-row partial
    # tile, so each wave's class count reaches its largest value (512 tenants
    # of one class per wave), the limit of the packed class-count fields
    M, N, K, T = 2048, 80, 128, 2048
    p = wl.make_problem(M, N, K, T, seed=28, multi_tenant=True, y_dtype="f32")
    p.tenant_ids = np.random.default_rng(29).permutation(T).astype(np.int32)
    log("grouped prefill: 2048 tenants of one row each")
    check(_grouped(p), oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)


def test_grouped_prefill_deterministic():
    p = wl.make_problem(700, 600, 512, 6, seed=27, multi_tenant=True)
    log("grouped prefill determinism")
    t = torch()
    y1 = run_matmul(p, path=PREFILL)
    y2 = run_matmul(p, path=PREFILL)
    assert t.equal(y1.view(t.int16), y2.view(t.int16))


def test_mt_prefill_workload_full():
    p = wl.mt_prefill(seed=0)
    log(f"multi-tenant prefill workload (full output): {p.name}, "
        f"tenants present {len(np.unique(p.tenant_ids))}")
    import paper_2609_36800_amd as bd
    assert bd.matmul_path(p.M, p.N, p.K, p.T, True) == PREFILL
    y = host_out(run_matmul(p))
    check(y, oracle_y(p), p.x, p.w, p.alpha, p.tenant_ids)
