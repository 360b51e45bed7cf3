"""Parity of the streaming decode kernel (one tenant, up to 16 rows, K a
multiple of 128 up to 16384) with the fp64 oracle.

The kernel streams W in 256-k tiles through a ring six tiles deep and never
issues a tile past the end of K: the last tiles run with waits that count only
the real tiles still in flight.  The cases cover K with fewer tiles than the
ring (128, 384), a last tile half full (384, 1152, 4224), K above 4096 (x then
copied per tile for every row count, and the larger sign staging area) and the
largest K, for each way x reaches LDS (one row or up to four rows staged up
front, sixteen rows per tile), ragged N, and fp16.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_util import log, host_out, run_matmul
from tolerance import check

pytestmark = pytest.mark.gpu

SKINNY = 1


@pytest.mark.parametrize("K", [128, 384, 1152, 2048, 4224, 16384])
@pytest.mark.parametrize("M", [1, 3, 16])
def test_stream_decode_k_range(M, K):
    N = 40 if K < 16384 else 24
    p = wl.make_problem(M, N, K, 1, seed=M * 31 + K, y_dtype="f32")
    log(f"stream decode M={M} N={N} K={K}")
    y = host_out(run_matmul(p, path=SKINNY))
    relf, _ = check(y, oracle.matmul(p.x, p.w, p.packed, p.alpha), p.x, p.w, p.alpha)
    assert relf < 1e-5, relf


@pytest.mark.parametrize("M,N,K", [(1, 17, 640), (16, 33, 896), (4, 1000, 1280)])
def test_stream_decode_ragged_n_bf16_out(M, N, K):
    p = wl.make_problem(M, N, K, 1, seed=M + N + K, y_dtype="bf16")
    log(f"stream decode bf16 out M={M} N={N} K={K}")
    y = host_out(run_matmul(p, path=SKINNY))
    check(y, oracle.matmul(p.x, p.w, p.packed, p.alpha), p.x, p.w, p.alpha)


@pytest.mark.parametrize("M,K", [(1, 384), (16, 1152)])
def test_stream_decode_f16(M, K):
    p = wl.make_problem(M, 40, K, 1, seed=M + K + 5, y_dtype="f32", dtype="f16")
    log(f"stream decode f16 M={M} K={K}")
    y = host_out(run_matmul(p, path=SKINNY))
    relf, _ = check(y, oracle.matmul(p.x, p.w, p.packed, p.alpha, dtype="f16"), p.x, p.w, p.alpha,
                    dtype="f16")
    assert relf < 1e-5, relf


def test_stream_decode_ones_zero_weight_exact():
    # x = 1, W = 0: y[m, n] = alpha * (2 popcount(S[n]) - K) exactly
    rng = np.random.default_rng(21)
    M, N, K = 16, 40, 1152
    packed = wl.uniform_words(rng, (1, N, K // 32))
    alpha = np.array([0.5], np.float32)
    p = wl.Problem("ones", np.full((M, K), 0x3F80, np.uint16), np.zeros((N, K), np.uint16),
                   alpha, packed=packed, y_dtype="f32")
    log("stream decode ones/zero-weight exact")
    y = host_out(run_matmul(p, path=SKINNY))
    pc = np.array([sum(int(v).bit_count() for v in packed[0, n]) for n in range(N)])
    assert np.array_equal(y, np.broadcast_to(0.5 * (2 * pc - K), (M, N)))
