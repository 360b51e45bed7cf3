"""The allocation-free entry point, bitdelta_matmul_noalloc, against
bitdelta_matmul_typed on the same inputs: two calls in a row that use its
scratch array (grouped prefill with output tiles split along K), the second
one smaller, so that what the first call left in the array must not leak into
the second's result."""
import ctypes

import numpy as np
import pytest

import workloads as wl
from gpu_util import dev_f32, dev_half, dev_i32, dev_words, host_out, log, torch
from tolerance import check

pytestmark = pytest.mark.gpu

PATH_AUTO = 0


def call(fn_name, p):
    import paper_2609_36800_amd as bd
    t = torch()
    lib = bd.load_library()
    x, w = dev_half(p.x, p.dtype), dev_half(p.w, p.dtype)
    pk, a, tid = dev_words(p.packed), dev_f32(p.alpha), dev_i32(p.tenant_ids)
    et = bd.F16 if p.dtype == "f16" else bd.BF16
    y = t.empty((p.M, p.N), dtype=t.float16 if p.dtype == "f16" else t.bfloat16, device="cuda")
    stream = ctypes.c_void_p(t.cuda.current_stream().cuda_stream)
    rc = getattr(lib, fn_name)(x.data_ptr(), p.M, p.K, w.data_ptr(), p.N, pk.data_ptr(), a.data_ptr(),
                               tid.data_ptr(), p.T, et, y.data_ptr(), et, PATH_AUTO, stream)
    assert rc == 0, bd.status_string(rc)
    t.cuda.synchronize()
    return y


def prompts_problem(M, N, K, T, seed, prompts):
    p = wl.make_problem(M, N, K, T, seed=seed, multi_tenant=True)
    p.tenant_ids = wl.prompt_tenant_ids(np.random.default_rng(seed + 1), M, T, prompts)
    tiles = sum(-(-int(c) // 256) for c in np.bincount(p.tenant_ids)) * -(-N // 256)
    return p, tiles


def test_noalloc_matches_typed_on_two_calls():
    t = torch()
    first, tiles1 = prompts_problem(4096, 4096, 512, 8, seed=51, prompts=16)
    second, tiles2 = prompts_problem(16640, 1024, 256, 5, seed=52, prompts=12)
    assert tiles1 > 256 and tiles2 > 256, (tiles1, tiles2)   # both split, so both use the scratch
    assert 2 * second.M * second.N * second.K < 2 * first.M * first.N * first.K
    for p, what in ((first, "first call"), (second, "second, smaller call")):
        log(f"no-alloc vs typed, {what}: M={p.M} N={p.N} K={p.K} T={p.T}")
        y_na = call("bitdelta_matmul_noalloc", p)
        y_ty = call("bitdelta_matmul_typed", p)
        # the tolerance bar against the existing entry point's output ...
        check(host_out(y_na), host_out(y_ty), p.x, p.w, p.alpha, p.tenant_ids)
        # ... which the two forms meet exactly: same kernels, same split
        assert t.equal(y_na.view(t.int16), y_ty.view(t.int16)), what


def test_noalloc_decode_and_prefill_paths():
    # the entry point serves every path (only the grouped prefill uses the scratch)
    t = torch()
    for (M, N, K, T) in ((16, 1000, 4096, 4), (300, 520, 576, 3)):
        p = wl.make_problem(M, N, K, T, seed=M + N, multi_tenant=True)
        log(f"no-alloc vs typed: M={M} N={N} K={K} T={T}")
        y_na = call("bitdelta_matmul_noalloc", p)
        y_ty = call("bitdelta_matmul_typed", p)
        assert t.equal(y_na.view(t.int16), y_ty.view(t.int16))
