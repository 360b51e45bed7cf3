"""Out-of-bounds write checks and direct calls of the standard entry point.

Every array of a call (inputs and outputs) is placed inside a larger device
buffer whose bytes on both sides hold a sentinel pattern.  After the call the
sentinels must be intact, the inputs unchanged and the outputs equal to the
oracle's: a kernel that writes one element past y (a 16-byte epilogue store at
a ragged N, a byte store of the packer) or into an input fails here even where
every in-range output is right.  A call only touches what it is given, which
the validity of a rewritten kernel requires along with its equivalence (Section
3.1, the safety condition next to Eq. 1).

The second part calls bitdelta_matmul itself (the bf16 entry point of the
boundary, not the typed or path-selecting variants the other tests use) on the
tiny and decode workloads.
"""
import ctypes

import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_util import host_out, log, torch
from tolerance import check

pytestmark = pytest.mark.gpu

GUARD = 4096          # sentinel bytes on each side (keeps 16-byte alignment)
SENTINEL = 0xA5
SKINNY, PREFILL, AUTO = 1, 2, 0


class Guarded:
    """nbytes of device memory between two GUARD-byte sentinel regions.  The
    payload starts filled with `fill` (bytes) or with the sentinel."""

    def __init__(self, payload: np.ndarray = None, nbytes: int = None):
        t = torch()
        if payload is not None:
            raw = np.ascontiguousarray(payload).view(np.uint8).reshape(-1)
            nbytes = raw.size
        self.nbytes = nbytes
        host = np.full(GUARD + nbytes + GUARD, SENTINEL, dtype=np.uint8)
        if payload is not None:
            host[GUARD:GUARD + nbytes] = raw
        self.initial = host.copy()
        self.buf = t.from_numpy(host).cuda()

    @property
    def ptr(self):
        return self.buf.data_ptr() + GUARD

    def host(self):
        return self.buf.cpu().numpy()

    def payload(self, dtype):
        return self.host()[GUARD:GUARD + self.nbytes].view(dtype)

    def assert_guards(self, name):
        h = self.host()
        lo = np.flatnonzero(h[:GUARD] != SENTINEL)
        hi = np.flatnonzero(h[GUARD + self.nbytes:] != SENTINEL)
        assert lo.size == 0, f"{name}: {lo.size} bytes written before the array (first at -{GUARD - lo[0]})"
        assert hi.size == 0, f"{name}: {hi.size} bytes written past the array (first at +{hi[0]})"

    def assert_unchanged(self, name):
        assert np.array_equal(self.host(), self.initial), f"{name}: input bytes were modified"


def stream():
    t = torch()
    return ctypes.c_void_p(t.cuda.current_stream().cuda_stream)


def to_f64(bits, y_dtype):
    if y_dtype == "f32":
        return bits.view(np.float32).astype(np.float64)
    return (bits.view(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def run_guarded_matmul(p, path, y_dtype):
    import paper_2609_36800_amd as bd
    lib = bd.load_library()
    ins = {"x": Guarded(p.x), "w": Guarded(p.w), "packed": Guarded(p.packed),
           "alpha": Guarded(p.alpha.astype(np.float32))}
    if p.tenant_ids is not None:
        ins["tenant_ids"] = Guarded(p.tenant_ids.astype(np.int32))
    ysize = 4 if y_dtype == "f32" else 2
    y = Guarded(nbytes=p.M * p.N * ysize)
    rc = lib.bitdelta_matmul_with_path(
        ins["x"].ptr, p.M, p.K, ins["w"].ptr, p.N, ins["packed"].ptr, ins["alpha"].ptr,
        ins["tenant_ids"].ptr if "tenant_ids" in ins else None, p.T, y.ptr,
        bd.F32 if y_dtype == "f32" else bd.BF16, path, stream())
    assert rc == 0, bd.status_string(rc)
    torch().cuda.synchronize()
    for name, g in ins.items():
        g.assert_guards(name)
        g.assert_unchanged(name)
    y.assert_guards("y")
    got = to_f64(y.payload(np.float32 if y_dtype == "f32" else np.uint16), y_dtype).reshape(p.M, p.N)
    return got


# (M, N, K, T, multi-tenant, path): each line reaches one kernel of the library
# with a ragged N (and ragged M where the kernel tiles rows)
MATMUL_CASES = [
    (1, 33, 256, 1, False, AUTO),        # streaming decode, x staged up front
    (16, 1001, 4224, 1, False, AUTO),    # streaming decode, x per tile, K above 4096
    (3, 19, 96, 1, False, AUTO),         # general decode (K not a multiple of 128)
    (40, 47, 544, 1, False, AUTO),       # skinny single-tenant kernel
    (40, 100, 512, 5, True, AUTO),       # batched kernel, 8 waves (one round)
    (20, 4100, 256, 5, True, AUTO),      # batched kernel, 4 waves (several rounds)
    (40, 10000, 640, 6, True, AUTO),     # wide batched kernel, 48 features (ragged last group)
    (24, 14300, 384, 8, True, AUTO),     # wide batched kernel, 64 features (ragged last group)
    (8, 70, 128, 20, True, AUTO),        # tenant-slot kernel (more than 16 tenants)
    (10, 50, 96, 3, True, AUTO),         # skinny multi-tenant kernel (K not a multiple of 128)
    (300, 520, 576, 1, False, PREFILL),  # fused prefill, streaming
    (70, 90, 96, 1, False, PREFILL),     # fused prefill, general (K not a multiple of 64)
    (300, 260, 256, 3, True, AUTO),      # grouped fused prefill
    (200, 37, 128, 4, True, SKINNY),     # batched request above 64 rows, 64 rows per launch
]


@pytest.mark.parametrize("M,N,K,T,multi,path", MATMUL_CASES)
@pytest.mark.parametrize("yd", ["bf16", "f32"])
def test_matmul_writes_only_y(M, N, K, T, multi, path, yd):
    p = wl.make_problem(M, N, K, T, seed=M * 3 + N + K + T, multi_tenant=multi, y_dtype=yd)
    if multi:
        p.tenant_ids[::7] = T            # out-of-range ids: those rows become NaN
    log(f"guarded matmul M={M} N={N} K={K} T={T} multi={multi} path={path} {yd}")
    got = run_guarded_matmul(p, path, yd)
    valid = np.ones(M, dtype=bool) if p.tenant_ids is None else (p.tenant_ids < T)
    assert np.all(np.isnan(got[~valid])), "rows with out-of-range tenant ids must be NaN"
    tid = None if p.tenant_ids is None else p.tenant_ids[valid]
    ref = oracle.matmul(p.x[valid], p.w, p.packed, p.alpha, tid)
    check(got[valid], ref, p.x, p.w, p.alpha, tid, rows=np.flatnonzero(valid))


@pytest.mark.parametrize("rows,K", [(1, 32), (7, 96), (33, 544), (130, 4128)])
def test_pack_unpack_write_only_their_outputs(rows, K):
    import paper_2609_36800_amd as bd
    lib = bd.load_library()
    rng = np.random.default_rng(rows + K)
    signs = rng.choice(np.array([-1.0, 1.0], dtype=np.float32), size=(rows, K))
    log(f"guarded pack/unpack rows={rows} K={K}")
    src = Guarded(signs)
    packed = Guarded(nbytes=rows * K // 8)
    assert lib.bitdelta_pack(src.ptr, bd.F32, rows, K, packed.ptr, stream()) == 0
    torch().cuda.synchronize()
    src.assert_guards("signs")
    src.assert_unchanged("signs")
    packed.assert_guards("packed")
    words = packed.payload(np.uint32).reshape(rows, K // 32)
    np.testing.assert_array_equal(words, oracle.pack(signs))
    for code, dt, size in ((bd.F32, np.float32, 4), (bd.BF16, np.uint16, 2), (bd.I8, np.int8, 1)):
        pin = Guarded(words)
        out = Guarded(nbytes=rows * K * size)
        assert lib.bitdelta_unpack(pin.ptr, rows, K, out.ptr, code, stream()) == 0
        torch().cuda.synchronize()
        pin.assert_guards("packed")
        pin.assert_unchanged("packed")
        out.assert_guards(f"signs ({dt.__name__})")
        vals = out.payload(dt).reshape(rows, K)
        if dt is np.uint16:
            vals = to_f64(vals, "bf16")
        np.testing.assert_array_equal(np.asarray(vals, dtype=np.float64),
                                      oracle.unpack(words, K).astype(np.float64))


@pytest.mark.parametrize("rows,K", [(1, 32), (9, 96), (130, 4128)])
def test_compress_writes_only_its_outputs(rows, K):
    import paper_2609_36800_amd as bd
    lib = bd.load_library()
    rng = np.random.default_rng(rows * 5 + K)
    base = wl.normal_bf16(rng, (rows, K), 0.02)
    fine = wl.f32_to_bf16_bits(wl.bf16_bits_to_f32(base)
                               + rng.standard_normal((rows, K)).astype(np.float32) * 5e-4)
    log(f"guarded compress rows={rows} K={K}")
    gf, gb = Guarded(fine), Guarded(base)
    packed, row_abs, alpha = Guarded(nbytes=rows * K // 8), Guarded(nbytes=rows * 4), Guarded(nbytes=4)
    assert lib.bitdelta_compress(gf.ptr, gb.ptr, rows, K, bd.BF16, packed.ptr, row_abs.ptr,
                                 alpha.ptr, stream()) == 0
    torch().cuda.synchronize()
    for name, g in (("w_fine", gf), ("w_base", gb)):
        g.assert_guards(name)
        g.assert_unchanged(name)
    for name, g in (("packed", packed), ("row_abs_sum", row_abs), ("alpha", alpha)):
        g.assert_guards(name)
    p_ref, r_ref, a_ref = oracle.compress(fine, base)
    np.testing.assert_array_equal(packed.payload(np.uint32).reshape(rows, K // 32), p_ref)
    np.testing.assert_allclose(row_abs.payload(np.float32), r_ref, rtol=1e-5)
    np.testing.assert_allclose(alpha.payload(np.float32)[0], a_ref, rtol=1e-5)


# ------------------------------------------------ the standard entry point itself

def call_standard(p):
    """bitdelta_matmul (bf16 x and W, path chosen by the library)."""
    import paper_2609_36800_amd as bd
    t = torch()
    lib = bd.load_library()
    x = t.from_numpy(p.x.view(np.int16)).cuda()
    w = t.from_numpy(p.w.view(np.int16)).cuda()
    pk = t.from_numpy(np.ascontiguousarray(p.packed).view(np.int32)).cuda()
    a = t.from_numpy(p.alpha.astype(np.float32)).cuda()
    tid = None if p.tenant_ids is None else t.from_numpy(p.tenant_ids.astype(np.int32)).cuda()
    y = t.empty((p.M, p.N), dtype=t.float32 if p.y_dtype == "f32" else t.bfloat16, device="cuda")
    rc = lib.bitdelta_matmul(x.data_ptr(), p.M, p.K, w.data_ptr(), p.N, pk.data_ptr(), a.data_ptr(),
                             None if tid is None else tid.data_ptr(), p.T, y.data_ptr(),
                             bd.F32 if p.y_dtype == "f32" else bd.BF16, stream())
    assert rc == 0, bd.status_string(rc)
    t.cuda.synchronize()
    return host_out(y)


def test_standard_entry_point_tiny():
    p = wl.tiny(seed=0)
    p.packed = np.stack([oracle.pack(s) for s in p.signs])
    log(f"bitdelta_matmul: {p.name}")
    got = call_standard(p)
    relf, _ = check(got, oracle.matmul(p.x, p.w, p.packed, p.alpha), p.x, p.w, p.alpha)
    assert relf < 1e-5, relf          # fp32 output, decode path: the sums are kept apart


@pytest.mark.parametrize("M", [1, 16])
def test_standard_entry_point_decode(M):
    p = wl.decode(M, seed=0)
    log(f"bitdelta_matmul: {p.name}")
    got = call_standard(p)
    check(got, oracle.matmul(p.x, p.w, p.packed, p.alpha), p.x, p.w, p.alpha)


def test_standard_entry_point_multi_tenant():
    p = wl.make_problem(32, 700, 1024, 16, seed=3, multi_tenant=True)
    log("bitdelta_matmul: 32 rows, 16 tenants, 700x1024")
    got = call_standard(p)
    check(got, oracle.matmul(p.x, p.w, p.packed, p.alpha, p.tenant_ids), p.x, p.w, p.alpha,
          p.tenant_ids)
