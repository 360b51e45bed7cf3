"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects bad arguments on the host before any launch."""
import ctypes
import os
import re

import pytest

import paper_2609_36800_amd as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bitdelta.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bitdelta_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(bd.LIB_PATH):
        pytest.fail("libbitdelta.so is not built (run __graft_entry__.build())")
    return bd.load_library()


def test_header_declares_expected_api():
    assert set(header_functions()) == set(bd.EXPORTED)


def test_library_exports_every_header_symbol(lib):
    for name in header_functions():
        assert hasattr(lib, name), name


def test_no_oracle_symbols_in_library():
    # the product library must not contain (or link) the test oracle
    data = open(bd.LIB_PATH, "rb").read()
    assert b"oracle_" not in data


def test_version_and_status_strings(lib):
    assert lib.bitdelta_version() >= 100
    for code in range(-8, 1):
        s = bd.status_string(code)
        assert s and s != "unknown status"
    assert bd.status_string(-99) == "unknown status"


# Fake, well-aligned device addresses: every call below must fail its host
# checks (or be a no-op) before anything could dereference them.
A = 0x10000000
B = 0x20000000
C = 0x30000000
D = 0x40000000
E = 0x50000000


def mm(lib, x=A, M=4, K=64, w=B, N=8, p=C, alpha=D, tid=None, T=1, y=E, yd=bd.BF16,
       path=bd.PATH_AUTO):
    return lib.bitdelta_matmul_with_path(x, M, K, w, N, p, alpha, tid, T, y, yd, path, None)


def test_matmul_shape_errors(lib):
    assert mm(lib, K=48) == -2            # K % 32
    assert mm(lib, M=-1) == -2
    assert mm(lib, N=-3) == -2
    assert mm(lib, K=-32) == -2
    assert mm(lib, T=0) == -2
    assert mm(lib, M=1 << 31) == -2


def test_matmul_null_errors(lib):
    assert mm(lib, x=None) == -1
    assert mm(lib, w=None) == -1
    assert mm(lib, p=None) == -1
    assert mm(lib, alpha=None) == -1
    assert mm(lib, y=None) == -1


def test_matmul_alignment_errors(lib):
    assert mm(lib, x=A + 2) == -3
    assert mm(lib, w=B + 8) == -3
    assert mm(lib, y=E + 4) == -3
    assert mm(lib, p=C + 2) == -3
    assert mm(lib, alpha=D + 1) == -3
    assert mm(lib, tid=D + 0x1000 + 2) == -3


def test_matmul_dtype_and_path_errors(lib):
    assert mm(lib, yd=bd.I8) == -4
    assert mm(lib, yd=7) == -4
    assert mm(lib, path=9) == -5
    # the grouped fused GEMM needs K a multiple of 64 and at most 2048 tenants
    assert mm(lib, K=96, tid=0x60000000, path=bd.PATH_PREFILL) == -5
    assert mm(lib, T=2049, tid=0x60000000, path=bd.PATH_PREFILL) == -5


def test_matmul_alias_errors(lib):
    # y overlapping x, w, packed, alpha or tenant ids
    assert mm(lib, y=A) == -7
    assert mm(lib, y=B + 256) == -7
    assert mm(lib, y=C) == -7
    assert mm(lib, y=D) == -7
    assert mm(lib, tid=0x60000000, y=0x60000000) == -7


def test_matmul_empty_is_noop(lib):
    assert mm(lib, M=0) == 0
    assert mm(lib, N=0) == 0
    assert mm(lib, M=0, x=None, y=None) == 0


def test_pack_unpack_errors(lib):
    assert lib.bitdelta_pack(A, bd.F32, 4, 48, B, None) == -2
    assert lib.bitdelta_pack(A, bd.F32, -1, 32, B, None) == -2
    assert lib.bitdelta_pack(A, 5, 4, 32, B, None) == -4
    assert lib.bitdelta_pack(None, bd.F32, 4, 32, B, None) == -1
    assert lib.bitdelta_pack(A, bd.F32, 4, 32, None, None) == -1
    assert lib.bitdelta_pack(A + 4, bd.F32, 4, 32, B, None) == -3   # f32 needs 16 B
    assert lib.bitdelta_pack(A + 4, bd.BF16, 4, 32, B, None) == -3   # bf16 needs 8 B
    assert lib.bitdelta_pack(A + 2, bd.I8, 4, 32, B, None) == -3    # i8 needs 4 B
    assert lib.bitdelta_pack(A, bd.F32, 4, 32, B + 2, None) == -3
    assert lib.bitdelta_pack(A, bd.F32, 4, 32, A + 64, None) == -7  # output inside input
    assert lib.bitdelta_pack(A, bd.F32, 0, 32, B, None) == 0
    assert lib.bitdelta_unpack(A, 4, 40, B, bd.F32, None) == -2
    assert lib.bitdelta_unpack(A, 4, 32, B, 9, None) == -4
    assert lib.bitdelta_unpack(None, 4, 32, B, bd.F32, None) == -1
    assert lib.bitdelta_unpack(A, 4, 32, B + 8, bd.F32, None) == -3
    assert lib.bitdelta_unpack(A, 4, 32, A, bd.F32, None) == -7
    assert lib.bitdelta_unpack(A, 4, 0, B, bd.F32, None) == 0


def test_compress_errors(lib):
    F, Bs, Pk, R, Al = A, B, C, D, E

    def cp(f, b, rows, K, pk, r, al, dt=bd.BF16):
        return lib.bitdelta_compress(f, b, rows, K, dt, pk, r, al, None)
    assert cp(F, Bs, 4, 48, Pk, R, Al) == -2        # K % 32
    assert cp(F, Bs, -1, 32, Pk, R, Al) == -2
    assert cp(F, Bs, 4, -32, Pk, R, Al) == -2
    assert cp(F, Bs, 4, 32, Pk, R, Al, dt=bd.F32) == -4
    assert cp(F, Bs, 4, 32, Pk, R, Al, dt=bd.I8) == -4
    assert cp(None, Bs, 4, 32, Pk, R, Al) == -1
    assert cp(F, None, 4, 32, Pk, R, Al) == -1
    assert cp(F, Bs, 4, 32, None, R, Al) == -1
    assert cp(F, Bs, 4, 32, Pk, None, Al) == -1      # row sums are required
    assert cp(F + 8, Bs, 4, 32, Pk, R, Al) == -3
    assert cp(F, Bs + 2, 4, 32, Pk, R, Al) == -3
    assert cp(F, Bs, 4, 32, Pk + 2, R, Al) == -3
    assert cp(F, Bs, 4, 32, Pk, R + 1, Al) == -3
    assert cp(F, Bs, 4, 32, Pk, R, Al + 2) == -3
    assert cp(F, Bs, 4, 32, F + 64, R, Al) == -7     # packed inside w_fine
    assert cp(F, Bs, 4, 32, Pk, Pk, Al) == -7        # row sums over packed
    assert cp(F, Bs, 4, 32, Pk, R, R) == -7          # alpha over row sums
    assert cp(F, Bs, 0, 32, Pk, R, Al) == 0
    assert cp(F, Bs, 4, 0, Pk, R, Al, dt=bd.F16) == 0


def test_typed_matmul_dtype_errors(lib):
    def mt(in_dt, y_dt):
        return lib.bitdelta_matmul_typed(A, 4, 64, B, 8, C, D, None, 1, in_dt, E, y_dt,
                                         bd.PATH_AUTO, None)
    assert mt(bd.F32, bd.F32) == -4          # inputs are 16-bit
    assert mt(bd.I8, bd.F32) == -4
    assert mt(bd.F16, bd.BF16) == -4         # a 16-bit output has the input type
    assert mt(bd.BF16, bd.F16) == -4
    assert mt(7, bd.F32) == -4
    assert lib.bitdelta_matmul_typed(A, 0, 64, B, 8, C, D, None, 1, bd.F16, E, bd.F16,
                                     bd.PATH_AUTO, None) == 0


def test_path_selection(lib):
    assert bd.matmul_path(1, 4096, 4096, 1, False) == bd.PATH_SKINNY
    assert bd.matmul_path(64, 4096, 4096, 1, False) == bd.PATH_SKINNY
    assert bd.matmul_path(65, 4096, 4096, 1, False) == bd.PATH_PREFILL
    assert bd.matmul_path(4096, 4096, 4096, 1, False) == bd.PATH_PREFILL
    assert bd.matmul_path(32, 11008, 4096, 16, True) == bd.PATH_SKINNY
    assert bd.matmul_path(255, 4096, 4096, 8, True) == bd.PATH_SKINNY
    assert bd.matmul_path(256, 4096, 4096, 8, True) == bd.PATH_PREFILL
    assert bd.matmul_path(4096, 4096, 4096, 8, True) == bd.PATH_PREFILL
    assert bd.matmul_path(4096, 4096, 4000, 8, True) == bd.PATH_SKINNY   # K % 64
    assert bd.matmul_path(4096, 4096, 4096, 2049, True) == bd.PATH_SKINNY


# The binding checks every shape before a pointer reaches the library (which
# sees raw pointers only and cannot tell an undersized buffer): a wrong shape
# raises ValueError before the device checks, so CPU tensors suffice here.

def _t():
    import torch
    return torch


def test_binding_matmul_rejects_bad_out_shape():
    t = _t()
    x = t.zeros((4, 64), dtype=t.bfloat16)
    w = t.zeros((8, 64), dtype=t.bfloat16)
    p = t.zeros((1, 8, 2), dtype=t.int32)
    a = t.zeros((1,), dtype=t.float32)
    for shape in [(4, 7), (3, 8), (32,), (4, 8, 1)]:
        with pytest.raises(ValueError, match="out has shape"):
            bd.matmul(x, w, p, a, out=t.zeros(shape, dtype=t.bfloat16))


def test_binding_matmul_rejects_bad_operand_shapes():
    t = _t()
    x = t.zeros((4, 64), dtype=t.bfloat16)
    w = t.zeros((8, 64), dtype=t.bfloat16)
    a = t.zeros((2,), dtype=t.float32)
    with pytest.raises(ValueError, match="shape mismatch"):
        bd.matmul(x, w, t.zeros((2, 8, 3), dtype=t.int32), a)          # K/32 words
    with pytest.raises(ValueError, match="shape mismatch"):
        bd.matmul(x, w, t.zeros((1, 8, 2), dtype=t.int32), a)          # T from alpha
    with pytest.raises(ValueError, match="shape mismatch"):
        bd.matmul(x, t.zeros((8, 96), dtype=t.bfloat16), t.zeros((2, 8, 2), dtype=t.int32), a)
    with pytest.raises(ValueError, match="shape mismatch"):
        bd.matmul(t.zeros((4, 48), dtype=t.bfloat16), t.zeros((8, 48), dtype=t.bfloat16),
                  t.zeros((2, 8, 1), dtype=t.int32), a)                 # K % 32
    with pytest.raises(ValueError, match="one entry per row"):
        bd.matmul(x, w, t.zeros((2, 8, 2), dtype=t.int32), a, tenant_ids=t.zeros((5,), dtype=t.int32))
    with pytest.raises(ValueError, match="2-D"):
        bd.matmul(x[None], w, t.zeros((2, 8, 2), dtype=t.int32), a)


def test_binding_pack_unpack_reject_bad_shapes():
    t = _t()
    with pytest.raises(ValueError, match="out has shape"):
        bd.pack(t.zeros((4, 64)), out=t.zeros((4, 1), dtype=t.int32))
    with pytest.raises(ValueError, match="out has shape"):
        bd.pack(t.zeros((4, 64)), out=t.zeros((3, 2), dtype=t.int32))
    with pytest.raises(ValueError, match="multiple of 32"):
        bd.pack(t.zeros((4, 48)))
    with pytest.raises(ValueError, match="rows, K"):
        bd.pack(t.zeros((256,)))
    packed = t.zeros((4, 2), dtype=t.int32)
    with pytest.raises(ValueError, match="words per row"):
        bd.unpack(packed, 96)                 # would read past packed
    with pytest.raises(ValueError, match="words per row"):
        bd.unpack(packed, 32)                 # would decode rows wrongly
    with pytest.raises(ValueError, match="out has shape"):
        bd.unpack(packed, 64, out=t.zeros((4, 32)))
    with pytest.raises(ValueError, match="out has shape"):
        bd.unpack(packed, 64, out=t.zeros((5, 64)))


def test_binding_compress_rejects_bad_shapes():
    t = _t()
    with pytest.raises(ValueError, match="same shape"):
        bd.compress(t.zeros((4, 64), dtype=t.bfloat16), t.zeros((4, 32), dtype=t.bfloat16))
    with pytest.raises(ValueError, match="multiple of 32"):
        bd.compress(t.zeros((4, 48), dtype=t.bfloat16), t.zeros((4, 48), dtype=t.bfloat16))


def test_plain_matmul_entry_host_errors(lib):
    # bitdelta_matmul itself (automatic path, bf16 inputs): same host checks
    def pm(x=A, M=4, K=64, w=B, N=8, p=C, alpha=D, tid=None, T=1, y=E, yd=bd.BF16):
        return lib.bitdelta_matmul(x, M, K, w, N, p, alpha, tid, T, y, yd, None)
    assert pm(K=48) == -2
    assert pm(M=-1) == -2
    assert pm(T=0) == -2
    assert pm(x=None) == -1
    assert pm(y=None) == -1
    assert pm(alpha=None) == -1
    assert pm(x=A + 2) == -3
    assert pm(tid=D + 0x1000 + 2) == -3
    assert pm(yd=bd.I8) == -4
    assert pm(yd=bd.F16) == -4            # bf16 inputs: a 16-bit output is bf16
    assert pm(y=B + 64) == -7
    assert pm(M=0) == 0
    assert pm(N=0, y=None) == 0


def test_library_shares_torchs_hip_runtime():
    # Loading the library before torch must not leave two HIP runtimes in the
    # process (the library's launches on torch's memory fail if it does).
    import subprocess
    import sys
    code = ("import paper_2609_36800_amd as bd; bd.load_library(); import torch; "
            "maps = open('/proc/self/maps').read(); "
            "print(len({l.split()[-1] for l in maps.splitlines() if 'libamdhip64' in l}))")
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True,
                         timeout=300)
    assert out.returncode == 0, out.stderr[-2000:]
    assert out.stdout.strip().splitlines()[-1] == "1", out.stdout
