"""Pack / unpack on the GPU: bit-exact against the oracle and numpy."""
import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_util import dev_words, host_words, log, torch

pytestmark = pytest.mark.gpu


def _dev(a):
    t = torch()
    if a.dtype == np.uint16:
        return t.from_numpy(a.view(np.int16)).view(t.bfloat16).cuda()
    return t.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("rows,K", [(1, 32), (3, 96), (512, 256), (37, 4096), (4096, 4096),
                                    (11008, 4096 // 32 * 32), (5, 11008)])
@pytest.mark.parametrize("dtype", ["f32", "i8", "bf16"])
def test_pack_matches_oracle(rows, K, dtype):
    import paper_2609_36800_amd as bd
    log(f"pack rows={rows} K={K} {dtype}")
    rng = np.random.default_rng(rows + K)
    s = wl.random_signs_i8(rng, (rows, K))
    if dtype == "f32":
        s = s.astype(np.float32)
    elif dtype == "bf16":
        s = wl.f32_to_bf16_bits(s.astype(np.float32))
    got = host_words(bd.pack(_dev(s)))
    torch().cuda.synchronize()
    np.testing.assert_array_equal(got, oracle.pack(s))


def test_pack_special_values():
    import paper_2609_36800_amd as bd
    log("pack special values")
    f = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, -np.nan, 1e-45, -1e-45,
                  3.5, -3.5, 1e38, -1e38] + [1.0, -1.0] * 10, dtype=np.float32)[None]
    f = np.repeat(f, 3, axis=0)
    np.testing.assert_array_equal(host_words(bd.pack(_dev(f))), oracle.pack(f))
    i8 = np.arange(-128, 128, dtype=np.int16).astype(np.int8).reshape(8, 32)
    np.testing.assert_array_equal(host_words(bd.pack(_dev(i8))), oracle.pack(i8))
    bits = np.arange(0, 65536, 64, dtype=np.uint16).reshape(32, 32)
    np.testing.assert_array_equal(host_words(bd.pack(_dev(bits))), oracle.pack(bits))


@pytest.mark.parametrize("rows,K", [(1, 32), (7, 160), (4096, 4096), (3, 11008)])
@pytest.mark.parametrize("dtype", ["f32", "i8", "bf16"])
def test_unpack_matches_oracle(rows, K, dtype):
    import paper_2609_36800_amd as bd
    t = torch()
    log(f"unpack rows={rows} K={K} {dtype}")
    rng = np.random.default_rng(rows * 7 + K)
    words = wl.uniform_words(rng, (rows, K // 32))
    tdt = {"f32": t.float32, "i8": t.int8, "bf16": t.bfloat16}[dtype]
    out = bd.unpack(dev_words(words), K, tdt)
    got = out.float().cpu().numpy().astype(np.float64)
    np.testing.assert_array_equal(got, oracle.unpack(words, K))
    # round trip on the device: pack(unpack(w)) == w
    np.testing.assert_array_equal(host_words(bd.pack(out)), words)


def test_empty_pack_is_noop():
    import paper_2609_36800_amd as bd
    t = torch()
    out = t.full((0, 1), 7, dtype=t.int32, device="cuda")
    bd.pack(t.empty((0, 32), dtype=t.float32, device="cuda"), out=out)
    t.cuda.synchronize()
