"""8-bit (E4M3) sparse values on the GPU, through the C ABI, against the oracle.

The page values are compared code for code (bit-exact), the indices and the
fp16 ring bit for bit, and decode outputs within 2e-3 (max |o - o_ref| /
max |o_ref| per query head), as for fp16 values.
"""
import sys

import numpy as np
import pytest

from oracle import swan_oracle as O
from tests import swan_cases as C
from tests.test_gpu_parity import TOL, _build, _decode_check

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _finite_fp16_rows():
    """Every finite fp16 bit pattern once, as 496 rows of 128 (63488 values)."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    x = bits.view(np.float16)
    x = x[np.isfinite(x)]
    assert x.size == 496 * 128
    return x.reshape(496, 128)


@pytest.mark.parametrize("single_appends", [False, True])
def test_e4m3_codes_of_every_fp16_value(gpu_device, swan_mod, torch_mod, single_appends):
    """P = identity, k = 128, b = 0: every token is pruned on arrival with all of its
    components kept, so the pages hold the E4M3 code of every input value: all finite
    fp16 values, through the prefill kernel (one append) or the decode-step insert
    (one token per append)."""
    torch = torch_mod
    _log(f"e4m3 codes of every fp16 value, single appends={single_appends}")
    X = _finite_fp16_rows()
    n = X.shape[0]
    eye = torch.eye(128, dtype=torch.float32, device=gpu_device)[None].contiguous()
    cache = swan_mod.SwanCache(1, 1, 1, 0, n, [128], torch.float16, gpu_device,
                               sparse_values="e4m3")
    xk = torch.tensor(X[None, None], device=gpu_device)
    xv = torch.tensor(X[None, None, ::-1].copy(), device=gpu_device)
    if single_appends:
        for t in range(n):
            cache.append(xk[:, :, t:t + 1].contiguous(), xv[:, :, t:t + 1].contiguous(), eye, eye)
    else:
        cache.append(xk, xv, eye, eye)
    torch.cuda.synchronize()
    for role, rows in ((0, X), (1, X[::-1])):
        idx, val, _, _ = C.unit_pages(cache, 0, 0, role, n, np.uint8)
        assert np.array_equal(idx, np.tile(np.arange(128), (n, 1)))
        # the stored value is the rotation by the identity, rounded to fp16: the
        # input itself, except that -0 becomes +0 (it is summed with +0 products)
        stored = O.to_storage(O.rotate(rows, np.eye(128)), np.float16)
        want = O.to_e4m3_codes(stored)
        bad = np.nonzero(val != want)
        assert bad[0].size == 0, (f"role {role}: {bad[0].size} codes differ, e.g. "
                                  f"fp16 {rows[bad][:4]} -> {val[bad][:4]} vs {want[bad][:4]}")


@pytest.mark.parametrize("L,b,k", [
    (1, 0, 48), (130, 0, 48), (200, 16, 1), (200, 16, 128), (333, 64, 13), (300, 16, 96),
    (129, 3, 5), (40, 64, 48),
])
def test_e4m3_compress_bit_exact(gpu_device, swan_mod, torch_mod, L, b, k):
    _log(f"e4m3 compress L={L} b={b} k={k}")
    cache, oc, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=2, Hkv=2, L=L, b=b,
                           k_active=[k, k], dtype="f16", values="e4m3")
    for bi in range(2):
        for h in range(2):
            C.compare_unit(cache, oc[bi][h], bi, h, L, np.float16, values="e4m3")


@pytest.mark.parametrize("chunks", [[1] * 150, [7, 1, 64, 13, 65]])
def test_e4m3_chunked_appends(gpu_device, swan_mod, torch_mod, chunks):
    _log(f"e4m3 chunks={chunks[:6]}")
    L = sum(chunks)
    cache, oc, *_ = _build(swan_mod, torch_mod, gpu_device, B=1, Hq=1, Hkv=1, L=L, b=16,
                           k_active=[24], dtype="f16", chunks=chunks, values="e4m3")
    C.compare_unit(cache, oc[0][0], 0, 0, L, np.float16, values="e4m3")


@pytest.mark.parametrize("L,b,k,Hq,Hkv", [
    (1, 16, 48, 4, 4), (700, 128, 48, 4, 4), (2049, 128, 64, 8, 2), (1000, 16, 128, 2, 2),
    (513, 5, 3, 2, 1), (1500, 64, 48, 16, 2), (900, 32, 32, 32, 2), (600, 16, 24, 6, 2),
])
def test_e4m3_decode_matches_oracle(gpu_device, swan_mod, torch_mod, L, b, k, Hq, Hkv):
    _log(f"e4m3 decode L={L} b={b} k={k} Hq={Hq} Hkv={Hkv}")
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=Hq,
                                                Hkv=Hkv, L=L, b=b, k_active=[k, k], dtype="f16",
                                                values="e4m3")
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, "f16")


def test_e4m3_ragged_batch_many_k(gpu_device, swan_mod, torch_mod):
    B = 24
    Ls = [1 + (53 * i) % 400 for i in range(B)]
    ks = [1 + (11 * i) % 128 for i in range(B)]
    _log(f"e4m3 ragged batch B={B}")
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=B, Hq=4,
                                                Hkv=2, L=Ls, b=16, k_active=ks, dtype="f16",
                                                capacity=400, values="e4m3")
    for bi in range(0, B, 5):
        C.compare_unit(cache, oc[bi][1], bi, 1, Ls[bi], np.float16, values="e4m3")
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, "f16")
