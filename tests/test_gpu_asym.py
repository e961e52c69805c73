"""Keys and values pruned to different k (the key/value ablation of Appendix A.5,
Table 2), on the GPU through the C ABI, against the oracle.

Compress: indices and stored values bit-exact for each role with its own k.
Decode: outputs within 2e-3 (max |o - o_ref| / max |o_ref| per query head).  A
sequence whose keys and values have different k_pad takes the decode kernels
specialised on the larger k_pad, with each role's own page size and group count;
one whose k differ within the same k_pad, the equal-k_pad kernels; a batch can
mix all of them.
"""
import sys

import numpy as np
import pytest

import swan_inputs as si
from oracle import swan_oracle as O
from tests import swan_cases as C
from tests.test_gpu_parity import TOL, _build, _decode_check

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _dt(fmt):
    """(storage dtype, sparse values) of a test format name."""
    return ("f16", "e4m3") if fmt == "e4m3" else (fmt, "same")


@pytest.mark.parametrize("fmt,L,b,kk,kv", [
    ("f16", 300, 16, 77, 51), ("f16", 200, 0, 13, 115), ("f16", 130, 16, 128, 1),
    ("f32", 300, 16, 64, 24), ("e4m3", 300, 16, 77, 51), ("e4m3", 129, 0, 96, 8),
    # the prefill kernel's page copy: one LDS round for k_pad 88, two for 96
    ("f16", 300, 16, 88, 96), ("f16", 300, 16, 96, 88),
])
def test_asym_compress_bit_exact(gpu_device, swan_mod, torch_mod, fmt, L, b, kk, kv):
    _log(f"asym compress fmt={fmt} L={L} b={b} k_key={kk} k_value={kv}")
    dtype, vals = _dt(fmt)
    cache, oc, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=2, Hkv=2, L=L, b=b,
                           k_active=[kk, kv], k_value=[kv, kk], dtype=dtype, values=vals)
    for bi in range(2):
        for h in range(2):
            C.compare_unit(cache, oc[bi][h], bi, h, L, si.np_dtype(dtype), values=vals)


@pytest.mark.parametrize("fmt,chunks", [("f16", [1] * 70 + [65, 3]), ("e4m3", [7, 1, 64, 13, 65])])
def test_asym_chunked_appends(gpu_device, swan_mod, torch_mod, fmt, chunks):
    _log(f"asym chunked fmt={fmt} chunks={chunks[:4]}...")
    dtype, vals = _dt(fmt)
    L = sum(chunks)
    cache, oc, *_ = _build(swan_mod, torch_mod, gpu_device, B=1, Hq=1, Hkv=1, L=L, b=16,
                           k_active=[40], k_value=[72], dtype=dtype, chunks=chunks, values=vals)
    C.compare_unit(cache, oc[0][0], 0, 0, L, si.np_dtype(dtype), values=vals)


@pytest.mark.parametrize("fmt,L,b,kk,kv,Hq,Hkv", [
    ("f16", 700, 128, 77, 51, 4, 4), ("f16", 1000, 0, 77, 51, 4, 4), ("f16", 1, 0, 77, 51, 2, 2),
    ("f16", 40, 64, 77, 51, 4, 4),  # buffer only: no sparse page in the group
    ("f16", 2049, 128, 13, 115, 8, 2),  # GQA, 4 heads per wave
    ("f16", 1500, 64, 51, 77, 16, 2),  # GQA, 8 heads per wave
    ("f16", 900, 32, 24, 40, 4, 2),  # GQA, 2 heads per wave
    ("f16", 600, 16, 24, 40, 6, 2),  # GQA group of 3: one wave per query head
    ("f16", 64, 0, 96, 32, 8, 2), ("f16", 3000, 16, 128, 8, 2, 2), ("f16", 3000, 16, 8, 128, 2, 2),
    ("f32", 512, 16, 64, 8, 1, 1), ("f32", 900, 32, 96, 40, 4, 1),
    ("e4m3", 1000, 128, 77, 51, 4, 4), ("e4m3", 1500, 64, 77, 51, 8, 2),
    ("e4m3", 700, 16, 20, 100, 16, 2),
])
def test_asym_decode_matches_oracle(gpu_device, swan_mod, torch_mod, fmt, L, b, kk, kv, Hq,
                                    Hkv):
    _log(f"asym decode fmt={fmt} L={L} b={b} k_key={kk} k_value={kv} Hq={Hq} Hkv={Hkv}")
    dtype, vals = _dt(fmt)
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=Hq,
                                                Hkv=Hkv, L=L, b=b, k_active=[kk, kk],
                                                k_value=[kv, kv], dtype=dtype, values=vals)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, dtype)


@pytest.mark.parametrize("fmt,Hq,Hkv", [("f16", 4, 4), ("f16", 8, 2), ("e4m3", 8, 2),
                                        ("f32", 2, 1)])
def test_asym_mixed_batch(gpu_device, swan_mod, torch_mod, fmt, Hq, Hkv):
    """One batch: symmetric k, equal k_pad with different k, and several different-k_pad
    pairs, at ragged lengths, launched side by side."""
    _log(f"asym mixed batch fmt={fmt} Hq={Hq} Hkv={Hkv}")
    dtype, vals = _dt(fmt)
    kk = [48, 77, 48, 13, 77, 128, 64]
    kv = [48, 51, 41, 115, 51, 8, 64]
    Ls = [3000, 1500, 64, 2500, 1, 700, 17]
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=7, Hq=Hq,
                                                Hkv=Hkv, L=Ls, b=16, k_active=kk, k_value=kv,
                                                dtype=dtype, values=vals, chunks=[1000, 1, 2000])
    for bi in range(7):
        C.compare_unit(cache, oc[bi][Hkv - 1], bi, Hkv - 1, Ls[bi], si.np_dtype(dtype),
                       values=vals)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, dtype)


def test_asym_decode_steps(gpu_device, swan_mod, torch_mod):
    """Append one token, then attend, several times (the decode loop)."""
    torch = torch_mod
    B, Hq, Hkv, L0, steps, b = 2, 8, 2, 700, 5, 32
    kk, kv = [77, 24], [51, 96]
    _log("asym decode steps")
    cache, _, Pqk, Pvo, tqk, tvo, K0, V0 = _build(swan_mod, torch_mod, gpu_device, B=B, Hq=Hq,
                                                   Hkv=Hkv, L=L0, b=b, k_active=kk, k_value=kv,
                                                   dtype="f16", capacity=L0 + steps)
    rng = si.rng_for(31337, 1)
    K = np.concatenate([K0, rng.standard_normal((B, Hkv, steps, 128)).astype(np.float16)], 2)
    V = np.concatenate([V0, rng.standard_normal((B, Hkv, steps, 128)).astype(np.float16)], 2)
    for s in range(steps):
        L = L0 + s + 1
        cache.append(torch.tensor(K[:, :, L - 1:L], device=gpu_device),
                     torch.tensor(V[:, :, L - 1:L], device=gpu_device), tqk, tvo)
        oc = [[O.compress_block(K[bi, h, :L], V[bi, h, :L], Pqk[h], Pvo[h], b, kk[bi],
                                np.float16, k_value=kv[bi]) for h in range(Hkv)]
              for bi in range(B)]
        _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, "f16",
                      seed=s)
    for bi in range(B):
        C.compare_unit(cache, oc[bi][0], bi, 0, L0 + steps, np.float16)


def test_explicit_equal_k_value_is_the_default(gpu_device, swan_mod, torch_mod):
    """k_value equal to k_active gives the same bytes and outputs as k_value = NULL."""
    torch = torch_mod
    _log("explicit k_value == k_active")
    outs, pages = [], []
    for kv in (None, [48, 96]):
        cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=4,
                                                    Hkv=2, L=[900, 300], b=16, k_active=[48, 96],
                                                    k_value=kv, dtype="f16")
        got, _ = _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo,
                               "f16")
        outs.append(got)
        pages.append((cache.k_pages.cpu().numpy(), cache.v_pages.cpu().numpy()))
        torch.cuda.synchronize()
    assert np.array_equal(outs[0], outs[1])
    assert np.array_equal(pages[0][0], pages[1][0]) and np.array_equal(pages[0][1], pages[1][1])
