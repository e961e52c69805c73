"""k changed for running sequences (swan_change_k) on the GPU, against the oracle.

The converted pages must equal the oracle's ``change_k_cache`` of the same cache bit
for bit (indices, values or E4M3 codes, and the padding), and decode on them must
stay within 2e-3 of the oracle (max |o - o_ref| / max |o_ref| per query head).
Appends after the change prune with the new k; the oracle for those is a
``UnitCache`` fed token by token with the same change in the middle.
"""
import sys

import numpy as np
import pytest

import swan_inputs as si
from oracle import swan_oracle as O
from tests import swan_cases as C
from tests import swan_layout as lay
from tests.test_gpu_parity import _build, _decode_check

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _dt(fmt):
    return ("f16", "e4m3") if fmt == "e4m3" else (fmt, "same")


@pytest.mark.parametrize("fmt,L,b,Hq,Hkv,k0,kv0,k1,kv1", [
    ("f16", 700, 16, 4, 4, 48, 48, 32, 32),     # lower
    ("f16", 700, 16, 4, 4, 32, 32, 64, 64),     # raise
    ("f16", 900, 0, 8, 2, 77, 51, 40, 64),      # per role: lower keys, raise values
    ("f16", 300, 64, 2, 2, 128, 128, 1, 8),     # extremes
    ("f16", 300, 64, 2, 2, 1, 8, 128, 120),
    ("f16", 513, 5, 4, 4, 48, 48, 48, 48),      # copy
    ("f16", 513, 5, 4, 4, 45, 47, 41, 48),      # within the same k_pad
    ("f32", 400, 16, 2, 1, 64, 24, 24, 64),
    ("e4m3", 700, 16, 8, 2, 64, 64, 24, 96),
    ("e4m3", 600, 0, 4, 4, 96, 48, 48, 20),
])
def test_change_k_matches_oracle(gpu_device, swan_mod, torch_mod, fmt, L, b, Hq, Hkv, k0, kv0,
                                 k1, kv1):
    _log(f"change_k fmt={fmt} L={L} b={b} Hq={Hq} Hkv={Hkv} ({k0},{kv0}) -> ({k1},{kv1})")
    dtype, vals = _dt(fmt)
    Ls = [L, L // 3, 1]  # the last one is all buffer when b > 0
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=3, Hq=Hq,
                                                Hkv=Hkv, L=Ls, b=b, k_active=[k0] * 3,
                                                k_value=[kv0] * 3, dtype=dtype, values=vals)
    cache.change_k([k1] * 3, [kv1] * 3)
    oc2 = [[O.change_k_cache(u, k1, kv1) for u in row] for row in oc]
    for bi in range(3):
        for h in range(Hkv):
            C.compare_unit(cache, oc2[bi][h], bi, h, Ls[bi], si.np_dtype(dtype), values=vals)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc2, Pqk, Pvo, tqk, tvo, dtype)


def test_change_k_per_sequence_in_a_ragged_batch(gpu_device, swan_mod, torch_mod):
    _log("change_k per sequence, ragged batch")
    k0, kv0 = [48, 96, 13, 64, 32], [48, 40, 13, 120, 8]
    k1, kv1 = [24, 96, 60, 8, 32], [64, 40, 5, 128, 16]
    Ls = [2000, 700, 65, 1, 1300]
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=5, Hq=8,
                                                Hkv=2, L=Ls, b=16, k_active=k0, k_value=kv0,
                                                dtype="f16", chunks=[500, 1, 1499])
    cache.change_k(k1, kv1)
    oc2 = [[O.change_k_cache(u, k1[bi], kv1[bi]) for u in oc[bi]] for bi in range(5)]
    for bi in range(5):
        for h in range(2):
            C.compare_unit(cache, oc2[bi][h], bi, h, Ls[bi], np.float16)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc2, Pqk, Pvo, tqk, tvo, "f16")


@pytest.mark.parametrize("k0,k1", [(48, 24), (24, 64)])
def test_appends_after_change_use_the_new_k(gpu_device, swan_mod, torch_mod, k0, k1):
    """Decode loop: prefill, change k, then one-token appends and a chunk, each checked
    against a UnitCache given the same tokens and the same change."""
    torch = torch_mod
    B, Hq, Hkv, L0, b = 2, 4, 2, 400, 32
    extra = [1, 1, 1, 70, 1]
    _log(f"appends after change_k {k0} -> {k1}")
    cache, _, Pqk, Pvo, tqk, tvo, K0, V0 = _build(swan_mod, torch_mod, gpu_device, B=B, Hq=Hq,
                                                   Hkv=Hkv, L=L0, b=b, k_active=[k0, k0],
                                                   dtype="f16", capacity=L0 + sum(extra))
    rng = si.rng_for(4711, k0, k1)
    n_more = sum(extra)
    K = np.concatenate([K0, rng.standard_normal((B, Hkv, n_more, 128)).astype(np.float16)], 2)
    V = np.concatenate([V0, rng.standard_normal((B, Hkv, n_more, 128)).astype(np.float16)], 2)
    units = [[O.UnitCache(Pqk[h], Pvo[h], b, k0, np.float16) for h in range(Hkv)]
             for _ in range(B)]
    for bi in range(B):
        for h in range(Hkv):
            for t in range(L0):
                units[bi][h].append(K[bi, h, t], V[bi, h, t])
    cache.change_k([k1, k1])
    for row in units:
        for u in row:
            u.change_k(k1)
    t0 = L0
    for i, n in enumerate(extra):
        cache.append(torch.tensor(K[:, :, t0:t0 + n], device=gpu_device),
                     torch.tensor(V[:, :, t0:t0 + n], device=gpu_device), tqk, tvo)
        for bi in range(B):
            for h in range(Hkv):
                for t in range(t0, t0 + n):
                    units[bi][h].append(K[bi, h, t], V[bi, h, t])
        t0 += n
        oc = [[u.sparse_arrays() for u in row] for row in units]
        _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, "f16",
                      seed=i)
    for bi in range(B):
        for h in range(Hkv):
            C.compare_unit(cache, oc[bi][h], bi, h, t0, np.float16)


def test_lower_then_raise(gpu_device, swan_mod, torch_mod):
    """Raising after lowering cannot bring pruned components back: the tokens keep the
    lower k's pairs and get zero-valued slots."""
    _log("lower then raise")
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=4,
                                                Hkv=2, L=[800, 333], b=16, k_active=[64, 64],
                                                dtype="f16")
    cache.change_k([16, 40])
    cache.change_k([96, 40])
    oc2 = [[O.change_k_cache(O.change_k_cache(u, k), 96 if bi == 0 else 40) for u in row]
           for bi, (row, k) in enumerate(zip(oc, [16, 40]))]
    for bi, L in enumerate([800, 333]):
        for h in range(2):
            C.compare_unit(cache, oc2[bi][h], bi, h, L, np.float16)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc2, Pqk, Pvo, tqk, tvo, "f16")


@pytest.mark.parametrize("fmt,k0,k1,k2", [
    ("f16", 32, 64, 48),     # lowering keeps the 32 pairs and the 16 lowest zero fills
    ("f16", 32, 64, 33),
    ("f32", 24, 60, 30),
    ("e4m3", 48, 96, 64),
])
def test_raise_then_lower(gpu_device, swan_mod, torch_mod, fmt, k0, k1, k2):
    """After a raise the stored pairs are the pairs kept at pruning, then the zero
    fills; lowering must still rank ties by index and write ascending indices."""
    _log(f"raise then lower fmt={fmt} {k0} -> {k1} -> {k2}")
    dtype, vals = _dt(fmt)
    Ls = [900, 333]
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=4,
                                                Hkv=2, L=Ls, b=16, k_active=[k0, k0],
                                                dtype=dtype, values=vals, seed=5)
    cache.change_k([k1, k1])
    cache.change_k([k2, k2])
    oc2 = [[O.change_k_cache(O.change_k_cache(u, k1), k2) for u in row] for row in oc]
    for bi, L in enumerate(Ls):
        for h in range(2):
            C.compare_unit(cache, oc2[bi][h], bi, h, L, si.np_dtype(dtype), values=vals)
            assert np.all(np.diff(oc2[bi][h]["k_idx"], axis=1) > 0)  # ascending indices
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc2, Pqk, Pvo, tqk, tvo, dtype)


@pytest.mark.parametrize("dtype,k0,steps", [
    (np.float16, 40, [(80, False), (50, True)]),   # raise, then lower into the fills
    (np.float16, 40, [(33, True)]),                # lower with ties at zero
    (np.float32, 24, [(64, False), (30, True)]),
    (np.float16, 8, [(128, False), (9, True)]),
])
def test_change_k_zero_ties_on_host_packed_pages(gpu_device, swan_mod, torch_mod, dtype, k0,
                                                 steps):
    """Pages packed on the host from pairs with many zero (+0 and -0) and equal
    magnitudes, so that the k'-th magnitude is tied between pairs kept at pruning
    and the zero fills of a raise: the converted pages equal the oracle's."""
    torch = torch_mod
    B, Hkv, S, b = 2, 2, 300, 4
    L = S + b
    rng = si.rng_for(4712, k0, len(steps))
    esize = np.dtype(dtype).itemsize
    cache = swan_mod.SwanCache(B, 2, Hkv, b, S, [k0] * B, torch.float16 if esize == 2
                               else torch.float32, gpu_device)
    npc = (S + 63) // 64
    kp_bytes = np.zeros(cache.k_pages.numel(), np.uint8)
    vp_bytes = np.zeros(cache.v_pages.numel(), np.uint8)
    oc = []
    for bi in range(B):
        row = []
        for h in range(Hkv):
            c = {"n_sparse": S, "k_buf": np.zeros((b, 128), dtype),
                 "v_buf": np.zeros((b, 128), dtype)}
            for r in ("k", "v"):
                idx = np.sort(np.stack([rng.choice(128, k0, replace=False) for _ in range(S)]),
                              axis=1)
                # magnitudes from a small set (many ties), a third of them zero, random signs
                mag = rng.choice([0.0, 0.0, 0.5, 1.0, 0.25, 2.0], size=(S, k0))
                val = (mag * rng.choice([-1.0, 1.0], size=(S, k0))).astype(dtype)
                c[f"{r}_idx"], c[f"{r}_val"] = idx, val
                s0, e0 = lay.unit_slice([k0] * B, Hkv, S, esize, bi, h)
                (kp_bytes if r == "k" else vp_bytes)[s0:e0] = lay.pack(idx, val, dtype, k0, npc)
            row.append(c)
        oc.append(row)
    cache.k_pages.copy_(torch.tensor(kp_bytes, device=gpu_device))
    cache.v_pages.copy_(torch.tensor(vp_bytes, device=gpu_device))
    cache.seq_len = [L] * B
    for k, _ in steps:
        cache.change_k([k] * B)
        oc = [[O.change_k_cache(u, k) for u in row] for row in oc]
    torch.cuda.synchronize()
    for bi in range(B):
        for h in range(Hkv):
            for role, r in enumerate(("k", "v")):
                idx, val, _, _ = C.unit_pages(cache, bi, h, role, S, dtype)
                assert np.array_equal(idx, oc[bi][h][f"{r}_idx"]), (bi, h, r)
                assert np.array_equal(val.view(np.uint8),
                                      np.asarray(oc[bi][h][f"{r}_val"], dtype).view(np.uint8))
