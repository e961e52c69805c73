"""GPU-vs-oracle parity through the C ABI (needs an MI355X).

Bars: top-k indices and stored values bit-exact (both sides round a float64
rotation once to the storage type, so selection is taken on identical values);
attention outputs within max_j |o - o_ref| / max_j |o_ref| <= 2e-3 per
(sequence, query head).
"""
import math
import sys

import numpy as np
import pytest

import swan_inputs as si
from oracle import swan_oracle as O
from tests import swan_cases as C
from tests import swan_layout as lay

pytestmark = pytest.mark.gpu
TOL = 2e-3


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


# --------------------------------------------------------------------------- #
# calibration (Sec. 4.1.2)
# --------------------------------------------------------------------------- #
def test_calibrate_matches_oracle(gpu_device, swan_mod):
    _log("calibrate: workload 0 and 1 rows")
    for wid, h, role in ((0, 0, si.ROLE_K), (0, 0, si.ROLE_V), (1, 5, si.ROLE_K)):
        rows = si.calibration_rows(wid, h, role)
        Pg, sg = C.gpu_calibrate(rows, gpu_device)
        Po, so = O.calibrate(rows)
        Pg64 = Pg.astype(np.float64)
        assert np.max(np.abs(Pg64.T @ Pg64 - np.eye(128))) < 2e-6
        assert np.allclose(sg, so, rtol=1e-5, atol=1e-6 * so[0])
        # columns with a clear spectral gap agree with the oracle's, signs included
        gap = np.minimum(np.r_[np.inf, so[:-1] - so[1:]], np.r_[so[:-1] - so[1:], np.inf])
        sep = gap > 1e-3 * so
        assert sep.sum() > 100
        err = np.max(np.abs(Pg64[:, sep] - Po[:, sep]), axis=0)
        assert np.max(err) < 1e-4, np.max(err)


def test_calibrate_constructed_basis(gpu_device):
    d, n = 128, 600
    V = si.random_orthogonal(40, d)
    U = si.random_orthogonal(41, n)[:, :d]
    sig = np.exp(-np.arange(d) / 40.0) * 10
    S = (U * sig) @ V.T
    Pg, sg = C.gpu_calibrate(S, gpu_device)
    assert np.allclose(sg, sig, rtol=1e-5)
    cos = np.abs(np.sum(Pg.astype(np.float64) * V, axis=0))
    assert np.min(cos) > 1 - 1e-6


# --------------------------------------------------------------------------- #
# compress-append: indices and values bit-exact
# --------------------------------------------------------------------------- #
def _build(swan_mod, torch_mod, device, *, B, Hq, Hkv, L, b, k_active, dtype, chunks=None,
           seed=0, capacity=None, wid=99, values="same", k_value=None, kv_hook=None):
    """GPU cache + oracle caches for synthetic rows of the recipe (kv_hook(K, V)
    may rewrite the rows in place first)."""
    torch = torch_mod
    np_dt = si.np_dtype(dtype)
    Pqk = np.stack([si.random_orthogonal(seed * 100 + h, 128) for h in range(Hkv)]).astype(
        np.float32)
    Pvo = np.stack([si.random_orthogonal(seed * 100 + 50 + h, 128) for h in range(Hkv)]).astype(
        np.float32)
    Ls = [L] * B if np.isscalar(L) else list(L)
    Lmax = max(Ls)
    K = np.zeros((B, Hkv, Lmax, 128), dtype=np_dt)
    V = np.zeros((B, Hkv, Lmax, 128), dtype=np_dt)
    for bi in range(B):
        for h in range(Hkv):
            R = si.haar_orthogonal(si.rng_for(wid, seed, h), 128)
            K[bi, h] = si.lowrank_rows(si.rng_for(wid, seed, bi, h, 0), Lmax, R).astype(np_dt)
            V[bi, h] = si.lowrank_rows(si.rng_for(wid, seed, bi, h, 1), Lmax, R).astype(np_dt)
    if kv_hook is not None:
        kv_hook(K, V)
    cap = capacity if capacity is not None else max(Lmax - b, 1)
    cache = swan_mod.SwanCache(B, Hq, Hkv, b, cap, k_active, C.torch_dtype(dtype), device,
                               sparse_values=values, k_value=k_value)
    tP_qk = torch.tensor(Pqk, device=device)
    tP_vo = torch.tensor(Pvo, device=device)
    # sequences of different lengths: each chunk appends min(n, what is left)
    # tokens per sequence
    if chunks is None:
        chunks = [Lmax]
    t0 = 0
    for n in chunks:
        n = min(n, Lmax - t0)
        if n <= 0:
            break
        per = [max(min(n, Lb - t0), 0) for Lb in Ls]
        kn = torch.tensor(K[:, :, t0:t0 + n], device=device)
        vn = torch.tensor(V[:, :, t0:t0 + n], device=device)
        cache.append(kn, vn, tP_qk, tP_vo, n_new_per_seq=per)
        t0 += n
    assert cache.seq_len == Ls
    torch.cuda.synchronize()
    ovals = "e4m3" if values == "e4m3" else "t"
    oc = [[O.compress_block(K[bi, h, :Ls[bi]], V[bi, h, :Ls[bi]], Pqk[h], Pvo[h], b,
                            k_active[bi], np_dt, values=ovals,
                            k_value=None if k_value is None else k_value[bi])
           for h in range(Hkv)]
          for bi in range(B)]
    return cache, oc, Pqk, Pvo, tP_qk, tP_vo, K, V


@pytest.mark.parametrize("dtype,L,b,k", [
    ("f16", 1, 0, 48), ("f16", 130, 0, 48), ("f16", 200, 16, 1), ("f16", 200, 16, 128),
    ("f16", 333, 64, 13), ("f16", 64, 64, 48), ("f16", 40, 64, 48),
    ("f32", 300, 16, 64), ("f32", 129, 3, 5),
    # pages that fit the prefill kernel's LDS copy (k_pad 88) and those that
    # take two rounds (k_pad 96)
    ("f16", 300, 16, 88), ("f16", 300, 16, 81), ("f16", 300, 16, 89), ("f16", 129, 0, 96),
])
def test_compress_prefill_bit_exact(gpu_device, swan_mod, torch_mod, dtype, L, b, k):
    _log(f"compress prefill dtype={dtype} L={L} b={b} k={k}")
    cache, oc, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=2, Hkv=2, L=L, b=b,
                           k_active=[k, k], dtype=dtype)
    for bi in range(2):
        for h in range(2):
            C.compare_unit(cache, oc[bi][h], bi, h, L, si.np_dtype(dtype))


def _extreme_rows(K, V):
    """Rows that reach the rotation's edge cases: elements far below the row's
    largest (they fall below its fixed-point resolution), fp16 subnormals, zeros,
    rows of small or large magnitude, all-zero rows and single-element rows."""
    rng = si.rng_for(4242)
    for X in (K, V):
        B, H, L, D = X.shape
        for bi in range(B):
            for h in range(H):
                x = X[bi, h].astype(np.float64)
                for t in range(L):
                    kind = t % 8
                    row = x[t]
                    m = np.max(np.abs(row))
                    if kind == 1:    # a few elements 2^-21 .. 2^-26 of the largest
                        idx = rng.choice(D, 6, replace=False)
                        row[idx] = m * np.ldexp(1.0, -rng.integers(21, 27, 6)) * rng.choice([-1, 1], 6)
                    elif kind == 2:  # fp16 subnormals and zeros
                        idx = rng.choice(D, 10, replace=False)
                        row[idx[:6]] = np.ldexp(rng.integers(1, 1024, 6).astype(np.float64), -24)
                        row[idx[6:]] = 0.0
                    elif kind == 3:  # small row: largest below 2^-8
                        row *= np.ldexp(1.0, -10) / max(m, 1e-30)
                    elif kind == 4:  # large row: rotated components up to ~3e4
                        row *= 3.0e4 / max(np.linalg.norm(row), 1e-30)
                    elif kind == 5 and t % 16 == 5:
                        row[:] = 0.0
                    elif kind == 6:  # one nonzero element
                        j = int(rng.integers(0, D))
                        v = row[j]
                        row[:] = 0.0
                        row[j] = v if v != 0 else 1.0
                X[bi, h] = x.astype(X.dtype)


@pytest.mark.parametrize("L,b,k", [(300, 16, 48), (200, 0, 13), (130, 64, 96)])
def test_compress_prefill_extreme_rows(gpu_device, swan_mod, torch_mod, L, b, k):
    _log(f"compress prefill extreme rows L={L} b={b} k={k}")
    cache, oc, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=2, Hkv=2, L=L, b=b,
                           k_active=[k, k], dtype="f16", kv_hook=_extreme_rows)
    for bi in range(2):
        for h in range(2):
            C.compare_unit(cache, oc[bi][h], bi, h, L, np.float16)


@pytest.mark.parametrize("chunks", [[1] * 150, [7, 1, 64, 13, 65], [100, 1, 1, 1, 47]])
def test_compress_chunked_equals_prefill(gpu_device, swan_mod, torch_mod, chunks):
    _log(f"compress chunks={chunks[:6]}")
    L = sum(chunks)
    cache, oc, *_ = _build(swan_mod, torch_mod, gpu_device, B=1, Hq=1, Hkv=1, L=L, b=16,
                           k_active=[24], dtype="f16", chunks=chunks)
    C.compare_unit(cache, oc[0][0], 0, 0, L, np.float16)


# --------------------------------------------------------------------------- #
# decode attention
# --------------------------------------------------------------------------- #
def _decode_check(swan_mod, torch_mod, device, cache, oc, Pqk, Pvo, tP_qk, tP_vo, dtype,
                  seed=0, scale=0.0):
    torch = torch_mod
    B, Hq = cache.desc.batch, cache.desc.n_q_heads
    q = si.rng_for(777, seed).standard_normal((B, Hq, 128)).astype(si.np_dtype(dtype))
    out = cache.decode(torch.tensor(q, device=device), tP_qk, tP_vo, scale=scale)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    ref = O.decode_batch(q.astype(np.float64), Pqk, Pvo, oc, scale if scale > 0 else None)
    err = C.max_rel_err(got, ref)
    _log(f"  decode max rel err {err:.3e}")
    assert err <= TOL
    return got, ref


@pytest.mark.parametrize("dtype,L,b,k,Hq,Hkv", [
    ("f16", 1, 0, 48, 4, 4), ("f16", 1, 16, 48, 4, 4), ("f16", 17, 16, 48, 4, 4),
    ("f16", 700, 0, 8, 4, 2), ("f16", 700, 128, 48, 4, 4), ("f16", 2049, 128, 64, 8, 2),
    ("f16", 1000, 16, 128, 2, 2), ("f16", 513, 5, 3, 2, 1), ("f32", 512, 16, 64, 1, 1),
    ("f32", 900, 32, 96, 4, 1),
    # GQA groups of 8 and 16 (MFMA value path, 8 heads per wave) and of 3
    # (one wave per query head), fp32 GQA (one wave per query head)
    ("f16", 1500, 64, 48, 16, 2), ("f16", 900, 32, 32, 32, 2), ("f16", 600, 16, 24, 6, 2),
    ("f32", 700, 16, 40, 8, 2), ("f16", 64, 0, 96, 8, 2),
])
def test_decode_matches_oracle(gpu_device, swan_mod, torch_mod, dtype, L, b, k, Hq, Hkv):
    _log(f"decode dtype={dtype} L={L} b={b} k={k} Hq={Hq} Hkv={Hkv}")
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=Hq,
                                                Hkv=Hkv, L=L, b=b, k_active=[k, k], dtype=dtype)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, dtype)


def test_decode_ragged_lengths_and_per_sequence_k(gpu_device, swan_mod, torch_mod):
    """Sequences of different lengths and k in one batch (per-sequence append counts)."""
    _log("decode ragged lengths, per-sequence k")
    torch = torch_mod
    Ls = [1, 130, 700, 64]
    ks = [32, 48, 96, 5]
    B, Hq, Hkv, b = 4, 4, 2, 16
    Lmax = max(Ls)
    cache = swan_mod.SwanCache(B, Hq, Hkv, b, 1000, ks, torch.float16, gpu_device)
    Pqk = np.stack([si.random_orthogonal(500 + h, 128) for h in range(Hkv)]).astype(np.float32)
    Pvo = np.stack([si.random_orthogonal(600 + h, 128) for h in range(Hkv)]).astype(np.float32)
    tqk, tvo = torch.tensor(Pqk, device=gpu_device), torch.tensor(Pvo, device=gpu_device)
    K = np.zeros((B, Hkv, Lmax, 128), np.float16)
    V = np.zeros((B, Hkv, Lmax, 128), np.float16)
    for bi in range(B):
        for h in range(Hkv):
            R = si.random_orthogonal(700 + h, 128)
            K[bi, h] = si.lowrank_rows(si.rng_for(88, bi, h, 0), Lmax, R).astype(np.float16)
            V[bi, h] = si.lowrank_rows(si.rng_for(88, bi, h, 1), Lmax, R).astype(np.float16)
    # prefill L_b - 1 tokens per sequence, then one decode-step append each
    pre = [L - 1 for L in Ls]
    cache.append(torch.tensor(K[:, :, :Lmax - 1], device=gpu_device),
                 torch.tensor(V[:, :, :Lmax - 1], device=gpu_device), tqk, tvo,
                 n_new_per_seq=pre)
    last_k = np.stack([K[bi, :, Ls[bi] - 1:Ls[bi]] for bi in range(B)])
    last_v = np.stack([V[bi, :, Ls[bi] - 1:Ls[bi]] for bi in range(B)])
    cache.append(torch.tensor(last_k, device=gpu_device), torch.tensor(last_v, device=gpu_device),
                 tqk, tvo)
    torch.cuda.synchronize()
    assert cache.seq_len == Ls
    oc = [[O.compress_block(K[bi, h, :Ls[bi]], V[bi, h, :Ls[bi]], Pqk[h], Pvo[h], b, ks[bi],
                            np.float16) for h in range(Hkv)] for bi in range(B)]
    for bi in range(B):
        for h in range(Hkv):
            C.compare_unit(cache, oc[bi][h], bi, h, Ls[bi], np.float16)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, "f16")


@pytest.mark.parametrize("Hq,Hkv", [(1, 1), (4, 2)])
def test_decode_max_batch_many_k(gpu_device, swan_mod, torch_mod, Hq, Hkv):
    """The largest batch, each sequence with its own length and k: on the MHA
    path one fused launch with every k_pad tier, on the GQA path up to 16
    attention launches spread over the library's side streams."""
    B = 64
    Ls = [1 + (37 * i) % 300 for i in range(B)]
    ks = [1 + (7 * i) % 128 for i in range(B)]
    _log(f"decode max batch B={B} Hq={Hq} Hkv={Hkv}, {len({(k + 7) // 8 for k in ks})} k groups")
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=B, Hq=Hq,
                                                Hkv=Hkv, L=Ls, b=16, k_active=ks, dtype="f16",
                                                capacity=300)
    for bi in range(0, B, 7):
        C.compare_unit(cache, oc[bi][0], bi, 0, Ls[bi], np.float16)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, "f16")


@pytest.mark.parametrize("Hq,Hkv", [(2, 2), (4, 2)])
def test_decode_largest_buffer(gpu_device, swan_mod, torch_mod, Hq, Hkv):
    """A dense buffer of 4096 tokens (the ring's maximum) next to sparse pages."""
    _log(f"decode with b=4096, Hq={Hq} Hkv={Hkv}")
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=1, Hq=Hq,
                                                Hkv=Hkv, L=4500, b=4096, k_active=[48],
                                                dtype="f16")
    C.compare_unit(cache, oc[0][0], 0, 0, 4500, np.float16)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, "f16")


def test_decode_only_on_oracle_packed_pages(gpu_device, swan_mod, torch_mod):
    """Decode alone: pages packed on the host from the oracle's own pairs."""
    _log("decode on oracle-packed pages")
    torch = torch_mod
    B, Hq, Hkv, L, b, k = 2, 4, 2, 1500, 32, 40
    Pqk = np.stack([si.random_orthogonal(800 + h, 128) for h in range(Hkv)]).astype(np.float32)
    Pvo = np.stack([si.random_orthogonal(900 + h, 128) for h in range(Hkv)]).astype(np.float32)
    cache = swan_mod.SwanCache(B, Hq, Hkv, b, L - b, [k] * B, torch.float16, gpu_device)
    npc = (L - b + 63) // 64
    oc = []
    kp_bytes = np.zeros(cache.k_pages.numel(), np.uint8)
    vp_bytes = np.zeros(cache.v_pages.numel(), np.uint8)
    kr = np.zeros(tuple(cache.k_ring.shape), np.float16)
    vr = np.zeros(tuple(cache.v_ring.shape), np.float16)
    for bi in range(B):
        row = []
        for h in range(Hkv):
            R = si.random_orthogonal(1000 + h, 128)
            Kr = si.lowrank_rows(si.rng_for(99, bi, h, 0), L, R).astype(np.float16)
            Vr = si.lowrank_rows(si.rng_for(99, bi, h, 1), L, R).astype(np.float16)
            c = O.compress_block(Kr, Vr, Pqk[h], Pvo[h], b, k, np.float16)
            row.append(c)
            s, e = lay.unit_slice([k] * B, Hkv, L - b, 2, bi, h)
            kp_bytes[s:e] = lay.pack(c["k_idx"], c["k_val"], np.float16, k, npc)
            vp_bytes[s:e] = lay.pack(c["v_idx"], c["v_val"], np.float16, k, npc)
            pos = np.arange(L - b, L)
            kr[bi, h, pos % b] = c["k_buf"]
            vr[bi, h, pos % b] = c["v_buf"]
        oc.append(row)
    cache.k_pages.copy_(torch.tensor(kp_bytes, device=gpu_device))
    cache.v_pages.copy_(torch.tensor(vp_bytes, device=gpu_device))
    cache.k_ring.copy_(torch.tensor(kr, device=gpu_device))
    cache.v_ring.copy_(torch.tensor(vr, device=gpu_device))
    cache.seq_len = [L] * B
    tqk, tvo = torch.tensor(Pqk, device=gpu_device), torch.tensor(Pvo, device=gpu_device)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, "f16")
    # explicit scale
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, "f16",
                  scale=0.05)


def test_decode_is_deterministic(gpu_device, swan_mod, torch_mod):
    _log("decode determinism")
    torch = torch_mod
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=4,
                                                Hkv=4, L=3000, b=128, k_active=[48, 48],
                                                dtype="f16")
    q = torch.tensor(si.rng_for(5).standard_normal((2, 4, 128)).astype(np.float16),
                     device=gpu_device)
    outs = [cache.decode(q, tqk, tvo).clone() for _ in range(10)]
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o, outs[0])


def test_decode_step_append_then_attend(gpu_device, swan_mod, torch_mod):
    """Algorithm 1 per decode step: append one token (evicting the oldest buffered
    one), then attend, for several consecutive steps."""
    _log("decode steps")
    torch = torch_mod
    B, Hq, Hkv, L0, b, k = 2, 4, 2, 200, 16, 32
    steps = 5
    cache, oc, Pqk, Pvo, tqk, tvo, K, V = _build(swan_mod, torch_mod, gpu_device, B=B, Hq=Hq,
                                                  Hkv=Hkv, L=L0 + steps, b=b, k_active=[k, k],
                                                  dtype="f16", chunks=[L0] + [1] * steps)
    # the chunked GPU cache equals the oracle at the final length
    for bi in range(B):
        for h in range(Hkv):
            C.compare_unit(cache, oc[bi][h], bi, h, L0 + steps, np.float16)
    _decode_check(swan_mod, torch_mod, gpu_device, cache, oc, Pqk, Pvo, tqk, tvo, "f16")


# --------------------------------------------------------------------------- #
# the small workloads, every unit
# --------------------------------------------------------------------------- #
def _workload_full(swan_mod, torch_mod, device, w):
    torch = torch_mod
    np_dt = si.np_dtype(w.dtype)
    Pqk, Pvo = C.rotations(w.wid, w.n_kv_heads, device)
    L = w.context
    ks = list(si.k_active_for(w))
    cache = swan_mod.SwanCache(w.batch, w.n_q_heads, w.n_kv_heads, w.buffer, max(L - w.buffer, 1),
                               ks, C.torch_dtype(w.dtype), device)
    K = np.stack([np.stack([si.kv_rows_host(w.wid, b, h, si.ROLE_K, L, w.dtype)
                            for h in range(w.n_kv_heads)]) for b in range(w.batch)])
    V = np.stack([np.stack([si.kv_rows_host(w.wid, b, h, si.ROLE_V, L, w.dtype)
                            for h in range(w.n_kv_heads)]) for b in range(w.batch)])
    tqk, tvo = torch.tensor(Pqk, device=device), torch.tensor(Pvo, device=device)
    # prefill L-1 tokens, then the decode step appends the current token
    cache.append(torch.tensor(K[:, :, :L - 1], device=device),
                 torch.tensor(V[:, :, :L - 1], device=device), tqk, tvo)
    cache.append(torch.tensor(K[:, :, L - 1:], device=device),
                 torch.tensor(V[:, :, L - 1:], device=device), tqk, tvo)
    q = si.queries_host(w.wid, w.batch, w.n_q_heads, w.dtype)
    out = cache.decode(torch.tensor(q, device=device), tqk, tvo)
    torch.cuda.synchronize()
    oc = [[O.compress_block(K[b, h], V[b, h], Pqk[h], Pvo[h], w.buffer, ks[b], np_dt)
           for h in range(w.n_kv_heads)] for b in range(w.batch)]
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            C.compare_unit(cache, oc[b][h], b, h, L, np_dt)
    ref = O.decode_batch(q.astype(np.float64), Pqk, Pvo, oc)
    err = C.max_rel_err(out.cpu().numpy(), ref)
    _log(f"  {w.name}: decode max rel err {err:.3e}")
    assert err <= TOL


def test_workload_tiny_fp32_all_units(gpu_device, swan_mod, torch_mod):
    _log("workload tiny_fp32_L512")
    _workload_full(swan_mod, torch_mod, gpu_device, si.WORKLOADS["tiny_fp32_L512"])


def test_workload_llama2_4k_all_units(gpu_device, swan_mod, torch_mod):
    _log("workload llama2_7b_L4k_b1")
    _workload_full(swan_mod, torch_mod, gpu_device, si.WORKLOADS["llama2_7b_L4k_b1"])
