"""Randomised parity sweep: many small caches with seeded random shapes (batch, heads,
GQA group, lengths, buffer, per-sequence k, values with their own k, storage, E4M3
values, append chunking, a change of k after the appends), each compared with the
oracle: pages and ring bit-exact, outputs within 2e-3."""
import os
import sys

import numpy as np
import pytest

import swan_inputs as si
from oracle import swan_oracle as O
from tests import swan_cases as C

pytestmark = pytest.mark.gpu
TOL = 2e-3
N_CASES = int(os.environ.get("SWAN_RANDOM_CASES", "64"))  # a wider sweep on request


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _case(i):
    r = si.rng_for(31337, i)
    Hkv = int(r.choice([1, 2, 3]))
    G = int(r.choice([1, 2, 3, 4, 8]))
    dtype = "f32" if r.random() < 0.2 else "f16"
    values = "e4m3" if (dtype == "f16" and r.random() < 0.4) else "same"
    B = int(r.integers(1, 6))
    b = int(r.choice([0, 1, 7, 16, 64, 130]))
    Ls = [int(x) for x in r.integers(1, 700, B)]
    ks = [int(x) for x in r.integers(1, 129, B)]
    chunking = str(r.choice(["one", "two", "steps"]))
    # drawn from a stream of their own, so the draws above stay those of earlier versions
    r2 = si.rng_for(31339, i)
    kvs = [int(x) for x in r2.integers(1, 129, B)] if r2.random() < 0.4 else None
    change = None
    if r2.random() < 0.4:
        change = ([int(x) for x in r2.integers(1, 129, B)],
                  [int(x) for x in r2.integers(1, 129, B)] if r2.random() < 0.5 else None)
    return dict(Hkv=Hkv, Hq=Hkv * G, dtype=dtype, values=values, B=B, b=b, Ls=Ls, ks=ks,
                kvs=kvs, change=change, chunking=chunking)


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_cache_matches_oracle(gpu_device, swan_mod, torch_mod, i):
    torch = torch_mod
    c = _case(i)
    _log(f"random case {i}: {c}")
    np_dt = si.np_dtype(c["dtype"])
    B, Hq, Hkv, b = c["B"], c["Hq"], c["Hkv"], c["b"]
    Ls, ks = c["Ls"], c["ks"]
    Lmax = max(Ls)
    Pqk = np.stack([si.random_orthogonal(7000 + 10 * i + h, 128) for h in range(Hkv)]).astype(
        np.float32)
    Pvo = np.stack([si.random_orthogonal(8000 + 10 * i + h, 128) for h in range(Hkv)]).astype(
        np.float32)
    K = np.zeros((B, Hkv, Lmax, 128), np_dt)
    V = np.zeros((B, Hkv, Lmax, 128), np_dt)
    for bi in range(B):
        for h in range(Hkv):
            R = si.haar_orthogonal(si.rng_for(9000, i, h), 128)
            K[bi, h] = si.lowrank_rows(si.rng_for(9001, i, bi, h), Lmax, R).astype(np_dt)
            V[bi, h] = si.lowrank_rows(si.rng_for(9002, i, bi, h), Lmax, R).astype(np_dt)
    kvs = c["kvs"]
    cache = swan_mod.SwanCache(B, Hq, Hkv, b, max(Lmax - b, 1), ks, C.torch_dtype(c["dtype"]),
                               gpu_device, sparse_values=c["values"], k_value=kvs)
    tqk = torch.tensor(Pqk, device=gpu_device)
    tvo = torch.tensor(Pvo, device=gpu_device)
    if c["chunking"] == "one":
        cuts = [0, Lmax]
    elif c["chunking"] == "two":
        cuts = [0, Lmax // 3, Lmax]
    else:  # a long prefill, then single-token steps
        cuts = [0, max(Lmax - 5, 0)] + list(range(max(Lmax - 4, 1), Lmax + 1))
    for t0, t1 in zip(cuts[:-1], cuts[1:]):
        if t1 <= t0:
            continue
        per = [max(min(t1, L) - t0, 0) for L in Ls]
        cache.append(torch.tensor(K[:, :, t0:t1], device=gpu_device),
                     torch.tensor(V[:, :, t0:t1], device=gpu_device), tqk, tvo, n_new_per_seq=per)
    torch.cuda.synchronize()
    assert cache.seq_len == Ls
    ov = "e4m3" if c["values"] == "e4m3" else "t"
    oc = [[O.compress_block(K[bi, h, :Ls[bi]], V[bi, h, :Ls[bi]], Pqk[h], Pvo[h], b, ks[bi], np_dt,
                            values=ov, k_value=None if kvs is None else kvs[bi])
           for h in range(Hkv)] for bi in range(B)]
    if c["change"] is not None:
        ks1, kvs1 = c["change"]
        cache.change_k(ks1, kvs1)
        oc = [[O.change_k_cache(u, ks1[bi], None if kvs1 is None else kvs1[bi]) for u in oc[bi]]
              for bi in range(B)]
    for bi in range(B):
        h = bi % Hkv
        C.compare_unit(cache, oc[bi][h], bi, h, Ls[bi], np_dt, values=c["values"])
    q = si.rng_for(31338, i).standard_normal((B, Hq, 128)).astype(np_dt)
    out = cache.decode(torch.tensor(q, device=gpu_device), tqk, tvo)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(got))
    ref = O.decode_batch(q.astype(np.float64), Pqk, Pvo, oc)
    err = C.max_rel_err(got, ref)
    _log(f"  max rel err {err:.2e}")
    assert err <= TOL
