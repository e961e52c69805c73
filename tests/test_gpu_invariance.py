"""Invariances of the decode path that the oracle cannot see directly.

* Split-count invariance: Algorithm 1's softmax runs over Concat(sparse cache,
  buffer) whatever the kernels cut the token axis into, so one cache decoded
  under several split plans (swan_set_decode_tuning) gives outputs within 1e-6 of
  each other (only the order of float32 additions differs) and within 2e-3 of the
  oracle.
* Cache round trip (checkpoint / resume): the library keeps no state between
  calls, so pages and ring copied to the host and back into new arrays continue
  exactly like the original: the next append and decode are bitwise equal.
* Two threads, each with its own stream and a batch that mixes page formats
  (one fused launch on the MHA path; on the GQA path each uses its thread's side
  streams), decode concurrently and both match the oracle.
"""
import sys
import threading

import numpy as np
import pytest

import swan_inputs as si
from oracle import swan_oracle as O
from tests import swan_cases as C
from tests.test_gpu_parity import _build

pytestmark = pytest.mark.gpu
TOL = 2e-3


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _oracle_err(out, q, oc, Pqk, Pvo, G):
    o = out.cpu().numpy().astype(np.float64)
    qn = q.cpu().numpy().astype(np.float64)
    worst = 0.0
    for b in range(q.shape[0]):
        for hq in range(q.shape[1]):
            ref = O.attend_arrays(qn[b, hq], Pqk[hq // G], Pvo[hq // G], oc[b][hq // G])
            worst = max(worst, C.max_rel_err(o[b, hq][None], ref[None]))
    return worst


PLANS = [
    dict(),                                   # the default plan
    dict(target_waves=1),                     # one split per (sequence, head)
    dict(target_waves=1 << 20),               # as many splits as the one-page rule allows
    dict(target_waves=97, short_split_pages=-1),
    dict(target_waves=5000, short_split_pages=1),
]


@pytest.mark.parametrize("dtype,Hq,Hkv,values", [
    ("f16", 4, 4, "same"), ("f16", 8, 2, "same"), ("f32", 2, 2, "same"), ("f16", 4, 2, "e4m3"),
])
def test_outputs_do_not_depend_on_the_split_plan(gpu_device, swan_mod, torch_mod, dtype, Hq,
                                                 Hkv, values):
    torch, swan = torch_mod, swan_mod
    Ls = [3000, 700, 130, 2049]
    ks = [48, 24, 64, 96]
    _log(f"split plans: {dtype} Hq={Hq} Hkv={Hkv} values={values} L={Ls} k={ks}")
    cache, oc, Pqk, Pvo, tP_qk, tP_vo, *_ = _build(
        swan, torch, gpu_device, B=4, Hq=Hq, Hkv=Hkv, L=Ls, b=16, k_active=ks, dtype=dtype,
        seed=7, wid=130, values=values)
    q = torch.tensor(si.queries_host(130, 4, Hq, dtype), device=gpu_device)
    outs, sizes = [], []
    try:
        for plan in PLANS:
            swan.set_decode_tuning(**plan)
            ws = torch.empty(swan.decode_workspace_bytes(cache.desc, cache.seq_len, ks),
                             dtype=torch.uint8, device=gpu_device)
            sizes.append(ws.numel())
            out = torch.empty_like(q)
            swan.decode_attention(cache.desc, cache.seq_len, ks, q, tP_qk, tP_vo, out, ws)
            torch.cuda.synchronize()
            outs.append(out.cpu().numpy().astype(np.float64))
    finally:
        swan.set_decode_tuning()
    assert len(set(sizes)) >= 3, sizes  # the plans really differ
    base = outs[0].reshape(-1, 128)
    for o in outs[1:]:
        d = C.max_rel_err(o.reshape(-1, 128), base)
        # fp32 accumulation in another order, then one rounding to the storage type:
        # at most one ulp of the output apart (fp16: 2^-11 of the row's largest |o|)
        bound = 1e-6 if dtype == "f32" else 2.0 ** -10
        assert d <= bound, (d, bound)
    for o in outs:
        err = _oracle_err(torch.tensor(o), q, oc, Pqk, Pvo, Hq // Hkv)
        assert err <= TOL
    _log(f"  workspace sizes {sizes}; outputs agree")


def test_split_plans_agree_to_1e6_before_output_rounding(gpu_device, swan_mod, torch_mod):
    """With the output left in fp32 (fp32 storage) the plans agree to 1e-6 relative."""
    torch, swan = torch_mod, swan_mod
    Ls = [5000, 64, 1000]
    cache, oc, Pqk, Pvo, tP_qk, tP_vo, *_ = _build(
        swan, torch, gpu_device, B=3, Hq=4, Hkv=2, L=Ls, b=32, k_active=[40, 40, 40],
        dtype="f32", seed=8, wid=131)
    q = torch.tensor(si.queries_host(131, 3, 4, "f32"), device=gpu_device)
    outs = []
    try:
        for plan in PLANS:
            swan.set_decode_tuning(**plan)
            outs.append(cache.decode(q, tP_qk, tP_vo).cpu().numpy().astype(np.float64))
            cache._ws = None
    finally:
        swan.set_decode_tuning()
    for o in outs[1:]:
        assert C.max_rel_err(o.reshape(-1, 128), outs[0].reshape(-1, 128)) <= 1e-6


def _clone_through_host(swan, torch, cache):
    """A new cache whose arrays hold the original's bytes, copied to the host and back."""
    c2 = swan.SwanCache(cache.batch, cache.desc.n_q_heads, cache.desc.n_kv_heads,
                        cache.desc.buffer_tokens, cache.desc.sparse_capacity, cache.k_active,
                        cache.dtype, cache.device, sparse_values=cache.sparse_values,
                        k_value=cache.k_value)
    for name in ("k_pages", "v_pages", "k_ring", "v_ring"):
        host = getattr(cache, name).cpu().numpy().copy()
        getattr(c2, name).copy_(torch.from_numpy(host).to(cache.device))
    c2.seq_len = list(cache.seq_len)
    return c2


@pytest.mark.parametrize("dtype,values,kv", [("f16", "same", None), ("f16", "e4m3", [30, 70]),
                                             ("f32", "same", None)])
def test_cache_round_trip_through_host_memory(gpu_device, swan_mod, torch_mod, dtype, values,
                                              kv):
    torch, swan = torch_mod, swan_mod
    Ls = [900, 150]
    _log(f"round trip: {dtype} values={values} k_value={kv}")
    cache, _, Pqk, Pvo, tP_qk, tP_vo, K, V = _build(
        swan, torch, gpu_device, B=2, Hq=4, Hkv=2, L=Ls, b=16, k_active=[48, 61], dtype=dtype,
        seed=9, wid=132, values=values, k_value=kv, capacity=1200)
    c2 = _clone_through_host(swan, torch, cache)
    np_dt = si.np_dtype(dtype)
    rng = si.rng_for(132, 99)
    for step in range(3):
        kn = torch.tensor(rng.standard_normal((2, 2, 5, 128)).astype(np_dt), device=gpu_device)
        vn = torch.tensor(rng.standard_normal((2, 2, 5, 128)).astype(np_dt), device=gpu_device)
        q = torch.tensor(rng.standard_normal((2, 4, 128)).astype(np_dt), device=gpu_device)
        for c in (cache, c2):
            c.append(kn, vn, tP_qk, tP_vo)
        o1 = cache.decode(q, tP_qk, tP_vo)
        o2 = c2.decode(q, tP_qk, tP_vo)
        torch.cuda.synchronize()
        assert cache.seq_len == c2.seq_len
        for name in ("k_pages", "v_pages", "k_ring", "v_ring"):
            a, b = getattr(cache, name), getattr(c2, name)
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), (step, name)
        assert torch.equal(o1.view(torch.uint8), o2.view(torch.uint8)), step


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (4, 2)])
def test_two_threads_on_two_streams(gpu_device, swan_mod, torch_mod, Hq, Hkv):
    """Two callers, each on its own thread and stream with a mixed-k batch (one
    fused launch for MHA; side streams of its own thread for GQA): both outputs
    match the oracle."""
    torch, swan = torch_mod, swan_mod
    _log(f"two threads Hq={Hq} Hkv={Hkv}")
    setups = []
    for i in range(2):
        cache, oc, Pqk, Pvo, tP_qk, tP_vo, *_ = _build(
            swan, torch, gpu_device, B=4, Hq=Hq, Hkv=Hkv, L=[2000 + 300 * i, 900, 1500, 400],
            b=16, k_active=[96, 64, 48, 24], dtype="f16", seed=10 + i, wid=133)
        q = torch.tensor(si.queries_host(133 + i, 4, Hq, "f16"), device=gpu_device)
        setups.append((cache, oc, Pqk, Pvo, tP_qk, tP_vo, q))
    outs = [None, None]
    errors = []

    def run(i):
        try:
            cache, _, _, _, tP_qk, tP_vo, q = setups[i]
            st = torch.cuda.Stream(device=gpu_device)
            with torch.cuda.stream(st):
                ws = cache.workspace()
                res = []
                for _ in range(20):
                    res.append(cache.decode(q, tP_qk, tP_vo, stream=st))
            st.synchronize()
            outs[i] = res
        except Exception as e:  # reported by the main thread
            errors.append(e)

    ts = [threading.Thread(target=run, args=(i,)) for i in range(2)]
    for t in ts:
        t.start()
    for t in ts:
        t.join(timeout=120)
    assert not errors, errors
    for i, (cache, oc, Pqk, Pvo, *_rest, q) in enumerate(setups):
        res = outs[i]
        for o in res[1:]:
            assert torch.equal(o, res[0])
        err = _oracle_err(res[0], q, oc, Pqk, Pvo, Hq // Hkv)
        _log(f"thread {i}: oracle err {err:.2e}")
        assert err <= TOL
