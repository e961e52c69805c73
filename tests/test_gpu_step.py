"""swan_decode_step, one decode step of Algorithm 1 in one call (the query
rotation runs inside the append launch), against the two calls it stands for
(compress-append of one token, then decode attention): outputs, pages and ring
bit for bit at every step, then the cache and the last output against the
oracle."""
import os
import sys

import numpy as np
import pytest

import swan_inputs as si
from oracle import swan_oracle as O
from tests import swan_cases as C
from tests.test_gpu_parity import TOL, _build

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _fresh_cache(swan_mod, torch_mod, device, K, V, tqk, tvo, *, Hq, Hkv, b, cap, ks, kv,
                 dtype, values, L0):
    cache = swan_mod.SwanCache(len(ks), Hq, Hkv, b, cap, ks, C.torch_dtype(dtype), device,
                               sparse_values=values, k_value=kv)
    if L0 > 0:
        cache.append(torch_mod.tensor(K[:, :, :L0], device=device),
                     torch_mod.tensor(V[:, :, :L0], device=device), tqk, tvo)
    return cache


CASES = [
    # Hq, Hkv, dtype, values, b, L0, k_active, k_value
    (4, 4, "f16", "same", 16, 200, [48, 64], None),      # MHA, an eviction every step
    (8, 2, "f16", "same", 16, 200, [32, 32], None),      # GQA, G = 4
    (6, 2, "f16", "same", 16, 150, [64, 40], None),      # G = 3
    (4, 2, "f16", "same", 16, 150, [1, 128], None),      # G = 2, extreme k
    (16, 2, "f16", "same", 16, 150, [48, 48], None),     # G = 8
    (32, 2, "f16", "same", 16, 150, [48, 40], None),     # G = 16: the separate query rotation
    (4, 4, "f32", "same", 8, 130, [48, 17], None),
    (8, 2, "f16", "e4m3", 16, 200, [64, 64], None),
    (4, 4, "f16", "e4m3", 16, 200, [48, 24], None),
    (4, 4, "f16", "same", 16, 200, [77, 48], [51, 48]),  # keys and values of their own k
    (4, 2, "f16", "same", 0, 150, [48, 48], None),       # no buffer: pruned on arrival
    (4, 4, "f16", "same", 64, 10, [48, 48], None),       # all in the buffer, no eviction
    (4, 4, "f16", "same", 16, 0, [48, 48], None),        # the first token of an empty cache
]


def _steps_against_two_calls(gpu_device, swan_mod, torch_mod, Hq, Hkv, dtype, values, b, L0, ks,
                             kv, steps=3):
    torch = torch_mod
    B, L = len(ks), L0 + steps
    np_dt = si.np_dtype(dtype)
    # the rows, rotations and oracle caches at the final length
    _, oc, Pqk, Pvo, tqk, tvo, K, V = _build(swan_mod, torch_mod, gpu_device, B=B, Hq=Hq,
                                             Hkv=Hkv, L=L, b=b, k_active=ks, dtype=dtype,
                                             values=values, k_value=kv)
    cap = max(L - b, 1)
    kw = dict(Hq=Hq, Hkv=Hkv, b=b, cap=cap, ks=ks, kv=kv, dtype=dtype, values=values, L0=L0)
    two = _fresh_cache(swan_mod, torch_mod, gpu_device, K, V, tqk, tvo, **kw)
    one = _fresh_cache(swan_mod, torch_mod, gpu_device, K, V, tqk, tvo, **kw)
    for s in range(steps):
        t = L0 + s
        kn = torch.tensor(K[:, :, t:t + 1], device=gpu_device)
        vn = torch.tensor(V[:, :, t:t + 1], device=gpu_device)
        q = si.queries_host(99, B, Hq, dtype, step=s)
        tq = torch.tensor(q, device=gpu_device)
        two.append(kn, vn, tqk, tvo)
        out_two = two.decode(tq, tqk, tvo)
        out_one = one.step(kn, vn, tq, tqk, tvo)
        torch.cuda.synchronize()
        assert one.seq_len == two.seq_len == [t + 1] * B
        assert torch.equal(out_one, out_two), f"step {s}: outputs differ"
    for name in ("k_pages", "v_pages", "k_ring", "v_ring"):
        assert torch.equal(getattr(one, name), getattr(two, name)), name
    for bi in range(B):
        for h in range(Hkv):
            C.compare_unit(one, oc[bi][h], bi, h, L, np_dt, values=values)
    ref = O.decode_batch(q.astype(np.float64), Pqk, Pvo, oc)
    err = C.max_rel_err(out_one.cpu().numpy().astype(np.float64), ref)
    _log(f"  last step vs oracle: max rel err {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("Hq,Hkv,dtype,values,b,L0,ks,kv", CASES)
def test_decode_step_equals_append_then_decode(gpu_device, swan_mod, torch_mod, Hq, Hkv, dtype,
                                               values, b, L0, ks, kv):
    _log(f"decode_step Hq={Hq} Hkv={Hkv} {dtype}/{values} b={b} L0={L0} k={ks} kv={kv}")
    _steps_against_two_calls(gpu_device, swan_mod, torch_mod, Hq, Hkv, dtype, values, b, L0, ks,
                             kv)


def test_decode_step_error_leaves_the_cache(gpu_device, swan_mod, torch_mod):
    """A workspace too small for the lengths after the step is rejected before the
    append is enqueued: pages, ring and lengths stay as they were."""
    torch = torch_mod
    B, Hq, Hkv, L0, b, ks = 2, 4, 2, 120, 16, [48, 48]
    _, oc, Pqk, Pvo, tqk, tvo, K, V = _build(swan_mod, torch_mod, gpu_device, B=B, Hq=Hq,
                                             Hkv=Hkv, L=L0 + 1, b=b, k_active=ks, dtype="f16")
    cache = _fresh_cache(swan_mod, torch_mod, gpu_device, K, V, tqk, tvo, Hq=Hq, Hkv=Hkv, b=b,
                         cap=L0 + 1 - b, ks=ks, kv=None, dtype="f16", values="same", L0=L0)
    torch.cuda.synchronize()
    before = {n: getattr(cache, n).clone() for n in ("k_pages", "v_pages", "k_ring", "v_ring")}
    need = swan_mod.decode_workspace_bytes(cache.desc, [L0 + 1] * B, ks)
    small = torch.empty(need - 256, dtype=torch.uint8, device=gpu_device)
    kn = torch.tensor(K[:, :, L0:L0 + 1], device=gpu_device)
    vn = torch.tensor(V[:, :, L0:L0 + 1], device=gpu_device)
    q = torch.tensor(si.queries_host(99, B, Hq, "f16"), device=gpu_device)
    out = torch.empty_like(q)
    with pytest.raises(swan_mod.SwanError) as ex:
        swan_mod.decode_step(cache.desc, cache.seq_len, ks, kn, vn, q, tqk, tvo, out, small)
    assert ex.value.status == swan_mod.SWAN_ERR_WORKSPACE
    torch.cuda.synchronize()
    for n, t in before.items():
        assert torch.equal(getattr(cache, n), t), n
    assert cache.seq_len == [L0] * B
    # the same step with a large enough workspace then matches the oracle
    out = cache.step(kn, vn, q, tqk, tvo)
    torch.cuda.synchronize()
    ref = O.decode_batch(q.cpu().numpy().astype(np.float64), Pqk, Pvo, oc)
    assert C.max_rel_err(out.cpu().numpy().astype(np.float64), ref) <= TOL


@pytest.mark.parametrize("Hq,Hkv,ks", [
    (4, 4, [48, 48]),  # one attention launch
    (8, 2, [48, 48]),  # one GQA launch
    (4, 4, [32, 96]),  # two k_pad, one fused launch
    (8, 2, [32, 96]),  # two GQA launches on side streams
])
def test_profile_events_time_the_attention(gpu_device, swan_mod, torch_mod, Hq, Hkv, ks):
    """The profiling hook times the attention launches inside a decode call, and
    what is computed does not change with it."""
    _log(f"profile events Hq={Hq} Hkv={Hkv} k={ks}")
    torch = torch_mod
    cache, oc, Pqk, Pvo, tqk, tvo, *_ = _build(swan_mod, torch_mod, gpu_device, B=2, Hq=Hq,
                                                Hkv=Hkv, L=700, b=16, k_active=ks, dtype="f16")
    q = torch.tensor(si.queries_host(99, 2, Hq, "f16"), device=gpu_device)
    ref = cache.decode(q, tqk, tvo)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in ev:  # torch creates the HIP events on their first record
        e.record()
    torch.cuda.synchronize()
    swan_mod.set_profile_events(ev[0], ev[1])
    try:
        ev[2].record()
        out = cache.decode(q, tqk, tvo)
        ev[3].record()
    finally:
        swan_mod.set_profile_events(None, None)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    t_attn, t_call = ev[0].elapsed_time(ev[1]), ev[2].elapsed_time(ev[3])
    _log(f"  attention {t_attn * 1e3:.1f} us of the call's {t_call * 1e3:.1f} us")
    assert 0.0 < t_attn <= t_call
    err = C.max_rel_err(out.cpu().numpy().astype(np.float64),
                        O.decode_batch(q.cpu().numpy().astype(np.float64), Pqk, Pvo, oc))
    assert err <= TOL


N_RANDOM = int(os.environ.get("SWAN_RANDOM_STEPS", "24"))  # a wider sweep on request


def _random_case(i):
    r = si.rng_for(42421, i)
    Hkv = int(r.choice([1, 2, 3]))
    G = int(r.choice([1, 2, 3, 4, 5, 8]))
    dtype = "f32" if r.random() < 0.2 else "f16"
    values = "e4m3" if (dtype == "f16" and r.random() < 0.4) else "same"
    B = int(r.integers(1, 5))
    b = int(r.choice([0, 1, 2, 7, 16, 64]))
    L0 = int(r.integers(0, 400))
    ks = [int(x) for x in r.integers(1, 129, B)]
    kv = [int(x) for x in r.integers(1, 129, B)] if r.random() < 0.3 else None
    return dict(Hq=Hkv * G, Hkv=Hkv, dtype=dtype, values=values, b=b, L0=L0, ks=ks, kv=kv)


@pytest.mark.parametrize("i", range(N_RANDOM))
def test_random_decode_steps(gpu_device, swan_mod, torch_mod, i):
    """Seeded random shapes: swan_decode_step against append + decode bit for bit over
    four steps (lengths crossing the buffer size on the way), then the oracle."""
    c = _random_case(i)
    _log(f"random decode steps {i}: {c}")
    _steps_against_two_calls(gpu_device, swan_mod, torch_mod, c["Hq"], c["Hkv"], c["dtype"],
                             c["values"], c["b"], c["L0"], c["ks"], c["kv"], steps=4)
