"""swan_decode_attention_noalloc: the decode entry point that takes no workspace
and allocates nothing (its scratch is a device array inside the library).

Through the C ABI it must give the same bytes as swan_decode_attention with a
caller workspace on the same cache, on two calls in a row, the second one
smaller, and match the oracle to 2e-3 per (sequence, query head).
"""
import sys

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


def _both(swan, torch, cache, q, tP_qk, tP_vo):
    """(output of swan_decode_attention with a workspace, output of the no-alloc call)."""
    ref = torch.full_like(q, float("nan"))
    got = torch.full_like(q, float("nan"))
    swan.decode_attention(cache.desc, cache.seq_len, cache.k_active, q, tP_qk, tP_vo, ref,
                          cache.workspace(), k_value=cache.k_value)
    swan.decode_attention_noalloc(cache.desc, cache.seq_len, cache.k_active, q, tP_qk, tP_vo,
                                  got, k_value=cache.k_value)
    torch.cuda.synchronize()
    return ref, got


def _against_oracle(out, q, oc, Pqk, Pvo, G):
    B, Hq, _ = q.shape
    o = out.cpu().numpy().astype(np.float64)
    qn = q.cpu().numpy().astype(np.float64)
    worst = 0.0
    for b in range(B):
        for hq in range(Hq):
            h = hq // G
            ref = O.attend_arrays(qn[b, hq], Pqk[h], Pvo[h], oc[b][h])
            worst = max(worst, C.max_rel_err(o[b, hq][None], ref[None]))
    return worst


def test_noalloc_matches_workspace_call_two_calls(gpu_device, swan_mod, torch_mod):
    torch = torch_mod
    # first call: GQA (2 query heads per KV head), fp16, ragged lengths and a k per
    # sequence in three page formats (several attention launches, all on one stream)
    _log("no-alloc decode, call 1: B=3, Hq=4, Hkv=2, fp16, L=[700, 300, 1000], k=[48, 32, 96]")
    cache, oc, Pqk, Pvo, tP_qk, tP_vo, *_ = _build(
        swan_mod, torch, gpu_device, B=3, Hq=4, Hkv=2, L=[700, 300, 1000], b=16,
        k_active=[48, 32, 96], dtype="f16", seed=3, wid=120)
    q = torch.tensor(si.queries_host(120, 3, 4, "f16"), device=gpu_device)
    ref, got = _both(swan_mod, torch, cache, q, tP_qk, tP_vo)
    assert torch.equal(ref.view(torch.int16), got.view(torch.int16))
    err = _against_oracle(got, q, oc, Pqk, Pvo, 2)
    _log(f"  bit-equal to the workspace call; oracle err {err:.2e}")
    assert err <= TOL
    # second call, smaller: MHA, fp32, two sequences (fewer units and partials)
    _log("no-alloc decode, call 2: B=2, Hq=Hkv=2, fp32, L=[200, 90], k=[24, 64]")
    cache2, oc2, Pqk2, Pvo2, tP_qk2, tP_vo2, *_ = _build(
        swan_mod, torch, gpu_device, B=2, Hq=2, Hkv=2, L=[200, 90], b=8, k_active=[24, 64],
        dtype="f32", seed=4, wid=121)
    q2 = torch.tensor(si.queries_host(121, 2, 2, "f32"), device=gpu_device)
    ref2, got2 = _both(swan_mod, torch, cache2, q2, tP_qk2, tP_vo2)
    assert torch.equal(ref2.view(torch.int32), got2.view(torch.int32))
    err2 = _against_oracle(got2, q2, oc2, Pqk2, Pvo2, 1)
    _log(f"  bit-equal to the workspace call; oracle err {err2:.2e}")
    assert err2 <= TOL
    # and the first cache again after the smaller call left its partials behind
    ref3, got3 = _both(swan_mod, torch, cache, q, tP_qk, tP_vo)
    assert torch.equal(ref.view(torch.int16), got3.view(torch.int16))
    assert torch.equal(ref3.view(torch.int16), got3.view(torch.int16))


def test_noalloc_rejects_a_batch_larger_than_its_scratch(gpu_device, swan_mod, torch_mod):
    """More partials than the scratch holds: SWAN_ERR_WORKSPACE, and the output untouched."""
    torch = torch_mod
    swan = swan_mod
    B, Hq = 64, 256
    desc = swan.CacheDesc(B, Hq, Hq, 128, 1, 0, swan.SWAN_F16, 0, None, None, None, None)
    ring = torch.zeros((B, Hq, 1, 128), dtype=torch.float16, device=gpu_device)
    desc.k_ring = desc.v_ring = ring.data_ptr()
    P = torch.zeros((Hq, 128, 128), dtype=torch.float32, device=gpu_device)
    q = torch.zeros((B, Hq, 128), dtype=torch.float16, device=gpu_device)
    out = torch.full_like(q, 7.0)
    need = swan.decode_workspace_bytes(desc, [1] * B, [48] * B)
    assert need > swan.NOALLOC_SCRATCH_BYTES
    with pytest.raises(swan.SwanError) as ei:
        swan.decode_attention_noalloc(desc, [1] * B, [48] * B, q, P, P, out)
    assert ei.value.status == swan.SWAN_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
