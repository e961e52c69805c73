"""Parity at the benchmark's full sizes, in the launch configuration bench.py times.

The GPU builds the whole cache (prefill compress of L-1 tokens, then the decode
step's append of the current token) and decodes every (sequence, query head);
the oracle recomputes a seeded sample of units one by one from the same input
bytes, copied back from the device: indices and values bit-exact, outputs
within 2e-3 (max |o - o_ref| / max |o_ref| per query head).
"""
import sys

import numpy as np
import pytest

import swan_inputs as si
from oracle import swan_oracle as O
from tests import swan_cases as C

pytestmark = pytest.mark.gpu
TOL = 2e-3


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _run(device, name: str, n_units: int):
    import torch

    from paper_2511_18936_amd import swan

    w = si.WORKLOADS[name]
    np_dt = si.np_dtype(w.dtype)
    ks = [int(k) for k in si.k_active_for(w)]
    kvs = si.k_value_for(w)
    kvs = None if kvs is None else [int(k) for k in kvs]
    L = w.context
    _log(f"[{name}] calibrating {2 * w.n_kv_heads} rotations")
    Pqk = torch.empty((w.n_kv_heads, 128, 128), dtype=torch.float32, device=device)
    Pvo = torch.empty_like(Pqk)
    for h in range(w.n_kv_heads):
        swan.calibrate_rotation(
            torch.tensor(si.calibration_rows(w.wid, h, si.ROLE_K), device=device), Pqk[h])
        swan.calibrate_rotation(
            torch.tensor(si.calibration_rows(w.wid, h, si.ROLE_V), device=device), Pvo[h])
    _log(f"[{name}] drawing K/V on the device, prefill {L - 1} + 1 token")
    K = si.kv_rows_device(w.wid, w.batch, w.n_kv_heads, si.ROLE_K, L - 1, w.dtype, device)
    V = si.kv_rows_device(w.wid, w.batch, w.n_kv_heads, si.ROLE_V, L - 1, w.dtype, device)
    K1 = si.kv_rows_device(w.wid, w.batch, w.n_kv_heads, si.ROLE_K, 1, w.dtype, device, block=1)
    V1 = si.kv_rows_device(w.wid, w.batch, w.n_kv_heads, si.ROLE_V, 1, w.dtype, device, block=1)
    q = si.queries_device(w.wid, w.batch, w.n_q_heads, w.dtype, device)
    cache = swan.SwanCache(w.batch, w.n_q_heads, w.n_kv_heads, w.buffer, L - w.buffer, ks,
                           C.torch_dtype(w.dtype), device, sparse_values=w.sparse_values,
                           k_value=kvs)
    vals = "e4m3" if w.sparse_values == "e4m3" else "t"
    cache.append(K, V, Pqk, Pvo)
    cache.append(K1, V1, Pqk, Pvo)
    out = cache.decode(q, Pqk, Pvo)
    torch.cuda.synchronize()
    assert cache.seq_len == [L] * w.batch
    assert bool(torch.isfinite(out).all())
    P_qk, P_vo = Pqk.cpu().numpy(), Pvo.cpu().numpy()
    out_np = out.cpu().numpy().astype(np.float64)
    q_np = q.cpu().numpy().astype(np.float64)
    rng = si.rng_for(4242, w.wid)
    units = [(int(u // w.n_kv_heads), int(u % w.n_kv_heads))
             for u in rng.choice(w.batch * w.n_kv_heads, size=n_units, replace=False)]
    G = w.group
    worst = 0.0
    for b, h in units:
        Kh = np.concatenate([K[b, h].cpu().numpy(), K1[b, h].cpu().numpy()])
        Vh = np.concatenate([V[b, h].cpu().numpy(), V1[b, h].cpu().numpy()])
        oc = O.compress_block(Kh, Vh, P_qk[h], P_vo[h], w.buffer, ks[b], np_dt, values=vals,
                              k_value=None if kvs is None else kvs[b])
        C.compare_unit(cache, oc, b, h, L, np_dt, values=w.sparse_values)
        for hq in range(h * G, (h + 1) * G):
            ref = O.attend_arrays(q_np[b, hq], P_qk[h], P_vo[h], oc)
            err = C.max_rel_err(out_np[b, hq][None], ref[None])
            worst = max(worst, err)
        kv_txt = "" if kvs is None else f"/{kvs[b]}"
        _log(f"[{name}] unit (b={b}, h={h}, k={ks[b]}{kv_txt}): pages and ring bit-exact, "
             f"worst output err so far {worst:.2e}")
    assert worst <= TOL


def test_llama2_7b_32k_batch16(gpu_device):
    _run(gpu_device, "llama2_7b_L32k_b16", 8)


def test_llama3_8b_gqa_128k_batch4(gpu_device):
    _run(gpu_device, "llama3_8b_gqa_L128k_b4", 8)


def test_prefill16k_batch8_per_sequence_k(gpu_device):
    _run(gpu_device, "llama2_7b_prefill16k_b8", 8)


def test_llama2_7b_32k_batch16_e4m3_values(gpu_device):
    _run(gpu_device, "llama2_7b_L32k_b16_e4m3", 8)


def test_llama2_7b_32k_batch16_keys77_values51(gpu_device):
    _run(gpu_device, "llama2_7b_L32k_b16_k77_v51", 8)


def test_llama3_8b_gqa_128k_batch4_keys77_values51(gpu_device):
    _run(gpu_device, "llama3_8b_gqa_L128k_b4_k77_v51", 8)
