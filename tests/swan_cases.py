"""Shared set-up for the GPU parity tests: build caches on the GPU through the
C ABI and the same caches with the oracle, from the same seeded input bytes."""
import numpy as np

import swan_inputs as si
from oracle import swan_oracle as O
from tests import swan_layout as lay


def torch_dtype(dtype: str):
    import torch

    return {"f16": torch.float16, "f32": torch.float32}[dtype]


def gpu_calibrate(rows_np, device):
    """P (float32 numpy) computed by swan_calibrate_rotation on the GPU."""
    import torch

    from paper_2511_18936_amd import swan

    rows = torch.tensor(np.ascontiguousarray(rows_np, dtype=np.float32), device=device)
    P = torch.empty((128, 128), dtype=torch.float32, device=device)
    sig = torch.empty(128, dtype=torch.float32, device=device)
    swan.calibrate_rotation(rows, P, sig)
    return P.cpu().numpy(), sig.cpu().numpy()


def rotations(wid: int, n_kv: int, device, use_gpu: bool = True):
    """P_qk, P_vo [n_kv][128][128] float32 from the recipe's calibration rows."""
    Pqk, Pvo = [], []
    for h in range(n_kv):
        for role, dst in ((si.ROLE_K, Pqk), (si.ROLE_V, Pvo)):
            rows = si.calibration_rows(wid, h, role)
            if use_gpu:
                P, _ = gpu_calibrate(rows, device)
            else:
                P, _ = O.calibrate_f32(rows)
            dst.append(P)
    return np.stack(Pqk), np.stack(Pvo)


def max_rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max_j |got - ref| / max_j |ref| per output row, maximised over rows."""
    got = np.asarray(got, dtype=np.float64).reshape(-1, ref.shape[-1])
    ref = np.asarray(ref, dtype=np.float64).reshape(-1, ref.shape[-1])
    num = np.max(np.abs(got - ref), axis=1)
    den = np.max(np.abs(ref), axis=1)
    return float(np.max(num / den))


def unit_pages(cache, b, h, role, n_tokens, dtype_np):
    """(idx, val, pad_idx, pad_val) of one unit's sparse tokens read back from the GPU."""
    esize = np.dtype(dtype_np).itemsize
    ks = role_k(cache, role)
    s, e = lay.unit_slice(ks, cache.desc.n_kv_heads, cache.desc.sparse_capacity, esize, b, h)
    pages = cache.k_pages if role == 0 else cache.v_pages
    raw = pages[s:e].cpu().numpy()
    return lay.unpack(raw, dtype_np, ks[b], n_tokens)


def role_k(cache, role):
    """Per-sequence k of the keys (role 0) or of the values (role 1)."""
    if role == 1 and getattr(cache, "k_value", None) is not None:
        return cache.k_value
    return cache.k_active


def ring_rows(cache, b, h, role, L):
    """The dense buffer rows of one unit in position order (oldest first)."""
    bb = cache.desc.buffer_tokens
    ring = (cache.k_ring if role == 0 else cache.v_ring)[b, h].cpu().numpy()
    nb = min(L, bb)
    pos = np.arange(L - nb, L)
    return ring[pos % bb] if bb else ring[:0]


def compare_unit(cache, oc, b, h, L, dtype_np, values: str = "same"):
    """Bit-exact comparison of one unit's GPU cache with the oracle's cache dict
    (values="e4m3": the sparse values as E4M3 codes, the ring in dtype_np)."""
    S = oc["n_sparse"]
    assert S == max(L - cache.desc.buffer_tokens, 0)
    e4m3 = values == "e4m3"
    for role, r in enumerate(("k", "v")):
        idx, val, pidx, pval = unit_pages(cache, b, h, role, S, np.uint8 if e4m3 else dtype_np)
        bad = np.nonzero(np.any(idx != oc[f"{r}_idx"], axis=1))[0]
        assert bad.size == 0, f"role {role}: {bad.size} of {S} tokens select other indices"
        want_val = oc[f"{r}_code"] if e4m3 else np.asarray(oc[f"{r}_val"], dtype_np)
        assert np.array_equal(val.view(np.uint8), np.asarray(want_val).view(np.uint8)), \
            f"role {role}: values differ"
        if pidx.size:  # padding: value +0 at the lowest dims not kept
            assert np.all(pval.view(np.uint8) == 0)
            free = np.ones((S, 128), dtype=bool)
            np.put_along_axis(free, np.asarray(oc[f"{r}_idx"], dtype=np.int64), False, axis=1)
            # the free dims of each token in ascending order (stable sort puts True first)
            lowest = np.argsort(~free, axis=1, kind="stable")[:, : pidx.shape[1]]
            bad = np.nonzero(np.any(pidx != lowest, axis=1))[0]
            assert bad.size == 0, f"role {role}: padding of tokens {bad[:5]}"
        buf = ring_rows(cache, b, h, role, L)
        want = oc[f"{r}_buf"]
        assert np.array_equal(np.asarray(buf).view(np.uint8),
                              np.asarray(want, dtype_np).view(np.uint8)), f"role {role}: ring"
