"""Test-side reader/writer of the page layout documented in include/swan.h
(values of 4, 2 or 1 byte: float32, float16 or E4M3 codes as uint8).

Independent of the library: it restates the documented byte layout so that the
tests can (a) read the GPU's pages back into (index, value) pairs and (b) pack
the oracle's pairs into pages for a decode-only parity check.
"""
import numpy as np


def kpad(k: int) -> int:
    return (k + 7) // 8 * 8


def chunk_bytes(esize: int) -> int:
    """Bytes of a value chunk: 16 for 2- and 4-byte values, 8 for one-byte E4M3 codes."""
    return 16 if esize >= 2 else 8


def page_bytes(esize: int, k: int) -> int:
    return 64 * kpad(k) * (esize + 1)


def seq_offsets(k_active, n_kv_heads: int, capacity: int, esize: int):
    npc = (capacity + 63) // 64
    offs, off = [], 0
    for k in k_active:
        offs.append(off)
        off += n_kv_heads * npc * page_bytes(esize, int(k))
    return offs, off


def unit_slice(k_active, n_kv_heads, capacity, esize, b, h):
    """Byte range [start, end) of the pages of (sequence b, kv head h)."""
    offs, _ = seq_offsets(k_active, n_kv_heads, capacity, esize)
    npc = (capacity + 63) // 64
    pb = page_bytes(esize, int(k_active[b]))
    start = offs[b] + h * npc * pb
    return start, start + npc * pb


def unpack(raw: np.ndarray, dtype, k: int, n_tokens: int):
    """(idx [n][k] int64, val [n][k] dtype, pad_idx, pad_val) from a unit's page bytes."""
    esize = np.dtype(dtype).itemsize
    kp = kpad(k)
    cb = chunk_bytes(esize)
    gv = cb // esize
    pb = page_bytes(esize, k)
    npages = (n_tokens + 63) // 64
    raw = np.asarray(raw, dtype=np.uint8)[: npages * pb].reshape(npages, pb)
    vals = raw[:, : 64 * kp * esize].reshape(npages, kp // gv, 64, cb)
    vals = np.ascontiguousarray(vals.transpose(0, 2, 1, 3)).reshape(npages * 64, kp * esize)
    vals = vals.view(dtype).reshape(npages * 64, kp)[:n_tokens]
    idx = raw[:, 64 * kp * esize:].reshape(npages, kp // 8, 64, 8)
    idx = np.ascontiguousarray(idx.transpose(0, 2, 1, 3)).reshape(npages * 64, kp)[:n_tokens]
    idx = idx.astype(np.int64)
    return idx[:, :k], vals[:, :k], idx[:, k:], vals[:, k:]


def pack(idx: np.ndarray, val: np.ndarray, dtype, k: int, n_pages: int) -> np.ndarray:
    """Page bytes of one unit from pairs idx/val [n][k] (ascending idx per row)."""
    esize = np.dtype(dtype).itemsize
    kp = kpad(k)
    cb = chunk_bytes(esize)
    gv = cb // esize
    n = idx.shape[0]
    vfull = np.zeros((n_pages * 64, kp), dtype=dtype)
    ifull = np.zeros((n_pages * 64, kp), dtype=np.uint8)
    vfull[:n, :k] = val
    ifull[:n, :k] = idx
    for t in range(n):  # padding: value 0 at the lowest dims not kept
        if kp > k:
            free = np.setdiff1d(np.arange(128), idx[t])[: kp - k]
            ifull[t, k:] = free
    vb = vfull.view(np.uint8).reshape(n_pages, 64, kp // gv, cb).transpose(0, 2, 1, 3)
    ib = ifull.reshape(n_pages, 64, kp // 8, 8).transpose(0, 2, 1, 3)
    out = np.concatenate([vb.reshape(n_pages, -1), ib.reshape(n_pages, -1)], axis=1)
    return np.ascontiguousarray(out).reshape(-1)
