"""Plain CPU oracle for SWAN decode attention (TEST INFRASTRUCTURE ONLY).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  The product path (``libswan.so`` and its
Python binding) never calls it and shares no code with it.

Everything is computed in float64 with numpy, step by step in the order the
paper states the method (SWAN: Sparse Winnowed Attention, arXiv 2511.18936):

* ``calibrate``            Sec. 4.1.2: the projection is the right singular
                           matrix of the joint activation matrix S, columns in
                           descending singular value.
* ``joint_matrices`` / ``calibrate_joint``  Sec. 4.1.1-4.1.2: per KV head, S_QK
                           stacks the grouped queries over the keys and S_VO the
                           values over the group's transposed W_O head blocks
                           (reading 14).
* ``rotate`` / ``to_storage``  Algorithm 1 (project the key; the value arrives
                           projected): x_hat = x . P, rounded once to the
                           storage type T when it enters the dense buffer.
* ``topk_indices``         Algorithm 1 (arg TopK of |x_hat_old|) and Sec. 4.3
                           (magnitude pruning), ranking the stored T values,
                           ties to the lower index.
* ``UnitCache.append``     Algorithm 1: append to the buffer, and while the
                           buffer holds more than b vectors pop the oldest, prune
                           it and append the (index, value) pairs to the sparse
                           cache (Sec. 5.1: values plus int8 indices).
* ``UnitCache.attend``     Algorithm 1 (scores over Concat(sparse, buffer),
                           softmax with 1/sqrt(d_h), weighted sum of values) and
                           Sec. 4.2 / Lemma 2: the rotated output is mapped back
                           with P_VO^T.
* ``space_bytes`` / ``flops_swan`` / ``break_even_length``  Sec. 5.1 and Sec. 5.2
                           with Appendix A.2.
* ``to_e4m3_codes``        8-bit sparse values (reading 9), by brute force over
                           the format's 127 finite magnitudes.
* ``k_value``              keys and values pruned to different k (reading 10,
                           the key/value ablation of Appendix A.5, Table 2).
* ``change_k_rows`` / ``UnitCache.change_k``  k changed for a running sequence
                           (reading 11: k_active is a run-time input of
                           Algorithm 1, Sec. 1 / Sec. 3).
* ``rope`` / ``absorbed_weights`` / ``layer_decode``  a Llama-shaped attention
                           layer around the cache: RoPE before the rotation
                           (Sec. 4.2), W_V and W_O absorbing P_VO (Sec. 4.2,
                           Lemma 2), readings 12-13.

Readings of the paper used here (where it is silent or ambiguous):
  1. top-k ranks the stored (T-rounded) buffer value, because Algorithm 1 pops
     the vector from the buffer;
  2. equal magnitudes go to the lower index; +0 and -0 tie;
  3. pairs are kept in ascending index order (the CSR convention of Sec. 5.1);
  4. the current token is appended before attention, so it attends to itself;
  5. with b = 0 every token, the current one included, is pruned at once;
  6. the scale is 1/sqrt(d_h) for the full head dimension, whatever k is;
  7. q_hat, scores, probabilities and the accumulator are never rounded to T;
  8. the output is returned un-rotated: o = o_hat . P_VO^T;
  9. 8-bit sparse values (Sec. 4.3, Sec. 5.1 name 8-bit values without a
     format) are OCP FP8 E4M3 without a scale: the kept T values, rounded to the
     nearest E4M3 value (ties to the even code, saturating at +-448); the
     selection still ranks the T values (reading 1) and the buffer stays T;
 10. Algorithm 1 prunes keys and values to the same k_active; the ablation of
     Appendix A.5 (Table 2) retains different fractions of the key and the value
     dimensions.  Here a key keeps its k_active largest components and a value
     its k_value largest, by the same rule (readings 1-3); k_value defaults to
     k_active.  A retention ratio r maps to round(r * d_h) components;
 11. k changed for a running sequence (Algorithm 1 takes k_active as an input
     at every step).  Lowering it to k' re-prunes the tokens already in the
     sparse cache: each keeps the k' largest of its stored values (ties to the
     lower index), which for values stored in T is exactly its top-k' (the
     top-k' of a top-k set, under one tie rule) and for 8-bit values ranks the
     stored codes.  Raising it keeps their pairs (they were pruned with the k of
     their step, as Algorithm 1 does) and fills the new slots with value 0 at
     the lowest dims not kept, after the kept pairs.  Tokens that leave the
     buffer afterwards are pruned with the new k;
 12. RoPE (the rotary embedding of the Llama models the paper evaluates): dims
     j and j + d/2 of a head rotate by pos * base^(-2j/d), computed in float64
     and rounded once to T; the SWAN rotation takes the rounded post-RoPE rows,
     as it would take a model's post-RoPE tensors;
 13. the absorbed layer: q, k and v_hat = x . W_V_hat are the model's tensors,
     each rounded once to T from a float64 product; W_V_hat = W_V . P_VO and
     W_O_hat = P_VO^T . W_O per head are formed in float64; the values enter
     the cache without a further rotation and the attention output leaves it
     rotated, straight into W_O_hat;
 14. the joint matrices (Sec. 4.1.1-4.1.2): KV head j serves query heads
     jG .. jG + G - 1 (the reshape of Q to N_kv x nG x d_h keeps consecutive
     heads together); W_O's head blocks are its consecutive d_h-row blocks; the
     tensors are stacked as they are, without scaling or mean removal, and the
     row order inside S does not change its right singular vectors.

Parity status: every function above is pinned by tests/test_oracle_pins.py;
nothing here is "parity unpinned" except the end-task accuracy of Tables 1-3,
which needs models and datasets and is not computed.
"""
from __future__ import annotations

import collections
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

F64 = np.float64


# --------------------------------------------------------------------------- #
# Sec. 4.1.2: projection matrices from the SVD of the joint matrix S
# --------------------------------------------------------------------------- #
def canonical_signs(P: np.ndarray) -> np.ndarray:
    """Make the largest-magnitude entry of every column positive (ties: lowest row).

    Singular vectors are defined up to sign; this only makes them reproducible.
    The attention output does not depend on the choice (|-x| = |x|).
    """
    P = np.array(P, dtype=F64, copy=True)
    for j in range(P.shape[1]):
        col = P[:, j]
        r = int(np.argmax(np.abs(col)))  # argmax returns the first (lowest) row on ties
        if col[r] < 0:
            P[:, j] = -col
    return P


def calibrate(S: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """P = right singular matrix of S (columns = basis vectors, descending sigma).

    S is the n x d joint matrix (rows stacked along the sequence axis, Sec. 4.1.2);
    no mean is removed.  Returns (P [d][d] float64, sigma [d] float64).
    """
    S = np.asarray(S, dtype=F64)
    n, d = S.shape
    # the right singular matrix is d x d either way; the thin factorisation skips
    # the n x n left factor, which only a short S (n < d) needs for a square V
    _, sig, vt = np.linalg.svd(S, full_matrices=n < d)
    sigma = np.zeros(d, dtype=F64)
    sigma[: sig.shape[0]] = sig
    P = vt.T  # columns are the right singular vectors, already in descending sigma
    return canonical_signs(P), sigma


def calibrate_f32(S: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """The fp32 rotation that both the oracle and the GPU path then consume."""
    P, sigma = calibrate(S)
    return P.astype(np.float32), sigma.astype(np.float32)


# --------------------------------------------------------------------------- #
# Sec. 4.1.1-4.1.2: the joint matrices of a layer's calibration activations
# --------------------------------------------------------------------------- #
def joint_matrices(Q: np.ndarray, K: np.ndarray, V: np.ndarray, W_o: np.ndarray,
                   n_kv_heads: int) -> Tuple[List[np.ndarray], List[np.ndarray]]:
    """S_QK and S_VO of every KV head j (Sec. 4.1.1-4.1.2), float64.

    Q [N_q][n][d_h]: post-RoPE queries of the calibration tokens, K [N_kv][n][d_h]
    post-RoPE keys, V [N_kv][n][d_h] values, W_o [N_q d_h][d] the output weights.
    The G = N_q / N_kv query heads of KV head j are heads jG .. jG + G - 1.  The
    query tensor is reshaped to Q_grouped [N_kv][n G][d_h]; W_O is sliced into
    its N_q head blocks W_O^(h) [d_h][d] (rows h d_h .. (h + 1) d_h - 1), grouped
    the same way.  S_QK^(j) stacks Q_grouped^(j) over K^(j); S_VO^(j) stacks V^(j)
    over the transposed blocks W_O^(h)^T [d][d_h] of the group's heads.
    """
    Q = np.asarray(Q, dtype=F64)
    K = np.asarray(K, dtype=F64)
    V = np.asarray(V, dtype=F64)
    W_o = np.asarray(W_o, dtype=F64)
    n_q, n, d_h = Q.shape
    G = n_q // n_kv_heads
    Q_grouped = Q.reshape(n_kv_heads, n * G, d_h)
    blocks = W_o.reshape(n_q, d_h, W_o.shape[1])  # W_O^(h)
    S_qk, S_vo = [], []
    for j in range(n_kv_heads):
        S_qk.append(np.concatenate([Q_grouped[j], K[j]], axis=0))
        wo_t = [blocks[h].T for h in range(j * G, (j + 1) * G)]
        S_vo.append(np.concatenate([V[j]] + wo_t, axis=0))
    return S_qk, S_vo


def calibrate_joint(Q: np.ndarray, K: np.ndarray, V: np.ndarray, W_o: np.ndarray,
                    n_kv_heads: int) -> Tuple[np.ndarray, np.ndarray]:
    """P_QK, P_VO [N_kv][d_h][d_h] (float64): the right singular matrices of each
    KV head's joint matrices (Sec. 4.1.2)."""
    S_qk, S_vo = joint_matrices(Q, K, V, W_o, n_kv_heads)
    return (np.stack([calibrate(S)[0] for S in S_qk]),
            np.stack([calibrate(S)[0] for S in S_vo]))


# --------------------------------------------------------------------------- #
# Algorithm 1: rotation, rounding to storage, magnitude top-k
# --------------------------------------------------------------------------- #
def rotate(x: np.ndarray, P: np.ndarray) -> np.ndarray:
    """x_hat = x . P for row vectors x (float64, not rounded)."""
    return np.asarray(x, dtype=F64) @ np.asarray(P, dtype=F64)


def to_storage(y: np.ndarray, dtype) -> np.ndarray:
    """Round once, to nearest-even, to the storage type T (the buffer's type)."""
    return np.asarray(y, dtype=F64).astype(dtype)


def topk_indices(y: np.ndarray, k: int) -> np.ndarray:
    """arg TopK(|y|, k): the k largest magnitudes, lower index first on ties.

    Returned in ascending index order (the order in which pairs are stored).
    """
    mag = np.abs(np.asarray(y, dtype=F64))
    d = mag.shape[0]
    order = np.lexsort((np.arange(d), -mag))  # primary key -|y|, secondary key index
    return np.sort(order[:k])


def topk_indices_rows(Y: np.ndarray, k: int) -> np.ndarray:
    """Row-wise ``topk_indices`` for a [n][d] block (stable sort keeps index order on ties)."""
    mag = np.abs(np.asarray(Y, dtype=F64))
    order = np.argsort(-mag, axis=1, kind="stable")[:, :k]
    return np.sort(order, axis=1)


def change_k_rows(idx: np.ndarray, val: np.ndarray, k_new: int, d: int,
                  code: Optional[np.ndarray] = None):
    """Stored pairs [n][k_old] of n tokens, laid out again for k_new (reading 11).

    k_new <= k_old: each token keeps its k_new largest stored magnitudes, lower
    index first on ties, in ascending index order.  k_new > k_old: each token
    keeps its pairs and gains k_new - k_old entries of value 0 at its lowest
    dims not kept, placed after them in ascending order.  ``code`` (8-bit
    values) follows ``val``.  Returns (idx, val, code).
    """
    idx = np.asarray(idx, dtype=np.int64)
    val = np.asarray(val)
    n, k_old = idx.shape
    if k_new <= k_old:
        mag = np.abs(val.astype(F64))
        keep = np.zeros((n, k_new), dtype=np.int64)
        for t in range(n):  # rank by (-|value|, index), keep the first k_new
            order = np.lexsort((idx[t], -mag[t]))[:k_new]
            keep[t] = order[np.argsort(idx[t][order])]
        pick = lambda a: None if a is None else np.take_along_axis(np.asarray(a), keep, 1)
        return pick(idx), pick(val), pick(code)
    extra = k_new - k_old
    fill = np.zeros((n, extra), dtype=np.int64)
    for t in range(n):
        fill[t] = np.setdiff1d(np.arange(d), idx[t])[:extra]
    zeros = np.zeros((n, extra), dtype=val.dtype)
    out_code = None if code is None else np.concatenate(
        [np.asarray(code), np.zeros((n, extra), dtype=np.asarray(code).dtype)], 1)
    return np.concatenate([idx, fill], 1), np.concatenate([val, zeros], 1), out_code


def change_k_cache(cache: Dict[str, np.ndarray], k_new: int, k_value_new: Optional[int] = None,
                   d: int = 128) -> Dict[str, np.ndarray]:
    """``change_k_rows`` applied to both roles of a cache dict (``compress_block``'s)."""
    out = dict(cache)
    for r, k in (("k", k_new), ("v", k_new if k_value_new is None else k_value_new)):
        i, v, c = change_k_rows(cache[f"{r}_idx"], cache[f"{r}_val"], k, d,
                                cache.get(f"{r}_code"))
        out[f"{r}_idx"], out[f"{r}_val"] = i, v
        if c is not None:
            out[f"{r}_code"] = c
    return out


# --------------------------------------------------------------------------- #
# Algorithm 1: hybrid cache of one (sequence, kv head) unit
# --------------------------------------------------------------------------- #
# 8-bit sparse values (Sec. 4.3, Sec. 5.1; reading 9: OCP FP8 E4M3, no scale)
# --------------------------------------------------------------------------- #
def e4m3_magnitudes() -> np.ndarray:
    """The 127 finite non-negative E4M3 values, indexed by their 7-bit code:
    exponent field e = code >> 3 (bias 7), mantissa m = code & 7; e = 0 is
    subnormal (m * 2^-9); code 127 (all ones) is NaN and not a value."""
    vals = []
    for code in range(127):
        e, m = code >> 3, code & 7
        vals.append(m * 2.0 ** -9 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7))
    return np.array(vals, dtype=F64)


def to_e4m3_codes(x: np.ndarray) -> np.ndarray:
    """Round each value to the nearest E4M3 value, ties to the even code,
    magnitudes above 448 saturating to 448; returns uint8 codes with the sign in
    bit 7 (-0 keeps its sign).  Brute force: the distance to every magnitude."""
    x = np.asarray(x, dtype=F64)
    flat = x.reshape(-1)
    tbl = e4m3_magnitudes()
    codes = np.empty(flat.shape, dtype=np.uint8)
    step = 1 << 16
    for s0 in range(0, flat.size, step):
        a = np.minimum(np.abs(flat[s0:s0 + step]), tbl[-1])
        dist = np.abs(a[:, None] - tbl[None, :])
        near = dist == dist.min(axis=1, keepdims=True)
        first = np.argmax(near, axis=1)  # the lower code of the nearest ones
        tie = near.sum(axis=1) == 2      # exactly between two codes
        c = np.where(tie & (first % 2 == 1), first + 1, first)
        codes[s0:s0 + step] = c.astype(np.uint8) | (np.signbit(flat[s0:s0 + step]) * 0x80).astype(np.uint8)
    return codes.reshape(x.shape)


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    """Values of E4M3 codes (sign in bit 7); code 0x7f / 0xff is NaN."""
    codes = np.asarray(codes, dtype=np.uint8)
    tbl = np.append(e4m3_magnitudes(), np.nan)
    mag = tbl[codes & 0x7F]
    return np.where(codes & 0x80, -mag, mag)


# --------------------------------------------------------------------------- #
class UnitCache:
    """Sparse cache + dense FIFO buffer of one (sequence, KV head), as in Algorithm 1.

    The buffer holds rotated vectors already rounded to T.  The sparse cache
    holds, per pruned token, ascending indices and the T values at them,
    separately for keys (k_active of them) and values (k_value, reading 10).
    """

    def __init__(self, P_qk: np.ndarray, P_vo: np.ndarray, buffer_tokens: int,
                 k_active: int, dtype=np.float16, values: str = "t",
                 k_value: Optional[int] = None):
        self.P_qk = np.asarray(P_qk, dtype=F64)
        self.P_vo = np.asarray(P_vo, dtype=F64)
        self.b = int(buffer_tokens)
        self.k = int(k_active)
        self.kv = int(k_active if k_value is None else k_value)
        self.dtype = dtype
        self.values = values  # "t": sparse values in T; "e4m3": 8-bit (reading 9)
        self.k_buf: collections.deque = collections.deque()
        self.v_buf: collections.deque = collections.deque()
        self.k_idx: List[np.ndarray] = []
        self.k_val: List[np.ndarray] = []
        self.v_idx: List[np.ndarray] = []
        self.v_val: List[np.ndarray] = []

    def __len__(self) -> int:
        return len(self.k_idx) + len(self.k_buf)

    def append(self, k_row: np.ndarray, v_row: np.ndarray) -> None:
        """Admit one token (Algorithm 1): its rotated key and value, rounded once
        to T, join the dense buffer, which keeps the b most recent tokens; a token
        pushed out of it is retired into the sparse cache."""
        self.k_buf.append(to_storage(rotate(k_row, self.P_qk), self.dtype))
        self.v_buf.append(to_storage(rotate(v_row, self.P_vo), self.dtype))
        while len(self.k_buf) > self.b:
            self._retire(self.k_buf.popleft(), self.v_buf.popleft())

    def _retire(self, k_old: np.ndarray, v_old: np.ndarray) -> None:
        """A token leaving the buffer keeps, per role, the (index, value) pairs of
        its largest stored magnitudes (Sec. 4.3): k of them for the key, k_value
        for the value (reading 10)."""
        for vec, keep, idx_l, val_l in ((k_old, self.k, self.k_idx, self.k_val),
                                        (v_old, self.kv, self.v_idx, self.v_val)):
            i = topk_indices(vec, keep)
            idx_l.append(i)
            val_l.append(self._sparse_value(vec[i]))

    def change_k(self, k_new: int, k_value_new: Optional[int] = None) -> None:
        """Reading 11: the stored tokens laid out again for the new k, which the
        tokens leaving the buffer from now on are pruned with."""
        d = self.P_qk.shape[0]
        kv_new = k_new if k_value_new is None else k_value_new
        for idx_l, val_l, k in ((self.k_idx, self.k_val, k_new), (self.v_idx, self.v_val, kv_new)):
            if idx_l:
                i, v, _ = change_k_rows(np.stack(idx_l), np.stack(val_l), k, d)
                idx_l[:] = list(i)
                val_l[:] = list(v)
        self.k, self.kv = int(k_new), int(kv_new)

    def _sparse_value(self, kept: np.ndarray) -> np.ndarray:
        if self.values == "e4m3":
            return e4m3_decode(to_e4m3_codes(kept))
        return kept

    def sparse_arrays(self) -> Dict[str, np.ndarray]:
        d = self.P_qk.shape[0]
        n = len(self.k_idx)
        def stack(lst, dt, width):
            return np.stack(lst) if lst else np.zeros((0, width), dtype=dt)
        vdt = F64 if self.values == "e4m3" else self.dtype
        return {
            "k_idx": stack(self.k_idx, np.int64, self.k),
            "k_val": stack(self.k_val, vdt, self.k),
            "v_idx": stack(self.v_idx, np.int64, self.kv),
            "v_val": stack(self.v_val, vdt, self.kv),
            "k_buf": np.stack(list(self.k_buf)) if self.k_buf else np.zeros((0, d), self.dtype),
            "v_buf": np.stack(list(self.v_buf)) if self.v_buf else np.zeros((0, d), self.dtype),
            "n_sparse": n,
        }

    def attend(self, q: np.ndarray, scale: Optional[float] = None) -> np.ndarray:
        return attend_arrays(q, self.P_qk, self.P_vo, self.sparse_arrays(), scale)


def compress_block(K_rows: np.ndarray, V_rows: np.ndarray, P_qk: np.ndarray,
                   P_vo: np.ndarray, buffer_tokens: int, k_active: int,
                   dtype=np.float16, values: str = "t",
                   k_value: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Algorithm 1 applied to n tokens of an empty unit, all at once.

    Equal, bit for bit, to n successive ``UnitCache.append`` calls (tested):
    the first max(n - b, 0) tokens end up pruned, the last min(n, b) stay dense.
    With values="e4m3" the kept values are stored as 8-bit codes (reading 9):
    "k_code"/"v_code" hold the codes and "k_val"/"v_val" their values.
    Values keep k_value components (reading 10; default k_active).
    """
    n = K_rows.shape[0]
    b = int(buffer_tokens)
    k_hat = to_storage(rotate(K_rows, P_qk), dtype)
    v_hat = to_storage(rotate(V_rows, P_vo), dtype)
    n_sparse = max(n - b, 0)
    k_idx = topk_indices_rows(k_hat[:n_sparse], k_active)
    v_idx = topk_indices_rows(v_hat[:n_sparse], k_active if k_value is None else k_value)
    out = {
        "k_idx": k_idx,
        "k_val": np.take_along_axis(k_hat[:n_sparse], k_idx, axis=1),
        "v_idx": v_idx,
        "v_val": np.take_along_axis(v_hat[:n_sparse], v_idx, axis=1),
        "k_buf": k_hat[n_sparse:],
        "v_buf": v_hat[n_sparse:],
        "n_sparse": n_sparse,
    }
    if values == "e4m3":
        for r in ("k", "v"):
            out[f"{r}_code"] = to_e4m3_codes(out[f"{r}_val"])
            out[f"{r}_val"] = e4m3_decode(out[f"{r}_code"])
    return out


def attend_arrays(q: np.ndarray, P_qk: np.ndarray, P_vo: np.ndarray,
                  cache: Dict[str, np.ndarray], scale: Optional[float] = None) -> np.ndarray:
    """Algorithm 1, attention part, for one query head on one unit's cache.

    q_hat = q . P_QK; scores = q_hat . K_cache^T over the sparse pairs and the
    dense buffer; softmax of scores / sqrt(d_h); o_hat = p . V_cache; and the
    output is returned to the model's coordinates with P_VO^T (Lemma 2).
    """
    P_qk = np.asarray(P_qk, dtype=F64)
    P_vo = np.asarray(P_vo, dtype=F64)
    d = P_qk.shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    q_hat = rotate(q, P_qk)
    k_idx, k_val = cache["k_idx"], np.asarray(cache["k_val"], dtype=F64)
    v_idx, v_val = cache["v_idx"], np.asarray(cache["v_val"], dtype=F64)
    k_buf = np.asarray(cache["k_buf"], dtype=F64)
    v_buf = np.asarray(cache["v_buf"], dtype=F64)
    # sparse-dense mat-vec: only the kept components of each key contribute
    s_sparse = scale * np.sum(q_hat[k_idx] * k_val, axis=1) if k_idx.shape[0] else np.zeros(0)
    s_buf = scale * (k_buf @ q_hat)
    s = np.concatenate([s_sparse, s_buf])
    if s.shape[0] == 0:
        raise ValueError("attention over an empty cache")
    m = np.max(s)
    w = np.exp(s - m)
    p = w / np.sum(w)
    p_sparse, p_buf = p[: s_sparse.shape[0]], p[s_sparse.shape[0]:]
    o_hat = np.zeros(d, dtype=F64)
    if v_idx.shape[0]:
        np.add.at(o_hat, v_idx.ravel(), (p_sparse[:, None] * v_val).ravel())
    o_hat += p_buf @ v_buf
    return o_hat @ P_vo.T


def decode_batch(q: np.ndarray, P_qk: np.ndarray, P_vo: np.ndarray,
                 caches: Sequence[Sequence[Dict[str, np.ndarray]]],
                 scale: Optional[float] = None) -> np.ndarray:
    """o[b][h_q] for q [B][H_q][d]; caches[b][h_kv]; P [H_kv][d][d].  GQA: h_kv = h_q // G."""
    B, Hq, d = q.shape
    Hkv = len(caches[0])
    G = Hq // Hkv
    out = np.zeros((B, Hq, d), dtype=F64)
    for b in range(B):
        for hq in range(Hq):
            g = hq // G
            out[b, hq] = attend_arrays(q[b, hq], P_qk[g], P_vo[g], caches[b][g], scale)
    return out


# --------------------------------------------------------------------------- #
# A Llama-shaped attention layer around the cache (readings 12-13)
# --------------------------------------------------------------------------- #
def rope(x: np.ndarray, pos: np.ndarray, base: float, dtype=None) -> np.ndarray:
    """Rotary embedding of rows x [..., n, d] at positions pos [n] (reading 12).

    Dims j and j + d/2 rotate by the angle pos * base^(-2j/d); float64, then
    rounded once to ``dtype`` if given.
    """
    x = np.asarray(x, dtype=F64)
    d = x.shape[-1]
    h = d // 2
    inv = base ** (-(2.0 * np.arange(h)) / d)
    ang = np.asarray(pos, dtype=F64)[:, None] * inv[None, :]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :h], x[..., h:]
    y = np.concatenate([a * c - b * s, b * c + a * s], axis=-1)
    return y if dtype is None else y.astype(dtype)


def absorbed_weights(W_v: np.ndarray, W_o: np.ndarray, P_vo: np.ndarray, n_heads: int,
                     n_kv_heads: int):
    """W_V_hat = W_V . P_VO per KV head and W_O_hat = P_VO^T . W_O per query head
    (Sec. 4.2), float64.  W_v [hidden][n_kv * d], W_o [n_q * d][hidden], P_vo [n_kv][d][d]."""
    d = P_vo.shape[-1]
    G = n_heads // n_kv_heads
    Wv = np.asarray(W_v, dtype=F64).copy()
    Wo = np.asarray(W_o, dtype=F64).copy()
    for h in range(n_kv_heads):
        Wv[:, h * d:(h + 1) * d] = Wv[:, h * d:(h + 1) * d] @ P_vo[h]
    for hq in range(n_heads):
        Wo[hq * d:(hq + 1) * d, :] = np.asarray(P_vo[hq // G], dtype=F64).T @ Wo[hq * d:(hq + 1) * d, :]
    return Wv, Wo


def layer_tensors(x: np.ndarray, W_q, W_k, W_v_hat, n_heads: int, n_kv_heads: int,
                  pos: np.ndarray, base: float, dtype):
    """The layer's post-RoPE q, k and absorbed v_hat for rows x [n][hidden] at
    positions pos: each product rounded once to T, RoPE rounded once (13)."""
    d = 128
    n = x.shape[0]
    x = np.asarray(x, dtype=F64)
    q = to_storage(x @ np.asarray(W_q, dtype=F64), dtype).reshape(n, n_heads, d)
    k = to_storage(x @ np.asarray(W_k, dtype=F64), dtype).reshape(n, n_kv_heads, d)
    v = to_storage(x @ np.asarray(W_v_hat, dtype=F64), dtype).reshape(n, n_kv_heads, d)
    q = rope(q.transpose(1, 0, 2), pos, base, dtype).transpose(1, 0, 2)
    k = rope(k.transpose(1, 0, 2), pos, base, dtype).transpose(1, 0, 2)
    return q, k, v


def layer_decode(x_seq: np.ndarray, W_q, W_k, W_v, W_o, P_qk, P_vo, n_heads: int,
                 n_kv_heads: int, base: float, buffer_tokens: int, k_active: int,
                 dtype=np.float16, k_value: Optional[int] = None) -> np.ndarray:
    """Output of the attention layer for the last of the rows x_seq [L][hidden]
    (positions 0..L-1), every row having been appended to the SWAN cache first
    (Algorithm 1 inside the layer, readings 12-13).  Returns y [hidden] float64."""
    L = x_seq.shape[0]
    d = 128
    G = n_heads // n_kv_heads
    W_v_hat, W_o_hat = absorbed_weights(W_v, W_o, P_vo, n_heads, n_kv_heads)
    q, k, v = layer_tensors(x_seq, W_q, W_k, W_v_hat, n_heads, n_kv_heads, np.arange(L), base,
                            dtype)
    eye = np.eye(d)
    o = np.zeros(n_heads * d, dtype=F64)
    for h in range(n_kv_heads):
        # values arrive rotated: the cache's value rotation is the identity
        c = compress_block(k[:, h], v[:, h], P_qk[h], eye, buffer_tokens, k_active, dtype,
                           k_value=k_value)
        for hq in range(h * G, (h + 1) * G):
            o[hq * d:(hq + 1) * d] = attend_arrays(q[L - 1, hq], P_qk[h], eye, c)
    return o @ W_o_hat


# --------------------------------------------------------------------------- #
# Sec. 5.1 space model and Sec. 5.2 / Appendix A.2 FLOP model
# --------------------------------------------------------------------------- #
def space_bytes_per_vector(k_active: int, value_bytes: int = 2, index_bytes: int = 1,
                           offset_bytes: int = 2) -> int:
    """M_sparse = k (sizeof(value) + sizeof(index)) + the 2-byte CSR offset."""
    return k_active * (value_bytes + index_bytes) + offset_bytes


def dense_bytes_per_vector(d_h: int = 128, value_bytes: int = 2) -> int:
    return d_h * value_bytes


def flops_standard(L: int, d_h: int) -> int:
    """C_std ~ 4 L d_h: two mat-vecs over the whole cache."""
    return 4 * L * d_h


def flops_swan(L: int, d_h: int, b: int, k_active: int) -> int:
    """C_SWAN ~ 4 d_h^2 + 4 (L - b) k + 4 b d_h (projections, sparse part, buffer part)."""
    return 4 * d_h * d_h + 4 * (L - b) * k_active + 4 * b * d_h


def break_even_length(d_h: int, k_active: int, b: int) -> float:
    """SWAN is cheaper than standard attention once L exceeds d_h^2 / (d_h - k) + b."""
    return d_h * d_h / (d_h - k_active) + b
