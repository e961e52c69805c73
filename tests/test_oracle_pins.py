"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests retypes the oracle's own formula: each checks it against an
independent route (exact rational arithmetic, a constructed SVD, brute-force
loops over a dense masked formulation, Lemma 1 / Lemma 2 of Appendix A.1, or
numbers printed in the paper), chosen so that a dropped term, a wrong sign or
index, a transposed operand or a wrong tie rule fails at least one of them.
"""
import fractions
import math
import os

import numpy as np
import pytest

import swan_inputs as si
from oracle import swan_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------- #
# Rounding to the storage type: exact nearest-even by rational arithmetic
# --------------------------------------------------------------------------- #
def _fp16_grid_neighbors(x: float):
    """All fp16 values as exact fractions around x (finite range only)."""
    h = np.float16(x)
    cands = set()
    bits = np.array([h], dtype=np.float16).view(np.uint16)[0]
    for dlt in (-2, -1, 0, 1, 2):
        b = (int(bits) + dlt) & 0xFFFF
        v = np.array([b], dtype=np.uint16).view(np.float16)[0]
        if np.isfinite(v):
            cands.add(float(v))
    return sorted(cands)


def _exact_nearest_even_fp16(x: float) -> float:
    fx = fractions.Fraction(x)
    best = None
    for c in _fp16_grid_neighbors(x):
        fc = fractions.Fraction(c)
        dist = abs(fc - fx)
        if best is None or dist < best[0]:
            best = (dist, [c])
        elif dist == best[0]:
            best[1].append(c)
    cands = best[1]
    if len(cands) == 1:
        return cands[0]
    # tie: pick the one with an even mantissa (last bit 0)
    for c in cands:
        if int(np.array([c], dtype=np.float16).view(np.uint16)[0]) % 2 == 0:
            return c
    raise AssertionError("no even candidate")


def test_to_storage_fp16_is_round_to_nearest_even():
    r = np.random.default_rng(1)
    xs = list(r.standard_normal(3000) * np.exp(r.uniform(-12, 8, 3000)))
    # exact midpoints between consecutive fp16 values, and doubles one ulp off them
    grid = np.array(r.integers(0x0400, 0x7B00, 400), dtype=np.uint16).view(np.float16)
    for g in grid.astype(np.float64):
        up = float(np.nextafter(np.float16(g), np.float16(np.inf)))
        mid = (g + up) / 2.0
        xs += [mid, -mid, np.nextafter(mid, 0.0), np.nextafter(mid, np.inf)]
    got = O.to_storage(np.array(xs), np.float16).astype(np.float64)
    want = np.array([_exact_nearest_even_fp16(x) for x in xs])
    assert np.array_equal(got, want)


# --------------------------------------------------------------------------- #
# Sec. 4.1.2 calibration: right singular vectors, descending sigma
# --------------------------------------------------------------------------- #
def test_calibrate_recovers_a_constructed_svd():
    d, n = 16, 40
    V = si.random_orthogonal(3, d)
    U = si.random_orthogonal(4, n)[:, :d]
    sig = np.linspace(9.0, 1.0, d) ** 1.5  # distinct, descending
    perm = si.rng_for(77).permutation(d)  # hand the SVD its columns shuffled
    S = (U[:, perm] * sig[perm]) @ V[:, perm].T
    P, sigma = O.calibrate(S)
    assert np.allclose(sigma, sig, rtol=1e-12, atol=0)
    # every column of P is +/- the matching column of V
    assert np.allclose(np.abs(np.sum(P * V, axis=0)), 1.0, atol=1e-12)
    # canonical sign: the largest-magnitude entry of each column is positive
    for j in range(d):
        assert P[np.argmax(np.abs(P[:, j])), j] > 0


def test_calibrate_orthogonal_columns_give_a_sorted_permutation():
    # S with orthogonal columns of distinct norms: the basis is the identity, sorted by norm
    norms = np.array([2.0, 7.0, 3.0, 5.0, 1.0, 4.0])
    S = np.zeros((10, 6))
    for j, nj in enumerate(norms):
        S[j, j] = -nj if j % 2 else nj
    P, sigma = O.calibrate(S)
    order = np.argsort(-norms)
    want = np.zeros((6, 6))
    want[order, np.arange(6)] = 1.0
    assert np.array_equal(P, want)
    assert np.allclose(sigma, norms[order])


def test_calibrate_on_the_synthetic_recipe():
    S = si.calibration_rows(0, 0, si.ROLE_K).astype(np.float64)
    P, sigma = O.calibrate(S)
    d = S.shape[1]
    assert np.max(np.abs(P.T @ P - np.eye(d))) < 1e-12
    # eigen-equation of the Gram matrix, checked column by column
    G = S.T @ S
    resid = np.linalg.norm(G @ P - P * sigma**2, axis=0) / sigma[0] ** 2
    assert np.max(resid) < 1e-12
    assert np.all(np.diff(sigma) <= 0)
    # closed form of the recipe: sigma_j ~ sqrt(n) s_j for the leading directions
    s = si.spectrum(d)
    ratio = sigma[:5] / (math.sqrt(S.shape[0]) * s[:5])
    assert np.all(np.abs(ratio - 1) < 0.05)
    # fp32 copy stays orthogonal to fp32 precision
    P32, _ = O.calibrate_f32(S)
    P32 = P32.astype(np.float64)
    assert np.max(np.abs(P32.T @ P32 - np.eye(d))) < 1e-6


# --------------------------------------------------------------------------- #
# Algorithm 1 arg TopK: brute force and special cases
# --------------------------------------------------------------------------- #
def _brute_topk(y, k):
    order = sorted(range(len(y)), key=lambda j: (-abs(float(y[j])), j))
    return sorted(order[:k])


# --------------------------------------------------------------------------- #
# Sec. 4.1.1-4.1.2: the joint matrices of a layer (reading 14)
# --------------------------------------------------------------------------- #
@pytest.mark.parametrize("n_q,n_kv", [(8, 2), (4, 4), (6, 3)])
def test_joint_matrices_brute_force_grouping(n_q, n_kv):
    """Each KV head's matrices, assembled row by row with explicit head and token
    loops: query head h belongs to KV head h // G, and W_O^(h) is rows h d_h ..
    (h + 1) d_h - 1 of W_O, entering S_VO transposed."""
    d_h, n, d = 8, 5, 6
    r = si.rng_for(9001, n_q, n_kv)
    Q = r.standard_normal((n_q, n, d_h))
    K = r.standard_normal((n_kv, n, d_h))
    V = r.standard_normal((n_kv, n, d_h))
    W_o = r.standard_normal((n_q * d_h, d))
    S_qk, S_vo = O.joint_matrices(Q, K, V, W_o, n_kv)
    G = n_q // n_kv
    for j in range(n_kv):
        rows = []
        for h in range(n_q):
            if h // G == j:
                for t in range(n):
                    rows.append([Q[h][t][c] for c in range(d_h)])
        for t in range(n):
            rows.append([K[j][t][c] for c in range(d_h)])
        assert np.array_equal(S_qk[j], np.array(rows))
        rows = [[V[j][t][c] for c in range(d_h)] for t in range(n)]
        for h in range(n_q):
            if h // G == j:
                for col in range(d):  # row col of W_O^(h)^T
                    rows.append([W_o[h * d_h + i][col] for i in range(d_h)])
        assert np.array_equal(S_vo[j], np.array(rows))


def test_joint_matrices_mark_each_head():
    """Constant marker rows: query head h's rows are (h + 1) e_h, W_O block h holds
    1000 (h + 1) + row; each KV head's matrices hold exactly its group's marks."""
    n_q, n_kv, d_h, n, d = 8, 2, 8, 3, 4
    Q = np.zeros((n_q, n, d_h))
    for h in range(n_q):
        Q[h, :, h] = h + 1
    K = np.zeros((n_kv, n, d_h))
    V = np.zeros((n_kv, n, d_h))
    W_o = np.zeros((n_q * d_h, d))
    for h in range(n_q):
        W_o[h * d_h:(h + 1) * d_h, :] = 1000 * (h + 1) + np.arange(d_h)[:, None]
    S_qk, S_vo = O.joint_matrices(Q, K, V, W_o, n_kv)
    for j, heads in enumerate(([0, 1, 2, 3], [4, 5, 6, 7])):
        marks = sorted({int(x) for x in S_qk[j].ravel() if x})
        assert marks == [h + 1 for h in heads]
        wo_part = S_vo[j][n:]
        assert wo_part.shape == (len(heads) * d, d_h)
        for gi, h in enumerate(heads):
            block = wo_part[gi * d:(gi + 1) * d]
            assert np.array_equal(block, np.tile(1000 * (h + 1) + np.arange(d_h), (d, 1)))


def test_joint_calibration_reduces_to_single_tensor_calibration():
    """Special cases with a plain answer: queries equal to the keys (each row
    twice) and zero output weights leave the right singular vectors of K and V
    alone, so calibrate_joint equals calibrate on K and on V; and the row order
    inside S does not matter."""
    n_kv, n, d_h = 2, 300, 16
    r = si.rng_for(9002)
    scales = np.exp(-np.arange(d_h) / 3.0)
    K = r.standard_normal((n_kv, n, d_h)) * scales
    V = r.standard_normal((n_kv, n, d_h)) * scales[::-1]
    Q = K.copy()  # G = 1, MHA
    W_o = np.zeros((n_kv * d_h, 7))
    P_qk, P_vo = O.calibrate_joint(Q, K, V, W_o, n_kv)
    for j in range(n_kv):
        assert np.allclose(P_qk[j], O.calibrate(K[j])[0], atol=1e-9)
        assert np.allclose(P_vo[j], O.calibrate(V[j])[0], atol=1e-9)
        S_qk, _ = O.joint_matrices(Q, K, V, W_o, n_kv)
        perm = r.permutation(S_qk[j].shape[0])
        assert np.allclose(O.calibrate(S_qk[j][perm])[0], P_qk[j], atol=1e-9)


@pytest.mark.parametrize("d", [4, 8, 16, 128])
def test_topk_brute_force_with_many_ties(d):
    r = si.rng_for(11, d)
    for trial in range(200):
        y = r.integers(-3, 4, d).astype(np.float64) * (0.5 if trial % 2 else 1.0)
        if trial % 3 == 0:
            y[r.integers(0, d, 2)] = -0.0
        for k in sorted({1, 2, d // 2, d - 1, d}):
            assert list(O.topk_indices(y, k)) == _brute_topk(y, k)
        Y = np.stack([y, -y, y[::-1]])
        for k in (1, d // 2, d):
            rows = O.topk_indices_rows(Y, k)
            for i in range(3):
                assert list(rows[i]) == _brute_topk(Y[i], k)


def test_topk_special_cases():
    y = np.array([1.0, -1.0] * 8)
    assert list(O.topk_indices(y, 5)) == [0, 1, 2, 3, 4]
    y = np.array([0.0, -0.0, 0.0, -0.0])
    assert list(O.topk_indices(y, 2)) == [0, 1]
    y = np.array([0.1, -0.7, 0.7, 0.2])
    assert list(O.topk_indices(y, 1)) == [1]  # argmax of |y|, lowest index on the tie
    assert list(O.topk_indices(y, 4)) == [0, 1, 2, 3]
    y = np.float16(np.array([3.0, -5.0, 1.0, 5.0, -2.0]))
    assert list(O.topk_indices(y, 3)) == [0, 1, 3]


# --------------------------------------------------------------------------- #
# Algorithm 1 end to end: brute force over a dense masked formulation
# --------------------------------------------------------------------------- #
def _brute_swan(q, K, V, Pqk, Pvo, b, k, dtype, kv=None):
    """Independent restatement with Python loops.

    Token t (0-based) of L is dense if t >= L - b, else its key is pruned to the
    k largest-magnitude rotated components (ties: lower index) and its value to
    the kv largest (kv = k unless given), the rest zeroed.
    """
    kv = k if kv is None else kv
    d = len(q)
    L = len(K)
    def rot(x, P):
        return [sum(float(x[i]) * float(P[i][j]) for i in range(d)) for j in range(d)]
    def rnd(v):
        return [float(np.asarray(x).astype(dtype)) for x in v]
    qh = rot(q, Pqk)
    scores, vrows = [], []
    for t in range(L):
        kh = rnd(rot(K[t], Pqk))
        vh = rnd(rot(V[t], Pvo))
        if t < L - b:
            for vec, kk in ((kh, k), (vh, kv)):
                keep = sorted(range(d), key=lambda j: (-abs(vec[j]), j))[:kk]
                for j in range(d):
                    if j not in keep:
                        vec[j] = 0.0
        scores.append(sum(qh[j] * kh[j] for j in range(d)) / math.sqrt(d))
        vrows.append(vh)
    m = max(scores)
    w = [math.exp(s - m) for s in scores]
    z = sum(w)
    oh = [sum(w[t] / z * vrows[t][j] for t in range(L)) for j in range(d)]
    return [sum(oh[j] * float(Pvo[i][j]) for j in range(d)) for i in range(d)]


@pytest.mark.parametrize("dtype", [np.float64, np.float16])
@pytest.mark.parametrize("d", [4, 8])
def test_attention_brute_force_tiny(d, dtype):
    for L in (1, 2, 5, 12):
        q, K, V = si.tiny_case(L * 10 + d, d, L)
        Pqk = si.random_orthogonal(L + 1, d)
        Pvo = si.random_orthogonal(L + 2, d)
        for k in range(1, d + 1):
            for b in range(0, L + 2):
                uc = O.UnitCache(Pqk, Pvo, b, k, dtype)
                for t in range(L):
                    uc.append(K[0, t], V[0, t])
                got = uc.attend(q[0])
                want = _brute_swan(q[0], K[0], V[0], Pqk, Pvo, b, k, dtype)
                assert np.allclose(got, want, rtol=1e-12, atol=1e-12), (L, k, b)


@pytest.mark.parametrize("dtype", [np.float64, np.float16])
@pytest.mark.parametrize("d", [4, 8])
def test_attention_brute_force_tiny_asymmetric_k(d, dtype):
    """Appendix A.5 (Table 2): keys and values pruned to different k (reading 10)."""
    pairs = [(kk, kv) for kk in range(1, d + 1) for kv in range(1, d + 1) if kk != kv]
    if d == 8:
        pairs = [(1, 8), (8, 1), (2, 7), (5, 3), (3, 6), (7, 4)]
    for L in (1, 5, 12):
        q, K, V = si.tiny_case(L * 13 + d, d, L)
        Pqk = si.random_orthogonal(L + 3, d)
        Pvo = si.random_orthogonal(L + 4, d)
        for kk, kv in pairs:
            for b in (0, 2, L):
                uc = O.UnitCache(Pqk, Pvo, b, kk, dtype, k_value=kv)
                for t in range(L):
                    uc.append(K[0, t], V[0, t])
                got = uc.attend(q[0])
                want = _brute_swan(q[0], K[0], V[0], Pqk, Pvo, b, kk, dtype, kv)
                assert np.allclose(got, want, rtol=1e-12, atol=1e-12), (L, kk, kv, b)
                arr = uc.sparse_arrays()
                assert arr["k_idx"].shape == (max(L - b, 0), kk)
                assert arr["v_idx"].shape == (max(L - b, 0), kv)


# --------------------------------------------------------------------------- #
# Appendix A.1, Lemma 1 and Lemma 2: the rotation itself is lossless
# --------------------------------------------------------------------------- #
def _textbook_attention(q, K, V):
    s = K @ q / math.sqrt(len(q))
    w = np.exp(s - s.max())
    return (w / w.sum()) @ V


@pytest.mark.parametrize("d,L", [(8, 30), (128, 300)])
def test_full_retention_equals_dense_attention(d, L):
    q, K, V = si.tiny_case(5, d, L)
    Pqk = si.random_orthogonal(6, d)
    Pvo = si.random_orthogonal(7, d)
    want = _textbook_attention(q[0], K[0], V[0])
    for b in (0, 3, L, L + 5):
        c = O.compress_block(K[0], V[0], Pqk, Pvo, b, d, np.float64)
        got = O.attend_arrays(q[0], Pqk, Pvo, c)
        assert np.allclose(got, want, rtol=0, atol=1e-12 * np.abs(want).max())
    # buffer covering the whole context: dense whatever k is
    c = O.compress_block(K[0], V[0], Pqk, Pvo, L, 1, np.float64)
    assert np.allclose(O.attend_arrays(q[0], Pqk, Pvo, c), want, atol=1e-12)
    # identity rotation, full retention
    I = np.eye(d)
    c = O.compress_block(K[0], V[0], I, I, 0, d, np.float64)
    assert np.allclose(O.attend_arrays(q[0], I, I, c), want, atol=1e-12)


def test_full_retention_fp16_equals_dense_on_rounded_rotated_rows():
    d, L = 128, 200
    q, K, V = si.tiny_case(8, d, L)
    Pqk = si.random_orthogonal(9, d)
    Pvo = si.random_orthogonal(10, d)
    c = O.compress_block(K[0], V[0], Pqk, Pvo, 16, d, np.float16)
    got = O.attend_arrays(q[0], Pqk, Pvo, c)
    Kh = (K[0] @ Pqk).astype(np.float16).astype(np.float64)
    Vh = (V[0] @ Pvo).astype(np.float16).astype(np.float64)
    want = _textbook_attention(q[0] @ Pqk, Kh, Vh) @ Pvo.T
    assert np.allclose(got, want, rtol=0, atol=1e-13)


# --------------------------------------------------------------------------- #
# Invariances
# --------------------------------------------------------------------------- #
@pytest.mark.parametrize("b,k", [(0, 5), (4, 3), (16, 64), (0, 128)])
def test_prefill_equals_token_by_token_appends(b, k):
    d = 128 if k > 8 else 8
    L = 70
    q, K, V = si.tiny_case(12 + b + k, d, L)
    K16, V16 = K.astype(np.float16), V.astype(np.float16)
    Pqk = si.random_orthogonal(13, d)
    Pvo = si.random_orthogonal(14, d)
    uc = O.UnitCache(Pqk, Pvo, b, k, np.float16)
    for t in range(L):
        uc.append(K16[0, t], V16[0, t])
    a = uc.sparse_arrays()
    c = O.compress_block(K16[0], V16[0], Pqk, Pvo, b, k, np.float16)
    for key in ("k_idx", "k_val", "v_idx", "v_val", "k_buf", "v_buf"):
        assert np.array_equal(a[key], c[key]), key
    assert a["n_sparse"] == c["n_sparse"] == max(L - b, 0)
    assert np.array_equal(uc.attend(q[0]), O.attend_arrays(q[0], Pqk, Pvo, c))


@pytest.mark.parametrize("b,kk,kv", [(0, 77, 51), (8, 13, 115), (4, 128, 1), (16, 51, 77)])
def test_asymmetric_prefill_equals_appends_and_splits_by_role(b, kk, kv):
    """Reading 10: the key side of a (k_key, k_value) cache is the k_key cache's,
    the value side the k_value cache's, and a block equals token-by-token appends."""
    d, L = 128, 70
    q, K, V = si.tiny_case(40 + kk + kv, d, L)
    K16, V16 = K.astype(np.float16), V.astype(np.float16)
    Pqk = si.random_orthogonal(41, d)
    Pvo = si.random_orthogonal(42, d)
    uc = O.UnitCache(Pqk, Pvo, b, kk, np.float16, k_value=kv)
    for t in range(L):
        uc.append(K16[0, t], V16[0, t])
    a = uc.sparse_arrays()
    c = O.compress_block(K16[0], V16[0], Pqk, Pvo, b, kk, np.float16, k_value=kv)
    ck = O.compress_block(K16[0], V16[0], Pqk, Pvo, b, kk, np.float16)
    cv = O.compress_block(K16[0], V16[0], Pqk, Pvo, b, kv, np.float16)
    for key in ("k_idx", "k_val", "v_idx", "v_val", "k_buf", "v_buf"):
        assert np.array_equal(a[key], c[key]), key
    for key in ("k_idx", "k_val"):
        assert np.array_equal(c[key], ck[key]), key
    for key in ("v_idx", "v_val"):
        assert np.array_equal(c[key], cv[key]), key
    assert np.array_equal(uc.attend(q[0]), O.attend_arrays(q[0], Pqk, Pvo, c))


def test_table2_ratios_map_to_components():
    """Appendix A.5, Table 2: the retention pairs sum to 1, so k_key + k_value = d_h."""
    for rk in range(1, 10):
        kk, kv = round(rk / 10 * 128), round((10 - rk) / 10 * 128)
        assert kk + kv == 128 and 1 <= kk <= 127


# --------------------------------------------------------------------------- #
# Reading 11: k changed for a running sequence
# --------------------------------------------------------------------------- #
def _brute_swan_k_schedule(q, K, V, Pqk, Pvo, b, changes, dtype):
    """Python loops: token t leaves the buffer at step t + b (when token t + b is
    appended) and is pruned with the k then in force; each later change to a smaller
    k re-prunes it, which the nested top-k makes equal to pruning its rotated vector
    at the smallest k in force from its eviction on.  changes: {step: (k, k_value)},
    in force from that step's append on (step 0 gives the initial k)."""
    d, L = len(q), len(K)
    def rot(x, P):
        return [sum(float(x[i]) * float(P[i][j]) for i in range(d)) for j in range(d)]
    def rnd(v):
        return [float(np.asarray(x).astype(dtype)) for x in v]
    def k_at(step):
        return changes[max(s for s in changes if s <= step)]
    eff = {}
    for t in range(L - b):
        ev = t + b  # the step whose append evicts token t
        ks = [k_at(ev)] + [changes[s] for s in changes if ev < s <= L - 1]
        eff[t] = (min(k for k, _ in ks), min(kv for _, kv in ks))
    qh = rot(q, Pqk)
    scores, vrows = [], []
    for t in range(L):
        kh, vh = rnd(rot(K[t], Pqk)), rnd(rot(V[t], Pvo))
        if t in eff:
            for vec, kk in ((kh, eff[t][0]), (vh, eff[t][1])):
                keep = sorted(range(d), key=lambda j: (-abs(vec[j]), j))[:kk]
                for j in range(d):
                    if j not in keep:
                        vec[j] = 0.0
        scores.append(sum(qh[j] * kh[j] for j in range(d)) / math.sqrt(d))
        vrows.append(vh)
    m = max(scores)
    w = [math.exp(s - m) for s in scores]
    z = sum(w)
    oh = [sum(w[t] / z * vrows[t][j] for t in range(L)) for j in range(d)]
    return [sum(oh[j] * float(Pvo[i][j]) for j in range(d)) for i in range(d)]


@pytest.mark.parametrize("dtype", [np.float64, np.float16])
def test_change_k_mid_sequence_brute_force(dtype):
    d, L = 8, 12
    q, K, V = si.tiny_case(61, d, L)
    Pqk = si.random_orthogonal(62, d)
    Pvo = si.random_orthogonal(63, d)
    schedules = [{0: (5, 5), 4: (2, 3)}, {0: (2, 3), 6: (7, 8)}, {0: (6, 2), 3: (3, 6), 8: (8, 1)},
                 {0: (4, 4), 11: (1, 1)}, {0: (8, 8), 1: (1, 8), 5: (8, 1)}]
    for changes in schedules:
        for b in (0, 2, 5):
            uc = O.UnitCache(Pqk, Pvo, b, changes[0][0], dtype, k_value=changes[0][1])
            for t in range(L):
                if t in changes and t > 0:
                    uc.change_k(*changes[t])
                uc.append(K[0, t], V[0, t])
            got = uc.attend(q[0])
            want = _brute_swan_k_schedule(q[0], K[0], V[0], Pqk, Pvo, b, changes, dtype)
            assert np.allclose(got, want, rtol=1e-12, atol=1e-12), (changes, b)
            arr = uc.sparse_arrays()
            assert arr["k_idx"].shape[1] == uc.k and arr["v_idx"].shape[1] == uc.kv


@pytest.mark.parametrize("k,kv,k2,kv2", [(48, 48, 32, 32), (77, 51, 40, 51), (128, 64, 1, 13)])
def test_lowering_k_equals_pruning_at_the_lower_k(k, kv, k2, kv2):
    """Nested top-k: re-pruning the stored top-k to k' is the top-k' of the vector."""
    d, L, b = 128, 90, 8
    _, K, V = si.tiny_case(70 + k2, d, L)
    Pqk = si.random_orthogonal(71, d)
    Pvo = si.random_orthogonal(72, d)
    K16, V16 = K[0].astype(np.float16), V[0].astype(np.float16)
    c = O.compress_block(K16, V16, Pqk, Pvo, b, k, np.float16, k_value=kv)
    got = O.change_k_cache(c, k2, kv2)
    want = O.compress_block(K16, V16, Pqk, Pvo, b, k2, np.float16, k_value=kv2)
    for key in ("k_idx", "k_val", "v_idx", "v_val", "k_buf", "v_buf"):
        assert np.array_equal(got[key], want[key]), key


def test_raising_k_keeps_pairs_and_attention():
    d, L, b = 128, 70, 4
    q, K, V = si.tiny_case(80, d, L)
    Pqk = si.random_orthogonal(81, d)
    Pvo = si.random_orthogonal(82, d)
    c = O.compress_block(K[0], V[0], Pqk, Pvo, b, 24, np.float16, k_value=40)
    up = O.change_k_cache(c, 40, 48)
    for r, k0, k1 in (("k", 24, 40), ("v", 40, 48)):
        assert np.array_equal(up[f"{r}_idx"][:, :k0], c[f"{r}_idx"])
        assert np.array_equal(up[f"{r}_val"][:, :k0], c[f"{r}_val"])
        assert np.all(up[f"{r}_val"][:, k0:] == 0)
        for t in range(up[f"{r}_idx"].shape[0]):  # the fillers: lowest dims not kept
            free = np.setdiff1d(np.arange(d), c[f"{r}_idx"][t])[: k1 - k0]
            assert np.array_equal(up[f"{r}_idx"][t, k0:], free)
    a0 = O.attend_arrays(q[0], Pqk, Pvo, c)
    a1 = O.attend_arrays(q[0], Pqk, Pvo, up)
    assert np.allclose(a0, a1, rtol=0, atol=1e-15 * np.abs(a0).max())


def test_lowering_k_of_e4m3_values_on_exact_values():
    """8-bit values rank the stored codes; where every value is exact in E4M3 this is
    the same selection as pruning the fp16 values at the lower k."""
    rng = np.random.default_rng(90)
    mags = O.e4m3_magnitudes()
    mags = mags[(mags > 0) & (mags <= 448)]
    X = (rng.choice(mags, size=(60, 128)) * rng.choice([-1.0, 1.0], size=(60, 128)))
    X = X.astype(np.float16)
    eye = np.eye(128)
    c = O.compress_block(X, X[::-1].copy(), eye, eye, 0, 64, np.float16, values="e4m3",
                         k_value=48)
    got = O.change_k_cache(c, 20, 33)
    want = O.compress_block(X, X[::-1].copy(), eye, eye, 0, 20, np.float16, values="e4m3",
                            k_value=33)
    for key in ("k_idx", "k_code", "v_idx", "v_code"):
        assert np.array_equal(got[key], want[key]), key


# --------------------------------------------------------------------------- #
# Readings 12-13: RoPE and the absorbed layer
# --------------------------------------------------------------------------- #
def test_rope_against_complex_rotation_and_closed_forms():
    rng = np.random.default_rng(101)
    x = rng.standard_normal((4, 9, 128))
    pos = np.array([0, 1, 2, 7, 100, 4095, 32767, 131071, 5])
    for base in (10000.0, 500000.0):
        y = O.rope(x, pos, base)
        # an independent form: dims (j, j + 64) as the complex number x_j + i x_{j+64},
        # multiplied by exp(i pos theta_j), theta_j = 1 / base^(j / 64)
        theta = 1.0 / np.power(base, np.arange(64) / 64.0)
        z = (x[..., :64] + 1j * x[..., 64:]) * np.exp(1j * pos[:, None] * theta[None, :])
        # theta rounds differently in the two forms; at position 131071 that moves the
        # angle by ~1e-11, so the bound is 1e-9 (far below an fp16 ulp)
        assert np.allclose(y[..., :64], z.real, rtol=0, atol=1e-9)
        assert np.allclose(y[..., 64:], z.imag, rtol=0, atol=1e-9)
        assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1))
        assert np.array_equal(y[:, 0], x[:, 0])  # position 0
    # relative positions: <rope(q, m), rope(k, n)> depends on m - n only
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    for m, n in ((5, 2), (1000, 997), (70000, 69997)):
        a = O.rope(q[None], np.array([m]), 10000.0)[0] @ O.rope(k[None], np.array([n]), 10000.0)[0]
        b = O.rope(q[None], np.array([3]), 10000.0)[0] @ O.rope(k[None], np.array([0]), 10000.0)[0]
        assert abs(a - b) < 1e-9 * max(1.0, abs(b))
    # e_0 at position 1 with theta_0 = 1: (cos 1, sin 1) on dims 0 and 64
    e0 = np.zeros((1, 128))
    e0[0, 0] = 1.0
    y = O.rope(e0, np.array([1]), 10000.0)[0]
    assert y[0] == math.cos(1.0) and y[64] == math.sin(1.0) and np.count_nonzero(y) == 2


def _textbook_layer(x_seq, W_q, W_k, W_v, W_o, n_heads, n_kv, base):
    """Standard attention of a Llama layer for the last row (no SWAN, float64)."""
    L, d, G = x_seq.shape[0], 128, n_heads // n_kv
    q = (x_seq @ W_q).reshape(L, n_heads, d)
    k = (x_seq @ W_k).reshape(L, n_kv, d)
    v = (x_seq @ W_v).reshape(L, n_kv, d)
    pos = np.arange(L)
    q = O.rope(q.transpose(1, 0, 2), pos, base).transpose(1, 0, 2)
    k = O.rope(k.transpose(1, 0, 2), pos, base).transpose(1, 0, 2)
    o = np.zeros(n_heads * d)
    for hq in range(n_heads):
        o[hq * d:(hq + 1) * d] = _textbook_attention(q[L - 1, hq], k[:, hq // G], v[:, hq // G])
    return o @ W_o


def _layer_weights(seed, hidden, n_heads, n_kv):
    r = np.random.default_rng(seed)
    d = 128
    W_q = r.standard_normal((hidden, n_heads * d)) / math.sqrt(hidden)
    W_k = r.standard_normal((hidden, n_kv * d)) / math.sqrt(hidden)
    W_v = r.standard_normal((hidden, n_kv * d)) / math.sqrt(hidden)
    W_o = r.standard_normal((n_heads * d, hidden)) / math.sqrt(n_heads * d)
    P_qk = np.stack([si.random_orthogonal(seed * 10 + h, d) for h in range(n_kv)])
    P_vo = np.stack([si.random_orthogonal(seed * 10 + 5 + h, d) for h in range(n_kv)])
    return W_q, W_k, W_v, W_o, P_qk, P_vo


@pytest.mark.parametrize("n_heads,n_kv", [(4, 2), (2, 2)])
def test_layer_with_full_retention_is_the_textbook_layer(n_heads, n_kv):
    """k = d or b >= L, float64 storage: SWAN with W_V / W_O absorbed (Lemma 2) equals
    the plain attention layer, RoPE and the GQA head mapping included."""
    hidden, L = 96, 40
    W_q, W_k, W_v, W_o, P_qk, P_vo = _layer_weights(3 + n_heads, hidden, n_heads, n_kv)
    x = np.random.default_rng(4).standard_normal((L, hidden))
    want = _textbook_layer(x, W_q, W_k, W_v, W_o, n_heads, n_kv, 10000.0)
    for b, k in ((0, 128), (4, 128), (L, 7)):
        got = O.layer_decode(x, W_q, W_k, W_v, W_o, P_qk, P_vo, n_heads, n_kv, 10000.0, b, k,
                             np.float64)
        assert np.allclose(got, want, rtol=0, atol=1e-11 * np.abs(want).max()), (b, k)


def test_absorbed_layer_equals_explicit_rotation_with_pruning():
    """Lemma 2 with pruning active: rotating v inside the cache and rotating the output
    back (the library's explicit form) equals absorbing P_VO into W_V and W_O."""
    hidden, L, n_heads, n_kv, b, k = 96, 60, 4, 2, 8, 40
    W_q, W_k, W_v, W_o, P_qk, P_vo = _layer_weights(11, hidden, n_heads, n_kv)
    x = np.random.default_rng(12).standard_normal((L, hidden))
    got = O.layer_decode(x, W_q, W_k, W_v, W_o, P_qk, P_vo, n_heads, n_kv, 10000.0, b, k,
                         np.float64)
    # explicit: v = x W_v, the cache rotates it with P_VO and attend rotates back
    q, kk, _ = O.layer_tensors(x, W_q, W_k, W_v, n_heads, n_kv, np.arange(L), 10000.0,
                               np.float64)
    v = (x @ W_v).reshape(L, n_kv, 128)
    o = np.zeros(n_heads * 128)
    for h in range(n_kv):
        c = O.compress_block(kk[:, h], v[:, h], P_qk[h], P_vo[h], b, k, np.float64)
        for hq in range(h * 2, (h + 1) * 2):
            o[hq * 128:(hq + 1) * 128] = O.attend_arrays(q[L - 1, hq], P_qk[h], P_vo[h], c)
    want = o @ W_o
    assert np.allclose(got, want, rtol=0, atol=1e-11 * np.abs(want).max())


def test_column_sign_flip_changes_nothing_but_signs():
    d, L, b, k = 128, 90, 8, 40
    q, K, V = si.tiny_case(15, d, L)
    K16, V16 = K.astype(np.float16), V.astype(np.float16)
    Pqk = si.random_orthogonal(16, d)
    Pvo = si.random_orthogonal(17, d)
    flip = np.where(si.rng_for(18).random(d) < 0.5, -1.0, 1.0)
    c1 = O.compress_block(K16[0], V16[0], Pqk, Pvo, b, k, np.float16)
    c2 = O.compress_block(K16[0], V16[0], Pqk * flip, Pvo * flip, b, k, np.float16)
    assert np.array_equal(c1["k_idx"], c2["k_idx"])
    assert np.array_equal(c1["v_idx"], c2["v_idx"])
    assert np.array_equal(np.abs(c1["k_val"]), np.abs(c2["k_val"]))
    o1 = O.attend_arrays(q[0], Pqk, Pvo, c1)
    o2 = O.attend_arrays(q[0], Pqk * flip, Pvo * flip, c2)
    assert np.allclose(o1, o2, rtol=0, atol=1e-14)


def test_gqa_query_heads_map_to_their_kv_head():
    d, L, b, k = 16, 40, 4, 6
    Hq, Hkv = 8, 2
    q, K, V = si.tiny_case(19, d, L, n_q=Hq, n_kv=Hkv)
    Pqk = np.stack([si.random_orthogonal(20 + h, d) for h in range(Hkv)])
    Pvo = np.stack([si.random_orthogonal(30 + h, d) for h in range(Hkv)])
    caches = [[O.compress_block(K[h], V[h], Pqk[h], Pvo[h], b, k, np.float16)
               for h in range(Hkv)]]
    out = O.decode_batch(q[None], Pqk, Pvo, caches)[0]
    for hq in range(Hq):
        g = hq // (Hq // Hkv)
        assert np.array_equal(out[hq], O.attend_arrays(q[hq], Pqk[g], Pvo[g], caches[0][g]))
    # permuting query heads inside a group permutes the outputs
    perm = np.array([1, 3, 0, 2, 6, 4, 7, 5])
    out_p = O.decode_batch(q[perm][None], Pqk, Pvo, caches)[0]
    assert np.array_equal(out_p, out[perm])
    # a query head of the other group gives a different answer
    assert not np.allclose(out[0], O.attend_arrays(q[0], Pqk[1], Pvo[1], caches[0][1]))


# --------------------------------------------------------------------------- #
# Sec. 5.1 space model, Sec. 5.2 / Appendix A.2 FLOP model, Sec. 1 sizes
# --------------------------------------------------------------------------- #
def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


def test_break_even_examples_match_the_paper():
    for d_h, k, b, printed in _rows("break_even.txt"):
        d_h, k, b, printed = int(d_h), int(k), int(b), int(printed)
        L = O.break_even_length(d_h, k, b)
        assert round(L) == printed
        # the bound is where the FLOP model of C_SWAN crosses C_std
        Lc = int(math.floor(L)) + 1
        assert O.flops_swan(Lc, d_h, b, k) < O.flops_standard(Lc, d_h)
        assert O.flops_swan(int(math.floor(L)) - 1, d_h, b, k) > O.flops_standard(
            int(math.floor(L)) - 1, d_h)


def test_space_model_matches_the_paper():
    g = {k: float(v) for k, v in _rows("space_model.txt")}
    assert O.dense_bytes_per_vector(128, 2) == g["dense_fp16_bytes_d128"]
    assert O.space_bytes_per_vector(1) == g["sparse_fp16_formula_k1"]
    assert O.space_bytes_per_vector(64) == g["sparse_fp16_formula_k64"]
    assert O.space_bytes_per_vector(64, value_bytes=1) == g["sparse_fp8_formula_k64"]
    # largest retention ratio that still saves memory with 16-bit values
    kmax = max(k for k in range(1, 129) if O.space_bytes_per_vector(k) < 256)
    assert round((kmax + 1) / 128, 2) == g["fp16_break_even_retention"] or \
        round(kmax / 128, 2) == g["fp16_break_even_retention"]


def test_motivating_kv_size_matches_the_paper():
    (layers, heads, d_h, nbytes, seq, batch, printed), = _rows("motivating_size.txt")
    total = 2 * int(layers) * int(heads) * int(d_h) * int(nbytes) * int(seq) * int(batch)
    assert round(total / 2**30) == int(printed)


def test_flops_swan_terms():
    # each term of C_SWAN checked separately: projections, sparse part, buffer part
    assert O.flops_swan(0, 128, 0, 48) == 4 * 128 * 128
    assert O.flops_swan(1000, 128, 0, 48) - O.flops_swan(999, 128, 0, 48) == 4 * 48
    assert O.flops_swan(1000, 128, 10, 48) - O.flops_swan(1000, 128, 9, 48) == 4 * (128 - 48)


# --------------------------------------------------------------------------- #
# 8-bit sparse values (reading 9: OCP FP8 E4M3, no scale)
# --------------------------------------------------------------------------- #
def _all_finite_fp16():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    x = bits.view(np.float16)
    return x[np.isfinite(x)]


def test_e4m3_table_is_the_format():
    """Closed form of E4M3: 2^-9 smallest subnormal, 2^-6 smallest normal, 448 largest,
    strictly increasing codes, every value exact in fp16 (so fp16 -> E4M3 -> fp16
    loses nothing more than the rounding)."""
    t = O.e4m3_magnitudes()
    assert t.shape == (127,)
    assert t[0] == 0.0 and t[1] == 2.0 ** -9 and t[7] == 7 * 2.0 ** -9
    assert t[8] == 2.0 ** -6 and t[126] == 448.0 and t[120] == 256.0
    assert np.all(np.diff(t) > 0)
    assert np.array_equal(t.astype(np.float16).astype(np.float64), t)
    # the spacing doubles at every binade from 2^-6 up
    for e in range(1, 16):
        seg = t[8 * e: 8 * e + 8] if e < 15 else t[120:127]
        assert np.all(np.diff(seg) == 2.0 ** (e - 10))


def test_e4m3_rounding_matches_torch_on_every_fp16_value():
    """A library routine: torch's float8_e4m3fn conversion (nearest, ties to even) on
    every finite fp16 value up to 464 in magnitude (above, torch gives NaN where the
    oracle saturates)."""
    torch = pytest.importorskip("torch")
    x = _all_finite_fp16()
    x = x[np.abs(x.astype(np.float64)) <= 464.0]
    want = torch.tensor(x.astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = O.to_e4m3_codes(x)
    assert np.array_equal(got, want)


def test_e4m3_ties_saturation_and_signed_zero():
    assert list(O.to_e4m3_codes(np.array([1.0625, 1.1875, 2.0 ** -10, 3 * 2.0 ** -10]))) == \
        [56, 58, 0, 2]                                   # ties to the even code
    assert list(O.to_e4m3_codes(np.array([448.0, 465.0, 1000.0, 65504.0, -1e4]))) == \
        [126, 126, 126, 126, 254]                        # saturating at +-448
    assert list(O.to_e4m3_codes(np.array([0.0, -0.0]))) == [0, 128]
    v = O.e4m3_decode(np.arange(256, dtype=np.uint8))
    assert np.isnan(v[127]) and np.isnan(v[255]) and v[254] == -448.0
    # decode(encode(x)) is the nearest value: no other code is strictly closer
    x = np.random.default_rng(5).uniform(-500, 500, 4000)
    d_best = np.abs(O.e4m3_decode(O.to_e4m3_codes(x)) - np.clip(x, -448, 448))
    t = O.e4m3_magnitudes()
    d_any = np.min(np.abs(np.abs(np.clip(x, -448, 448))[:, None] - t[None, :]), axis=1)
    assert np.all(d_best <= d_any)


def test_e4m3_values_keep_the_fp16_selection():
    """Reading 9: the indices are those of fp16 storage (selection ranks the stored fp16
    values), the values are the E4M3 rounding of the kept fp16 values, the buffer is
    unchanged, and token-by-token appends give the same codes as the block form."""
    rng = si.rng_for(9100, 0)
    R = si.haar_orthogonal(rng, 128)
    K = si.lowrank_rows(si.rng_for(9100, 1), 90, R)
    V = si.lowrank_rows(si.rng_for(9100, 2), 90, R)
    Pk, Pv = si.random_orthogonal(91, 128), si.random_orthogonal(92, 128)
    for k in (1, 13, 48, 128):
        a = O.compress_block(K, V, Pk, Pv, 16, k, np.float16)
        e = O.compress_block(K, V, Pk, Pv, 16, k, np.float16, values="e4m3")
        for r in ("k", "v"):
            assert np.array_equal(a[f"{r}_idx"], e[f"{r}_idx"])
            assert np.array_equal(e[f"{r}_code"], O.to_e4m3_codes(a[f"{r}_val"]))
            assert np.array_equal(a[f"{r}_buf"].view(np.uint16), e[f"{r}_buf"].view(np.uint16))
        uc = O.UnitCache(Pk, Pv, 16, k, np.float16, values="e4m3")
        for t in range(90):
            uc.append(K[t], V[t])
        sa = uc.sparse_arrays()
        for r in ("k", "v"):
            assert np.array_equal(sa[f"{r}_idx"], e[f"{r}_idx"])
            assert np.array_equal(sa[f"{r}_val"], e[f"{r}_val"])


def test_e4m3_values_with_k_equal_d_are_dense_attention_on_rounded_vectors():
    """k = d, b = 0: every component kept, so attention is textbook softmax attention on
    the E4M3-rounded rotated keys and values (written out here), rotated back."""
    rng = si.rng_for(9200, 0)
    d, L = 8, 12
    Pk, Pv = si.random_orthogonal(93, d), si.random_orthogonal(94, d)
    K = rng.standard_normal((L, d))
    V = rng.standard_normal((L, d))
    q = rng.standard_normal(d)
    c = O.compress_block(K, V, Pk, Pv, 0, d, np.float16, values="e4m3")
    got = O.attend_arrays(q, Pk, Pv, c)
    kh = O.e4m3_decode(O.to_e4m3_codes((K @ Pk).astype(np.float16)))
    vh = O.e4m3_decode(O.to_e4m3_codes((V @ Pv).astype(np.float16)))
    s = (kh @ (q @ Pk)) / math.sqrt(d)
    p = np.exp(s - s.max())
    want = (p / p.sum()) @ vh @ Pv.T
    assert np.allclose(got, want, rtol=1e-12, atol=1e-12)
