"""Host-only checks of the C ABI: the library loads, exports every declared entry
point, and rejects bad arguments before touching the GPU (no compute calls)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

swan = pytest.importorskip("paper_2511_18936_amd.swan")

FAKE = 0x10000  # never dereferenced: every call below fails validation first


def _declared_functions():
    with open(os.path.join(ROOT, "include", "swan.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:swan_status|const char\*|int32_t)\s+(swan_\w+)\(",
                                 text, re.M)))


def test_header_and_binding_agree_on_exports():
    declared = _declared_functions()
    assert len(declared) == 15
    assert sorted(swan.EXPORTED) == declared
    lib = swan.lib()
    for name in declared:
        assert hasattr(lib, name), name


def test_version_is_the_current_abi():
    """2.04: swan_set_decode_tuning; 2.03: swan_decode_attention_noalloc; 2.02: swan_change_k, swan_rope; 2.00: keys
    and values with their own k."""
    assert swan.lib().swan_version() == 205


def test_nm_shows_exported_symbols():
    import subprocess

    out = subprocess.run(["nm", "-D", "--defined-only", swan.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    for name in _declared_functions():
        assert re.search(rf"\bT {name}\b", out), name


def _desc(**kw):
    d = dict(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128, buffer_tokens=16,
             sparse_capacity=1000, dtype=swan.SWAN_F16, reserved=0,
             k_pages=FAKE, v_pages=FAKE, k_ring=FAKE, v_ring=FAKE)
    d.update(kw)
    return swan.CacheDesc(**d)


def test_page_and_cache_sizes():
    assert swan.page_bytes(swan.SWAN_F16, 48) == 64 * 48 * 3
    assert swan.page_bytes(swan.SWAN_F16, 45) == 64 * 48 * 3  # k padded to 8
    assert swan.page_bytes(swan.SWAN_F32, 64) == 64 * 64 * 5
    kb, vb, rb = swan.cache_bytes(_desc(), [48, 64])
    npc = (1000 + 63) // 64
    assert kb == vb == 2 * npc * 64 * 3 * (48 + 64)
    assert rb == 2 * 2 * 16 * 128 * 2
    # keys and values with their own k (k_pad 80 / 56 and 8 / 128)
    kb, vb, rb2 = swan.cache_bytes(_desc(), [77, 1], [51, 128])
    assert kb == 2 * npc * 64 * 3 * (80 + 8)
    assert vb == 2 * npc * 64 * 3 * (56 + 128)
    assert rb2 == rb
    # E4M3 sparse values: one byte per value plus one per index; the ring stays fp16
    assert swan.page_bytes(swan.SWAN_F16_E4M3, 48) == 64 * 48 * 2
    assert swan.page_bytes(swan.SWAN_F16_E4M3, 41) == 64 * 48 * 2
    kb8, vb8, rb8 = swan.cache_bytes(_desc(dtype=swan.SWAN_F16_E4M3), [48, 64])
    assert kb8 == vb8 == 2 * npc * 64 * 2 * (48 + 64)
    assert rb8 == rb
    with pytest.raises(swan.SwanError):
        swan.page_bytes(3, 48)


@pytest.mark.parametrize("kw,status", [
    (dict(batch=0), swan.SWAN_ERR_INVALID_ARG),
    (dict(batch=65), swan.SWAN_ERR_INVALID_ARG),
    (dict(n_q_heads=6, n_kv_heads=4), swan.SWAN_ERR_INVALID_ARG),
    (dict(head_dim=64), swan.SWAN_ERR_UNSUPPORTED),
    (dict(buffer_tokens=-1), swan.SWAN_ERR_INVALID_ARG),
    (dict(buffer_tokens=5000), swan.SWAN_ERR_UNSUPPORTED),
    (dict(buffer_tokens=4097), swan.SWAN_ERR_UNSUPPORTED),  # one past the largest buffer
    (dict(dtype=7), swan.SWAN_ERR_UNSUPPORTED),
    (dict(reserved=1), swan.SWAN_ERR_INVALID_ARG),
    (dict(k_pages=None), swan.SWAN_ERR_INVALID_ARG),
    (dict(v_ring=FAKE + 4), swan.SWAN_ERR_INVALID_ARG),
])
def test_compress_rejects_bad_descriptors(kw, status):
    lib = swan.lib()
    d = _desc(**kw)
    n = max(1, min(d.batch, 64))
    seq = swan._i32_array([0] * n)
    kk = swan._i32_array([48] * n)
    st = lib.swan_compress_append(ctypes.byref(d), seq, kk, None, FAKE, FAKE, 1, None, FAKE,
                                  FAKE, None)
    assert st == status, swan.last_error()
    assert swan.last_error()


def test_compress_rejects_bad_arguments():
    lib = swan.lib()
    d = _desc()
    ok_seq = swan._i32_array([10, 20])
    ok_k = swan._i32_array([48, 64])
    E = swan.SWAN_ERR_INVALID_ARG
    assert lib.swan_compress_append(ctypes.byref(d), ok_seq, swan._i32_array([0, 48]), None, FAKE,
                                    FAKE, 1, None, FAKE, FAKE, None) == E
    assert lib.swan_compress_append(ctypes.byref(d), ok_seq, swan._i32_array([48, 129]), None, FAKE,
                                    FAKE, 1, None, FAKE, FAKE, None) == E
    assert lib.swan_compress_append(ctypes.byref(d), None, ok_k, None, FAKE, FAKE, 1, None, FAKE,
                                    FAKE, None) == E
    assert lib.swan_compress_append(ctypes.byref(d), ok_seq, ok_k, None, FAKE, FAKE, 2,
                                    swan._i32_array([1, 3]), FAKE, FAKE, None) == E
    assert lib.swan_compress_append(ctypes.byref(d), ok_seq, ok_k, None, FAKE, FAKE, -1, None, FAKE,
                                    FAKE, None) == E
    assert lib.swan_compress_append(ctypes.byref(d), ok_seq, ok_k, None, None, FAKE, 1, None, FAKE,
                                    FAKE, None) == E
    assert lib.swan_compress_append(ctypes.byref(d), ok_seq, ok_k, None, FAKE, FAKE, 1, None, None,
                                    FAKE, None) == E
    assert lib.swan_compress_append(ctypes.byref(d), ok_seq, ok_k, None, FAKE, FAKE, 1, None, FAKE + 8,
                                    FAKE, None) == E
    assert lib.swan_compress_append(ctypes.byref(d), swan._i32_array([-1, 0]), ok_k, None, FAKE, FAKE,
                                    1, None, FAKE, FAKE, None) == E
    # capacity: 1000 + 16 tokens fit, one more does not
    st = lib.swan_compress_append(ctypes.byref(d), swan._i32_array([1016, 0]), ok_k, None, FAKE, FAKE,
                                  1, None, FAKE, FAKE, None)
    assert st == swan.SWAN_ERR_CAPACITY


def test_decode_rejects_bad_arguments():
    lib = swan.lib()
    d = _desc()
    ok_k = swan._i32_array([48, 64])
    seq = swan._i32_array([100, 200])
    need = swan.decode_workspace_bytes(d, [100, 200], [48, 64])
    assert need > 0
    E = swan.SWAN_ERR_INVALID_ARG
    args = lambda seq_, ws, wsb, scale=0.0: (ctypes.byref(d), seq_, ok_k, None, FAKE, FAKE,
                                            FAKE, scale, FAKE, ws, wsb, None)
    assert lib.swan_decode_attention(*args(swan._i32_array([0, 5]), FAKE, need)) == E
    assert lib.swan_decode_attention(*args(seq, None, need)) == swan.SWAN_ERR_WORKSPACE
    assert lib.swan_decode_attention(*args(seq, FAKE, need - 1)) == swan.SWAN_ERR_WORKSPACE
    assert lib.swan_decode_attention(*args(seq, FAKE + 16, need)) == E  # misaligned
    assert lib.swan_decode_attention(*args(seq, FAKE, need, float("nan"))) == E
    assert lib.swan_decode_attention(*args(swan._i32_array([1017, 5]), FAKE, 1 << 30)) == \
        swan.SWAN_ERR_CAPACITY
    assert lib.swan_decode_attention(ctypes.byref(d), seq, ok_k, None, None, FAKE, FAKE, 0.0,
                                     FAKE, FAKE, need, None) == E
    # k_value outside 1..128
    for bad in ([48, 0], [129, 48]):
        assert lib.swan_decode_attention(ctypes.byref(d), seq, ok_k, swan._i32_array(bad), FAKE,
                                         FAKE, FAKE, 0.0, FAKE, FAKE, 1 << 30, None) == E


def test_decode_step_checks_both_parts_on_the_host():
    """swan_decode_step rejects whatever the append or the decode would, before
    anything is enqueued; its workspace is sized for the lengths after the step."""
    lib = swan.lib()
    d = _desc()
    ok_k = swan._i32_array([48, 64])
    need = swan.decode_workspace_bytes(d, [101, 201], [48, 64])
    E = swan.SWAN_ERR_INVALID_ARG

    def step(seq=(100, 200), k_new=FAKE, q=FAKE, P_qk=FAKE, scale=0.0, ws=FAKE, wsb=need,
             k_value=None):
        return lib.swan_decode_step(ctypes.byref(d), swan._i32_array(list(seq)), ok_k, k_value,
                                    k_new, FAKE, q, P_qk, FAKE, scale, FAKE, ws, wsb, None)

    assert step(k_new=None) == E                    # append part
    assert step(k_new=FAKE + 8) == E                # misaligned new rows
    assert step(seq=(-1, 0)) == E
    assert step(seq=(1016, 0)) == swan.SWAN_ERR_CAPACITY  # 1017 - 16 sparse tokens > 1000
    assert step(P_qk=None) == E
    assert step(q=None) == E                        # decode part
    assert step(scale=float("inf")) == E
    assert step(ws=None) == swan.SWAN_ERR_WORKSPACE
    assert step(wsb=need - 1) == swan.SWAN_ERR_WORKSPACE
    assert step(ws=FAKE + 16) == E                  # misaligned workspace
    assert step(k_value=swan._i32_array([48, 0])) == E
    assert swan.last_error()


def test_calibrate_rejects_bad_arguments():
    lib = swan.lib()
    need = swan.calibrate_workspace_bytes(128)
    assert need >= 2 * 8 * 128 * 128
    assert lib.swan_calibrate_rotation(FAKE, 100, 64, FAKE, None, FAKE, need, None) == \
        swan.SWAN_ERR_UNSUPPORTED
    assert lib.swan_calibrate_rotation(FAKE, 0, 128, FAKE, None, FAKE, need, None) == \
        swan.SWAN_ERR_INVALID_ARG
    assert lib.swan_calibrate_rotation(None, 10, 128, FAKE, None, FAKE, need, None) == \
        swan.SWAN_ERR_INVALID_ARG
    assert lib.swan_calibrate_rotation(FAKE, 10, 128, FAKE, None, FAKE, need - 1, None) == \
        swan.SWAN_ERR_WORKSPACE


def test_profile_hook_needs_both_events():
    lib = swan.lib()
    assert lib.swan_set_profile_events(FAKE, None) == swan.SWAN_ERR_INVALID_ARG
    assert lib.swan_set_profile_events(None, None) == swan.SWAN_OK


def test_workspace_grows_with_splits():
    d = _desc(batch=1, n_q_heads=1, n_kv_heads=1, sparse_capacity=1 << 20)
    small = swan.decode_workspace_bytes(d, [100], [48])
    large = swan.decode_workspace_bytes(d, [1 << 19], [48])
    assert large > small > 0


def test_asymmetric_k_workspace():
    """Keys and values with their own k need no extra workspace: the token splits
    follow the bytes of both roles, so (48, 32) plans like (40, 40)."""
    d = _desc(batch=2, n_q_heads=8, n_kv_heads=2, buffer_tokens=16, sparse_capacity=1 << 16)
    L = [5000, 3000]
    base = swan.decode_workspace_bytes(d, L, [48, 48])
    assert swan.decode_workspace_bytes(d, L, [48, 48], [48, 48]) == base
    assert swan.decode_workspace_bytes(d, L, [48, 48], [41, 47]) == base  # same k_pad
    assert swan.decode_workspace_bytes(d, L, [48, 48], [32, 48]) == \
        swan.decode_workspace_bytes(d, L, [40, 48])


def test_change_k_rejects_bad_arguments():
    lib = swan.lib()
    d = _desc()
    seq = swan._i32_array([100, 200])
    ks = swan._i32_array([48, 64])
    E = swan.SWAN_ERR_INVALID_ARG
    B2 = 0x20000000  # another page region, far from FAKE
    dst = _desc(k_pages=B2, v_pages=B2 + (1 << 24))
    call = lambda src_, dst_, kd=ks, seq_=seq: lib.swan_change_k(
        ctypes.byref(src_), ks, None, ctypes.byref(dst_), kd, None, seq_, None)
    assert call(d, _desc(batch=1, k_pages=B2, v_pages=B2 + (1 << 24))) == E  # other batch
    assert call(d, _desc(buffer_tokens=8, k_pages=B2, v_pages=B2 + (1 << 24))) == E
    assert call(d, _desc(dtype=swan.SWAN_F32, k_pages=B2, v_pages=B2 + (1 << 24))) == E
    assert call(d, _desc(k_ring=FAKE + 256, k_pages=B2, v_pages=B2 + (1 << 24))) == E  # ring
    assert call(d, d) == E  # dst pages overlap src pages
    assert call(d, dst, kd=swan._i32_array([0, 48])) == E
    assert call(d, dst, kd=swan._i32_array([48, 129])) == E
    assert call(d, dst, seq_=swan._i32_array([-1, 5])) == E
    assert lib.swan_change_k(ctypes.byref(d), ks, None, ctypes.byref(dst), ks, None, None,
                             None) == E
    # the sparse tokens must fit the destination's capacity
    assert call(d, _desc(sparse_capacity=50, k_pages=B2, v_pages=B2 + (1 << 24))) == \
        swan.SWAN_ERR_CAPACITY


def test_rope_rejects_bad_arguments():
    lib = swan.lib()
    pos = swan._i32_array([0, 5])
    E = swan.SWAN_ERR_INVALID_ARG
    assert lib.swan_rope(FAKE, FAKE, swan.SWAN_F16, 2, 4, 3, 64, pos, 1e4, None) == \
        swan.SWAN_ERR_UNSUPPORTED
    assert lib.swan_rope(FAKE, FAKE, 9, 2, 4, 3, 128, pos, 1e4, None) == swan.SWAN_ERR_UNSUPPORTED
    assert lib.swan_rope(FAKE, FAKE, swan.SWAN_F16, 0, 4, 3, 128, pos, 1e4, None) == E
    assert lib.swan_rope(FAKE, FAKE, swan.SWAN_F16, 2, 4, 3, 128, pos, 1.0, None) == E
    assert lib.swan_rope(FAKE, FAKE, swan.SWAN_F16, 2, 4, 3, 128, None, 1e4, None) == E
    assert lib.swan_rope(None, FAKE, swan.SWAN_F16, 2, 4, 3, 128, pos, 1e4, None) == E
    assert lib.swan_rope(FAKE + 8, FAKE, swan.SWAN_F16, 2, 4, 3, 128, pos, 1e4, None) == E
    assert lib.swan_rope(FAKE, FAKE, swan.SWAN_F16, 2, 4, 3, 128, swan._i32_array([0, -1]), 1e4,
                         None) == E
    assert lib.swan_rope(None, None, swan.SWAN_F16, 2, 4, 0, 128, pos, 1e4, None) == swan.SWAN_OK


def test_noalloc_decode_checks_arguments_and_its_scratch_limit_on_the_host():
    """The allocation-free decode rejects bad arguments, and a batch whose partials
    exceed its scratch array, before it looks the array up on a device."""
    lib = swan.lib()
    seq = swan._i32_array([10, 20])
    kk = swan._i32_array([48, 64])
    st = lib.swan_decode_attention_noalloc(ctypes.byref(_desc(batch=0)), seq, kk, None, FAKE,
                                           FAKE, FAKE, 0.0, FAKE, None)
    assert st == swan.SWAN_ERR_INVALID_ARG, swan.last_error()
    st = lib.swan_decode_attention_noalloc(ctypes.byref(_desc()), seq, kk, None, None, FAKE,
                                           FAKE, 0.0, FAKE, None)
    assert st == swan.SWAN_ERR_INVALID_ARG, swan.last_error()
    B, H = 64, 256
    d = _desc(batch=B, n_q_heads=H, n_kv_heads=H, buffer_tokens=1, sparse_capacity=0)
    lens, ks = [1] * B, [48] * B
    assert swan.decode_workspace_bytes(d, lens, ks) > swan.NOALLOC_SCRATCH_BYTES
    st = lib.swan_decode_attention_noalloc(ctypes.byref(d), swan._i32_array(lens),
                                           swan._i32_array(ks), None, FAKE, FAKE, FAKE, 0.0,
                                           FAKE, None)
    assert st == swan.SWAN_ERR_WORKSPACE, swan.last_error()
    assert "scratch" in swan.last_error()


def test_decode_tuning_changes_the_plan_and_checks_its_ranges():
    """swan_set_decode_tuning: the workspace follows the thread's split plan (one
    split per sequence with a target of one wave), bad values are rejected and leave
    the tuning as it was, and all-zero restores the defaults."""
    d = _desc(batch=2, n_q_heads=4, n_kv_heads=4, buffer_tokens=16, sparse_capacity=40000)
    lens, ks = [30000, 20000], [48, 48]
    default = swan.decode_workspace_bytes(d, lens, ks)
    try:
        swan.set_decode_tuning(target_waves=1)
        one = swan.decode_workspace_bytes(d, lens, ks)
        units = 2 * 4
        assert one == (units * 128 * 4 + 255) // 256 * 256 + units * 2 * 132 * 4
        assert one < default
        for kw in (dict(target_waves=-1), dict(short_split_pages=-2), dict(merge_pct=101),
                   dict(side_streams=4), dict(side_streams=-2)):
            with pytest.raises(swan.SwanError) as ei:
                swan.set_decode_tuning(**kw)
            assert ei.value.status == swan.SWAN_ERR_INVALID_ARG
            assert swan.decode_workspace_bytes(d, lens, ks) == one
        # a large target is capped by the one-page rule (30 splits for 469 pages)
        swan.set_decode_tuning(target_waves=1 << 20)
        assert swan.decode_workspace_bytes(d, lens, ks) == default
    finally:
        swan.set_decode_tuning()
    assert swan.decode_workspace_bytes(d, lens, ks) == default


def test_binding_checks_tensors_before_the_call():
    """The library sees only device pointers, so the binding checks dtype, shape,
    layout and device of every tensor against the descriptor first (CPU tensors
    here: each case fails before any device pointer is taken)."""
    import torch

    d = _desc()  # batch 2, 8 query / 2 KV heads, fp16
    P = torch.zeros((2, 128, 128), dtype=torch.float32)
    k = torch.zeros((2, 2, 3, 128), dtype=torch.float16)
    q = torch.zeros((2, 8, 128), dtype=torch.float16)
    ws = torch.zeros(16, dtype=torch.uint8)

    def rejects(fn, what):
        with pytest.raises(swan.SwanError) as ei:
            fn()
        assert what in str(ei.value), str(ei.value)

    app = lambda kn, vn, Pq=P, Pv=P: swan.compress_append(d, [0, 0], [48, 48], kn, vn, Pq, Pv)
    rejects(lambda: app(k.float(), k), "dtype")
    rejects(lambda: app(k, k[:, :1].contiguous()), "shape")
    rejects(lambda: app(k, k.transpose(2, 3).contiguous().transpose(2, 3)), "contiguous")
    rejects(lambda: app(k, k, P.double()), "P_qk")
    rejects(lambda: app(k, k, P, P[:1]), "P_vo")
    rejects(lambda: app(k, k), "not on a GPU")
    dec = lambda qq, oo, Pq=P: swan.decode_attention(d, [5, 5], [48, 48], qq, Pq, P, oo, ws)
    rejects(lambda: dec(q.float(), q), "dtype")
    rejects(lambda: dec(q, q[:, :4].contiguous()), "shape")
    rejects(lambda: dec(q, q.transpose(0, 1).contiguous().transpose(0, 1)), "contiguous")
    rejects(lambda: dec(q, q, P.transpose(1, 2)), "P_qk")
    rejects(lambda: dec(q, q), "not on a GPU")
    rejects(lambda: swan.decode_attention_noalloc(d, [5, 5], [48, 48], q, P, P, q[:1]), "shape")
    d32 = _desc(dtype=swan.SWAN_F32)
    rejects(lambda: swan.decode_attention(d32, [5, 5], [48, 48], q, P, P, q, ws), "float32")


def test_bench_library_exports_its_header():
    """libswanbench.so (the streaming-read ceiling bench.py measures) exports what
    include/swan_bench.h declares."""
    import subprocess

    with open(os.path.join(ROOT, "include", "swan_bench.h")) as f:
        declared = re.findall(r"^\s*int32_t\s+(swan_\w+)\(", f.read(), re.M)
    assert declared == ["swan_stream_read"]
    path = os.path.join(ROOT, "paper_2511_18936_amd", "libswanbench.so")
    out = subprocess.run(["nm", "-D", "--defined-only", path], capture_output=True, text=True,
                         check=True).stdout
    for name in declared:
        assert re.search(rf"\bT {name}\b", out), name
