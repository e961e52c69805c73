"""ctypes binding of libswan (include/swan.h), plus a small cache holder.

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  PyTorch provides device memory and the current stream.  If the
library is missing the import fails loudly; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("SWAN_LIB", os.path.join(_HERE, "libswan.so"))

SWAN_OK = 0
SWAN_ERR_INVALID_ARG = 1
SWAN_ERR_UNSUPPORTED = 2
SWAN_ERR_CAPACITY = 3
SWAN_ERR_WORKSPACE = 4
SWAN_ERR_HIP = 5
SWAN_ERR_NO_CONVERGENCE = 6
SWAN_F32 = 0
SWAN_F16 = 1
SWAN_F16_E4M3 = 2  # fp16 everywhere, sparse values as OCP FP8 E4M3
MAX_BATCH = 64
HEAD_DIM = 128
PAGE_TOKENS = 64

EXPORTED = (
    "swan_last_error", "swan_version", "swan_page_bytes", "swan_cache_bytes",
    "swan_calibrate_workspace_bytes", "swan_calibrate_rotation", "swan_compress_append",
    "swan_decode_workspace_bytes", "swan_decode_attention", "swan_decode_attention_noalloc",
    "swan_decode_step", "swan_change_k", "swan_rope", "swan_set_decode_tuning", "swan_set_profile_events",
)
NOALLOC_SCRATCH_BYTES = 16 << 20


class SwanError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"swan status {status}: {message}")
        self.status = status


class DecodeTuning(ctypes.Structure):
    _fields_ = [
        ("target_waves", ctypes.c_int32),
        ("short_split_pages", ctypes.c_int32),
        ("merge_pct", ctypes.c_int32),
        ("side_streams", ctypes.c_int32),
    ]


class CacheDesc(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("buffer_tokens", ctypes.c_int32),
        ("sparse_capacity", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
        ("k_pages", ctypes.c_void_p),
        ("v_pages", ctypes.c_void_p),
        ("k_ring", ctypes.c_void_p),
        ("v_ring", ctypes.c_void_p),
    ]


def _load() -> ctypes.CDLL:
    # torch first: its HIP runtime (soname libamdhip64.so.7) then also serves
    # libswan, so the process holds a single runtime and a single device context
    import torch  # noqa: F401

    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"libswan.so not found at {LIB_PATH}; build it with "
            "`python -m paper_2511_18936_amd.build` (there is no fallback path)")
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, sz, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p
    pi32, psz, pdesc = ctypes.POINTER(i32), ctypes.POINTER(sz), ctypes.POINTER(CacheDesc)
    lib.swan_last_error.restype = ctypes.c_char_p
    lib.swan_last_error.argtypes = []
    lib.swan_version.restype = i32
    lib.swan_version.argtypes = []
    sigs = {
        "swan_page_bytes": [i32, i32, psz],
        "swan_cache_bytes": [pdesc, pi32, pi32, psz, psz, psz],
        "swan_calibrate_workspace_bytes": [i32, psz],
        "swan_calibrate_rotation": [vp, i64, i32, vp, vp, vp, sz, vp],
        "swan_compress_append": [pdesc, pi32, pi32, pi32, vp, vp, i32, pi32, vp, vp, vp],
        "swan_decode_workspace_bytes": [pdesc, pi32, pi32, pi32, psz],
        "swan_decode_attention": [pdesc, pi32, pi32, pi32, vp, vp, vp, ctypes.c_float, vp, vp, sz,
                                  vp],
        "swan_decode_attention_noalloc": [pdesc, pi32, pi32, pi32, vp, vp, vp, ctypes.c_float,
                                          vp, vp],
        "swan_decode_step": [pdesc, pi32, pi32, pi32, vp, vp, vp, vp, vp, ctypes.c_float, vp, vp,
                             sz, vp],
        "swan_change_k": [pdesc, pi32, pi32, pdesc, pi32, pi32, pi32, vp],
        "swan_rope": [vp, vp, i32, i32, i32, i32, i32, pi32, ctypes.c_double, vp],
        "swan_set_decode_tuning": [ctypes.POINTER(DecodeTuning)],
        "swan_set_profile_events": [vp, vp],
    }
    for name, args in sigs.items():
        f = getattr(lib, name)
        f.restype = i32
        f.argtypes = args
    return lib


_lib = _load()


def lib() -> ctypes.CDLL:
    return _lib


def last_error() -> str:
    return _lib.swan_last_error().decode()


def _check(status: int) -> None:
    if status != SWAN_OK:
        raise SwanError(status, last_error())


_I32_TYPES: dict = {}


def _i32_array(values: Sequence[int]):
    n = len(values)
    ty = _I32_TYPES.get(n)
    if ty is None:
        ty = _I32_TYPES[n] = ctypes.c_int32 * n
    return ty(*values)


def _opt_i32_array(values: Optional[Sequence[int]]):
    return None if values is None else _i32_array(values)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream, device_index: Optional[int] = None) -> Optional[int]:
    """The HIP stream handle: the given torch stream's, else the current stream of
    device_index (default: the current device)."""
    import torch

    if stream is not None:
        return stream.cuda_stream
    raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
    if raw is not None:
        return raw(torch.cuda.current_device() if device_index is None else device_index)
    return torch.cuda.current_stream().cuda_stream


def _elem_torch_dtype(code: int):
    import torch

    return torch.float32 if code == SWAN_F32 else torch.float16


def _tensor(t, name: str, dtype, shape) -> None:
    """The library sees only a device pointer: check what it assumes about the
    tensor behind it (dtype, shape, dense row-major layout, a GPU) before the call.
    A None entry of `shape` matches any size."""
    if t is None:
        raise SwanError(SWAN_ERR_INVALID_ARG, f"{name} is None")
    if t.dtype != dtype:
        raise SwanError(SWAN_ERR_INVALID_ARG, f"{name} has dtype {t.dtype}, expected {dtype}")
    ts = tuple(t.shape)
    if ts != shape and (len(ts) != len(shape) or
                        any(w is not None and g != w for g, w in zip(ts, shape))):
        want = "x".join("*" if w is None else str(w) for w in shape)
        raise SwanError(SWAN_ERR_INVALID_ARG,
                        f"{name} has shape {ts}, expected [{want}]")
    if not t.is_contiguous():
        raise SwanError(SWAN_ERR_INVALID_ARG, f"{name} must be contiguous (row-major)")


def _on_gpu(**tensors) -> None:
    for name, t in tensors.items():
        if t is not None and not t.is_cuda:
            raise SwanError(SWAN_ERR_INVALID_ARG, f"{name} is on {t.device}, not on a GPU")


def _rotations(desc: CacheDesc, P_qk, P_vo) -> None:
    import torch

    shape = (desc.n_kv_heads, desc.head_dim, desc.head_dim)
    _tensor(P_qk, "P_qk", torch.float32, shape)
    if P_vo is not None:
        _tensor(P_vo, "P_vo", torch.float32, shape)


def dtype_code(torch_dtype, sparse_values: str = "same") -> int:
    import torch

    if sparse_values not in ("same", "e4m3"):
        raise SwanError(SWAN_ERR_INVALID_ARG, f"sparse_values {sparse_values!r}")
    if sparse_values == "e4m3":
        if torch_dtype != torch.float16:
            raise SwanError(SWAN_ERR_UNSUPPORTED, "E4M3 sparse values need float16 storage")
        return SWAN_F16_E4M3
    if torch_dtype == torch.float16:
        return SWAN_F16
    if torch_dtype == torch.float32:
        return SWAN_F32
    raise SwanError(SWAN_ERR_UNSUPPORTED, f"dtype {torch_dtype} not supported")


def page_bytes(dtype: int, k_active: int) -> int:
    out = ctypes.c_size_t()
    _check(_lib.swan_page_bytes(dtype, k_active, ctypes.byref(out)))
    return out.value


def cache_bytes(desc: CacheDesc, k_active: Sequence[int],
                k_value: Optional[Sequence[int]] = None):
    """(key page bytes, value page bytes, ring bytes); k_value None: as k_active."""
    kb, vb, rb = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    _check(_lib.swan_cache_bytes(ctypes.byref(desc), _i32_array(k_active),
                                 _opt_i32_array(k_value), ctypes.byref(kb), ctypes.byref(vb),
                                 ctypes.byref(rb)))
    return kb.value, vb.value, rb.value


def calibrate_workspace_bytes(d: int = HEAD_DIM) -> int:
    out = ctypes.c_size_t()
    _check(_lib.swan_calibrate_workspace_bytes(d, ctypes.byref(out)))
    return out.value


def calibrate_rotation(rows, P_out, sigma_out=None, workspace=None, stream=None) -> None:
    """Sec. 4.1.2 basis of `rows` ([n][d] float32, cuda) into P_out ([d][d] float32)."""
    import torch

    n, d = rows.shape
    if workspace is None:
        workspace = torch.empty(calibrate_workspace_bytes(d), dtype=torch.uint8,
                                device=rows.device)
    _check(_lib.swan_calibrate_rotation(_ptr(rows), n, d, _ptr(P_out), _ptr(sigma_out),
                                        _ptr(workspace), workspace.numel(), _stream(stream)))


def compress_append(desc: CacheDesc, seq_len: Sequence[int], k_active: Sequence[int], k_new,
                    v_new, P_qk, P_vo, n_new_per_seq: Optional[Sequence[int]] = None,
                    stream=None, k_value: Optional[Sequence[int]] = None) -> None:
    n_new = 0 if k_new is None else int(k_new.shape[2])
    if k_new is not None or v_new is not None:
        et = _elem_torch_dtype(desc.dtype)
        shape = (desc.batch, desc.n_kv_heads, n_new, desc.head_dim)
        _tensor(k_new, "k_new", et, shape)
        _tensor(v_new, "v_new", et, shape)
    _rotations(desc, P_qk, P_vo)
    _on_gpu(k_new=k_new, v_new=v_new, P_qk=P_qk, P_vo=P_vo)
    per = None if n_new_per_seq is None else _i32_array(n_new_per_seq)
    _check(_lib.swan_compress_append(ctypes.byref(desc), _i32_array(seq_len),
                                     _i32_array(k_active), _opt_i32_array(k_value), _ptr(k_new),
                                     _ptr(v_new), n_new, per, _ptr(P_qk), _ptr(P_vo),
                                     _stream(stream, P_qk.get_device())))


def decode_workspace_bytes(desc: CacheDesc, seq_len: Sequence[int], k_active: Sequence[int],
                           k_value: Optional[Sequence[int]] = None) -> int:
    out = ctypes.c_size_t()
    _check(_lib.swan_decode_workspace_bytes(ctypes.byref(desc), _i32_array(seq_len),
                                            _i32_array(k_active), _opt_i32_array(k_value),
                                            ctypes.byref(out)))
    return out.value


def decode_attention(desc: CacheDesc, seq_len: Sequence[int], k_active: Sequence[int], q,
                     P_qk, P_vo, out, workspace, scale: float = 0.0, stream=None,
                     k_value: Optional[Sequence[int]] = None) -> None:
    _decode_tensors(desc, q, P_qk, P_vo, out)
    if workspace is None or not workspace.is_cuda or not workspace.is_contiguous():
        raise SwanError(SWAN_ERR_WORKSPACE, "workspace must be a contiguous GPU tensor")
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(_lib.swan_decode_attention(ctypes.byref(desc), _i32_array(seq_len),
                                      _i32_array(k_active), _opt_i32_array(k_value), _ptr(q),
                                      _ptr(P_qk), _ptr(P_vo), float(scale), _ptr(out),
                                      _ptr(workspace), ws_bytes, _stream(stream, q.get_device())))


def _decode_tensors(desc: CacheDesc, q, P_qk, P_vo, out) -> None:
    et = _elem_torch_dtype(desc.dtype)
    shape = (desc.batch, desc.n_q_heads, desc.head_dim)
    _tensor(q, "q", et, shape)
    _tensor(out, "out", et, shape)
    _rotations(desc, P_qk, P_vo)
    _on_gpu(q=q, out=out, P_qk=P_qk, P_vo=P_vo)


def decode_attention_noalloc(desc: CacheDesc, seq_len: Sequence[int], k_active: Sequence[int],
                             q, P_qk, P_vo, out, scale: float = 0.0, stream=None,
                             k_value: Optional[Sequence[int]] = None) -> None:
    """swan_decode_attention with the library's own scratch instead of a workspace."""
    _decode_tensors(desc, q, P_qk, P_vo, out)
    _check(_lib.swan_decode_attention_noalloc(ctypes.byref(desc), _i32_array(seq_len),
                                              _i32_array(k_active), _opt_i32_array(k_value),
                                              _ptr(q), _ptr(P_qk), _ptr(P_vo), float(scale),
                                              _ptr(out), _stream(stream, q.get_device())))


def decode_step(desc: CacheDesc, seq_len: Sequence[int], k_active: Sequence[int], k_new, v_new,
                q, P_qk, P_vo, out, workspace, scale: float = 0.0, stream=None,
                k_value: Optional[Sequence[int]] = None) -> None:
    """swan_decode_step: append one token per sequence (seq_len: lengths before it), then
    decode q over the cache with it; workspace sized for the lengths after the step."""
    et = _elem_torch_dtype(desc.dtype)
    shape = (desc.batch, desc.n_kv_heads, 1, desc.head_dim)
    _tensor(k_new, "k_new", et, shape)
    _tensor(v_new, "v_new", et, shape)
    _decode_tensors(desc, q, P_qk, P_vo, out)
    _on_gpu(k_new=k_new, v_new=v_new)
    if workspace is None or not workspace.is_cuda or not workspace.is_contiguous():
        raise SwanError(SWAN_ERR_WORKSPACE, "workspace must be a contiguous GPU tensor")
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(_lib.swan_decode_step(ctypes.byref(desc), _i32_array(seq_len), _i32_array(k_active),
                                 _opt_i32_array(k_value), _ptr(k_new), _ptr(v_new), _ptr(q),
                                 _ptr(P_qk), _ptr(P_vo), float(scale), _ptr(out),
                                 _ptr(workspace), ws_bytes, _stream(stream, q.get_device())))


def change_k(src: CacheDesc, k_active_src: Sequence[int], k_value_src: Optional[Sequence[int]],
             dst: CacheDesc, k_active_dst: Sequence[int], k_value_dst: Optional[Sequence[int]],
             seq_len: Sequence[int], stream=None) -> None:
    """Lay src's sparse caches out again in dst for the new k (see swan_change_k)."""
    _check(_lib.swan_change_k(ctypes.byref(src), _i32_array(k_active_src),
                              _opt_i32_array(k_value_src), ctypes.byref(dst),
                              _i32_array(k_active_dst), _opt_i32_array(k_value_dst),
                              _i32_array(seq_len), _stream(stream)))


def rope(x, pos0: Sequence[int], base: float, out=None, stream=None):
    """RoPE of rows x [B][H][n][128] (float16 or float32, cuda) at positions pos0[b] + i;
    out=None writes a new tensor, out=x works in place."""
    import torch

    if out is None:
        out = torch.empty_like(x)
    B, H, n, d = x.shape
    code = SWAN_F16 if x.dtype == torch.float16 else SWAN_F32
    _check(_lib.swan_rope(_ptr(x), _ptr(out), code, B, H, n, d, _i32_array(pos0), float(base),
                          _stream(stream)))
    return out


def set_decode_tuning(target_waves: int = 0, short_split_pages: int = 0, merge_pct: int = 0,
                      side_streams: int = 0) -> None:
    """Split plan and launch grouping of the decode calls on this thread
    (swan_set_decode_tuning; 0 = the default, -1 = off where the header allows it).
    With every argument 0 the defaults are restored."""
    t = DecodeTuning(target_waves, short_split_pages, merge_pct, side_streams)
    _check(_lib.swan_set_decode_tuning(ctypes.byref(t)))


def set_profile_events(start=None, stop=None) -> None:
    """Record start/stop (events with a .cuda_event HIP handle: torch.cuda.Event, or one
    made for timing only) around the attention kernels of the next decode calls on
    this thread (None, None disables)."""
    _check(_lib.swan_set_profile_events(None if start is None else start.cuda_event,
                                        None if stop is None else stop.cuda_event))


class SwanCache:
    """Owns the device arrays of one layer's hybrid cache and the host-side lengths.

    The arrays are plain torch tensors (uint8 pages, storage-typed ring); the
    library only ever receives their device pointers.  sparse_values="e4m3"
    (float16 only) stores the pruned values as one-byte E4M3 codes.  k_value
    (one per sequence) prunes the values to other k than the keys (k_active);
    None keeps both at k_active.
    """

    def __init__(self, batch: int, n_q_heads: int, n_kv_heads: int, buffer_tokens: int,
                 sparse_capacity: int, k_active: Sequence[int], dtype, device,
                 head_dim: int = HEAD_DIM, sparse_values: str = "same",
                 k_value: Optional[Sequence[int]] = None):
        import torch

        self.dtype = dtype
        self.sparse_values = sparse_values
        self.device = torch.device(device)
        self.k_active = [int(k) for k in k_active]
        if len(self.k_active) != batch:
            raise ValueError("k_active needs one entry per sequence")
        self.k_value = None if k_value is None else [int(k) for k in k_value]
        if self.k_value is not None and len(self.k_value) != batch:
            raise ValueError("k_value needs one entry per sequence")
        self.seq_len = [0] * batch
        self.desc = CacheDesc(batch, n_q_heads, n_kv_heads, head_dim, buffer_tokens,
                              sparse_capacity, dtype_code(dtype, sparse_values), 0, None, None,
                              None, None)
        kb, vb, rb = cache_bytes(self.desc, self.k_active, self.k_value)
        # torch's caching allocator returns 256-byte aligned blocks
        self.k_pages = torch.zeros(max(kb, 16), dtype=torch.uint8, device=self.device)
        self.v_pages = torch.zeros(max(vb, 16), dtype=torch.uint8, device=self.device)
        shape = (batch, n_kv_heads, buffer_tokens, head_dim)
        self.k_ring = torch.zeros(shape, dtype=dtype, device=self.device)
        self.v_ring = torch.zeros(shape, dtype=dtype, device=self.device)
        self.desc.k_pages = self.k_pages.data_ptr()
        self.desc.v_pages = self.v_pages.data_ptr()
        self.desc.k_ring = self.k_ring.data_ptr() if buffer_tokens > 0 else None
        self.desc.v_ring = self.v_ring.data_ptr() if buffer_tokens > 0 else None
        self._ws = None

    @property
    def batch(self) -> int:
        return self.desc.batch

    def append(self, k_new, v_new, P_qk, P_vo, n_new_per_seq=None, stream=None) -> None:
        """Compress-append k_new / v_new ([B][H_kv][n][d]) and advance the lengths.

        n_new_per_seq optionally appends only the first n_b rows of sequence b.
        """
        compress_append(self.desc, self.seq_len, self.k_active, k_new, v_new, P_qk, P_vo,
                        n_new_per_seq, stream, self.k_value)
        n = int(k_new.shape[2])
        per = [n] * self.batch if n_new_per_seq is None else [int(x) for x in n_new_per_seq]
        self.seq_len = [L + m for L, m in zip(self.seq_len, per)]

    def change_k(self, k_active: Sequence[int], k_value: Optional[Sequence[int]] = None,
                 stream=None) -> None:
        """Change k of the running sequences (swan_change_k): new page arrays for the new
        k, the stored tokens converted into them, the dense buffer kept.  Tokens that
        leave the buffer from now on are pruned with the new k."""
        import torch

        k_active = [int(k) for k in k_active]
        k_value = None if k_value is None else [int(k) for k in k_value]
        dst = CacheDesc(*[getattr(self.desc, f) for f, _ in CacheDesc._fields_])
        kb, vb, _ = cache_bytes(dst, k_active, k_value)
        k_pages = torch.zeros(max(kb, 16), dtype=torch.uint8, device=self.device)
        v_pages = torch.zeros(max(vb, 16), dtype=torch.uint8, device=self.device)
        dst.k_pages = k_pages.data_ptr()
        dst.v_pages = v_pages.data_ptr()
        change_k(self.desc, self.k_active, self.k_value, dst, k_active, k_value, self.seq_len,
                 stream)
        # the old pages stay alive until the conversion on the stream has read them
        (stream or torch.cuda.current_stream()).synchronize()
        self.desc, self.k_pages, self.v_pages = dst, k_pages, v_pages
        self.k_active, self.k_value = k_active, k_value
        self._ws = None

    def workspace(self):
        import torch

        need = decode_workspace_bytes(self.desc, self.seq_len, self.k_active, self.k_value)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        return self._ws

    def decode(self, q, P_qk, P_vo, out=None, scale: float = 0.0, stream=None):
        import torch

        if out is None:
            out = torch.empty_like(q)
        decode_attention(self.desc, self.seq_len, self.k_active, q, P_qk, P_vo, out,
                         self.workspace(), scale, stream, self.k_value)
        return out

    def step(self, k_new, v_new, q, P_qk, P_vo, out=None, scale: float = 0.0, stream=None):
        """One decode step (swan_decode_step): append k_new / v_new ([B][H_kv][1][d]),
        advance the lengths, and return the attention of q ([B][H_q][d]) over the cache."""
        import torch

        if out is None:
            out = torch.empty_like(q)
        after = [L + 1 for L in self.seq_len]
        need = decode_workspace_bytes(self.desc, after, self.k_active, self.k_value)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        decode_step(self.desc, self.seq_len, self.k_active, k_new, v_new, q, P_qk, P_vo, out,
                    self._ws, scale, stream, self.k_value)
        self.seq_len = after
        return out
