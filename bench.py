#!/usr/bin/env python3
"""Benchmark of the SWAN decode hot path on one MI355X.

One step = Algorithm 1 for one decode token of every sequence: compress-append
of the new key/value (rotate, append to the buffer, evict and prune the oldest
buffered token) followed by decode attention over the sparse pages and the
dense buffer (q rotation, sparse split-K attention, buffer partial, merge and
inverse rotation).  Inputs are synthetic (the seeded low-rank recipe of
swan_inputs), already resident in HBM before the timed region.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
import argparse
import ctypes
import hashlib
import json
import math
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MALL_BYTES = 256 << 20  # MI355X last-level (Infinity) cache
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_traffic_{wl}.txt")
# sources of the decode attention kernels: counter summaries are valid only for these bytes
ATTN_SOURCES = ("decode.hip", "decode_gqa.hip", "decode_asym.hip", "decode_gqa_asym.hip",
                "decode_fused.hip", "decode_mha.h", "decode_gqa.h", "decode_common.h", "decode_gqa_common.h",
                "swan_device.h", "swan_internal.h")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama2_7b_L32k_b16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="seconds of oracle work per host core in the CPU baseline")
    ap.add_argument("--change-k", type=int, default=0,
                    help="also time swan_change_k of the cache from the workload's k to this k")
    ap.add_argument("--layer", action="store_true",
                    help="also time decode steps of the whole attention layer (synthetic weights)")
    ap.add_argument("--replicas", type=int, default=0,
                    help="caches the steps rotate over (0: 8 when one step's attention bytes "
                         "fit the GPU's 256 MB last-level cache, else 1)")
    ap.add_argument("--probe-copy", type=int, default=0,
                    help="also run a device copy of this many bytes (HBM counter calibration)")
    return ap.parse_args()


class TimingEvent:
    """A HIP event made for timing only (hipEventDisableSystemFence): the library's
    record of it before and after the attention launches then adds no system-scope
    release to the step, which torch's events do (a few microseconds per record on
    a short step).  The same .cuda_event / elapsed_time(end) as torch.cuda.Event."""
    FLAGS = 0x20000000  # hipEventDisableSystemFence
    _hip = None

    @classmethod
    def _runtime(cls):
        if cls._hip is None:  # the HIP runtime this process (torch, the library) runs on
            path = next(ln.split()[-1] for ln in open("/proc/self/maps") if "libamdhip64" in ln)
            hip = ctypes.CDLL(path)
            hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p),
                                                    ctypes.c_uint]
            hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                ctypes.c_void_p]
            hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
            cls._hip = hip
        return cls._hip

    def __init__(self):
        self._ev = ctypes.c_void_p()
        st = self._runtime().hipEventCreateWithFlags(ctypes.byref(self._ev), self.FLAGS)
        if st != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({st})")
        self.cuda_event = self._ev.value

    def elapsed_time(self, end) -> float:
        ms = ctypes.c_float()
        st = self._runtime().hipEventElapsedTime(ctypes.byref(ms), self._ev, end._ev)
        if st != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({st})")
        return ms.value

    def __del__(self):
        if self._hip is not None and self._ev.value:
            self._hip.hipEventDestroy(self._ev)


def source_digest() -> str:
    h = hashlib.sha256()
    for name in ATTN_SOURCES:
        with open(os.path.join(ROOT, "paper_2511_18936_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(wl: str, digest: str):
    """HBM bytes of one step's attention launches from the committed counter summary,
    if it was taken on the current kernel source (else None)."""
    path = TRAFFIC_FILE.format(wl=wl)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for ln in f:
            if ":" in ln and not ln.startswith("#"):
                k, v = ln.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("source_digest") != digest:
        return None
    try:
        return float(vals["hbm_bytes_per_step"])
    except (KeyError, ValueError):
        return None


def value_bytes(w, esize):
    """Bytes of one stored sparse value (one for 8-bit E4M3 values)."""
    return 1 if w.sparse_values == "e4m3" else esize


def attention_bytes(w, seq_len, k_key, k_val, esize):
    """Algorithmic bytes of one step's attention: every sparse (value, index) pair of
    the keys (k_key per token) and of the values (k_val) once, plus the dense buffer
    of keys and values once."""
    total = 0
    vb = value_bytes(w, esize)
    for b in range(w.batch):
        L = seq_len[b]
        S = max(L - w.buffer, 0)
        nb = min(L, w.buffer)
        per_head = S * (k_key[b] + k_val[b]) * (vb + 1) + 2 * nb * w.head_dim * esize
        total += w.n_kv_heads * per_head
    return total


def kpad(k: int) -> int:
    return (k + 7) // 8 * 8


def fused_path(w) -> bool:
    """MHA on fp16 storage: a batch with several k_pad takes one launch in which
    each sequence's waves are specialised on its own k_pad."""
    return w.dtype == "f16" and w.n_q_heads == w.n_kv_heads


def attention_launches(k_key, k_val, merge_pct: int = 66, fused: bool = False):
    """The library's attention launches for these per-sequence k: [(kp8, same_k_pad)].
    Sequences are grouped by (key, value) k_pad.  fused (fused_path): several groups
    make one launch.  Otherwise, from the largest k_pad down, a group joins the
    launch before it when its k_pad is at least merge_pct % of that launch's (the
    library's default, 66; <= 0 merges nothing), and a launch whose sequences do
    not all have its k_pad for both roles runs the instances for different k_pad."""
    pct = merge_pct
    groups = sorted({(kpad(a) // 8, kpad(b) // 8) for a, b in zip(k_key, k_val)},
                    key=lambda g: (-max(g), -g[0], -g[1]))
    if fused and len(groups) > 1:
        return [(max(groups[0]), False)]
    launches = []
    for pk, pv in groups:
        kp = max(pk, pv)
        if launches and pct > 0 and kp * 100 >= launches[-1][0] * pct:
            launches[-1] = (launches[-1][0], False)
        else:
            launches.append((kp, pk == pv))
    return launches


def attn_kernel_name(w, k_key, k_val) -> str:
    """The decode attention kernel the library launches for this shape."""
    g = w.n_q_heads // w.n_kv_heads
    launches = attention_launches(k_key, k_val, fused=fused_path(w))
    if fused_path(w) and len({(kpad(a), kpad(b)) for a, b in zip(k_key, k_val)}) > 1:
        return ("attn_fused_kernel (one query head per wave, each sequence's waves specialised "
                "on its own k_pad; sparse split-K + dense buffer)")
    asym = not all(same for _, same in launches)
    note = ("; launches mixing k_pad (keys and values, or merged sequences): specialised on "
            "the largest, each role and sequence at its own page size" if asym else "")
    if w.dtype == "f16" and g > 1 and g % 2 == 0:
        hpw = 8 if g % 8 == 0 else 4 if g % 4 == 0 else 2
        return (f"attn_gqa_kernel ({hpw} query heads per wave, sparse split-K + dense buffer"
                f"{note})")
    return f"attn_kernel (one query head per wave, sparse split-K + dense buffer{note})"


def launches_per_step(w, k_key, k_val) -> int:
    return len(attention_launches(k_key, k_val, fused=fused_path(w)))


def time_change_k(swan, torch, w, cache, ks, kvs, k_new, esize, reps=5):
    """swan_change_k of the whole cache from the workload's k to k_new (both roles),
    timed with HIP events on the stream it runs on; bytes = the pages read (old k_pad)
    plus the pages written (new k_pad)."""
    kd = [k_new] * w.batch
    dst = swan.CacheDesc(*[getattr(cache.desc, f) for f, _ in swan.CacheDesc._fields_])
    kb, vb, _ = swan.cache_bytes(dst, kd, None)
    kp = torch.empty(kb, dtype=torch.uint8, device=cache.device)
    vp = torch.empty(vb, dtype=torch.uint8, device=cache.device)
    dst.k_pages, dst.v_pages = kp.data_ptr(), vp.data_ptr()
    swan.change_k(cache.desc, ks, kvs, dst, kd, None, cache.seq_len)  # warm-up
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        swan.change_k(cache.desc, ks, kvs, dst, kd, None, cache.seq_len)
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) * 1e-3 / reps
    vbytes = value_bytes(w, esize) + 1
    kvl = ks if kvs is None else kvs
    nbytes = 0
    for b in range(w.batch):
        S = max(cache.seq_len[b] - w.buffer, 0)
        n = w.n_kv_heads * S * vbytes
        nbytes += n * (kpad(ks[b]) + kpad(kvl[b]) + 2 * kpad(k_new))
    return {"from": [ks[0], kvl[0]], "to": k_new, "ms": t * 1e3, "bytes": nbytes,
            "gbps": nbytes / t / 1e9, "frac": nbytes / t / 1e9 / HBM_PEAK_GBPS,
            "kernel": "change_k_kernel (one launch per role)"}


def time_layer(swan, torch, si, w, Pqk, Pvo, ks, kvs, dev, warmup, steps):
    """Decode steps of the attention layer around the cache (RoPE, W_V / W_O absorbing
    P_VO, paper_2511_18936_amd.layer) at the workload's shape: synthetic float16
    weights, hidden = n_heads * 128, the cache filled to the workload's context; each
    step = q/k/v GEMMs, RoPE, append, decode, output GEMM, timed with HIP events."""
    import math

    from paper_2511_18936_amd.layer import SwanAttentionLayer

    hidden = w.n_q_heads * w.head_dim
    base = 500000.0 if "llama3" in w.name else 10000.0
    gen = torch.Generator(device=dev)
    gen.manual_seed(si.torch_seed_for(w.wid, 9000))
    def weight(n_in, n_out):
        m = torch.randn(n_in, n_out, generator=gen, device=dev, dtype=torch.float32)
        return (m / math.sqrt(n_in)).to(torch.float16 if w.dtype == "f16" else torch.float32)
    d = w.head_dim
    L0 = w.context - 1
    cap = max(w.context + warmup + steps - w.buffer, 1)
    layer = SwanAttentionLayer(weight(hidden, w.n_q_heads * d), weight(hidden, w.n_kv_heads * d),
                               weight(hidden, w.n_kv_heads * d), weight(w.n_q_heads * d, hidden),
                               Pqk, Pvo, w.n_q_heads, w.n_kv_heads, base, w.batch, w.buffer, cap,
                               ks, kvs, w.sparse_values)
    K = si.kv_rows_device(w.wid, w.batch, w.n_kv_heads, si.ROLE_K, L0, w.dtype, dev)
    V = si.kv_rows_device(w.wid, w.batch, w.n_kv_heads, si.ROLE_V, L0, w.dtype, dev)
    layer.cache.append(K, V, layer.P_qk, None)  # the context, its values taken as rotated
    del K, V
    torch.cuda.empty_cache()
    xs = [torch.randn(w.batch, 1, hidden, generator=gen, device=dev).to(layer.dtype)
          for _ in range(warmup + steps)]
    for i in range(warmup):
        layer(xs[i])
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for i in range(steps):
        y = layer(xs[warmup + i])
    e1.record()
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y).all())
    t = e0.elapsed_time(e1) * 1e-3 / steps
    return {"hidden": hidden, "rope_base": base, "step_ms": t * 1e3,
            "tokens_per_s": w.batch / t,
            "weights_bytes": 2 * hidden * d * (2 * w.n_q_heads + 2 * w.n_kv_heads)}


def streaming_ceiling(torch, caches, dev, reps: int = 5):
    """Bandwidth of a read-only streaming kernel over the caches' page arrays (the
    bytes the attention kernels stream), with their load form: swan_stream_read of
    libswanbench.so, timed with HIP events on the current stream; the best of a
    sweep over wave counts and loads in flight."""
    import ctypes

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2511_18936_amd", "libswanbench.so"))
    lib.swan_stream_read.restype = ctypes.c_int32
    lib.swan_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32,
                                     ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    sink = torch.empty(16384, dtype=torch.int32, device=dev)
    arrays = [t for c in caches for t in (c.k_pages, c.v_pages)]
    stream = torch.cuda.current_stream().cuda_stream
    nbytes = sum(t.numel() // 1024 * 1024 for t in arrays)

    def one_pass(waves, u):
        for t in arrays:
            st = lib.swan_stream_read(t.data_ptr(), t.numel(), waves, u, sink.data_ptr(), stream)
            if st != 0:
                raise RuntimeError(f"swan_stream_read returned {st}")

    best = None
    for waves in (1024, 2048, 4096, 8192, 16384):
        for u in (8, 16):
            one_pass(waves, u)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                one_pass(waves, u)
            e1.record()
            torch.cuda.synchronize()
            t = e0.elapsed_time(e1) * 1e-3 / reps
            if best is None or t < best[0]:
                best = (t, waves, u)
    t, waves, u = best
    return {"gbps": nbytes / t / 1e9, "bytes": nbytes, "ms": t * 1e3, "waves": waves,
            "loads_in_flight": u, "launches_per_pass": len(arrays)}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.machine()


def _oracle_unit(args):
    """One (sequence, KV head) unit for the oracle's timing: its caches after the
    step's append (the attention input) and just before it (the append input)."""
    import numpy as np

    import swan_inputs as si
    from oracle import swan_oracle as O

    wname, u = args
    w = si.WORKLOADS[wname]
    ks = si.k_active_for(w)
    kvs = si.k_value_for(w)
    kvs = ks if kvs is None else kvs
    np_dt = si.np_dtype(w.dtype)
    vals = "e4m3" if w.sparse_values == "e4m3" else "t"
    L = w.context
    b, h = (u // w.n_kv_heads) % w.batch, u % w.n_kv_heads
    Pqk, _ = O.calibrate_f32(si.calibration_rows(w.wid, h, si.ROLE_K))
    Pvo, _ = O.calibrate_f32(si.calibration_rows(w.wid, h, si.ROLE_V))
    K = si.kv_rows_host(w.wid, b, h, si.ROLE_K, L, w.dtype)
    V = si.kv_rows_host(w.wid, b, h, si.ROLE_V, L, w.dtype)
    c = O.compress_block(K, V, Pqk, Pvo, w.buffer, int(ks[b]), np_dt, values=vals,
                         k_value=int(kvs[b]))
    c_prev = O.compress_block(K[L - 1 - w.buffer:L - 1], V[L - 1 - w.buffer:L - 1], Pqk, Pvo,
                              w.buffer, int(ks[b]), np_dt, values=vals, k_value=int(kvs[b]))
    qs = si.queries_host(w.wid, 1, w.group, w.dtype)[0].astype(np.float64)
    return (Pqk, Pvo, c, c_prev, K[L - 1], V[L - 1], qs, int(ks[b]), int(kvs[b]), np_dt, vals,
            w.buffer)


def _oracle_unit_steps(unit, reps: int):
    """reps decode steps of one unit with the oracle: append the current token
    (Algorithm 1: rotate, buffer, evict and prune the oldest) and attend for each of
    the unit's query heads.  Returns (append seconds, attention seconds) in total."""
    import time as _t

    from oracle import swan_oracle as O

    Pqk, Pvo, c, c_prev, kl, vl, qs, k, kv, np_dt, vals, bb = unit
    t_app = t_att = 0.0
    for _ in range(reps):
        uc = O.UnitCache(Pqk, Pvo, bb, k, np_dt, values=vals, k_value=kv)
        uc.k_buf.extend(list(c_prev["k_buf"]))
        uc.v_buf.extend(list(c_prev["v_buf"]))
        t0 = _t.perf_counter()
        uc.append(kl, vl)
        t1 = _t.perf_counter()
        for q in qs:
            O.attend_arrays(q, Pqk, Pvo, c)
        t2 = _t.perf_counter()
        t_app += t1 - t0
        t_att += t2 - t1
    return t_app, t_att


def _oracle_worker(args):
    """Pool worker: build a unit, wait for every worker, then time `reps` steps on
    one thread; returns (start, end, reps) on the shared monotonic clock."""
    import numpy  # noqa: F401  (loaded before the limit, which covers loaded libraries only)
    from threadpoolctl import threadpool_limits

    import swan_inputs  # noqa: F401
    from oracle import swan_oracle  # noqa: F401

    wname, u, reps, barrier = args
    with threadpool_limits(limits=1):
        unit = _oracle_unit((wname, u))
        barrier.wait()
        t0 = time.perf_counter()
        _oracle_unit_steps(unit, reps)
        t1 = time.perf_counter()
    return t0, t1, reps


def cpu_baseline(w, seconds: float = 8.0):
    """The oracle, as it stands, timed on the host's cores on a bounded sample of the
    workload: one (sequence, KV head) unit per worker process, each worker doing
    whole decode steps of its unit (append + attention for the unit's query heads)
    on one thread for about `seconds`; all workers start together and the rate is
    their steps over the wall time.  A one-thread run of the same unit comes first
    and sets the repetition count."""
    import multiprocessing as mp

    import numpy  # noqa: F401  (loaded before the limit, which covers loaded libraries only)
    from threadpoolctl import threadpool_limits

    import swan_inputs  # noqa: F401
    from oracle import swan_oracle  # noqa: F401

    cores = max(1, min(len(os.sched_getaffinity(0)), 16))
    units_per_step = w.batch * w.n_kv_heads  # one append + G attentions each
    with threadpool_limits(limits=1):
        unit = _oracle_unit((w.name, 0))
        _oracle_unit_steps(unit, 1)  # warm-up
        t0 = time.perf_counter()
        ta, tt = _oracle_unit_steps(unit, 3)
        one = (time.perf_counter() - t0) / 3
    reps = max(1, int(seconds / one))
    one_thread = w.batch / (units_per_step * one)
    ctx = mp.get_context("spawn")
    with ctx.Manager() as mgr:
        barrier = mgr.Barrier(cores)
        with ctx.Pool(cores) as pool:
            res = pool.map(_oracle_worker, [(w.name, u, reps, barrier) for u in range(cores)])
    wall = max(r[1] for r in res) - min(r[0] for r in res)
    unit_steps = sum(r[2] for r in res)
    value = w.batch * unit_steps / (units_per_step * wall)
    return {
        "value": value,
        "unit": "decode tokens/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"{cores} (sequence, KV head) units at L={w.context}, one per worker process "
                   f"on one thread each, {reps} decode steps per unit (append of the current "
                   f"token {ta / 3 * 1e3:.2f} ms + {w.group} attention(s) {tt / 3 * 1e3:.1f} ms "
                   f"on one thread), {wall:.1f} s wall; scaled to the step's "
                   f"{units_per_step} units; numpy float64"),
        "one_thread": {"value": one_thread, "unit": "decode tokens/s", "cores": 1},
        "host_cpu": cpu_model(),
        "host_threads_available": len(os.sched_getaffinity(0)),
    }


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the SWAN path "
              "here is a single-GPU kernel set and has no multi-GPU mode.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import swan_inputs as si
    from paper_2511_18936_amd import swan

    w = si.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    tdt = {"f16": torch.float16, "f32": torch.float32}[w.dtype]
    esize = 2 if w.dtype == "f16" else 4
    ks = [int(k) for k in si.k_active_for(w)]
    kvs = si.k_value_for(w)  # None: values keep the keys' k
    kvs = None if kvs is None else [int(k) for k in kvs]
    kv_list = ks if kvs is None else kvs
    # warm-up steps, timed steps, then a few steps that also time compress and decode
    # apart (their events stay out of the timed region)
    n_detail = min(args.steps, 10)
    n_extra = args.warmup + args.steps + n_detail
    L0 = w.context - 1  # tokens cached before the first measured step

    # ---- rotations (Sec. 4.1.2), on the GPU ----
    t = time.perf_counter()
    Pqk = torch.empty((w.n_kv_heads, 128, 128), dtype=torch.float32, device=dev)
    Pvo = torch.empty_like(Pqk)
    for h in range(w.n_kv_heads):
        for role, P in ((si.ROLE_K, Pqk), (si.ROLE_V, Pvo)):
            rows = torch.tensor(si.calibration_rows(w.wid, h, role), device=dev)
            swan.calibrate_rotation(rows, P[h])
    log(f"[bench] calibrated {2 * w.n_kv_heads} rotations in {time.perf_counter() - t:.1f}s")

    # ---- synthetic K/V on the device and the cache ----
    t = time.perf_counter()
    Kp = si.kv_rows_device(w.wid, w.batch, w.n_kv_heads, si.ROLE_K, L0, w.dtype, dev)
    Vp = si.kv_rows_device(w.wid, w.batch, w.n_kv_heads, si.ROLE_V, L0, w.dtype, dev)
    Ks = si.kv_rows_device(w.wid, w.batch, w.n_kv_heads, si.ROLE_K, n_extra, w.dtype, dev,
                           block=1)
    Vs = si.kv_rows_device(w.wid, w.batch, w.n_kv_heads, si.ROLE_V, n_extra, w.dtype, dev,
                           block=1)
    step_k = [Ks[:, :, i:i + 1].contiguous() for i in range(n_extra)]
    step_v = [Vs[:, :, i:i + 1].contiguous() for i in range(n_extra)]
    qs = [si.queries_device(w.wid, w.batch, w.n_q_heads, w.dtype, dev, step=i)
          for i in range(n_extra)]
    capacity = max(w.context + n_extra - w.buffer, 1)
    # A step whose bytes fit the 256 MB last-level (MALL) cache would be timed
    # partly out of that cache if it read the same cache every step; the steps then
    # rotate over replicas, whose pages together exceed it.
    step_bytes = attention_bytes(w, [w.context] * w.batch, ks, kv_list, esize)
    n_rep = args.replicas or (8 if step_bytes < MALL_BYTES else 1)
    caches = [swan.SwanCache(w.batch, w.n_q_heads, w.n_kv_heads, w.buffer, capacity, ks, tdt,
                             dev, sparse_values=w.sparse_values, k_value=kvs)
              for _ in range(n_rep)]
    cache = caches[0]
    torch.cuda.synchronize()
    log(f"[bench] inputs ready in {time.perf_counter() - t:.1f}s "
        f"(raw K/V {2 * Kp.numel() * esize / 1e9:.2f} GB, "
        f"pages {(cache.k_pages.numel() + cache.v_pages.numel()) / 1e9:.2f} GB)")

    # ---- prefill compress (Algorithm 1 over L0 tokens at once), timed ----
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    cache.append(Kp, Vp, Pqk, Pvo)
    e1.record()
    torch.cuda.synchronize()
    t_prefill = e0.elapsed_time(e1) * 1e-3
    prefill_bytes = 2 * Kp.numel() * esize + sum(
        w.n_kv_heads * max(L0 - w.buffer, 0) * (k + kv) * (value_bytes(w, esize) + 1)
        for k, kv in zip(ks, kv_list))
    log(f"[bench] prefill compress of {L0} tokens: {t_prefill * 1e3:.2f} ms "
        f"({prefill_bytes / t_prefill / 1e9:.0f} GB/s algorithmic)")
    for c in caches[1:]:
        c.append(Kp, Vp, Pqk, Pvo)
    del Kp, Vp
    torch.cuda.empty_cache()

    # workspace sized for the longest step, allocated before timing
    final_len = [L + n_extra for L in cache.seq_len]  # every replica appends at most n_extra
    ws = torch.empty(swan.decode_workspace_bytes(cache.desc, final_len, ks, kvs),
                     dtype=torch.uint8, device=dev)
    ws_need = max(swan.decode_workspace_bytes(cache.desc, [L + i for L in cache.seq_len], ks, kvs)
                  for i in range(1, n_extra + 1))
    assert ws.numel() >= ws_need
    out = torch.empty((w.batch, w.n_q_heads, 128), dtype=tdt, device=dev)

    def step(i, evs=None, breakdown=False):
        """One decode step on replica i % n_rep: one swan_decode_step call (the
        compress-append of the new token, then decode attention); evs[2] / evs[3]
        bracket the attention launches (recorded by the library on their stream).
        With breakdown the step is the two calls it stands for instead, evs[0], [1],
        [4] bracketing the compress-append and the whole decode call."""
        cache = caches[i % n_rep]
        if evs is not None:
            swan.set_profile_events(evs[2], evs[3])
        if breakdown:
            evs[0].record()
            cache.append(step_k[i], step_v[i], Pqk, Pvo)
            evs[1].record()
            swan.decode_attention(cache.desc, cache.seq_len, ks, qs[i], Pqk, Pvo, out, ws,
                                  k_value=kvs)
            evs[4].record()
        else:
            swan.decode_step(cache.desc, cache.seq_len, ks, step_k[i], step_v[i], qs[i], Pqk,
                             Pvo, out, ws, k_value=kvs)
            cache.seq_len = [L + 1 for L in cache.seq_len]
        if evs is not None:
            swan.set_profile_events(None, None)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    def events(n):
        """Per step: [0], [1], [4] recorded here (torch), [2], [3] by the library."""
        return [[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
                 TimingEvent(), TimingEvent(), torch.cuda.Event(enable_timing=True)]
                for _ in range(n)]

    evs = events(args.steps)
    lens = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for j in range(args.steps):
        step(args.warmup + j, evs[j])
        lens.append(list(caches[(args.warmup + j) % n_rep].seq_len))
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    # untimed steps for the compress / decode breakdown
    devs = events(n_detail)
    for j in range(n_detail):
        step(args.warmup + args.steps + j, devs[j], breakdown=True)
    torch.cuda.synchronize()

    wall = t1 - t0
    t_comp = [e[0].elapsed_time(e[1]) * 1e-3 for e in devs]
    t_attn = [e[2].elapsed_time(e[3]) * 1e-3 for e in evs]
    t_dec = [e[1].elapsed_time(e[4]) * 1e-3 for e in devs]
    bytes_attn = [attention_bytes(w, L, ks, kv_list, esize) for L in lens]
    attn_avg = float(np.mean(t_attn))
    bytes_avg = float(np.mean(bytes_attn))
    achieved = bytes_avg / attn_avg / 1e9
    digest = source_digest()
    traffic = read_traffic(w.name, digest)
    dec_avg = float(np.mean(t_dec))
    log(f"[bench] step {wall / args.steps * 1e3:.3f} ms wall; compress {np.mean(t_comp) * 1e3:.3f} ms, "
        f"decode {dec_avg * 1e3:.3f} ms, attention kernel {attn_avg * 1e3:.3f} ms "
        f"= {achieved:.0f} GB/s ({achieved / HBM_PEAK_GBPS * 100:.1f}% of 8 TB/s)")
    ceiling = streaming_ceiling(torch, caches, dev)
    log(f"[bench] streaming-read ceiling over the same page arrays: {ceiling['gbps']:.0f} GB/s "
        f"({ceiling['gbps'] / HBM_PEAK_GBPS * 100:.1f}% of 8 TB/s); attention kernel at "
        f"{achieved / ceiling['gbps'] * 100:.1f}% of it")

    if args.probe_copy:
        n = args.probe_copy // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for _ in range(3):
            dst.copy_(src)
        c0.record()
        for _ in range(10):
            dst.copy_(src)
        c1.record()
        torch.cuda.synchronize()
        tc = c0.elapsed_time(c1) * 1e-3 / 10
        log(f"[bench] probe copy of {args.probe_copy} bytes: {tc * 1e3:.3f} ms, "
            f"{2 * args.probe_copy / tc / 1e9:.0f} GB/s read+write")

    change_k = None
    if args.change_k:
        change_k = time_change_k(swan, torch, w, cache, ks, kvs, args.change_k, esize)
        log(f"[bench] change_k {change_k['from']} -> {change_k['to']}: {change_k['ms']:.3f} ms, "
            f"{change_k['gbps']:.0f} GB/s read+write ({change_k['frac'] * 100:.1f}% of 8 TB/s)")

    layer = None
    if args.layer:
        del cache, caches
        torch.cuda.empty_cache()
        layer = time_layer(swan, torch, si, w, Pqk, Pvo, ks, kvs, dev, args.warmup, args.steps)
        log(f"[bench] layer decode step (hidden {layer['hidden']}): {layer['step_ms']:.3f} ms, "
            f"{layer['tokens_per_s']:.0f} tokens/s (attention alone {dec_avg * 1e3:.3f} ms)")

    cpu = None
    if not args.no_cpu_baseline:
        t = time.perf_counter()
        cpu = cpu_baseline(w, args.cpu_seconds)
        log(f"[bench] cpu baseline in {time.perf_counter() - t:.1f}s: {cpu['value']:.2f} tokens/s")

    result = {
        "metric": "decode-attention tokens/s + achieved HBM GB/s (% of peak), 7B shape, 32k ctx",
        "value": w.batch * args.steps / wall,
        "unit": "decode tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",  # the arithmetic: scores, softmax and accumulation in float32
        "storage_dtype": w.dtype if w.sparse_values != "e4m3" else f"{w.dtype}+e4m3",
        "data": "synthetic (seeded low-rank K/V recipe, N(0,1) queries; no dataset or weights)",
        "config": {
            "workload": w.name, "batch": w.batch, "n_q_heads": w.n_q_heads,
            "n_kv_heads": w.n_kv_heads, "head_dim": w.head_dim, "context": w.context,
            "buffer": w.buffer, "k_active": ks if not w.k_active else w.k_active,
            "k_value": None if kvs is None else (kvs if not w.k_value else w.k_value),
            "storage": w.dtype, "index": "u8",
            "sparse_values": "e4m3" if w.sparse_values == "e4m3" else w.dtype,
        },
        "roofline": {
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": traffic,
            "kernel": attn_kernel_name(w, ks, kv_list),
            # one launch per distinct (key, value) padded k in the batch; bytes and
            # time cover all of a step's attention launches together
            "launches_per_step": launches_per_step(w, ks, kv_list),
            "algorithmic_bytes_per_launch": bytes_avg,
            "avg_launch_ms": attn_avg * 1e3,
            "source_digest": digest,
            "replicas": n_rep,
            # the same page arrays read by a kernel that only streams them with the
            # attention kernels' load form (libswanbench.so, swan_stream_read)
            "ceiling_gbps": ceiling["gbps"],
            "frac_of_ceiling": achieved / ceiling["gbps"],
            "ceiling_bytes": ceiling["bytes"],
            "ceiling_shape": {k: ceiling[k] for k in ("waves", "loads_in_flight",
                                                     "launches_per_pass")},
        },
        "cpu_baseline": cpu,
        "detail": {
            "compress_append_ms": float(np.mean(t_comp)) * 1e3,
            "decode_attention_ms": dec_avg * 1e3,
            "decode_attention_gbps": bytes_avg / dec_avg / 1e9,
            "prefill_tokens": L0,
            "prefill_compress_ms": t_prefill * 1e3,
            "prefill_compress_gbps": prefill_bytes / t_prefill / 1e9,
            "kv_tokens_per_s": float(np.mean([sum(L) for L in lens])) / dec_avg,
            "change_k": change_k,
            "layer": layer,
        },
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
