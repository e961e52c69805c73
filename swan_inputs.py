"""Seeded synthetic inputs for the SWAN decode path.

This module is shared by the tests, ``bench.py`` and ``__graft_entry__.smoke``.
It draws random numbers and nothing else: it holds none of SWAN's arithmetic
(no rotation, pruning, packing or attention), so neither the oracle nor the
HIP path depends on the other through it.

Recipe (the low-rank key/value structure that the method exploits, Sec. 1 and
Sec. 4.1.2 of the paper): for every KV head h and role r in {K, V},
rows = Z . diag(s) . R_h with Z ~ N(0, 1), s_j = exp(-j/16) for j = 0..d-1 and
R_h a Haar-random orthogonal matrix, independent per head and shared by K and
V.  Queries are N(0, I).  The first 4096 rows of each (head, role) calibrate
the rotation; cached tokens are further draws of the same recipe.  These
stand in for the post-RoPE activations of a calibration corpus, which are not
available here.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Optional, Sequence, Tuple

import numpy as np

HEAD_DIM = 128
DECAY = 1.0 / 16.0
CALIB_ROWS = 4096
BASE_SEED = 0
ROLE_K, ROLE_V, ROLE_Q = 0, 1, 2


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload shape.

    ``context`` is the number of cached tokens L at the measured decode step,
    the current token included.  ``prefill`` > 0 means the cache is built by a
    single compress-append of that many tokens before decoding.
    """

    wid: int
    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    context: int
    buffer: int
    k_active: int          # 0 means "drawn per sequence from k_choices"
    dtype: str             # "f32" or "f16"
    prefill: int = 0
    k_choices: Tuple[int, ...] = ()
    description: str = ""
    sparse_values: str = "same"  # "same" (values stored in dtype) or "e4m3" (8-bit)
    k_value: int = 0       # k of the values; 0 means the same k as the keys

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


WORKLOADS = {
    w.name: w
    for w in (
        Workload(0, "tiny_fp32_L512", 1, 1, 1, 128, 512, 16, 64, "f32",
                 description="1 head, d=128, fp32 storage, L=512, b=16, k=64"),
        Workload(1, "llama2_7b_L4k_b1", 1, 32, 32, 128, 4096, 128, 64, "f16",
                 description="Llama-2-7B layer, 32 MHA heads, B=1, L=4096, b=128, k=64, fp16"),
        Workload(2, "llama2_7b_L32k_b16", 16, 32, 32, 128, 32768, 128, 48, "f16",
                 description="Llama-2-7B layer, 32 MHA heads, B=16, L=32768, b=128, k=48, fp16"),
        Workload(3, "llama3_8b_gqa_L128k_b4", 4, 32, 8, 128, 131072, 256, 64, "f16",
                 description="Llama-3-8B layer, 32 q / 8 kv heads, B=4, L=131072, b=256, k=64, fp16"),
        Workload(4, "llama2_7b_prefill16k_b8", 8, 32, 32, 128, 16385, 128, 0, "f16",
                 prefill=16384, k_choices=(32, 48, 64, 96),
                 description="Llama-2-7B layer, B=8, prefill 16384 then decode, k per sequence "
                             "from {32,48,64,96}, b=128, fp16"),
        Workload(5, "llama2_7b_L32k_b16_e4m3", 16, 32, 32, 128, 32768, 128, 48, "f16",
                 sparse_values="e4m3",
                 description="the 32k x 16 Llama-2-7B layer with 8-bit (E4M3) sparse values, "
                             "fp16 buffer, k=48"),
        Workload(6, "llama3_8b_gqa_L128k_b4_e4m3", 4, 32, 8, 128, 131072, 256, 64, "f16",
                 sparse_values="e4m3",
                 description="the 128k x 4 Llama-3-8B GQA layer with 8-bit (E4M3) sparse "
                             "values, fp16 buffer, k=64"),
        # key/value retention 0.6 / 0.4 of d_h (the asymmetric rows of the
        # Appendix A.5 ablation): k = 77 for keys, 51 for values
        Workload(7, "llama2_7b_L32k_b16_k77_v51", 16, 32, 32, 128, 32768, 128, 77, "f16",
                 k_value=51,
                 description="the 32k x 16 Llama-2-7B layer, keys keep 77 and values 51 "
                             "components, b=128, fp16"),
        Workload(8, "llama3_8b_gqa_L128k_b4_k77_v51", 4, 32, 8, 128, 131072, 256, 77, "f16",
                 k_value=51,
                 description="the 128k x 4 Llama-3-8B GQA layer, keys keep 77 and values 51 "
                             "components, b=256, fp16"),
    )
}
WORKLOAD_BY_ID = {w.wid: w for w in WORKLOADS.values()}


def np_dtype(dtype: str):
    return {"f32": np.float32, "f16": np.float16, "f64": np.float64}[dtype]


def _seed_words(*keys: int) -> list:
    return [BASE_SEED] + [int(k) for k in keys]


def rng_for(*keys: int) -> np.random.Generator:
    """Independent numpy stream for a tuple of integer keys."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(_seed_words(*keys))))


def torch_seed_for(*keys: int) -> int:
    """63-bit seed for a torch.Generator, derived from the same keys."""
    h = hashlib.sha256(repr(_seed_words(*keys)).encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def spectrum(d: int = HEAD_DIM, decay: float = DECAY) -> np.ndarray:
    return np.exp(-decay * np.arange(d, dtype=np.float64))


def haar_orthogonal(rng: np.random.Generator, d: int) -> np.ndarray:
    """Haar-distributed orthogonal matrix: QR of a Gaussian with the sign of diag(R) fixed."""
    a = rng.standard_normal((d, d))
    q, r = np.linalg.qr(a)
    return q * np.sign(np.diag(r))[None, :]


def head_rotation(wid: int, h: int, d: int = HEAD_DIM) -> np.ndarray:
    return haar_orthogonal(rng_for(wid, 1000, h), d)


def lowrank_rows(rng: np.random.Generator, n: int, R: np.ndarray,
                 s: Optional[np.ndarray] = None) -> np.ndarray:
    d = R.shape[0]
    if s is None:
        s = spectrum(d)
    z = rng.standard_normal((n, d))
    return (z * s[None, :]) @ R


def calibration_rows(wid: int, h: int, role: int, n: int = CALIB_ROWS,
                     d: int = HEAD_DIM) -> np.ndarray:
    """fp32 calibration rows for (workload, kv head, role); role K rows calibrate P_QK."""
    R = head_rotation(wid, h, d)
    return lowrank_rows(rng_for(wid, 2000, h, role), n, R).astype(np.float32)


def kv_rows_host(wid: int, b: int, h: int, role: int, n: int, dtype: str,
                 d: int = HEAD_DIM, block: int = 0) -> np.ndarray:
    """Cached-token rows for one (sequence, kv head, role), rounded to the storage dtype."""
    R = head_rotation(wid, h, d)
    return lowrank_rows(rng_for(wid, 3000, b, h, role, block), n, R).astype(np_dtype(dtype))


def queries_host(wid: int, batch: int, n_q_heads: int, dtype: str, d: int = HEAD_DIM,
                 step: int = 0) -> np.ndarray:
    return rng_for(wid, 4000, step).standard_normal((batch, n_q_heads, d)).astype(np_dtype(dtype))


def k_active_for(w: Workload) -> np.ndarray:
    if w.k_active:
        return np.full(w.batch, w.k_active, dtype=np.int32)
    r = rng_for(w.wid, 5000)
    return r.choice(np.array(w.k_choices, dtype=np.int32), size=w.batch)


def k_value_for(w: Workload) -> Optional[np.ndarray]:
    """Per-sequence k of the values, or None when the values keep the keys' k."""
    if not w.k_value:
        return None
    return np.full(w.batch, w.k_value, dtype=np.int32)


def kv_rows_device(wid: int, batch: int, n_kv_heads: int, role: int, n: int, dtype: str,
                   device, d: int = HEAD_DIM, block: int = 0):
    """[batch][n_kv_heads][n][d] rows drawn on the GPU (same recipe, torch's generator).

    Used for the large workloads, whose raw rows (up to 8.6 GB) are too large to
    draw on the host.  Tests copy back the bytes of the units they check.
    """
    import torch

    tdt = {"f32": torch.float32, "f16": torch.float16}[dtype]
    out = torch.empty((batch, n_kv_heads, n, d), dtype=tdt, device=device)
    s = torch.tensor(spectrum(d), dtype=torch.float32, device=device)
    for h in range(n_kv_heads):
        R = torch.tensor(head_rotation(wid, h, d), dtype=torch.float32, device=device)
        for b in range(batch):
            g = torch.Generator(device=device)
            g.manual_seed(torch_seed_for(wid, 6000, b, h, role, block))
            # draw in slabs to bound the fp32 temporaries
            for r0 in range(0, n, 32768):
                r1 = min(n, r0 + 32768)
                z = torch.randn((r1 - r0, d), generator=g, device=device, dtype=torch.float32)
                out[b, h, r0:r1] = ((z * s) @ R).to(tdt)
    return out


def queries_device(wid: int, batch: int, n_q_heads: int, dtype: str, device,
                   d: int = HEAD_DIM, step: int = 0):
    import torch

    tdt = {"f32": torch.float32, "f16": torch.float16}[dtype]
    g = torch.Generator(device=device)
    g.manual_seed(torch_seed_for(wid, 7000, step))
    return torch.randn((batch, n_q_heads, d), generator=g, device=device,
                       dtype=torch.float32).to(tdt)


def tiny_case(seed: int, d: int, L: int, n_q: int = 1, n_kv: int = 1,
              dtype=np.float64) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Small dense random (q, K, V) for brute-force checks: q [n_q][d], K/V [n_kv][L][d]."""
    r = rng_for(9000, seed, d, L)
    q = r.standard_normal((n_q, d)).astype(dtype)
    K = r.standard_normal((n_kv, L, d)).astype(dtype)
    V = r.standard_normal((n_kv, L, d)).astype(dtype)
    return q, K, V


def random_orthogonal(seed: int, d: int) -> np.ndarray:
    return haar_orthogonal(rng_for(9100, seed, d), d)


def stack_seq(values: Sequence[int]) -> np.ndarray:
    return np.asarray(list(values), dtype=np.int32)
