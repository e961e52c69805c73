"""A Llama-shaped attention layer on the SWAN cache, in the paper's model-side form.

Sec. 4.2: queries and keys take RoPE first and are then rotated by P_QK at run
time (RoPE keeps P_QK out of W_Q and W_K), while P_VO is absorbed into the
weights, W_V_hat = W_V . P_VO per KV head and W_O_hat = P_VO^T . W_O per query
head, so the values enter the cache already rotated and the attention output
leaves it rotated, straight into W_O_hat (Lemma 2).

One call with n new tokens per sequence, on the current stream:
  [q | k | v_hat] = x . [W_Q | W_K | W_V_hat]    one dense GEMM (torch: the GEMM library)
  swan_rope on q and k at each sequence's next positions
  a prompt (n > 1): swan_compress_append(k, v_hat, P_QK, P_VO = NULL)
  a decode step (n = 1): swan_decode_step(k, v_hat, q, P_QK, P_VO = NULL) -> o_hat
  (the append, then the attention, in one call), and
  y = o_hat . W_O_hat                             dense GEMM
The SWAN steps run in libswan's kernels; attention over a prompt is the dense,
standard kind and is not part of this layer (a prompt call only fills the cache).
Weights are [in][out] row-major, x . W.
"""
from __future__ import annotations

from typing import Optional, Sequence

from . import swan

HEAD_DIM = swan.HEAD_DIM


def calibrate_joint(q, k, v, W_o, n_kv_heads: int, P_qk_out, P_vo_out, stream=None) -> None:
    """The layer's rotations from calibration activations (Sec. 4.1.1-4.1.2).

    q [N_q][n][128]: post-RoPE queries of n calibration tokens; k [N_kv][n][128]
    post-RoPE keys; v [N_kv][n][128] values (x . W_V, before any rotation);
    W_o [N_q 128][hidden] (cuda tensors, float16 or float32).  For each KV head j
    (query heads jG .. jG + G - 1) the joint matrices are stacked in device
    memory as float32, S_QK = [Q_grouped^(j); K^(j)] and S_VO = [V^(j); W_O^(h)^T
    for the group's heads], W_O^(h) being rows 128 h .. 128 h + 127 of W_o, and
    swan_calibrate_rotation writes their right singular matrices to P_qk_out[j]
    and P_vo_out[j] ([N_kv][128][128] float32)."""
    import torch

    n_q, n, d = q.shape
    if d != HEAD_DIM or n_q % n_kv_heads != 0:
        raise ValueError("q must be [N_q][n][128] with N_q a multiple of n_kv_heads")
    if tuple(k.shape) != (n_kv_heads, n, d) or tuple(v.shape) != (n_kv_heads, n, d):
        raise ValueError("k and v must be [n_kv_heads][n][128]")
    if W_o.dim() != 2 or W_o.shape[0] != n_q * d:
        raise ValueError("W_o must be [N_q * 128][hidden]")
    G = n_q // n_kv_heads
    hidden = W_o.shape[1]
    q_grouped = q.reshape(n_kv_heads, n * G, d)
    blocks = W_o.reshape(n_q, d, hidden)  # W_O^(h)
    ws = torch.empty(swan.calibrate_workspace_bytes(d), dtype=torch.uint8, device=q.device)
    for j in range(n_kv_heads):
        s_qk = torch.cat([q_grouped[j], k[j]], dim=0).float().contiguous()
        swan.calibrate_rotation(s_qk, P_qk_out[j], workspace=ws, stream=stream)
        wo_t = blocks[j * G:(j + 1) * G].transpose(1, 2).reshape(G * hidden, d)
        s_vo = torch.cat([v[j], wo_t], dim=0).float().contiguous()
        swan.calibrate_rotation(s_vo, P_vo_out[j], workspace=ws, stream=stream)


class SwanAttentionLayer:
    def __init__(self, W_q, W_k, W_v, W_o, P_qk, P_vo, n_heads: int, n_kv_heads: int,
                 rope_base: float, batch: int, buffer_tokens: int, capacity: int,
                 k_active: Sequence[int], k_value: Optional[Sequence[int]] = None,
                 sparse_values: str = "same"):
        """W_q [hidden][n_heads*128], W_k and W_v [hidden][n_kv*128], W_o
        [n_heads*128][hidden] (float16 or float32, cuda); P_qk, P_vo [n_kv][128][128]
        float32 (swan_calibrate_rotation of post-RoPE keys and of values)."""
        import torch

        d = HEAD_DIM
        self.n_heads, self.n_kv_heads = n_heads, n_kv_heads
        self.rope_base = float(rope_base)
        self.dtype = W_q.dtype
        self.P_qk = P_qk.contiguous()
        G = n_heads // n_kv_heads
        # absorbed weights, formed once in float64 and rounded to the weights' type
        Wv = W_v.double().clone()
        Wo = W_o.double().clone()
        P = P_vo.double()
        for h in range(n_kv_heads):
            Wv[:, h * d:(h + 1) * d] = Wv[:, h * d:(h + 1) * d] @ P[h]
        for hq in range(n_heads):
            Wo[hq * d:(hq + 1) * d, :] = P[hq // G].T @ Wo[hq * d:(hq + 1) * d, :]
        # the three projections as one GEMM: [W_Q | W_K | W_V_hat], [hidden][(n_q + 2 n_kv) 128]
        self.W_qkv = torch.cat([W_q, W_k, Wv.to(self.dtype)], dim=1).contiguous()
        self.W_o_hat = Wo.to(self.dtype).contiguous()
        self.cache = swan.SwanCache(batch, n_heads, n_kv_heads, buffer_tokens, capacity,
                                    k_active, self.dtype, W_q.device,
                                    sparse_values=sparse_values, k_value=k_value)

    def project(self, x):
        """Post-RoPE q [B][H_q][n][128], k and v_hat [B][H_kv][n][128] of new rows x
        [B][n][hidden] at each sequence's next positions."""
        B, n, _ = x.shape
        d = HEAD_DIM
        pos0 = list(self.cache.seq_len)
        qkv = x @ self.W_qkv
        nq, nkv = self.n_heads * d, self.n_kv_heads * d
        q = qkv[..., :nq].reshape(B, n, self.n_heads, d).transpose(1, 2).contiguous()
        k = qkv[..., nq:nq + nkv].reshape(B, n, self.n_kv_heads, d).transpose(1, 2).contiguous()
        v = qkv[..., nq + nkv:].reshape(B, n, self.n_kv_heads, d).transpose(1, 2).contiguous()
        swan.rope(q, pos0, self.rope_base, out=q)
        swan.rope(k, pos0, self.rope_base, out=k)
        return q, k, v

    def __call__(self, x):
        """x [B][n][hidden]: append the n rows of every sequence to the cache; for a
        decode step (n = 1) return y [B][hidden], the layer's attention output."""
        q, k, v = self.project(x)
        if x.shape[1] != 1:
            self.cache.append(k, v, self.P_qk, None)
            return None
        B = x.shape[0]
        o_hat = self.cache.step(k, v, q[:, :, 0].contiguous(), self.P_qk, None)
        return o_hat.view(B, self.n_heads * HEAD_DIM) @ self.W_o_hat
