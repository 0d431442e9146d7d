"""Seeded synthetic attention workloads (post-RoPE Q/K/V with real model shapes).

This module only draws inputs.  It holds none of MomentKV's arithmetic, and both the
HIP path and the fp64 oracle consume exactly the tensors it returns (the oracle via
host copies).  Keys and values share a planted rank-4 component so that the
value-key covariance of any evicted set is far from zero:

    U_k, U_v in R^{d x 4} orthonormal (QR of a Gaussian), per (layer, KV head)
    c_j ~ N(0, I_4)                     shared by k_j and v_j
    k_j = z_j + 3 U_k c_j,  v_j = z'_j + 3 U_v c_j,   z, z' ~ N(0, I_d)

Keys are rotated by RoPE (half-split pairs, no frequency scaling) at their absolute
positions when the workload models a rotary model; queries are generated directly
in post-RoPE space:
  * "mean" queries: the mean of 4 uniformly drawn context keys of the query head's
    KV head plus N(0, 0.5^2) noise;
  * "needle" queries: 64 needle positions are planted uniformly among the eviction
    candidates of every (sequence, KV head); each query is one uniformly chosen
    needle key plus N(0, 0.5^2) noise, which concentrates attention.
Decode-time appended tokens follow the key/value law at positions N, N+1, ...
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import torch


@dataclass(frozen=True)
class Workload:
    """One attention layer shape plus the run recipe around it."""
    name: str
    dtype: torch.dtype
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ctx_len: int
    budgets: tuple
    window: int
    layers: int
    decode_steps: int
    rope_base: float | None
    queries: str = "mean"          # "mean" or "needle"
    n_sink: int = 1
    chunk: int = 4
    seed_base: int = 0
    n_needles: int = 64

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def seed(self, layer: int, seq: int) -> int:
        return self.seed_base + 100 * layer + seq


WORKLOADS = {
    # Tiny single layer in fp32: GQA 4, d=64, context 2048, budget 128, window 32.
    "tiny_fp32_n2048": Workload("tiny_fp32_n2048", torch.float32, 1, 4, 1, 64, 2048,
                                (128,), 32, 1, 16, None, "mean", seed_base=0),
    # LLaMA-3.1-8B attention shape, one layer, context 8K, budget 512.
    "llama31_8b_layer_n8192": Workload("llama31_8b_layer_n8192", torch.bfloat16, 1, 32, 8,
                                       128, 8192, (512,), 32, 1, 256, 5.0e5, "mean",
                                       seed_base=20000),
    # Qwen3-4B attention shape, 36-layer stack, context 32K, five budgets.
    "qwen3_4b_stack_n32768": Workload("qwen3_4b_stack_n32768", torch.bfloat16, 1, 32, 8, 128,
                                      32768, (128, 256, 512, 1024, 2048), 32, 36, 128,
                                      1.0e6, "mean", seed_base=30000),
    # LLaMA-3.1-8B attention shape, 32 layers, batch 8, context 32K, budget 256, needles.
    "llama31_8b_stack_b8_n32768": Workload("llama31_8b_stack_b8_n32768", torch.bfloat16, 8,
                                           32, 8, 128, 32768, (256,), 32, 32, 128, 5.0e5,
                                           "needle", seed_base=40000),
    # Long-context stress: context 128K, budget 1024, window 64, needles, 32 seeds.
    "ruler_n131072": Workload("ruler_n131072", torch.bfloat16, 1, 32, 8, 128, 131072,
                              (1024,), 64, 32, 128, 5.0e5, "needle", seed_base=50000),
}


def shrink(wl: Workload, **kw) -> Workload:
    """A copy of `wl` with some fields replaced (reduced sizes for quick parity runs)."""
    return replace(wl, **kw)


def rope(x: torch.Tensor, positions: torch.Tensor, base: float) -> torch.Tensor:
    """Rotate x[..., n, d] by RoPE at integer positions[n] (half-split pairs)."""
    d = x.shape[-1]
    half = d // 2
    inv = base ** (-torch.arange(half, dtype=torch.float64, device=x.device) * 2.0 / d)
    ang = positions.to(torch.float64)[:, None] * inv[None, :]
    cos = torch.cos(ang).to(torch.float32)
    sin = torch.sin(ang).to(torch.float32)
    x1, x2 = x[..., :half].float(), x[..., half:].float()
    return torch.cat([x1 * cos - x2 * sin, x1 * sin + x2 * cos], dim=-1)


def _planted_basis(gen, n_heads, d, device):
    """Per-head orthonormal d x 4 bases for keys and values (QR on the host)."""
    g_host = torch.Generator(device="cpu").manual_seed(int(gen.initial_seed()) ^ 0x5F3759DF)
    a = torch.randn(2, n_heads, d, 4, generator=g_host, dtype=torch.float64)
    qm, _ = torch.linalg.qr(a)
    return qm[0].float().to(device), qm[1].float().to(device)


def _kv(gen, U_k, U_v, n, d, device):
    """n keys/values per head under the planted rank-4 law; returns [H, n, d] fp32 x2."""
    H = U_k.shape[0]
    c = torch.randn(H, n, 4, generator=gen, device=device)
    k = torch.randn(H, n, d, generator=gen, device=device) + 3.0 * c @ U_k.transpose(1, 2)
    v = torch.randn(H, n, d, generator=gen, device=device) + 3.0 * c @ U_v.transpose(1, 2)
    return k, v


def make_layer(wl: Workload, layer: int = 0, device="cpu", decode_steps: int | None = None):
    """Draw one layer's inputs for all sequences of the batch.

    Returns a dict of tensors on `device` in the workload dtype:
      q_win [B, Hq, w, d]   window queries (post-RoPE)
      k, v  [B, Hkv, N, d]  prefill keys (post-RoPE) and values
      q_dec [T, B, Hq, d]   decode queries
      k_new, v_new [T, B, Hkv, d]  appended tokens for the T decode steps
      needles [B, Hkv, P] (needle workloads only) planted positions
    """
    T = wl.decode_steps if decode_steps is None else decode_steps
    B, Hq, Hkv, d, N, w, G = (wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                              wl.ctx_len, wl.window, wl.group)
    out = {k: [] for k in ("q_win", "k", "v", "q_dec", "k_new", "v_new", "needles")}
    for b in range(B):
        gen = torch.Generator(device=device).manual_seed(wl.seed(layer, b))
        U_k, U_v = _planted_basis(gen, Hkv, d, device)
        k, v = _kv(gen, U_k, U_v, N, d, device)
        kn, vn = _kv(gen, U_k, U_v, max(T, 1), d, device)
        if wl.rope_base is not None:
            k = rope(k, torch.arange(N, device=device), wl.rope_base)
            kn = rope(kn, torch.arange(N, N + max(T, 1), device=device), wl.rope_base)
        kq = k.to(wl.dtype).float()   # queries are built from the stored (rounded) keys
        if wl.queries == "needle":
            lo, hi = wl.n_sink, N - w
            needles = torch.randint(lo, hi, (Hkv, wl.n_needles), generator=gen, device=device)
            pick_w = torch.randint(0, wl.n_needles, (Hq, w), generator=gen, device=device)
            pick_d = torch.randint(0, wl.n_needles, (Hq, max(T, 1)), generator=gen, device=device)
            hk = torch.arange(Hq, device=device) // G
            src_w = needles[hk[:, None], pick_w]                     # [Hq, w]
            src_d = needles[hk[:, None], pick_d]                     # [Hq, T]
            q_win = kq[hk[:, None], src_w]                           # [Hq, w, d]
            q_dec = kq[hk[:, None], src_d]                           # [Hq, T, d]
            out["needles"].append(needles)
        else:
            hk = torch.arange(Hq, device=device) // G
            src_w = torch.randint(0, N, (Hq, w, 4), generator=gen, device=device)
            src_d = torch.randint(0, N, (Hq, max(T, 1), 4), generator=gen, device=device)
            q_win = kq[hk[:, None, None], src_w].mean(dim=2)
            q_dec = kq[hk[:, None, None], src_d].mean(dim=2)
        q_win = q_win + 0.5 * torch.randn(q_win.shape, generator=gen, device=device)
        q_dec = q_dec + 0.5 * torch.randn(q_dec.shape, generator=gen, device=device)
        out["q_win"].append(q_win)
        out["k"].append(k)
        out["v"].append(v)
        out["q_dec"].append(q_dec.transpose(0, 1))                    # [T, Hq, d]
        out["k_new"].append(kn.transpose(0, 1))                       # [T, Hkv, d]
        out["v_new"].append(vn.transpose(0, 1))
        del k, v, kq
    res = {
        "q_win": torch.stack(out["q_win"]).to(wl.dtype).contiguous(),
        "k": torch.stack(out["k"]).to(wl.dtype).contiguous(),
        "v": torch.stack(out["v"]).to(wl.dtype).contiguous(),
        "q_dec": torch.stack(out["q_dec"], dim=1)[:T].to(wl.dtype).contiguous(),
        "k_new": torch.stack(out["k_new"], dim=1)[:T].to(wl.dtype).contiguous(),
        "v_new": torch.stack(out["v_new"], dim=1)[:T].to(wl.dtype).contiguous(),
    }
    if out["needles"]:
        res["needles"] = torch.stack(out["needles"]).contiguous()
    return res
