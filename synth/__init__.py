"""Seeded synthetic inputs shaped like LLaMA-3.1-8B prompts (32 query heads,
8 KV heads, head_dim 128, bf16), with planted attention structure.

This module is input data only.  It holds none of the eviction arithmetic and
is shared by the CPU oracle, the tests and the benchmark, so that both sides of
every parity check read the same bf16 arrays.

Recipe, per (workload id, sequence, layer):

1. A NumPy PCG64 stream seeded by SeedSequence([20260615, workload, seq, layer]).
2. Draw the window queries Q [Hq, w, d], keys K [Hkv, L, d] and values
   V [Hkv, L, d] as float32 N(0, 1), in that order.
3. For each KV head h, take the mean query direction of its query group,
   qbar = mean over the group's heads and the last min(w, 64) query rows (the
   whole window of the window-scored workloads, w <= 64; the last 64 positions
   of a full-span workload, whose queries cover all L positions, where a mean
   over every position would be near zero and u enormous), and the unit-logit step
   u = sqrt(d) * qbar / |qbar|^2.  Adding a*u to a key raises the mean query's
   scaled logit (q.k / sqrt(d)) by exactly a, i.e. by a standard deviations of
   an N(0,1) logit.
   * sink:          K[h, 0]          += 3u
   * heavy hitters: K[h, p]          += 2u  for n_hh distinct p in [1, L - 64)
   * recency:       K[h, L-64 : L]   += 1u
4. Round to bf16 (round to nearest even).

Decode-step inputs (one new query per query head and one new key/value per KV
head per step) are unshifted N(0, 1) from their own stream.

bf16 tensors are carried on the host as uint16 bit patterns.
"""
from __future__ import annotations

import numpy as np

SEED_BASE = 20260615

# Planted-structure constants (in units of the mean query's logit std).
SINK_SHIFT = 3.0
HEAVY_SHIFT = 2.0
RECENT_SHIFT = 1.0
RECENT_SPAN = 64
PLANT_ROWS = 64   # query rows (the last ones) whose mean sets the planted direction


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_BASE, *key])))


def planted_positions(L: int, n_hh: int, recent: int = RECENT_SPAN):
    """Effective recency span and heavy-hitter range for a context of L keys."""
    rec = min(recent, max(L - 1, 0))
    hi = L - rec  # heavy hitters are drawn from [1, hi)
    n = min(n_hh, max(hi - 1, 0))
    return rec, hi, n


def prefill_layer(workload: int, seq: int, layer: int, *, seq_len: int, n_q_heads: int = 32,
                  n_kv_heads: int = 8, head_dim: int = 128, window: int = 32, n_hh: int = 16,
                  plant: bool = True):
    """One (sequence, layer) of prefill inputs.

    Returns dict with uint16 bf16 bits: q [Hq, w, d], k [Hkv, L, d], v [Hkv, L, d],
    and the planted heavy-hitter positions hh [Hkv, n] (int64).
    """
    L, Hq, Hkv, d, w = seq_len, n_q_heads, n_kv_heads, head_dim, window
    if Hq % Hkv:
        raise ValueError("n_q_heads must be a multiple of n_kv_heads")
    G = Hq // Hkv
    g = _rng(workload, seq, layer)
    q = g.standard_normal((Hq, w, d), dtype=np.float32)
    k = g.standard_normal((Hkv, L, d), dtype=np.float32)
    v = g.standard_normal((Hkv, L, d), dtype=np.float32)
    rec, hi, n = planted_positions(L, n_hh)
    hh = np.zeros((Hkv, n), dtype=np.int64)
    if plant and L > 0:
        for h in range(Hkv):
            qbar = q[h * G:(h + 1) * G, max(0, w - PLANT_ROWS):].astype(np.float64).mean(axis=(0, 1))
            u = (np.sqrt(d) * qbar / np.dot(qbar, qbar)).astype(np.float32)
            k[h, 0] += np.float32(SINK_SHIFT) * u
            if n > 0:
                hh[h] = np.sort(g.choice(np.arange(1, hi), size=n, replace=False))
                k[h, hh[h]] += np.float32(HEAVY_SHIFT) * u
            if rec > 0:
                k[h, L - rec:] += np.float32(RECENT_SHIFT) * u
    return {"q": f32_to_bf16_bits(q), "k": f32_to_bf16_bits(k), "v": f32_to_bf16_bits(v), "hh": hh}


def prefill_batch(workload: int, layer: int, *, batch: int, **kw):
    """Stack `batch` independent sequences (distinct seeds) of one layer: leading batch dim."""
    parts = [prefill_layer(workload, s, layer, **kw) for s in range(batch)]
    return {key: np.stack([p[key] for p in parts]) for key in ("q", "k", "v", "hh")}


def decode_steps(workload: int, seq: int, layer: int, *, steps: int, n_q_heads: int = 32,
                 n_kv_heads: int = 8, head_dim: int = 128):
    """Unshifted N(0,1) decode inputs for `steps` steps: q [T, Hq, d], k/v [T, Hkv, d] (bf16 bits)."""
    g = _rng(workload, seq, layer, 1)
    q = g.standard_normal((steps, n_q_heads, head_dim), dtype=np.float32)
    k = g.standard_normal((steps, n_kv_heads, head_dim), dtype=np.float32)
    v = g.standard_normal((steps, n_kv_heads, head_dim), dtype=np.float32)
    return {"q": f32_to_bf16_bits(q), "k": f32_to_bf16_bits(k), "v": f32_to_bf16_bits(v)}


# --------------------------------------------------------------------------------------
# Device-side generator for the large workloads (batch 8 at 8K, batch 4 at 32K, decode
# with 64 sequences).  Same recipe, torch's seeded device RNG instead of PCG64, so the
# values differ from the NumPy stream; both sides of a parity check read the arrays this
# produces (copied back to the host for the oracle).
# --------------------------------------------------------------------------------------

def prefill_layer_torch(workload: int, layer: int, *, batch: int, seq_len: int, n_q_heads: int = 32,
                        n_kv_heads: int = 8, head_dim: int = 128, window: int = 32, n_hh: int = 16,
                        device="cuda"):
    """Returns bf16 device tensors q [B,Hq,w,d], k/v [B,Hkv,L,d] and hh [B,Hkv,n] (int64, device)."""
    import torch
    L, Hq, Hkv, d, w = seq_len, n_q_heads, n_kv_heads, head_dim, window
    G = Hq // Hkv
    gen = torch.Generator(device=device)
    gen.manual_seed((SEED_BASE * 1_000_003 + workload * 10_007 + layer) % (2 ** 63))
    q = torch.randn((batch, Hq, w, d), generator=gen, device=device, dtype=torch.float32)
    k = torch.randn((batch, Hkv, L, d), generator=gen, device=device, dtype=torch.float32)
    v = torch.randn((batch, Hkv, L, d), generator=gen, device=device, dtype=torch.float32)
    rec, hi, n = planted_positions(L, n_hh)
    qbar = q.view(batch, Hkv, G, w, d)[:, :, :, max(0, w - PLANT_ROWS):].double().mean(dim=(2, 3))   # [B,Hkv,d]
    u = (d ** 0.5 * qbar / (qbar * qbar).sum(-1, keepdim=True)).float()     # [B,Hkv,d]
    k[:, :, 0] += SINK_SHIFT * u
    hh = torch.zeros((batch, Hkv, n), dtype=torch.int64, device=device)
    if n > 0:
        keys = torch.rand((batch, Hkv, hi - 1), generator=gen, device=device)
        hh = torch.sort(torch.topk(keys, n, dim=-1).indices + 1, dim=-1).values
        k.scatter_add_(2, hh.unsqueeze(-1).expand(-1, -1, -1, d),
                       (HEAVY_SHIFT * u).unsqueeze(2).expand(-1, -1, n, -1).contiguous())
    if rec > 0:
        k[:, :, L - rec:] += RECENT_SHIFT * u.unsqueeze(2)
    return {"q": q.to(torch.bfloat16), "k": k.to(torch.bfloat16), "v": v.to(torch.bfloat16), "hh": hh}


def decode_steps_torch(workload: int, layer: int, *, batch: int, steps: int, n_q_heads: int = 32,
                       n_kv_heads: int = 8, head_dim: int = 128, device="cuda"):
    """Device bf16 decode inputs q [T,B,Hq,d], k/v [T,B,Hkv,d]."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed((SEED_BASE * 1_000_003 + workload * 10_007 + layer + 7_777_777) % (2 ** 63))
    q = torch.randn((steps, batch, n_q_heads, head_dim), generator=gen, device=device)
    k = torch.randn((steps, batch, n_kv_heads, head_dim), generator=gen, device=device)
    v = torch.randn((steps, batch, n_kv_heads, head_dim), generator=gen, device=device)
    return {"q": q.to(torch.bfloat16), "k": k.to(torch.bfloat16), "v": v.to(torch.bfloat16)}
