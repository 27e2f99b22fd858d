"""Named workloads: shapes, route tables and allocation inputs (configuration data only).

Rule codes: 0 Full, 1 StreamingLLM, 2 SnapKV, 3 H2O.
Budgets are not stored here: each side derives them from `pyramid_weights`,
the aggregate total and b_min with its own allocator.
"""
from __future__ import annotations

FULL, STREAMING, SNAPKV, H2O = 0, 1, 2, 3

LLAMA8B = dict(n_layers=32, n_q_heads=32, n_kv_heads=8, head_dim=128)


def mixed_route(n_layers: int = 32):
    """StreamingLLM on layers 0-1, SnapKV 2-15, H2O 16-27, SnapKV 28-31."""
    assert n_layers == 32
    return [STREAMING] * 2 + [SNAPKV] * 14 + [H2O] * 12 + [SNAPKV] * 4


def pyramid_weights(n_layers: int = 32, top: float = 1024.0, bottom: float = 128.0):
    """PyramidKV-style linearly decreasing layer weights, top at layer 0, bottom at the last layer."""
    return [top - (top - bottom) * l / (n_layers - 1) for l in range(n_layers)]


B_MIN = 48

# name -> description used by tests and the benchmark
WORKLOADS = {
    # one layer, L=1024, SnapKV, budget 128, w=32, pool 7, 16 planted heavy hitters
    "c1_single_layer_1k": dict(workload_id=1, batch=1, seq_len=1024, window=32, pool_kernel=7,
                               n_hh=16, budget=128, rule=SNAPKV, **LLAMA8B),
    # 32-layer mixed route, L=8192, aggregate capacity 32 x 512, PyramidKV ramp
    "c2_mixed_route_8k": dict(workload_id=2, batch=1, seq_len=8192, window=32, pool_kernel=7,
                              n_hh=16, avg_budget=512, **LLAMA8B),
    # budget sweep on the mixed route, batch 8 distinct sequences
    "c3_sweep_8k_b8": dict(workload_id=3, batch=8, seq_len=8192, window=32, pool_kernel=7,
                           n_hh=16, avg_budgets=(128, 256, 512, 1024, 2048), **LLAMA8B),
    # long context, batch 4, w=64, average budget 1024, three routes
    "c4_long_32k_b4": dict(workload_id=4, batch=4, seq_len=32768, window=64, pool_kernel=7,
                           n_hh=64, avg_budget=1024, routes=("snapkv", "h2o", "mixed"), **LLAMA8B),
    # decode H2O: 64 sequences, 8K prompt compressed to a 1024-slot cache, 256 steps
    "c5_decode_h2o_b64": dict(workload_id=5, batch=64, seq_len=8192, window=32, pool_kernel=7,
                              n_hh=16, budget=1024, steps=256, **LLAMA8B),
}


def route_by_name(name: str, n_layers: int = 32):
    if name == "mixed":
        return mixed_route(n_layers)
    if name == "snapkv":
        return [SNAPKV] * n_layers
    if name == "h2o":
        return [H2O] * n_layers
    raise KeyError(name)
