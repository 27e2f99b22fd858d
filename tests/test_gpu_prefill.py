"""GPU parity of the prefill eviction path (through the C ABI) against the CPU oracle."""
import json
import os

import numpy as np
import pytest

from oracle import prefill as OP
from parity import (bits_to_torch, check_gather, check_retained, check_scores, oracle_unpooled,
                    torch_to_bits)
from synth import f32_to_bf16_bits, prefill_layer
from synth.workloads import B_MIN, mixed_route, pyramid_weights

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def run_case(rules, budgets, layers, *, window, pool_kernel=7, n_sink=4, num=1, den=2, check_acc=True,
             label="", status=0):
    """layers: list (per layer) of list (per sequence) of dicts with q/k/v bits.  `status`: the
    workspace status word the call must leave (0, or RKV_STATUS_REPAIRED for a repaired job)."""
    import torch
    import paper_2606_15157_amd as rkv
    plan = rkv.Plan(rules, budgets, window=window, pool_kernel=pool_kernel, n_sink=n_sink, recent_num=num,
                    recent_den=den)
    q_t, k_t, v_t = [], [], []
    for l, seqs in enumerate(layers):
        q_t.append(bits_to_torch(np.stack([x["q"] for x in seqs])))
        k_t.append(bits_to_torch(np.stack([x["k"] for x in seqs])))
        v_t.append(bits_to_torch(np.stack([x["v"] for x in seqs])))
    out = rkv.evict_prefill(plan, q_t, k_t, v_t, score_out=True, acc_out=True)
    torch.cuda.synchronize()
    assert rkv.prefill_check(out["workspace"]) == status, "unexpected status word"
    n_amb = 0
    for l, seqs in enumerate(layers):
        idx = out["idx"][l].cpu().numpy()
        sc = out["scores"][l].cpu().numpy()
        acc = out["acc"][l].cpu().numpy()
        ko = torch_to_bits(out["k_out"][l])
        vo = torch_to_bits(out["v_out"][l])
        for s, x in enumerate(seqs):
            ora = OP.evict_layer(rules[l], budgets[l], x["q"], x["k"], x["v"], window=window,
                                 pool_kernel=pool_kernel, n_sink=n_sink, recent_num=num, recent_den=den)
            L = x["k"].shape[1]
            su = oracle_unpooled(x["q"], x["k"]) if rules[l] in (OP.SNAPKV, OP.H2O) else None
            if rules[l] == OP.TOVA:
                su = ora["scores"]   # TOVA's score covers every position; acc carries it
            for h in range(x["k"].shape[0]):
                what = f"{label} layer {l} seq {s} head {h}"
                if ora["scores"] is not None:
                    n = ora["scores"].shape[1]
                    check_scores(sc[s, h, :n], ora["scores"][h], what)
                n_amb += check_retained(idx[s, h], ora, h, L, what)
                check_gather(ko[s, h], vo[s, h], x["k"][h], x["v"][h], idx[s, h], what)
                if check_acc and su is not None:
                    check_scores(acc[s, h], su[h, idx[s, h]], what + " acc")
                if check_acc and su is None:
                    assert (acc[s, h] == 0).all()
    return out, n_amb


def gen(workload, seq, layer, L, w=32, Hq=32, Hkv=8, n_hh=16):
    return prefill_layer(workload, seq, layer, seq_len=L, n_q_heads=Hq, n_kv_heads=Hkv, window=w, n_hh=n_hh)


@pytest.mark.parametrize("rule", [OP.SNAPKV, OP.H2O, OP.STREAMING, OP.FULL])
def test_single_layer_1k(rule):
    """Single layer, L=1024, 32/8 heads, w=32, pool 7, budget 128."""
    run_case([rule], [128], [[gen(1, 0, 0, 1024)]], window=32, label="c1")


@pytest.mark.parametrize("L", [33, 300, 777, 1000, 2049])
def test_ragged_lengths(L):
    """Context lengths that are not multiples of the 128-key slice (several slices + a tail)."""
    b = min(100, L - 1)
    rules = [OP.SNAPKV, OP.H2O, OP.STREAMING]
    run_case(rules, [b, b, b], [[gen(7, 0, l, L)] for l in range(3)], window=32, label=f"L{L}")


@pytest.mark.parametrize("budget", [0, 1, 2, 5, 31, 32, 33, 511, 512, 513, 4096])
def test_degenerate_budgets(budget):
    """Budgets around the window size, the context length and zero."""
    L = 512
    rules = [OP.SNAPKV, OP.H2O, OP.STREAMING, OP.FULL]
    run_case(rules, [budget] * 4, [[gen(8, 0, l, L)] for l in range(4)], window=32, label=f"b{budget}")


@pytest.mark.parametrize("L,w", [(32, 32), (100, 1), (129, 64)], ids=["window_is_prompt", "w1", "w64_L129"])
def test_window_edge_shapes(L, w, monkeypatch):
    """A window covering the whole prompt (SnapKV has no candidates: the window is kept), a
    one-row window (padded row tiles) and a 64-row window over one slice and a one-key tail
    (eight row tiles), through the default path and the window kernels."""
    b = min(L, 20)
    rules = [OP.SNAPKV, OP.H2O, OP.STREAMING]
    layers = [[gen(9, 0, l, L, w=w)] for l in range(3)]
    run_case(rules, [b] * 3, layers, window=w, label=f"edge_L{L}_w{w}")
    monkeypatch.setenv("RKV_FORCE_WINDOW", "1")
    run_case(rules, [b] * 3, layers, window=w, label=f"edge_L{L}_w{w}_window")


def test_window_totals_sum_to_w():
    """H2O keeping every position reports the unpooled group-mean score on all of [0, L):
    every window row's softmax sums to 1, so each KV head's scores sum to w."""
    import paper_2606_15157_amd as rkv
    import torch
    x = gen(9, 0, 0, 1536)
    plan = rkv.Plan([OP.H2O], [4096], window=32)
    out = rkv.evict_prefill(plan, [bits_to_torch(x["q"][None])], [bits_to_torch(x["k"][None])],
                            [bits_to_torch(x["v"][None])], score_out=True)
    torch.cuda.synchronize()
    tot = out["scores"][0].double().sum(-1).cpu().numpy()
    np.testing.assert_allclose(tot, 32.0, rtol=1e-4)


def test_uniform_keys_break_ties_by_position():
    """Equal keys give exactly equal prefix scores; the lowest positions must win."""
    L, w, b = 1024, 32, 200
    rng = np.random.default_rng(5)
    q = f32_to_bf16_bits(rng.standard_normal((32, w, 128)).astype(np.float32))
    k = f32_to_bf16_bits(np.tile(rng.standard_normal(128).astype(np.float32), (8, L, 1)))
    v = f32_to_bf16_bits(rng.standard_normal((8, L, 128)).astype(np.float32))
    x = {"q": q, "k": k, "v": v}
    out, _ = run_case([OP.SNAPKV, OP.H2O], [b, b], [[x], [x]], window=w, label="uniform")
    idx = out["idx"][0].cpu().numpy()
    for h in range(8):
        assert idx[0, h].tolist() == list(range(b - w)) + list(range(L - w, L))
    idx = out["idx"][1].cpu().numpy()
    for h in range(8):
        assert idx[0, h].tolist() == list(range(b - b // 2)) + list(range(L - b // 2, L))


def test_batch_of_distinct_sequences():
    L = 2048
    rules = [OP.SNAPKV, OP.H2O]
    layers = [[gen(3, s, l, L) for s in range(3)] for l in range(2)]
    run_case(rules, [300, 300], layers, window=32, label="batch3")


def test_window_64_two_tile_groups():
    """w = 64: each query head spans two 32-row tiles (the 8-tile scoring kernel)."""
    L = 4096
    rules = [OP.SNAPKV, OP.H2O]
    layers = [[gen(4, 0, l, L, w=64, n_hh=64)] for l in range(2)]
    run_case(rules, [1024, 1024], layers, window=64, label="w64")


def test_odd_window_and_group_shapes():
    """w = 20 (padded rows), G = 2 (16 query heads on 8 KV heads), pool kernel 5."""
    L = 1500
    rules = [OP.SNAPKV, OP.H2O]
    layers = [[gen(6, 0, l, L, w=20, Hq=16)] for l in range(2)]
    run_case(rules, [150, 150], layers, window=20, pool_kernel=5, label="w20g2")


@pytest.mark.parametrize("w,Hq,Hkv", [(64, 16, 8), (100, 8, 8)], ids=["w64_g2", "w100_g1"])
def test_wide_windows_few_heads(w, Hq, Hkv):
    """Windows of two and four 32-row tiles per head with two and one query heads per KV head
    (four row tiles in all: the pipelined kernel's two- and four-tile forms, the second with
    padding rows), L = 5000 and four layers: more than four items per workgroup, so the
    long-run form of the kernel."""
    L = 5000
    rules = [OP.SNAPKV, OP.H2O, OP.SNAPKV, OP.H2O]
    layers = [[gen(13, 0, l, L, w=w, Hq=Hq, Hkv=Hkv)] for l in range(4)]
    run_case(rules, [400] * 4, layers, window=w, label=f"w{w}_Hq{Hq}")


def test_prompt_between_8k_and_16k():
    """L = 12345 (ragged, 97 slices): the window kernels with the rows kernel's keys split over
    workgroups, and the selection with 16 scores per thread; SnapKV, H2O and TOVA layers."""
    L = 12345
    rules = [OP.SNAPKV, OP.H2O, OP.TOVA]
    layers = [[gen(12, 0, l, L)] for l in range(3)]
    run_case(rules, [1024, 1024, 1024], layers, window=32, label="L12345")


@pytest.mark.parametrize("L,Hq,Hkv", [(33000, 32, 8), (28000, 32, 4)], ids=["L33000_g4", "L28000_g8"])
def test_long_prompts_general_selection(L, Hq, Hkv):
    """The selection kernel for what the register-resident one cannot hold: more than 32K keys
    (L = 33000, ragged, its scores past the LDS cache), and eight query heads per KV head at 28K
    keys, whose slice-edge sums do not fit beside the registers (scores in the LDS cache); both
    score through the window kernels (more than 64 slices)."""
    rules = [OP.SNAPKV, OP.H2O]
    layers = [[gen(11, 0, l, L, Hq=Hq, Hkv=Hkv)] for l in range(2)]
    run_case(rules, [1024, 1024], layers, window=32, label=f"L{L}_Hq{Hq}_Hkv{Hkv}")


@pytest.mark.parametrize("Hq,Hkv", [(8, 8), (32, 4)], ids=["g1", "g8"])
def test_group_sizes_one_and_eight(Hq, Hkv):
    """G = 1 (one row tile of 32, padded to four in the pipelined kernel) and G = 8 (eight row
    tiles, the other scoring kernel), SnapKV and H2O, ragged L."""
    L = 1100
    rules = [OP.SNAPKV, OP.H2O]
    layers = [[gen(7, s, l, L, Hq=Hq, Hkv=Hkv) for s in range(2)] for l in range(2)]
    run_case(rules, [200, 200], layers, window=32, label=f"g{Hq // Hkv}")


def test_full_route_8k_matches_oracle():
    """The 32-layer mixed route at L=8192 (StreamingLLM 0-1, SnapKV 2-15, H2O 16-27,
    SnapKV 28-31), PyramidKV-ramp budgets summing to 32 x 512, full size, every layer."""
    g = json.load(open(os.path.join(GOLDEN, "budgets.json")))
    budgets = g["pyramid_512"]
    rules = mixed_route()
    layers = [[gen(2, 0, l, 8192)] for l in range(32)]
    out, n_amb = run_case(rules, budgets, layers, window=32, label="route8k")
    print(f"positions in tie bands: {n_amb}")


def test_repeat_runs_are_bitwise_identical():
    """Race detector: two runs on the same inputs give identical scores, indices and rows."""
    import paper_2606_15157_amd as rkv
    import torch
    L = 4096
    rules = [OP.SNAPKV, OP.H2O, OP.STREAMING]
    xs = [gen(11, 0, l, L) for l in range(3)]
    plan = rkv.Plan(rules, [400, 400, 400], window=32)
    q = [bits_to_torch(x["q"][None]) for x in xs]
    k = [bits_to_torch(x["k"][None]) for x in xs]
    v = [bits_to_torch(x["v"][None]) for x in xs]
    a = rkv.evict_prefill(plan, q, k, v, score_out=True, acc_out=True)
    b = rkv.evict_prefill(plan, q, k, v, score_out=True, acc_out=True)
    torch.cuda.synchronize()
    for key in ("idx", "scores", "acc", "k_out", "v_out"):
        for l in range(3):
            assert torch.equal(a[key][l], b[key][l]), (key, l)


def test_window_kernels_match_oracle_on_short_prompts(monkeypatch):
    """The window scoring kernels (row normalisers, then column sums: prompts of more than 64
    slices, eight row tiles), forced through the test hook on layouts the pipelined kernel would
    otherwise take: the 1K case and a ragged length."""
    monkeypatch.setenv("RKV_FORCE_WINDOW", "1")
    run_case([OP.SNAPKV, OP.H2O], [128, 128], [[gen(1, 0, 0, 1024)], [gen(1, 0, 1, 1024)]], window=32,
             label="win_1k")
    run_case([OP.SNAPKV, OP.H2O], [100, 100], [[gen(7, 0, 0, 777)], [gen(7, 0, 1, 777)]], window=32,
             label="win_777")


@pytest.mark.parametrize("L", [4096, 3000])
def test_window_kernels_split_keys(monkeypatch, L):
    """Few jobs (two layers x 8 KV heads): the rows kernel splits each job's keys over several
    workgroups (4 parts at L = 4096; 3 at L = 3000, the last with the ragged tail) and the columns
    kernel adds their row sums."""
    monkeypatch.setenv("RKV_FORCE_WINDOW", "1")
    run_case([OP.SNAPKV, OP.H2O], [300, 300], [[gen(15, 0, 0, L)], [gen(15, 0, 1, L)]], window=32,
             label=f"win_split_{L}")


def overflow_input(L=1024, w=32):
    """One window row (query head 5, row 7) set to 4 in every dimension and one prefix key
    (position 300) to 4 in every dimension: that row's logit there is 4 * 4 * 128 / sqrt(128) =
    181, about 170 natural-log units above the row's reference (its logits with its own key and
    with key 0), beyond the fp32 exponent range of the scoring kernels' row sums."""
    x = gen(12, 0, 0, L, w=w)
    q = x["q"].copy()
    k = x["k"].copy()
    four = f32_to_bf16_bits(np.full(128, 4.0, np.float32))
    q[5, 7, :] = four
    k[:, 300, :] = four
    return {"q": q, "k": k, "v": x["v"]}


def test_reference_overflow_is_repaired(monkeypatch):
    """The overflowing job is flagged by the scoring kernel and rescored exactly by its selection
    workgroup: scores, retained sets, rows and acc match the oracle, and the status word says
    RKV_STATUS_REPAIRED (outputs valid).  Through the pipelined kernel (the default here) and the
    window kernels (test hook)."""
    y = overflow_input()
    run_case([OP.SNAPKV, OP.H2O], [128, 128], [[y], [y]], window=32, label="ref_overflow", status=4)
    monkeypatch.setenv("RKV_FORCE_WINDOW", "1")
    run_case([OP.SNAPKV, OP.H2O], [128, 128], [[y], [y]], window=32, label="ref_overflow_window", status=4)


def test_reference_overflow_is_repaired_at_eight_row_tiles():
    """w = 64 with four query heads per KV head: 256 window rows per job (eight row tiles), which
    the window kernels score and the exact rescoring must cover in full."""
    y = overflow_input(L=1536, w=64)
    run_case([OP.SNAPKV, OP.H2O], [200, 200], [[y], [y]], window=64, label="ref_overflow_w64", status=4)


def test_status_word_spans_every_launch_group():
    """33 layers take two launch groups.  The overflow planted in layer 0 (first group) must still
    be visible in the status word after the second group ran, and both groups' layers (0, the
    repaired one, and 32) match the oracle."""
    L = 1024
    y = overflow_input(L)
    layers = [[y]] + [[gen(14, 0, l, L)] for l in range(1, 33)]
    run_case([OP.SNAPKV] * 33, [128] * 33, layers, window=32, label="two_groups", status=4)


def test_bench_call_matches_debug_call_at_full_size():
    """bench.py's exact call at the 8K route (no score or acc output: the pipelined kernel stores no
    unpooled scores, the selection writes no scores) gives indices and rows bitwise equal to the
    call with debug outputs, whose results the full-route test checks against the oracle; and
    here every layer's retained set is checked against the oracle too."""
    import paper_2606_15157_amd as rkv
    import torch
    g = json.load(open(os.path.join(GOLDEN, "budgets.json")))
    budgets = g["pyramid_512"]
    rules = mixed_route()
    xs = [gen(2, 0, l, 8192) for l in range(32)]
    plan = rkv.Plan(rules, budgets, window=32, pool_kernel=7)
    q = [bits_to_torch(x["q"][None]) for x in xs]
    k = [bits_to_torch(x["k"][None]) for x in xs]
    v = [bits_to_torch(x["v"][None]) for x in xs]
    out = rkv.alloc_outputs(plan, 1, 8, 8192, 128, "cuda")
    ws = rkv.alloc_workspace(plan, 1, 8192, 32, 8, "cuda")
    call = rkv.PreparedPrefill(plan, q, k, v, out, ws)
    for _ in range(3):   # as bench.py: repeated passes over one workspace
        call(torch.cuda.current_stream())
    torch.cuda.synchronize()
    assert rkv.prefill_check(ws) == 0
    dbg = rkv.evict_prefill(plan, q, k, v, score_out=True, acc_out=True)
    torch.cuda.synchronize()
    for l in range(32):
        for key in ("idx", "k_out", "v_out"):
            assert torch.equal(out[key][l], dbg[key][l]), (key, l)
        ora = OP.evict_layer(rules[l], budgets[l], xs[l]["q"], xs[l]["k"], xs[l]["v"], window=32, pool_kernel=7)
        idx = out["idx"][l].cpu().numpy()
        for h in range(8):
            check_retained(idx[0, h], ora, h, 8192, f"bench call layer {l} head {h}")


@pytest.mark.parametrize("case", range(40))
def test_random_shapes_against_oracle(case):
    """Seeded random shapes: batch 1-2, 1-8 KV heads, 1-8 query heads per KV head (3 included),
    windows of 1 up to the row-tile limit, prompts of a few keys up to 6000 (ragged slices), odd
    pools up to 15, sink counts and recent fractions of H2O varied, and 1-4 layers mixing SnapKV,
    H2O, StreamingLLM, Full and TOVA with budgets from 0 past the prompt length."""
    rng = np.random.default_rng(9000 + case)
    batch = int(rng.integers(1, 3))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 3, 4, 8]))
    w = int(rng.integers(1, 32 * (8 // G) + 1))
    L = int(np.exp(rng.uniform(np.log(max(w, 2)), np.log(6000))))
    pool = int(rng.choice([1, 3, 5, 7, 9, 15]))
    n_sink = int(rng.integers(0, 9))
    num, den = [(1, 2), (1, 3), (2, 3), (0, 1)][int(rng.integers(0, 4))]
    choices = [OP.SNAPKV, OP.H2O, OP.STREAMING, OP.FULL] + ([OP.TOVA] if G != 3 else [])
    n_layers = int(rng.integers(1, 5))
    rules = [int(rng.choice(choices)) for _ in range(n_layers)]
    budgets = []
    for _ in range(n_layers):
        kind = int(rng.integers(0, 8))
        budgets.append([0, 1, L, L + 5][kind] if kind < 4 else int(rng.integers(1, L + 1)))
    layers = [[gen(60 + case, s, l, L, w=w, Hq=G * Hkv, Hkv=Hkv) for s in range(batch)] for l in range(n_layers)]
    label = (f"case {case}: B{batch} Hkv{Hkv} G{G} w{w} L{L} pool{pool} sink{n_sink} recent {num}/{den} "
             f"rules {rules} budgets {budgets}")
    print(label, flush=True)
    run_case(rules, budgets, layers, window=w, pool_kernel=pool, n_sink=n_sink, num=num, den=den, label=label)


def test_graph_replay_matches_eager():
    """A prefill call captured in a HIP graph (kernels only: no allocation, no memset node) and
    replayed three times, with eager work between the replays (the outputs zeroed), gives the
    eager call's outputs bit for bit each time."""
    import torch
    import paper_2606_15157_amd as rkv
    L, w = 1000, 32
    rules = [OP.STREAMING, OP.SNAPKV, OP.H2O]
    budgets = [64, 150, 150]
    xs = [gen(70, 0, l, L) for l in range(3)]
    q = [bits_to_torch(x["q"][None]) for x in xs]
    k = [bits_to_torch(x["k"][None]) for x in xs]
    v = [bits_to_torch(x["v"][None]) for x in xs]
    plan = rkv.Plan(rules, budgets, window=w)
    out = rkv.alloc_outputs(plan, 1, 8, L, 128, "cuda")
    ws = rkv.alloc_workspace(plan, 1, L, 32, 8, "cuda")
    call = rkv.PreparedPrefill(plan, q, k, v, out, ws)
    call(torch.cuda.current_stream())
    torch.cuda.synchronize()
    names = ("idx", "k_out", "v_out")
    ref = {n: [t.clone() for t in out[n]] for n in names}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        call(side)
    torch.cuda.synchronize()
    for rep in range(3):
        for n in names:
            for t in out[n]:
                t.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert rkv.prefill_check(ws) == 0, f"replay {rep}: status word"
        for n in names:
            for l in range(3):
                assert torch.equal(out[n][l], ref[n][l]), f"replay {rep}: {n} of layer {l}"
    # the retained sets are the oracle's
    for l in range(3):
        ora = OP.evict_layer(rules[l], budgets[l], xs[l]["q"], xs[l]["k"], xs[l]["v"], window=w)
        for h in range(8):
            check_retained(out["idx"][l][0, h].cpu().numpy(), ora, h, L, f"graph layer {l} head {h}")
