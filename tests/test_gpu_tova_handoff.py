"""GPU parity of TOVA prompt compression, tied both-phase plans and the prefill -> decode hand-off
(Sections 3.1 and 3.4; Appendix E's H2O / TOVA composition) against the CPU oracle."""
import ctypes as C

import numpy as np
import pytest

from oracle import decode as OD
from oracle import prefill as OP
from parity import bits_to_torch, check_gather, check_retained, check_scores, torch_to_bits
from synth import decode_steps, f32_to_bf16_bits, prefill_layer
from test_gpu_decode import _decode_and_check, snapshot_opt
from test_gpu_prefill import run_case

pytestmark = pytest.mark.gpu


def gen(workload, seq, layer, L, w=32, Hq=32, Hkv=8):
    return prefill_layer(workload, seq, layer, seq_len=L, n_q_heads=Hq, n_kv_heads=Hkv, window=w)


# ----------------------------------------------------------------------------- TOVA prefill

@pytest.mark.parametrize("L", [1024, 777, 33, 8192])
def test_tova_prefill_single_layer(L):
    """The last query's group-mean attention over every key: scores, retained sets, rows, acc."""
    b = min(128, L - 1)
    run_case([OP.TOVA], [b], [[gen(40, 0, 0, L)]], window=32, label=f"tova L{L}")


@pytest.mark.parametrize("budget", [0, 1, 2, 500, 1023, 1024, 1500])
def test_tova_prefill_budgets(budget):
    L = 1024
    run_case([OP.TOVA, OP.SNAPKV], [budget, max(budget, 40)], [[gen(41, 0, 0, L)], [gen(41, 0, 1, L)]], window=32,
             label=f"tova b{budget}")


@pytest.mark.parametrize("Hq,Hkv", [(8, 8), (16, 8), (32, 4)])
def test_tova_prefill_group_sizes(Hq, Hkv):
    L, B = 1100, 2
    layers = [[gen(42, s, 0, L, Hq=Hq, Hkv=Hkv) for s in range(B)]]
    run_case([OP.TOVA], [300], layers, window=32, label=f"tova G{Hq // Hkv}")


def test_tova_uniform_keys_keep_the_lowest_positions():
    """Equal keys: every position scores exactly 1/L; ties keep the lowest positions."""
    import paper_2606_15157_amd as rkv
    import torch
    L, b = 2048, 300
    rng = np.random.default_rng(43)
    q = f32_to_bf16_bits(rng.standard_normal((32, 32, 128)).astype(np.float32))
    k = f32_to_bf16_bits(np.tile(rng.standard_normal(128).astype(np.float32), (8, L, 1)))
    v = f32_to_bf16_bits(rng.standard_normal((8, L, 128)).astype(np.float32))
    plan = rkv.Plan([OP.TOVA], [b], window=32)
    out = rkv.evict_prefill(plan, [bits_to_torch(q[None])], [bits_to_torch(k[None])], [bits_to_torch(v[None])],
                            score_out=True)
    torch.cuda.synchronize()
    assert rkv.prefill_check(out["workspace"]) == 0
    np.testing.assert_allclose(out["scores"][0].cpu().numpy(), 1.0 / L, rtol=1e-5)
    idx = out["idx"][0].cpu().numpy()
    for h in range(8):
        assert idx[0, h].tolist() == list(range(b))


def test_mixed_route_with_tova_batch():
    """StreamingLLM, SnapKV, H2O, full-span H2O and TOVA layers in one call, batch 2, L = 1500."""
    L, B = 1500, 2
    rules = [OP.STREAMING, OP.SNAPKV, OP.TOVA, OP.H2O, OP.TOVA]
    budgets = [64, 200, 150, 200, 400]
    layers = [[gen(44, s, l, L) for s in range(B)] for l in range(len(rules))]
    run_case(rules, budgets, layers, window=32, label="tova mixed")


# ----------------------------------------------------------------------------- hand-off and tied plans

def test_appendix_e_composition_tied_both_phases():
    """Appendix E's composition as a tied both-phase plan: H2O on layers 0-15 and TOVA on 16-31,
    512 positions per layer in both phases, an 8192-token prompt.  Prefill (H2O window scoring
    and TOVA prompt compression) is checked against the oracle on every layer, the hand-off must
    copy the compacted cache and the acc seed exactly, and three decode steps are checked per
    (layer, head) against the oracle's step of each layer's rule."""
    import paper_2606_15157_amd as rkv
    import torch
    L, C, n = 8192, 512, 32
    rules = [OP.H2O] * 16 + [OP.TOVA] * 16
    plan = rkv.Plan.from_scoped_route(rules, [rkv.SCOPE_BOTH] * n, [C] * n, window=32)
    xs = [gen(45, 0, l, L) for l in range(n)]
    q = [bits_to_torch(x["q"][None]) for x in xs]
    k = [bits_to_torch(x["k"][None]) for x in xs]
    v = [bits_to_torch(x["v"][None]) for x in xs]
    out = rkv.evict_prefill(plan, q, k, v, acc_out=True, check_status=True)
    state = rkv.decode_init_from_prefill(plan, out)
    torch.cuda.synchronize()
    for l in range(n):
        ora = OP.evict_layer(rules[l], C, xs[l]["q"], xs[l]["k"], xs[l]["v"], window=32)
        idx = out["idx"][l].cpu().numpy()
        acc = out["acc"][l].cpu().numpy()
        ko, vo = torch_to_bits(out["k_out"][l]), torch_to_bits(out["v_out"][l])
        for h in range(8):
            what = f"layer {l} ({OP.RULE_NAMES[rules[l]]}) head {h}"
            check_retained(idx[0, h], ora, h, L, what)
            check_gather(ko[0, h], vo[0, h], xs[l]["k"][h], xs[l]["v"][h], idx[0, h], what)
            su = OP.group_mean(OP.window_scores(OP.bf16_to_f64(xs[l]["q"][:, -1:] if rules[l] == OP.TOVA
                                                               else xs[l]["q"]), OP.bf16_to_f64(xs[l]["k"])), 4)
            check_scores(acc[0, h], su[h, idx[0, h]], what + " acc")
        # the hand-off: the decode cache is the compacted prompt cache, bit for bit
        assert torch.equal(state["k_cache"][l], out["k_out"][l])
        assert torch.equal(state["v_cache"][l], out["v_out"][l])
        assert torch.equal(state["pos"][l], out["idx"][l])
        if rules[l] == OP.H2O:
            assert torch.equal(state["acc"][l], out["acc"][l])
        else:
            assert state["acc"][l] is None
    n_close = _decode_and_check(plan, state, rules, C, L, 1, 3, n, seed_workload=46)
    print(f"victims chosen differently inside the 1e-3 tie band: {n_close}")


def test_handoff_zero_seed_and_in_place_state():
    """A StreamingLLM prefill layer handing over to decode H2O gets a zero accumulator seed; a
    state that aliases the prefill outputs is left as it is (in-place decoding)."""
    import paper_2606_15157_amd as rkv
    import torch
    L, C = 700, 96
    plan = rkv.Plan([OP.STREAMING, OP.SNAPKV], [C, C], [rkv.H2O, rkv.H2O], [C, C], window=32)
    xs = [gen(47, 0, l, L) for l in range(2)]
    out = rkv.evict_prefill(plan, [bits_to_torch(x["q"][None]) for x in xs], [bits_to_torch(x["k"][None]) for x in xs],
                            [bits_to_torch(x["v"][None]) for x in xs], acc_out=True, check_status=True)
    state = rkv.decode_init_from_prefill(plan, out)
    torch.cuda.synchronize()
    assert (state["acc"][0] == 0).all()
    assert torch.equal(state["acc"][1], out["acc"][1])
    alias = {"k_cache": out["k_out"], "v_cache": out["v_out"], "pos": out["idx"], "acc": out["acc"]}
    before = [t.clone() for t in out["k_out"]]
    rkv.decode_init_from_prefill(plan, out, alias)
    torch.cuda.synchronize()
    for a, b in zip(before, out["k_out"]):
        assert torch.equal(a, b)


def test_prefill_then_decode_through_the_c_abi_only():
    """Every call through ctypes on the C ABI (no binding helper): rkv_plan_from_route (tied H2O
    and TOVA layers), rkv_prefill_workspace_size, rkv_prefill_evict, rkv_prefill_check,
    rkv_decode_init_from_prefill and one rkv_decode_step; results checked against the oracle.
    torch only allocates device memory and provides the stream."""
    import torch
    from paper_2606_15157_amd import _abi
    lib = _abi.lib()
    L, cap, Hq, Hkv, d, n = 1024, 200, 32, 8, 128, 2
    rules = [OP.H2O, OP.TOVA]
    xs = [gen(48, 0, l, L) for l in range(n)]
    dev = "cuda"
    q = [bits_to_torch(x["q"][None]) for x in xs]
    k = [bits_to_torch(x["k"][None]) for x in xs]
    v = [bits_to_torch(x["v"][None]) for x in xs]
    mk = lambda shape, dt: [torch.empty(shape, dtype=dt, device=dev) for _ in range(n)]
    k_out, v_out = mk((1, Hkv, cap, d), torch.bfloat16), mk((1, Hkv, cap, d), torch.bfloat16)
    idx, acc = mk((1, Hkv, cap), torch.int32), mk((1, Hkv, cap), torch.float32)
    k_c, v_c = mk((1, Hkv, cap, d), torch.bfloat16), mk((1, Hkv, cap, d), torch.bfloat16)
    pos_c, acc_c = mk((1, Hkv, cap), torch.int32), mk((1, Hkv, cap), torch.float32)

    def arr(ts):
        a = (C.c_void_p * len(ts))()
        for i, t in enumerate(ts):
            a[i] = t.data_ptr() if t is not None else None
        return C.cast(a, C.POINTER(C.c_void_p))

    route = (_abi.RouteLayer * n)(*[_abi.RouteLayer(r, 2, cap) for r in rules])
    params = _abi.Params(32, 7, 4, 1, 2)
    plan = C.c_void_p()
    assert lib.rkv_plan_from_route(route, n, C.byref(params), C.byref(plan)) == 0
    shape = _abi.Shape(1, L, Hq, Hkv, d)
    nbytes = C.c_size_t()
    assert lib.rkv_prefill_workspace_size(plan, C.byref(shape), C.byref(nbytes)) == 0
    ws = torch.empty(nbytes.value, dtype=torch.uint8, device=dev)
    keep = [arr(q), arr(k), arr(v), arr(k_out), arr(v_out), arr(idx), arr(acc)]
    io = _abi.PrefillIO(keep[0], keep[1], keep[2], keep[3], keep[4], keep[5], None, keep[6])
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert lib.rkv_prefill_evict(plan, C.byref(shape), C.byref(io), C.c_void_p(ws.data_ptr()), ws.numel(), stream) == 0
    st_keep = [arr(k_c), arr(v_c), arr(pos_c), arr([acc_c[0], None])]
    state = _abi.DecodeState(*st_keep)
    assert lib.rkv_decode_init_from_prefill(plan, C.byref(shape), C.byref(io), C.byref(state), stream) == 0
    torch.cuda.synchronize()
    status = C.c_int32()
    assert lib.rkv_prefill_check(C.c_void_p(ws.data_ptr()), ws.numel(), C.byref(status)) == 0 and status.value == 0
    for l in range(n):
        ora = OP.evict_layer(rules[l], cap, xs[l]["q"], xs[l]["k"], xs[l]["v"], window=32)
        ii = idx[l].cpu().numpy()
        for h in range(Hkv):
            check_retained(ii[0, h], ora, h, L, f"c-abi layer {l} head {h}")
        assert torch.equal(k_c[l], k_out[l]) and torch.equal(pos_c[l], idx[l])
    assert torch.equal(acc_c[0], acc[0])
    # one decode step on both layers, checked against the oracle step of each rule
    dsteps = [decode_steps(49, 0, l, steps=1) for l in range(n)]
    qd = [bits_to_torch(ds["q"][0][None]) for ds in dsteps]
    kd = [bits_to_torch(ds["k"][0][None]) for ds in dsteps]
    vd = [bits_to_torch(ds["v"][0][None]) for ds in dsteps]
    vic = mk((1, Hkv), torch.int32)
    before = [{"k": torch_to_bits(k_c[l]), "pos": pos_c[l].cpu().numpy().copy(),
               "acc": acc_c[l].cpu().numpy().copy()} for l in range(n)]
    inp = _abi.DecodeInput(arr(qd), arr(kd), arr(vd), arr(vic))
    dshape = _abi.Shape(1, 1, Hq, Hkv, d)
    assert lib.rkv_decode_step(plan, C.byref(dshape), C.byref(state), C.byref(inp), L, stream) == 0
    torch.cuda.synchronize()
    for l in range(n):
        vv = vic[l].cpu().numpy()
        for h in range(Hkv):
            kc = OP.bf16_to_f64(before[l]["k"][0, h])
            qg = OP.bf16_to_f64(dsteps[l]["q"][0][4 * h:4 * h + 4])
            kt = OP.bf16_to_f64(dsteps[l]["k"][0][h])
            e = vv[0, h] if vv[0, h] >= 0 else cap
            if rules[l] == OP.TOVA:
                score, _ = OD.tova_step(kc, before[l]["pos"][0, h], qg, kt, L)
                assert score[e] <= score.min() * (1 + 1e-3) + 1e-30
            else:
                score, _, cand = OD.h2o_step(kc, before[l]["pos"][0, h], before[l]["acc"][0, h].astype(np.float64),
                                             qg, kt, L, cap // 2)
                assert cand[e] and score[e] <= score[cand].min() * (1 + 1e-3) + 1e-30
    lib.rkv_plan_destroy(plan)
