"""rkv_prefill_evict_noalloc (the entry point that allocates nothing: its workspace is the
library's static device array) against rkv_prefill_evict with a caller workspace, through the
C ABI, on two calls in a row, the second with a smaller input; plus the size limit."""
import ctypes as C

import numpy as np
import pytest

from oracle import prefill as OP
from parity import bits_to_torch, check_retained, check_scores
from synth import prefill_layer

pytestmark = pytest.mark.gpu


def _arr(ts):
    a = (C.c_void_p * len(ts))()
    for i, t in enumerate(ts):
        a[i] = t.data_ptr() if t is not None else None
    return C.cast(a, C.POINTER(C.c_void_p))


def _run_noalloc(plan, xs, L, Hq=32, Hkv=8, d=128):
    """Outputs of rkv_prefill_evict_noalloc (ctypes) and of rkv_prefill_evict (caller workspace)."""
    import torch
    import paper_2606_15157_amd as rkv
    from paper_2606_15157_amd import _abi
    lib = _abi.lib()
    q = [bits_to_torch(x["q"][None]) for x in xs]
    k = [bits_to_torch(x["k"][None]) for x in xs]
    v = [bits_to_torch(x["v"][None]) for x in xs]
    out = rkv.alloc_outputs(plan, 1, Hkv, L, d, "cuda", score_out=True, acc_out=True)
    keep = [_arr(q), _arr(k), _arr(v), _arr(out["k_out"]), _arr(out["v_out"]), _arr(out["idx"]),
            _arr(out["scores"]), _arr(out["acc"])]
    io = _abi.PrefillIO(*keep)
    shape = _abi.Shape(1, L, Hq, Hkv, d)
    status = torch.full((1,), 0x7fffffff, dtype=torch.int32, device="cuda")
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    rc = lib.rkv_prefill_evict_noalloc(plan.handle, C.byref(shape), C.byref(io), C.c_void_p(status.data_ptr()),
                                       stream)
    assert rc == 0, lib.rkv_last_error()
    ref = rkv.evict_prefill(plan, q, k, v, score_out=True, acc_out=True)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert rkv.prefill_check(ref["workspace"]) == 0
    return out, ref


def _compare(plan, rules, budgets, xs, L):
    out, ref = _run_noalloc(plan, xs, L)
    import torch
    for l, r in enumerate(rules):
        for key in ("idx", "k_out", "v_out"):
            assert torch.equal(out[key][l], ref[key][l]), (key, l)
        ora = OP.evict_layer(r, budgets[l], xs[l]["q"], xs[l]["k"], xs[l]["v"], window=32)
        idx = out["idx"][l].cpu().numpy()
        sc = out["scores"][l].cpu().numpy()
        sr = ref["scores"][l].cpu().numpy()
        for h in range(8):
            what = f"no-alloc layer {l} head {h}"
            check_retained(idx[0, h], ora, h, L, what)
            if ora["scores"] is not None:
                n = ora["scores"].shape[1]
                check_scores(sc[0, h, :n], sr[0, h, :n].astype(np.float64), what + " vs workspace call")
        if r in (OP.SNAPKV, OP.H2O, OP.TOVA):
            a, b = out["acc"][l].cpu().numpy(), ref["acc"][l].cpu().numpy()
            check_scores(a, b.astype(np.float64), f"no-alloc acc layer {l}")


def test_noalloc_matches_workspace_call_twice_second_smaller():
    import paper_2606_15157_amd as rkv
    rules1, budgets1, L1 = [OP.SNAPKV, OP.H2O, OP.TOVA, OP.STREAMING], [400, 300, 200, 100], 4096
    xs1 = [prefill_layer(60, 0, l, seq_len=L1, window=32) for l in range(4)]
    _compare(rkv.Plan(rules1, budgets1, window=32), rules1, budgets1, xs1, L1)
    rules2, budgets2, L2 = [OP.H2O, OP.SNAPKV], [128, 100], 1024
    xs2 = [prefill_layer(61, 0, l, seq_len=L2, window=32) for l in range(2)]
    _compare(rkv.Plan(rules2, budgets2, window=32), rules2, budgets2, xs2, L2)


def test_noalloc_rejects_a_workspace_above_its_limit():
    import paper_2606_15157_amd as rkv
    from paper_2606_15157_amd import _abi
    from synth.workloads import mixed_route, pyramid_weights
    lib = _abi.lib()
    budgets = rkv.allocate_budgets(pyramid_weights(32), 32 * 512, 48)
    plan = rkv.Plan(mixed_route(32), budgets, window=32)
    fake = _arr([None] * 32)
    io = _abi.PrefillIO(fake, fake, fake, fake, fake, fake, None, None)
    shape = _abi.Shape(8, 8192, 32, 8, 128)   # batch 8 needs about 265 MiB
    assert lib.rkv_prefill_evict_noalloc(plan.handle, C.byref(shape), C.byref(io), None, None) == 5
    assert b"no-allocation scratch" in lib.rkv_last_error()
