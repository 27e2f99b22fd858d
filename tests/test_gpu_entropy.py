"""GPU parity of the attention-entropy layer score (Section 3.3) against the CPU oracle.

Tolerance: row entropies within 1e-3 relative plus 1e-4 absolute (fp32 sums of bf16 logits;
H = ln 2 (log2 Z - T / Z) cancels for nearly one-hot rows, hence the absolute term); the layer
means within 1e-4 relative."""
import numpy as np
import pytest

from oracle import alloc as OA
from oracle import entropy as OE
from parity import bits_to_torch
from synth import f32_to_bf16_bits, prefill_layer

pytestmark = pytest.mark.gpu


def run(layers_qk, n_q):
    import paper_2606_15157_amd as rkv
    import torch
    q = [bits_to_torch(np.stack([x[0] for x in seqs])) for seqs in layers_qk]
    k = [bits_to_torch(np.stack([x[1] for x in seqs])) for seqs in layers_qk]
    out = rkv.entropy_profile(q, k)
    torch.cuda.synchronize()
    return out["h"].cpu().numpy(), out["rows"].cpu().numpy(), int(out["status"].item())


def check(layers_qk, n_q, label):
    h, rows, status = run(layers_qk, n_q)
    assert status == 0, label
    for l, seqs in enumerate(layers_qk):
        ora = [OE.row_entropies(qb, kb) for qb, kb in seqs]
        for s, r in enumerate(ora):
            err = np.abs(rows[l, s] - r)
            bad = err > 1e-3 * np.abs(r) + 1e-4
            assert not bad.any(), f"{label} layer {l} seq {s}: {bad.sum()} rows off, worst {err.max():.3e}"
        np.testing.assert_allclose(h[l], np.mean(ora), rtol=1e-4, err_msg=f"{label} layer {l} mean")
    return h


def gen(workload, seq, layer, L, n_q, Hq=32, Hkv=8):
    x = prefill_layer(workload, seq, layer, seq_len=L, n_q_heads=Hq, n_kv_heads=Hkv, window=n_q)
    return x["q"], x["k"]


def test_full_profile_1k():
    """Every query of a 1024-token calibration sequence, two layers, 32 / 8 heads."""
    L = 1024
    check([[gen(20, 0, l, L, L)] for l in range(2)], L, "full1k")


@pytest.mark.parametrize("Hq,Hkv,L,n_q,B", [(16, 8, 777, 100, 2), (8, 8, 300, 300, 1), (32, 4, 513, 77, 1)])
def test_ragged_shapes_and_groups(Hq, Hkv, L, n_q, B):
    """G = 2, 1, 8; query blocks with a ragged tail; prompts that are not a multiple of 128."""
    check([[gen(21, s, l, L, n_q, Hq, Hkv) for s in range(B)] for l in range(2)], n_q, f"g{Hq // Hkv}")


def test_more_than_one_launch_group():
    """More layers than one launch takes (33)."""
    L, n_q = 256, 64
    check([[gen(22, 0, l, L, n_q)] for l in range(33)], n_q, "33layers")


def test_uniform_rows_closed_form():
    """q = 0: row t has entropy ln(t + 1) exactly (checked on the device output directly)."""
    rng = np.random.default_rng(7)
    L, n_q = 640, 640
    q = np.zeros((32, n_q, 128), dtype=np.uint16)
    k = f32_to_bf16_bits(rng.standard_normal((8, L, 128)).astype(np.float32))
    h, rows, status = run([[(q, k)]], n_q)
    assert status == 0
    expect = np.log(np.arange(1, L + 1, dtype=np.float64))
    np.testing.assert_allclose(rows[0, 0], np.broadcast_to(expect, (32, n_q)), rtol=2e-6, atol=2e-6)


def test_entropy_budgets_match_oracle_allocation():
    """Entropy allocation (identity transform, b_min 32) from the device scores equals the
    oracle's allocation from its own scores."""
    import paper_2606_15157_amd as rkv
    L, n_q, n_layers = 512, 128, 8
    layers = [[gen(23, 0, l, L, n_q)] for l in range(n_layers)]
    h = check(layers, n_q, "alloc")
    h_ora = [OE.layer_score([x[0]], [x[1]]) for x in (seqs[0] for seqs in layers)]
    total = n_layers * 512
    got = rkv.entropy_budgets(h, total, 32)
    ref = OA.allocate_from_scores(h_ora, OA.IDENTITY, total, 32)
    assert sum(got) == total and min(got) >= 32
    assert np.abs(np.array(got) - np.array(ref)).max() <= 1   # a remainder tie may go either way
    print(f"budgets {got}")


def test_overflow_is_reported():
    """A row whose logit with one key beats its reference (own key, key 0) by ~180 natural-log
    units overflows fp32; the status word says so."""
    rng = np.random.default_rng(8)
    L, n_q = 512, 64
    q = f32_to_bf16_bits(rng.standard_normal((32, n_q, 128)).astype(np.float32))
    k = f32_to_bf16_bits(rng.standard_normal((8, L, 128)).astype(np.float32))
    four = f32_to_bf16_bits(np.full(128, 4.0, np.float32))
    q[5, 7] = four
    k[1, 100] = four
    _, _, status = run([[(q, k)]], n_q)
    assert status == 1
