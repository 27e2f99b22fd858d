"""Layer-routed KV-cache eviction on AMD MI355X (gfx950): Python binding of librkv.so.

Argument marshalling only: every step of the eviction path runs in the HIP kernels of
librkv.so.  PyTorch provides device memory and the current HIP stream.

    plan = Plan(rules, budgets, window=32, pool_kernel=7)
    out = evict_prefill(plan, q_win, k, v)      # per-layer lists of bf16 device tensors
    out["k_out"][l], out["v_out"][l], out["idx"][l]
"""
from __future__ import annotations

import ctypes as C
from typing import Sequence

from . import _abi
from ._abi import FULL, STREAMING, SNAPKV, H2O, TOVA, H2O_FULL, PHASE_PREFILL, PHASE_DECODE, T_IDENTITY, T_PPL_CAP  # noqa: F401
from ._abi import SCOPE_PREFILL, SCOPE_DECODE, SCOPE_BOTH, STATUS_TIMEOUT, STATUS_INVALID, STATUS_REPAIRED  # noqa: F401
from ._abi import RkvError, check

__all__ = ["Plan", "allocate_budgets", "evict_prefill", "decode_step", "decode_init_from_prefill", "prefill_check",
           "rule_phases", "version", "entropy_profile", "entropy_budgets",
           "FULL", "STREAMING", "SNAPKV", "H2O", "TOVA", "H2O_FULL", "SCOPE_PREFILL", "SCOPE_DECODE", "SCOPE_BOTH",
           "RkvError"]


def version() -> int:
    return _abi.lib().rkv_version()


def rule_phases(rule: int) -> int:
    """Phases operator `rule` declares (Section 3.4): bit 0 prefill, bit 1 decode."""
    m = C.c_int32()
    check(_abi.lib().rkv_rule_phases(int(rule), C.byref(m)))
    return m.value


def allocate_budgets(scores: Sequence[float], total: int, b_min: int, transform: int = T_IDENTITY):
    """Per-layer integer budgets summing to `total`, each >= b_min (Section 3.3, Eq. 3)."""
    n = len(scores)
    arr = (C.c_double * n)(*[float(x) for x in scores])
    out = (C.c_int32 * n)()
    check(_abi.lib().rkv_allocate_budgets(arr, n, transform, int(total), int(b_min), out))
    return list(out)


class Plan:
    """Immutable execution plan: per layer an operator and capacity for prefill and decode (Eq. 1)."""

    def __init__(self, rules_prefill, budgets_prefill, rules_decode=None, budgets_decode=None, *,
                 window=32, pool_kernel=7, n_sink=4, recent_num=1, recent_den=2):
        n = len(rules_prefill)
        rules_decode = list(rules_decode) if rules_decode is not None else [FULL] * n
        budgets_decode = list(budgets_decode) if budgets_decode is not None else [0] * n
        if not (len(budgets_prefill) == len(rules_decode) == len(budgets_decode) == n):
            raise ValueError("per-layer lists must have equal length")
        layers = (_abi.Layer * n)()
        for i in range(n):
            layers[i] = _abi.Layer(int(rules_prefill[i]), int(budgets_prefill[i]), int(rules_decode[i]),
                                   int(budgets_decode[i]))
        self.params = _abi.Params(window, pool_kernel, n_sink, recent_num, recent_den)
        handle = C.c_void_p()
        check(_abi.lib().rkv_plan_create(layers, n, C.byref(self.params), C.byref(handle)))
        self._h = handle
        self.n_layers = n
        self.rules_prefill = [int(r) for r in rules_prefill]
        self.rules_decode = rules_decode
        self.window = window

    @classmethod
    def from_route(cls, rules_prefill, weights, total: int, b_min: int, rules_decode=None, *,
                   transform: int = T_IDENTITY, **params):
        """Plan whose per-layer capacities split `total` by allocation `weights` (Eq. 3); decode
        capacities equal the prefill ones."""
        budgets = allocate_budgets(weights, total, b_min, transform)
        return cls(rules_prefill, budgets, rules_decode, budgets if rules_decode is not None else None, **params)

    @classmethod
    def from_scoped_route(cls, rules, scopes, budgets, **params) -> "Plan":
        """Plan of a completed route (Sections 3.1-3.2): layer l runs rules[l] at capacity
        budgets[l] in the phases of scopes[l] (SCOPE_PREFILL, SCOPE_DECODE or SCOPE_BOTH, a tied
        both-phase route) and FULL in the other phase; validated by rkv_plan_from_route."""
        n = len(rules)
        if not (len(scopes) == len(budgets) == n):
            raise ValueError("per-layer lists must have equal length")
        route = (_abi.RouteLayer * n)()
        for i in range(n):
            route[i] = _abi.RouteLayer(int(rules[i]), int(scopes[i]), int(budgets[i]))
        p = dict(window=32, pool_kernel=7, n_sink=4, recent_num=1, recent_den=2)
        p.update(params)
        prm = _abi.Params(p["window"], p["pool_kernel"], p["n_sink"], p["recent_num"], p["recent_den"])
        handle = C.c_void_p()
        check(_abi.lib().rkv_plan_from_route(route, n, C.byref(prm), C.byref(handle)))
        self = cls.__new__(cls)
        self._h = handle
        self.n_layers = n
        self.params = prm
        self.rules_prefill = [int(r) if s != SCOPE_DECODE else FULL for r, s in zip(rules, scopes)]
        self.rules_decode = [int(r) if s != SCOPE_PREFILL else FULL for r, s in zip(rules, scopes)]
        self.window = p["window"]
        return self

    def to_bytes(self) -> bytes:
        """The plan's serialized record (rkv_plan_serialize)."""
        size = C.c_size_t()
        check(_abi.lib().rkv_plan_serialize(self._h, None, 0, C.byref(size)))
        buf = C.create_string_buffer(size.value)
        check(_abi.lib().rkv_plan_serialize(self._h, buf, size.value, C.byref(size)))
        return buf.raw[:size.value]

    @classmethod
    def from_bytes(cls, data: bytes) -> "Plan":
        """A plan from a serialized record, validated by the library (rkv_plan_deserialize)."""
        import struct
        handle = C.c_void_p()
        check(_abi.lib().rkv_plan_deserialize(C.c_char_p(bytes(data)), len(data), C.byref(handle)))
        words = struct.unpack("<%di" % (len(data) // 4), data)
        n = words[2]
        self = cls.__new__(cls)
        self._h = handle
        self.n_layers = n
        self.params = _abi.Params(*words[3:8])
        lay = words[8:]
        self.rules_prefill = [lay[4 * i] for i in range(n)]
        self.rules_decode = [lay[4 * i + 2] for i in range(n)]
        self.window = words[3]
        return self

    @property
    def handle(self):
        return self._h

    def close(self):
        if getattr(self, "_h", None):
            _abi.lib().rkv_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def retained_counts(self, seq_len: int, phase: int = PHASE_PREFILL):
        out = (C.c_int32 * self.n_layers)()
        check(_abi.lib().rkv_plan_retained_counts(self._h, phase, seq_len, out))
        return list(out)

    def workspace_size(self, batch, seq_len, n_q_heads, n_kv_heads, head_dim=128) -> int:
        shape = _abi.Shape(batch, seq_len, n_q_heads, n_kv_heads, head_dim)
        nb = C.c_size_t()
        check(_abi.lib().rkv_prefill_workspace_size(self._h, C.byref(shape), C.byref(nb)))
        return nb.value


def _ptr(t):
    return t.data_ptr() if t is not None else None


def _parr(ptrs):
    return C.cast(_abi.ptr_array(ptrs), C.POINTER(C.c_void_p))


def _stream_handle(stream, device):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return s.cuda_stream


def alloc_workspace(plan: Plan, batch, seq_len, n_q_heads, n_kv_heads, device="cuda"):
    import torch
    nb = plan.workspace_size(batch, seq_len, n_q_heads, n_kv_heads)
    return torch.empty(nb, dtype=torch.uint8, device=device)


def evict_prefill(plan: Plan, q_win, k, v, *, out=None, workspace=None, score_out=False, acc_out=False,
                  stream=None, check_status=False):
    """Compress every layer's prompt cache.

    q_win[l]: bf16 [B, Hq, w, d] ([B, Hq, L, d] for H2O_FULL layers; None allowed for FULL /
    STREAMING layers);
    k[l], v[l]: bf16 [B, Hkv, L, d].  Returns dict of per-layer lists: k_out, v_out (bf16
    [B, Hkv, n_l, d]), idx (int32 [B, Hkv, n_l], ascending), and optionally scores (fp32
    [B, Hkv, L]) and acc (fp32 [B, Hkv, n_l]).  Outputs are valid after the stream syncs and
    when the workspace status word (prefill_check) has neither STATUS_TIMEOUT nor STATUS_INVALID;
    check_status=True synchronises and raises RkvError otherwise.
    """
    import torch
    n = plan.n_layers
    if not (len(k) == len(v) == len(q_win) == n):
        raise ValueError("need one q_win / k / v entry per layer")
    B, Hkv, L, d = k[0].shape
    Hq = next((q.shape[1] for q in q_win if q is not None), Hkv)
    dev = k[0].device
    for t in list(k) + list(v) + [q for q in q_win if q is not None]:
        if t.dtype != torch.bfloat16 or not t.is_contiguous() or t.device != dev:
            raise ValueError("inputs must be contiguous bf16 tensors on one device")
    for t in list(k) + list(v):
        if tuple(t.shape) != (B, Hkv, L, d):
            raise ValueError("every k / v must have shape [B, Hkv, L, d]")
    for q, r in zip(q_win, plan.rules_prefill):
        rows = L if r == H2O_FULL else plan.window
        if q is not None and tuple(q.shape) != (B, Hq, rows, d):
            raise ValueError("q_win must have shape [B, Hq, w, d] ([B, Hq, L, d] for H2O_FULL layers)")
    counts = plan.retained_counts(L)
    if out is None:
        out = {
            "k_out": [torch.empty((B, Hkv, c, d), dtype=torch.bfloat16, device=dev) for c in counts],
            "v_out": [torch.empty((B, Hkv, c, d), dtype=torch.bfloat16, device=dev) for c in counts],
            "idx": [torch.empty((B, Hkv, c), dtype=torch.int32, device=dev) for c in counts],
        }
        if score_out:
            out["scores"] = [torch.zeros((B, Hkv, L), dtype=torch.float32, device=dev) for _ in range(n)]
        if acc_out:
            out["acc"] = [torch.empty((B, Hkv, c), dtype=torch.float32, device=dev) for c in counts]
    if workspace is None:
        workspace = alloc_workspace(plan, B, L, Hq, Hkv, dev)
    call = PreparedPrefill(plan, q_win, k, v, out, workspace)
    call(stream)
    out["workspace"] = workspace
    out["io"] = call   # keeps the marshalled pointer tables (decode_init_from_prefill uses them)
    if check_status:
        torch.cuda.synchronize(dev)
        st = prefill_check(workspace)
        if st & (STATUS_TIMEOUT | STATUS_INVALID):
            raise RkvError(7, f"prefill status word {st:#x}: outputs invalid")
    return out


class PreparedPrefill:
    """A prefill call with its pointer tables marshalled once; calling it enqueues the whole
    eviction pass on the stream with a single C call (for loops, benchmarks and graphs)."""

    def __init__(self, plan: Plan, q_win, k, v, out, workspace):
        B, Hkv, L, d = k[0].shape
        Hq = next((q.shape[1] for q in q_win if q is not None), Hkv)
        self._keep = (q_win, k, v, out, workspace)
        self._arrays = [_parr([_ptr(q) for q in q_win]), _parr([_ptr(t) for t in k]), _parr([_ptr(t) for t in v]),
                        _parr([_ptr(t) for t in out["k_out"]]), _parr([_ptr(t) for t in out["v_out"]]),
                        _parr([_ptr(t) for t in out["idx"]]),
                        _parr([_ptr(t) for t in out["scores"]]) if "scores" in out else None,
                        _parr([_ptr(t) for t in out["acc"]]) if "acc" in out else None]
        self.io = _abi.PrefillIO(*self._arrays)
        self.shape = _abi.Shape(B, L, Hq, Hkv, d)
        self.plan = plan
        self.ws_ptr = C.c_void_p(workspace.data_ptr())
        self.ws_bytes = workspace.numel()
        self.device = k[0].device
        self._fn = _abi.lib().rkv_prefill_evict

    def __call__(self, stream=None):
        check(self._fn(self.plan.handle, C.byref(self.shape), C.byref(self.io), self.ws_ptr, self.ws_bytes,
                       C.c_void_p(_stream_handle(stream, self.device))))


def alloc_outputs(plan: Plan, B, Hkv, L, d=128, device="cuda", score_out=False, acc_out=False):
    import torch
    counts = plan.retained_counts(L)
    out = {
        "k_out": [torch.empty((B, Hkv, c, d), dtype=torch.bfloat16, device=device) for c in counts],
        "v_out": [torch.empty((B, Hkv, c, d), dtype=torch.bfloat16, device=device) for c in counts],
        "idx": [torch.empty((B, Hkv, c), dtype=torch.int32, device=device) for c in counts],
    }
    if score_out:
        out["scores"] = [torch.zeros((B, Hkv, L), dtype=torch.float32, device=device) for _ in counts]
    if acc_out:
        out["acc"] = [torch.empty((B, Hkv, c), dtype=torch.float32, device=device) for c in counts]
    return out


STAGE_ZERO, STAGE_SCORE, STAGE_SELECT, STAGE_GATHER, STAGE_DECODE = 0, 1, 2, 3, 4


def profile_enable(stage: int):
    """Record HIP events around every following launch of `stage` (-1 disables)."""
    check(_abi.lib().rkv_profile_enable(int(stage)))


def profile_read():
    """(number of recorded launches, summed milliseconds); synchronises and clears."""
    n = C.c_int32()
    ms = C.c_double()
    check(_abi.lib().rkv_profile_read(C.byref(n), C.byref(ms)))
    return n.value, ms.value


def prefill_check(workspace) -> int:
    """Status word a previous prefill left in `workspace` (0 = clean).  Synchronous."""
    st = C.c_int32()
    check(_abi.lib().rkv_prefill_check(C.c_void_p(workspace.data_ptr()), workspace.numel(), C.byref(st)))
    return st.value


def entropy_profile(q, k, *, stream=None):
    """Attention-entropy layer scores H_l (Section 3.3): q[l] bf16 [B, Hq, n_q, d] (queries of the
    last n_q positions), k[l] bf16 [B, Hkv, L, d].  Returns {"h": fp32 [n_layers] (nats),
    "rows": fp32 [n_layers, B, Hq, n_q], "status": int32 [1] (nonzero: a row was not finite)}.
    Outputs are valid after the stream is synchronised."""
    import torch
    n = len(q)
    assert n == len(k) and n >= 1
    B, Hq, n_q, d = q[0].shape
    Hkv, L = k[0].shape[1], k[0].shape[2]
    dev = k[0].device
    rows = torch.empty((n, B, Hq, n_q), dtype=torch.float32, device=dev)
    h = torch.empty((n,), dtype=torch.float32, device=dev)
    status = torch.empty((1,), dtype=torch.int32, device=dev)
    shape = _abi.Shape(B, L, Hq, Hkv, d)
    nbytes = C.c_size_t()
    check(_abi.lib().rkv_entropy_workspace_size(C.byref(shape), n, n_q, C.byref(nbytes)))
    ws = torch.empty((max(nbytes.value, 8) + 7) // 8, dtype=torch.float64, device=dev)
    check(_abi.lib().rkv_entropy_profile(C.byref(shape), n, n_q, _parr([_ptr(t) for t in q]),
                                         _parr([_ptr(t) for t in k]), C.c_void_p(rows.data_ptr()),
                                         C.c_void_p(h.data_ptr()), C.c_void_p(status.data_ptr()),
                                         C.c_void_p(ws.data_ptr()), ws.numel() * 8,
                                         C.c_void_p(_stream_handle(stream, dev))))
    return {"h": h, "rows": rows, "status": status, "workspace": ws}


def entropy_budgets(h, total: int, b_min: int = 32):
    """Entropy allocation: per-layer capacities from H_l by Eq. 3 with the identity transform."""
    return allocate_budgets([float(x) for x in h], total, b_min, T_IDENTITY)


def decode_init_from_prefill(plan: Plan, prefill_out, state=None, *, stream=None):
    """Prefill -> decode hand-off (Section 3.4, rkv_decode_init_from_prefill): the compacted prompt
    cache of an evict_prefill result becomes the decode state of every layer whose decode operator
    is not FULL.  `state` (per-layer lists "k_cache", "v_cache", "pos", "acc") is allocated when
    None; entries of FULL-decode layers stay None, "acc" only for decode H2O layers.  Returns the
    state; valid after the stream syncs."""
    import torch
    call = prefill_out["io"]
    B, L, Hq, Hkv, d = (call.shape.batch, call.shape.seq_len, call.shape.n_q_heads, call.shape.n_kv_heads,
                        call.shape.head_dim)
    dev = call.device
    caps = plan.retained_counts(L, PHASE_DECODE)
    n = plan.n_layers
    if state is None:
        state = {"k_cache": [], "v_cache": [], "pos": [], "acc": []}
        for l in range(n):
            r, c = plan.rules_decode[l], caps[l]
            live = r != FULL
            state["k_cache"].append(torch.empty((B, Hkv, c, d), dtype=torch.bfloat16, device=dev) if live else None)
            state["v_cache"].append(torch.empty((B, Hkv, c, d), dtype=torch.bfloat16, device=dev) if live else None)
            state["pos"].append(torch.empty((B, Hkv, c), dtype=torch.int32, device=dev) if live else None)
            state["acc"].append(torch.empty((B, Hkv, c), dtype=torch.float32, device=dev) if r == H2O else None)
    st = _abi.DecodeState(_parr([_ptr(t) for t in state["k_cache"]]), _parr([_ptr(t) for t in state["v_cache"]]),
                          _parr([_ptr(t) for t in state["pos"]]), _parr([_ptr(t) for t in state["acc"]]))
    check(_abi.lib().rkv_decode_init_from_prefill(plan.handle, C.byref(call.shape), C.byref(call.io), C.byref(st),
                                                  C.c_void_p(_stream_handle(stream, dev))))
    return state


def decode_step(plan: Plan, state, q, k, v, position: int, *, victim_out=None, stream=None):
    """One decode step for every layer with a decode operator.

    state: dict of per-layer lists "k_cache", "v_cache" (bf16 [B, Hkv, C_l, d]), "pos" (int32
    [B, Hkv, C_l]), "acc" (fp32 [B, Hkv, C_l]; None allowed for layers whose decode operator is
    not H2O); updated in place.  q[l]: bf16 [B, Hq, d];
    k[l], v[l]: bf16 [B, Hkv, d].  victim_out: optional per-layer int32 [B, Hkv] tensors.
    """
    n = plan.n_layers
    B, Hkv = k[0].shape[0], k[0].shape[1]
    Hq = q[0].shape[1]
    d = k[0].shape[-1]
    st = _abi.DecodeState(_parr([_ptr(t) for t in state["k_cache"]]), _parr([_ptr(t) for t in state["v_cache"]]),
                          _parr([_ptr(t) for t in state["pos"]]), _parr([_ptr(t) for t in state["acc"]]))
    inp = _abi.DecodeInput(_parr([_ptr(t) for t in q]), _parr([_ptr(t) for t in k]), _parr([_ptr(t) for t in v]),
                           _parr([_ptr(t) for t in victim_out]) if victim_out is not None else None)
    shape = _abi.Shape(B, 1, Hq, Hkv, d)
    dev = k[0].device
    assert len(q) == len(k) == len(v) == n
    check(_abi.lib().rkv_decode_step(plan.handle, C.byref(shape), C.byref(st), C.byref(inp), int(position),
                                     C.c_void_p(_stream_handle(stream, dev))))
