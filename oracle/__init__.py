"""CPU oracle for layer-routed KV-cache eviction.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, float64 NumPy
restatement of what the eviction path computes, written from the paper
("Exploring a Layer-Wise Design Space for KV Cache Eviction"): the execution
plan of Eq. 1 (Section 3.1), the fixed-total capacity allocator of Section 3.3
(Eq. 3 with the shift, the b_min clamp and largest-remainder rounding) and its
attention-entropy layer score, and the
retention rules the paper composes across layers (SnapKV window scoring, H2O
accumulated attention, StreamingLLM sinks plus recent tokens, Full), whose
arithmetic the paper cites rather than restates.

Only tests, the smoke check and the benchmark's CPU-baseline leg may import it.
It shares no code with the HIP path and imports nothing from it.

Points the paper leaves open are fixed here as stated readings; each function
names the reading it takes.  Functions with no independent pin say
"parity unpinned" in their docstring.
"""
from . import alloc, prefill, decode, entropy  # noqa: F401
from .prefill import FULL, STREAMING, SNAPKV, H2O  # noqa: F401
