"""MI355X-native proactive expert cache for MoE inference (after ProMoE,
arXiv 2410.22134).  The hot path is libpromoe.so (HIP for gfx950, C ABI in
include/promoe.h); this package is its ctypes binding plus the synthetic-model
harness that drives it."""
from ._abi import (Config, Context, HostBuffer, PromoeError, FLAG_FILL_BY_DEADLINE, FLAG_NO_CHUNK,  # noqa: F401
                   FLAG_NO_PREEMPT, FLAG_NO_PREFETCH, FLAG_NO_REORDER, FLAG_PROFILE, FLAG_STATIC, PRIO_HIGH,
                   PRIO_LOW,
                   PROMOE_BF16, PROMOE_F32, lib)

# The paper's ablation steps (LRU baseline, then prefetch, chunked prefetch, early
# preemption and reordered inference added in turn) and its static baseline, as flags.
ABLATION = {
    "lru": FLAG_NO_PREFETCH | FLAG_NO_CHUNK | FLAG_NO_PREEMPT | FLAG_NO_REORDER,
    "+p": FLAG_NO_CHUNK | FLAG_NO_PREEMPT | FLAG_NO_REORDER,
    "+pc": FLAG_NO_PREEMPT | FLAG_NO_REORDER,
    "+pce": FLAG_NO_REORDER,
    "+pcer": 0,
    "static": FLAG_STATIC | FLAG_NO_PREFETCH | FLAG_NO_CHUNK | FLAG_NO_PREEMPT | FLAG_NO_REORDER,
}
