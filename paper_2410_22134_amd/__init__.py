"""MI355X-native proactive expert cache for MoE inference (after ProMoE,
arXiv 2410.22134).  The hot path is libpromoe.so (HIP for gfx950, C ABI in
include/promoe.h); this package is its ctypes binding plus the synthetic-model
harness that drives it."""
from ._abi import (Config, Context, HostBuffer, PromoeError, FLAG_NO_PREFETCH, FLAG_PROFILE, PRIO_HIGH,  # noqa: F401
                   PRIO_LOW, PROMOE_BF16, PROMOE_F32, lib)
