"""MI355X (gfx950) implementation of NaCl's one-shot encoding-phase KV-cache
eviction (arXiv 2408.03675): HIP kernels behind the C ABI of include/nacl.h,
with a thin ctypes binding."""

from .nacl import (  # noqa: F401
    NaclError, Problem, SAMPLE_PROPORTIONAL, SAMPLE_SOFTMAX, SAMPLE_UNIFORM, EXPORTED,
    LIB_PATH, load_library, workspace_bytes, workspace, score, select, compact, compact_slots, evict,
    evict_slots, attention,
)
