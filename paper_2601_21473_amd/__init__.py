"""MI355X-native hot path of an invocation-distance memory manager for
multi-agent LLM simulation: per-step eviction/prefetch planning and the
movement of agents' paged prefix-KV and LoRA adapter memory between an HBM
pool and pinned host memory (libscalesim, HIP for gfx950).

``binding`` is the ctypes binding of the C ABI (include/scalesim.h);
``memory`` allocates a pool's device and pinned host buffers through the
library's own allocation calls (the HIP runtime it is linked with), not
through PyTorch.
"""
from . import binding  # noqa: F401  (loads the library lazily, on first call)
