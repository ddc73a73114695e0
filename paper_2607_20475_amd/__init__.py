"""MI355X-native fused LLM sampler (SonicSampler hot path, arXiv 2607.20475).

The computation lives in ``libss.so`` (hand-written HIP for gfx950, C ABI in
``include/ss.h``); :mod:`.binding` marshals torch tensors to it.
"""
from . import binding  # noqa: F401
from .binding import topk, sample, verify, process_logits, Params, workspace  # noqa: F401
