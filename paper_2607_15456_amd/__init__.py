"""MI355X-native hot path of Looped Latent Attention (arxiv 2607.15456).

liblla.so holds the HIP kernels (gfx950) behind the C ABI of include/lla.h;
``paper_2607_15456_amd.lla`` is its thin ctypes binding.
"""

from . import lla  # noqa: F401
from .lla import (  # noqa: F401
    LLAError,
    alloc_cache,
    cache_bytes,
    decode_attn,
    decode_workspace_bytes,
    encode,
    from_paged,
    new_workspace,
    prefill_attn,
    rho,
    rope_rotate,
    rope_write,
    to_paged,
)
