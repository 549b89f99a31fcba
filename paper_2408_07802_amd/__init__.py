"""MI355X-native (gfx950) Kraken prefill: HIP kernels behind a C ABI, with a thin binding.

Kraken (arXiv 2408.07802) layers hold N parallel pre-LN sub-layers whose outputs
are summed before the next layer's FFN LayerNorm.  ``kraken.Kraken`` wraps the
C ABI in ``include/kraken.h``; ``synth`` draws seeded synthetic workloads.
"""

from .kraken import Config, Kraken, KrakenError, cu_from_lens, pack_weights  # noqa: F401
