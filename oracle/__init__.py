"""Plain CPU oracle for the MiKV decode path (arXiv 2402.18096).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  It shares no
code with the HIP path in ``paper_2402_18096_amd`` and imports nothing from
it; the two meet only in the seeded input generators.

The oracle is a direct, slow, readable transcription of what the paper
computes: the Eq. 1 quantizer (quant), the Eq. 2-4 channel balancer (balance),
decode attention over the cache (attention), the H2O importance score and
the top-k plus recent-window selection (policy), and the decode step that
ties them together (cache).  Floating-point work is fp64 where the paper
fixes nothing (attention) and fp32 where the stored format demands an exact,
reproducible rounding (the quantizer, the balancer, the score sums).

Every function is pinned in ``tests/test_oracle_*.py`` against values and
properties that do not come from the oracle itself.
"""
from .attention import attention
from .balance import balance_keys, balance_query, balancer
from .cache import OracleCache
from .policy import accumulate, heavy_budget, heavy_list, prefill_importance, select
from .quant import (bits_per_element, dequantize, encode, f16_bits, f16_value, pack, quantize, quantize_channels,
                    unpack)

__all__ = [
    "attention", "balance_keys", "balance_query", "balancer", "OracleCache", "accumulate",
    "heavy_budget", "heavy_list", "prefill_importance", "select", "bits_per_element", "dequantize", "f16_bits", "f16_value", "pack",
    "quantize", "unpack", "encode", "quantize_channels",
]
