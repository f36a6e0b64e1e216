"""CPU oracle for the AgentKVShift reuse prefill.

TEST INFRASTRUCTURE ONLY. This package is a plain, slow, fp64 NumPy statement of
what the reuse-prefill path computes (the decoder, full prefill, standalone unit
caching, the first decode step over the reused caches, the probe-guided residual correction of Sec. 3.3 / Algorithm 1, and the
group-64 cache quantisers: 2/4-bit integer and FP8 E4M3). Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import it; the library path never does, and it shares no
code with the HIP kernels.

Every function cites the passage of the paper it follows; where the paper leaves a
step open, the function's docstring states the reading it takes.
"""
from .model import (ModelDims, dims_from, rms_norm, rope_cos_sin, rotate, attention,
                    decoder_layer, full_prefill, cache_units, split_layer, lm_logits,
                    greedy_token, decode_step)
from .reuse import (F_NO_CORRECTION, F_UNIT_WEIGHTS, F_FRESH_IF_RECOMPUTED,
                    F_NO_PREFIX_RECOMPUTE, F_PRE_ROPE_OFFSETS, probe_budget, chunk_starts,
                    rerotate, divergence, select_top, correction_weights, probe_offset,
                    probe_offset_pre_rope, correct_chunk, correct_chunk_pre_rope,
                    reuse_prefill)
from .quant import (quantize_g64, dequantize_g64, pack_codes, unpack_codes, E4M3_MAX,
                    e4m3_value, e4m3_code, quantize_e4m3_g64, dequantize_e4m3_g64)
