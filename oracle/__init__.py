"""Test infrastructure only: a plain float64 CPU forward of the dense decoder.

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this
package.  It shares no code with the GPU path and imports nothing from it.
"""

from .model import (DecoderOracle, attend, bf16_round, greedy, rms_norm, rope_rotate,
                    silu, softmax)
from .quant import dequantize_q8, q8_model_f64, quantize_q8, quantize_q8_loops

__all__ = ["DecoderOracle", "attend", "bf16_round", "greedy", "rms_norm", "rope_rotate",
           "silu", "softmax", "quantize_q8", "dequantize_q8", "quantize_q8_loops", "q8_model_f64"]
