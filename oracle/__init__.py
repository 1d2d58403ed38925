"""CPU oracle of the batch-1 Llama decode step, and (schedule_sim) an
independent safety oracle for its task schedules (test infrastructure only).

Only tests, the smoke check and the benchmark's CPU-baseline leg use this
package; the product path never imports it.
"""
from .decode import (  # noqa: F401
    OracleModel, argmax_first, attention, bf16_decode, bf16_round, decode_step, dequantize, dequantize_int4,
    greedy, linear, rmsnorm, rope, rope_angles, silu, softmax, top2_margin, unpack_int4)
