"""Seeded synthetic workloads (shapes, weights, visual tokens, prompts, sampling uniforms).

Shared by the oracle and the device path; holds none of the method's arithmetic.
"""
from .configs import (Shape, Workload, ALL, C1, C2, C3, C5, S1, S_T5, S_LLAMA, S_LLAMA_F32, c4_points,
                      TINY_T5, FLANT5_BASE, FLANT5_XL, LLAVA_7B, SMALL_T5_BF16, SMALL_LLAMA_BF16,
                      SMALL_LLAMA_F32)
from .generate import (make_weights, workload_weights, make_visual, make_prompts, round_to_bf16,
                       tensor_list, tensor_shape, make_uniforms)
