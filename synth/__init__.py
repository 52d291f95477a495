"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the benchmark."""
from .configs import CONFIGS, ORDER, DESCRIPTION, Config
from .batch import (make_batch, make_trees, make_attention_inputs, target_for_slots,
                    f32_to_bf16_bits, bf16_bits_to_f32)
from .micro import micro_pool, TIE_LOGQ
