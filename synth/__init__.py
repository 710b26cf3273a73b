"""Seeded synthetic inputs (workload shapes, factorized caches, router
features).  Shared by the tests, the benchmark and the oracle checks; holds
no arithmetic of the method."""
from .workloads import Workload, ALL, TINY, LLAMA8B_32K, LLAMA8B_64K, BATCH16, LLAMA70B_128K
from .generate import CompressedCache, generate, router_inputs, rng_for, f32_to_bf16_bits, f16_bits
