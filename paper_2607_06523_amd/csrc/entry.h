// Device routines that decode the routed residual storage (library private).
// Used by the fused decode kernel and by the residual-map test hook, so the
// hook checks exactly the decoding the decode kernel runs.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dwkv {

// 4-bit two's complement: nibble 0..7 -> 0..7, 8..15 -> -8..-1.
__device__ __forceinline__ int int4_value(uint32_t nibble) {
  return (int)((nibble & 0xFu) ^ 0x8u) - 8;
}

// Code of residual entry e, given the byte that holds it: entry e sits in byte
// e/2, low nibble when e is even.
__device__ __forceinline__ int entry_code(uint32_t byte, int64_t e) {
  return int4_value(byte >> ((uint32_t)(e & 1) * 4u));
}

__device__ __forceinline__ float half_bits_to_float(uint16_t b) {
  return (float)__builtin_bit_cast(_Float16, b);
}

__device__ __forceinline__ float bf16_bits_to_float(uint16_t b) {
  return __builtin_bit_cast(float, (uint32_t)b << 16);
}

}  // namespace dwkv
