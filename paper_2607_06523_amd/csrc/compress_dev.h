// Compression of one token's key or value vector (Sec. 3, the storage half
// of Eq. 1), shared by the append/compress kernel and the decode that appends
// the new token in its own launch.  One wave takes one vector; the window
// basis rows sit in LDS (rows of kBRow halves) and the wave owns small LDS
// arrays for its input, coefficients and entries.
//   A_i   = fp16( sum_j x_j B_ij )                    lane i (or the 8-bit
//           blockwise form: per block of 16, S = fp16(max |A| / 127),
//           code = rne(A / S), A_i = code * S from here on)
//   r_c   = x_c - sum_i A_i B_ic                      lanes own channels 2l, 2l+1
//   (each sum left to right over its index, one chain per lane and sum)
//   kept  = rho largest |r_c|, ties to the lower channel (threshold search on
//           64-bit keys, one ballot pair per key bit)
//   S     = max |r| / 7,  code = rne(r_c / S) in [-7, 7],  scale = fp16(g S)
//   entries in storage order (|code| descending, then channel) via ballots.
// Every sum is rounded to float32 term by term, left to right; products of
// two fp16 values are exact in float32, so they are accumulated with fused
// multiply-adds (the same numbers as separately rounded products and sums) and
// nothing else is contracted, so the integer results are exact functions of
// the inputs.
#pragma once
#include "entry.h"
#include "internal.h"

namespace dwkv {
namespace cdev {

constexpr int D = kHeadDim;
constexpr int kBRow = D + 8;             // LDS basis row in halves: a 16-byte pad keeps
                                         // the per-lane row reads of the projection
                                         // spread over all banks
constexpr int kMaxRB = 128;

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ uint16_t float_to_half_bits(float v) {
  return __builtin_bit_cast(uint16_t, (_Float16)v);      // round to nearest even
}

// acc + x*b for fp16 values x, b.  Their product is exact in float32, so one
// fused multiply-add (a single mixed-precision instruction) gives the same
// number as the product rounded to float32 followed by a rounded sum.  The
// first term of a sum is fma(x, b, -0), which is the product itself, signed
// zero included.
__device__ __forceinline__ float fma_exact(float x_f16_valued, uint16_t b_bits, float acc) {
  return __builtin_fmaf(x_f16_valued, half_bits_to_float(b_bits), acc);
}

__device__ __forceinline__ int mbcnt64(unsigned long long m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// The per-(KV head, Z) views of the layer's arrays that one workgroup writes.
struct Slab {
  const uint8_t* code;         // [T]
  const uint32_t* off;         // [T+1]
  uint16_t* coef;              // fp16: key tiles (key_index) or value blocks (value_index)
  uint8_t* coef8;              // int8: key tiles [T16/16][rb/16][16][16] or value blocks [T16/16][rb][16]
  uint16_t* cscale;            // int8: block scales [rb/16][T]
  uint8_t* res_idx;            // [res_stride]
  uint8_t* res_val;            // [res_stride/2]
  uint16_t* res_scale;         // [T]
};

// Global inputs of one token, loaded ahead of its arithmetic.
struct TokenIn {
  uint32_t xw;                 // x[2 lane], x[2 lane + 1] (fp16 pair)
  uint32_t lvl;                // routed level index
  int64_t e0, e1;              // its residual entries [e0, e1)
  float g;                     // gate
};

// The wave's LDS: basis rows (rb rows of kBRow halves), its input vector [d],
// its coefficients [rb] (as rebuilt: fp16 values, or code * S), and its
// entries in storage order (channel byte, int4 nibble) [d].
struct CWave {
  const uint16_t* bas;
  float* xs;
  float* as;
  uint8_t* ech;
  uint8_t* ecode;
};

// What a compressed token leaves besides its stored factors: the routed rank
// (0 for rank 0 or a malformed level) and the stored scale bits fp16(g S).
struct TokOut {
  int rho;
  uint16_t scale;
};

__device__ __forceinline__ TokOut compress_token(const CompressArgs& a, const Slab& sl, const CWave& w, int lane,
                                                 int z, int64_t t, const TokenIn& in) {
#pragma clang fp contract(off)
  const int rb = a.rb;
  const float x0 = half_bits_to_float((uint16_t)(in.xw & 0xffffu));
  const float x1 = half_bits_to_float((uint16_t)(in.xw >> 16));
  const uint32_t lvl = in.lvl;
  const int64_t e0 = in.e0, e1 = in.e1;
  const float g = in.g;
  wave_lds_sync();                       // the previous token is done with the wave's arrays
  *reinterpret_cast<float2*>(&w.xs[2 * lane]) = make_float2(x0, x1);
  wave_lds_sync();

  // ---- coefficients: lane i sums x_j B_ij over the channels, left to right
  for (int i = lane; i < rb; i += 64) {
    const uint16_t* row = w.bas + i * kBRow;
    float s = -0.0f;
#pragma unroll 4
    for (int j0 = 0; j0 < D; j0 += 8) {
      const uint4 bw = *reinterpret_cast<const uint4*>(row + j0);
      const float4 xa = *reinterpret_cast<const float4*>(&w.xs[j0]);
      const float4 xb = *reinterpret_cast<const float4*>(&w.xs[j0 + 4]);
      const float xv8[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
      const uint32_t bw4[4] = {bw.x, bw.y, bw.z, bw.w};
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t w = bw4[j >> 1];
        const uint16_t bij = (uint16_t)((j & 1) ? (w >> 16) : (w & 0xffffu));
        s = fma_exact(xv8[j], bij, s);
      }
    }
    if (a.c8) {
      // 8-bit blockwise: the 16 lanes of coefficient block i / 16 share
      // S = fp16(max |A| / 127); code = rne(A / S) in [-127, 127] (0 when S
      // is 0); the residual below uses the rebuilt code * S (exact)
      float mx = fabsf(s);
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
      const uint16_t sb = float_to_half_bits(mx / 127.0f);
      const float S = half_bits_to_float(sb);
      int q = 0;
      if (S > 0.f) q = (int)fminf(fmaxf(__builtin_rintf(s / S), -127.f), 127.f);
      w.as[i] = (float)q * S;
      const int64_t pos = z == 0 ? (((t >> 4) * (rb >> 4) + (i >> 4)) << 8) + ((t & 15) << 4) + (i & 15)
                                 : (((t >> 4) * rb + i) << 4) + (t & 15);
      sl.coef8[pos] = (uint8_t)(int8_t)q;
      if ((i & 15) == 0) sl.cscale[(int64_t)(i >> 4) * a.T + t] = sb;
    } else {
      const uint16_t ab = float_to_half_bits(s);
      w.as[i] = half_bits_to_float(ab);
      if (z == 0)
        sl.coef[key_index(t, i, rb)] = ab;
      else
        sl.coef[value_index(t, i, rb)] = ab;
    }
  }
  wave_lds_sync();

  // ---- residual of channels c0 = 2 lane, c1 = 2 lane + 1: the basis term
  // summed over the basis rows, left to right
  float p0 = -0.0f, p1 = -0.0f;
#pragma unroll 2
  for (int i0 = 0; i0 < rb; i0 += 4) {
    const float4 a4 = *reinterpret_cast<const float4*>(&w.as[i0]);
    const float av[4] = {a4.x, a4.y, a4.z, a4.w};
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const uint32_t bw = *reinterpret_cast<const uint32_t*>(w.bas + (i0 + v) * kBRow + 2 * lane);
      if (a.c8) {
        // int8 rows code * S carry up to 18 significant bits: their products
        // with the fp16 basis are not exact in float32, so each product is
        // rounded on its own before the sum (no contraction in this function)
        p0 = p0 + av[v] * half_bits_to_float((uint16_t)(bw & 0xffffu));
        p1 = p1 + av[v] * half_bits_to_float((uint16_t)(bw >> 16));
      } else {
        p0 = fma_exact(av[v], (uint16_t)(bw & 0xffffu), p0);
        p1 = fma_exact(av[v], (uint16_t)(bw >> 16), p1);
      }
    }
  }
  const float r0 = x0 - p0, r1 = x1 - p1;

  // ---- routed rank of the token (shared by the window's layers and K/V)
  const int rho = lvl < (uint32_t)a.n_levels ? a.levels[lvl] : -1;
  const bool entries_ok = rho > 0 && e1 - e0 == rho && e1 <= a.res_stride && (e0 & 1) == 0;
  if (rho <= 0) {                        // rank 0 (or a malformed code): no entries, scale 0
    if (lane == 0) sl.res_scale[t] = 0;
    return TokOut{0, 0};
  }

  // ---- scale: max |r| over every channel / 7, gate folded in
  float mx = fmaxf(fabsf(r0), fabsf(r1));
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  const float S = mx / 7.0f;
  // g * S is rounded to float32 before the fp16 conversion (the value is
  // uniform; taking it through readfirstlane keeps the two roundings apart
  // instead of one mixed-precision multiply that would round once)
  const float gS = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, g * S)));
  const uint16_t gsb = float_to_half_bits(gS);
  if (lane == 0) sl.res_scale[t] = gsb;

  // ---- kept channels: the rho largest keys (|r| bits, then 127 - channel;
  // keys are distinct and below 2^38).  The rho-th largest key is the largest
  // threshold that at least rho keys reach; its bits are fixed from the top.
  const int c0 = 2 * lane, c1 = 2 * lane + 1;
  const unsigned long long k0 =
      ((unsigned long long)__builtin_bit_cast(uint32_t, fabsf(r0)) << 7) | (uint32_t)(D - 1 - c0);
  const unsigned long long k1 =
      ((unsigned long long)__builtin_bit_cast(uint32_t, fabsf(r1)) << 7) | (uint32_t)(D - 1 - c1);
  // Stops as soon as exactly rho keys reach the threshold (then they are the
  // rho largest); rho == d stops at once.
  unsigned long long thr = 0;
  if (rho < D) {
    for (int bit = 37; bit >= 0; --bit) {
      const unsigned long long cand = thr | (1ull << bit);
      const int cnt = __popcll(__ballot(k0 >= cand)) + __popcll(__ballot(k1 >= cand));
      if (cnt >= rho) thr = cand;
      if (cnt == rho) break;
    }
  }
  const bool sel0 = k0 >= thr, sel1 = k1 >= thr;

  // ---- codes and storage order (|code| descending, then channel ascending)
  int q0 = 0, q1 = 0;
  if (S > 0.f) {
    q0 = (int)fminf(fmaxf(__builtin_rintf(r0 / S), -7.f), 7.f);
    q1 = (int)fminf(fmaxf(__builtin_rintf(r1 / S), -7.f), 7.f);
  }
  const int m0 = q0 < 0 ? -q0 : q0, m1 = q1 < 0 ? -q1 : q1;
  int pos0 = 0, pos1 = 0;
#pragma unroll
  for (int v = 7; v >= 0; --v) {
    const unsigned long long b0 = __ballot(sel0 && m0 == v);
    const unsigned long long b1 = __ballot(sel1 && m1 == v);
    const int tot = __popcll(b0) + __popcll(b1);
    const int below = mbcnt64(b0) + mbcnt64(b1);   // channels of lower lanes in this bucket
    pos0 += m0 < v ? tot : (m0 == v ? below : 0);
    pos1 += m1 < v ? tot : (m1 == v ? below + ((sel0 && m0 == v) ? 1 : 0) : 0);
  }
  if (sel0) { w.ech[pos0] = (uint8_t)c0; w.ecode[pos0] = (uint8_t)(q0 & 0xF); }
  if (sel1) { w.ech[pos1] = (uint8_t)c1; w.ecode[pos1] = (uint8_t)(q1 & 0xF); }
  wave_lds_sync();
  if (!entries_ok) return TokOut{rho, gsb};   // offsets disagree with the rank: leave the slab alone
  for (int j = lane; j < rho / 2; j += 64) {
    const uint16_t ch2 = (uint16_t)(w.ech[2 * j] | (w.ech[2 * j + 1] << 8));
    *reinterpret_cast<uint16_t*>(sl.res_idx + e0 + 2 * j) = ch2;
    sl.res_val[(e0 >> 1) + j] = (uint8_t)(w.ecode[2 * j] | (w.ecode[2 * j + 1] << 4));
  }
  return TokOut{rho, gsb};
}

}  // namespace cdev
}  // namespace dwkv
