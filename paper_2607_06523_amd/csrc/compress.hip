// Append/compress (Sec. 3, the storage half of Eq. 1) on gfx950: dense
// key/value vectors of new tokens become their coefficient rows, routed
// residual entries and gate-folded scales, written in place into the cache.
//
// One workgroup (4 waves) takes up to 64 tokens of one (KV head, Z) and holds
// the window basis of the tokens' sequence in LDS; each wave compresses one
// token at a time:
//   A_i   = fp16( x_0 B_i0 + x_1 B_i1 + ... )        lane i, left to right over d
//   r_c   = x_c - (A_0 B_0c + A_1 B_1c + ...)         lanes own channels 2l, 2l+1
//   kept  = rho largest |r_c|, ties to the lower channel (rank by a 64-bit key)
//   S     = max |r| / 7,  code = rne(r_c / S) in [-7, 7],  scale = fp16(g S)
//   entries in storage order (|code| descending, then channel) via ballots.
// Every product and sum is rounded to float32 on its own (no contraction), so
// the integer results do not depend on the compiler's choice of instructions.
#include "entry.h"
#include "internal.h"

namespace dwkv {
namespace {

constexpr int D = kHeadDim;
constexpr int kCW = 4;                   // waves per workgroup
constexpr int kCT = 64;                  // tokens per workgroup
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

__device__ __forceinline__ int mbcnt64(unsigned long long m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

struct Smem {
  uint16_t bas[kMaxRB * kBRow];          // basis rows of (sequence, window, head, Z)
  float xs[kCW][D];                      // the wave's input vector
  float as[kCW][kMaxRB];                 // its fp16-rounded coefficients
  unsigned long long key[kCW][D];        // selection keys
  uint8_t ech[kCW][D];                   // entries in storage order: channel
  uint8_t ecode[kCW][D];                 //                          int4 nibble
};

// Largest b with cu[b] <= t (t < cu[batch]): the sequence holding packed token t.
__device__ __forceinline__ int sequence_of(const int32_t* cu, int batch, int64_t t) {
  int lo = 0, hi = batch;                // invariant: cu[lo] <= t < cu[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if ((int64_t)cu[mid] <= t) lo = mid; else hi = mid;
  }
  return lo;
}

// The per-(KV head, Z) views of the layer's arrays that one workgroup writes.
struct Slab {
  const uint8_t* code;         // [T]
  const uint32_t* off;         // [T+1]
  uint16_t* coef;              // keys [T][rb]; values [T16/16][rb][16]
  uint8_t* res_idx;            // [res_stride]
  uint8_t* res_val;            // [res_stride/2]
  uint16_t* res_scale;         // [T]
};

__device__ __forceinline__ void compress_token(const CompressArgs& a, const Slab& sl, Smem& sm, int wv,
                                               int lane, int h, int z, int64_t t) {
#pragma clang fp contract(off)
  const int64_t k = t - a.t0;
  const int rb = a.rb;
  const uint16_t* X = (z ? a.xv : a.xk) + (k * a.n_kv_heads + h) * D;
  const uint32_t xw = reinterpret_cast<const uint32_t*>(X)[lane];
  const float x0 = half_bits_to_float((uint16_t)(xw & 0xffffu));
  const float x1 = half_bits_to_float((uint16_t)(xw >> 16));
  wave_lds_sync();                       // the previous token is done with the wave's arrays
  *reinterpret_cast<float2*>(&sm.xs[wv][2 * lane]) = make_float2(x0, x1);
  wave_lds_sync();

  // ---- coefficients: lane i sums x_j B_ij left to right over the d channels
  for (int i = lane; i < rb; i += 64) {
    const uint16_t* row = sm.bas + i * kBRow;
    float acc = 0.f;
#pragma unroll 2
    for (int q = 0; q < D / 8; ++q) {
      const uint4 bw = *reinterpret_cast<const uint4*>(row + 8 * q);
      const float4 xa = *reinterpret_cast<const float4*>(&sm.xs[wv][8 * q]);
      const float4 xb = *reinterpret_cast<const float4*>(&sm.xs[wv][8 * q + 4]);
      const float xv8[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
      const uint32_t bw4[4] = {bw.x, bw.y, bw.z, bw.w};
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t w = bw4[j >> 1];
        const float bij = half_bits_to_float((uint16_t)((j & 1) ? (w >> 16) : (w & 0xffffu)));
        const float prod = xv8[j] * bij;
        acc = (q == 0 && j == 0) ? prod : acc + prod;
      }
    }
    const uint16_t ab = float_to_half_bits(acc);
    sm.as[wv][i] = half_bits_to_float(ab);
    if (z == 0)
      sl.coef[t * rb + i] = ab;
    else
      sl.coef[((t >> 4) * rb + i) * 16 + (t & 15)] = ab;
  }
  wave_lds_sync();

  // ---- residual of channels c0 = 2 lane, c1 = 2 lane + 1
  float p0 = 0.f, p1 = 0.f;
  for (int i0 = 0; i0 < rb; i0 += 4) {
    const float4 a4 = *reinterpret_cast<const float4*>(&sm.as[wv][i0]);
    const float av[4] = {a4.x, a4.y, a4.z, a4.w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint32_t bw = *reinterpret_cast<const uint32_t*>(sm.bas + (i0 + u) * kBRow + 2 * lane);
      const float q0 = av[u] * half_bits_to_float((uint16_t)(bw & 0xffffu));
      const float q1 = av[u] * half_bits_to_float((uint16_t)(bw >> 16));
      if (i0 == 0 && u == 0) { p0 = q0; p1 = q1; } else { p0 = p0 + q0; p1 = p1 + q1; }
    }
  }
  const float r0 = x0 - p0, r1 = x1 - p1;

  // ---- routed rank of the token (shared by the window's layers and K/V)
  const uint32_t lvl = sl.code[t];
  const int rho = lvl < (uint32_t)a.n_levels ? a.levels[lvl] : -1;
  const int64_t e0 = sl.off[t], e1 = sl.off[t + 1];
  const bool entries_ok = rho > 0 && e1 - e0 == rho && e1 <= a.res_stride && (e0 & 1) == 0;
  if (rho <= 0) {                        // rank 0 (or a malformed code): no entries, scale 0
    if (lane == 0) sl.res_scale[t] = 0;
    return;
  }

  // ---- scale: max |r| over every channel / 7, gate folded in
  float mx = fmaxf(fabsf(r0), fabsf(r1));
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  const float S = mx / 7.0f;
  const float g = a.gate ? a.gate[(int64_t)(z * a.n_kv_heads + h) * a.n + k] : 1.0f;
  // g * S is rounded to float32 before the fp16 conversion (the value is
  // uniform; taking it through readfirstlane keeps the two roundings apart
  // instead of one mixed-precision multiply that would round once)
  const float gS = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, g * S)));
  if (lane == 0) sl.res_scale[t] = float_to_half_bits(gS);

  // ---- kept channels: rank of each channel under (|r| descending, channel ascending)
  const int c0 = 2 * lane, c1 = 2 * lane + 1;
  const unsigned long long k0 =
      ((unsigned long long)__builtin_bit_cast(uint32_t, fabsf(r0)) << 7) | (uint32_t)(D - 1 - c0);
  const unsigned long long k1 =
      ((unsigned long long)__builtin_bit_cast(uint32_t, fabsf(r1)) << 7) | (uint32_t)(D - 1 - c1);
  sm.key[wv][c0] = k0;
  sm.key[wv][c1] = k1;
  wave_lds_sync();
  int rank0 = 0, rank1 = 0;
#pragma unroll 4
  for (int c = 0; c < D; c += 2) {
    const ulonglong2 kk = *reinterpret_cast<const ulonglong2*>(&sm.key[wv][c]);
    rank0 += (kk.x > k0) + (kk.y > k0);
    rank1 += (kk.x > k1) + (kk.y > k1);
  }
  const bool sel0 = rank0 < rho, sel1 = rank1 < rho;

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
  if (sel0) { sm.ech[wv][pos0] = (uint8_t)c0; sm.ecode[wv][pos0] = (uint8_t)(q0 & 0xF); }
  if (sel1) { sm.ech[wv][pos1] = (uint8_t)c1; sm.ecode[wv][pos1] = (uint8_t)(q1 & 0xF); }
  wave_lds_sync();
  if (!entries_ok) return;               // offsets disagree with the rank: leave the slab alone
  for (int j = lane; j < rho / 2; j += 64) {
    const uint16_t ch2 = (uint16_t)(sm.ech[wv][2 * j] | (sm.ech[wv][2 * j + 1] << 8));
    *reinterpret_cast<uint16_t*>(sl.res_idx + e0 + 2 * j) = ch2;
    sl.res_val[(e0 >> 1) + j] = (uint8_t)(sm.ecode[wv][2 * j] | (sm.ecode[wv][2 * j + 1] << 4));
  }
}

// grid (ceil(n / 64), Hkv, 2)
__global__ __launch_bounds__(kCW * 64) void compress_kernel(const CompressArgs a) {
  __shared__ __align__(16) Smem sm;
  const int h = blockIdx.y, z = blockIdx.z;
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t slab = (int64_t)z * a.n_kv_heads + h;
  Slab sl;
  sl.code = a.code + (int64_t)h * a.T;
  sl.off = a.off + (int64_t)h * (a.T + 1);
  sl.coef = z == 0 ? a.coef_k + (int64_t)h * a.T * a.rb : a.coef_v + (int64_t)h * a.T16 * a.rb;
  sl.res_idx = a.res_idx + slab * a.res_stride;
  sl.res_val = a.res_val + slab * (a.res_stride / 2);
  sl.res_scale = a.res_scale + slab * a.T;
  const int64_t c0 = a.t0 + (int64_t)blockIdx.x * kCT;
  const int64_t c1 = min(c0 + (int64_t)kCT, a.t0 + a.n);
  const int rb = a.rb;
  for (int b = sequence_of(a.cu, a.batch, c0); b < a.batch && (int64_t)a.cu[b] < c1; ++b) {
    const int64_t s0 = max(c0, (int64_t)a.cu[b]), s1 = min(c1, (int64_t)a.cu[b + 1]);
    if (s1 <= s0) continue;              // empty sequence (uniform over the workgroup)
    __syncthreads();                     // every wave is done with the previous basis
    const uint16_t* src = a.basis + (int64_t)b * a.basis_b_stride + (int64_t)(h * 2 + z) * rb * D;
    for (int e = threadIdx.x; e < rb * (D / 8); e += kCW * 64) {
      const int i = e / (D / 8), q = e % (D / 8);
      *reinterpret_cast<uint4*>(sm.bas + i * kBRow + 8 * q) =
          *reinterpret_cast<const uint4*>(src + (int64_t)i * D + 8 * q);
    }
    __syncthreads();
    for (int64_t t = s0 + wv; t < s1; t += kCW) compress_token(a, sl, sm, wv, lane, h, z, t);
  }
}

}  // namespace

hipError_t launch_compress(const CompressArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  const unsigned nb = (unsigned)((a.n + kCT - 1) / kCT);
  hipLaunchKernelGGL(compress_kernel, dim3(nb, a.n_kv_heads, 2), dim3(kCW * 64), 0, s, a);
  return hipGetLastError();
}

}  // namespace dwkv
