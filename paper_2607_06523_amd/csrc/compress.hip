// Append/compress (Sec. 3, the storage half of Eq. 1) on gfx950: dense
// key/value vectors of new tokens become their coefficient rows, routed
// residual entries and gate-folded scales, written in place into the cache.
//
// One workgroup (4 waves) takes up to 64 tokens of one (KV head, Z) and holds
// the window basis of the tokens' sequence in LDS; each wave compresses one
// token at a time (the arithmetic of one token is in compress_dev.h).
#include "compress_dev.h"

namespace dwkv {
namespace {

using namespace cdev;

constexpr int kCW = 4;                   // waves per workgroup
constexpr int kCT = 64;                  // tokens per workgroup
struct Smem {
  uint16_t bas[kMaxRB * kBRow];          // basis rows of (sequence, window, head, Z)
  float xs[kCW][D];                      // the wave's input vector
  float as[kCW][kMaxRB];                 // its fp16-rounded coefficients
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

__device__ __forceinline__ TokenIn load_token(const CompressArgs& a, const Slab& sl, int lane, int h, int z,
                                              int64_t t) {
  const int64_t k = t - a.t0;
  const uint16_t* X = (z ? a.xv : a.xk) + (k * a.n_kv_heads + h) * D;
  TokenIn in;
  in.xw = reinterpret_cast<const uint32_t*>(X)[lane];
  in.lvl = sl.code[t];
  in.e0 = sl.off[t];
  in.e1 = sl.off[t + 1];
  in.g = a.gate ? a.gate[(int64_t)(z * a.n_kv_heads + h) * a.gate_ld + a.gate_k0 + k] : 1.0f;
  return in;
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
  sl.coef = (z == 0 ? a.coef_k : a.coef_v) + (int64_t)h * a.T16 * a.rb;
  sl.coef8 = reinterpret_cast<uint8_t*>(z == 0 ? a.coef_k : a.coef_v) + (int64_t)h * a.T16 * a.rb;
  sl.cscale = a.c8 ? (z == 0 ? a.cscale_k : a.cscale_v) + (int64_t)h * (a.rb / 16) * a.T : nullptr;
  sl.res_idx = a.res_idx + slab * a.res_stride;
  sl.res_val = a.res_val + slab * (a.res_stride / 2);
  sl.res_scale = a.res_scale + slab * a.T;
  const int64_t c0 = a.t0 + (int64_t)blockIdx.x * kCT;
  const int64_t c1 = min(c0 + (int64_t)kCT, a.t0 + a.n);
  const int rb = a.rb;
  for (int b = sequence_of(a.cu, a.batch, c0); b < a.batch && (int64_t)a.cu[b] < c1; ++b) {
    const int64_t s0 = max(c0, (int64_t)a.cu[b]), s1 = min(c1, (int64_t)a.cu[b + 1]);
    if (s1 <= s0) continue;              // empty sequence (uniform over the workgroup)
    int64_t t = s0 + wv;
    TokenIn cur = {};
    if (t < s1) cur = load_token(a, sl, lane, h, z, t);   // in flight while the basis loads
    __syncthreads();                     // every wave is done with the previous basis
    const uint16_t* src = a.basis + (int64_t)b * a.basis_b_stride + (int64_t)(h * 2 + z) * rb * D;
    for (int e = threadIdx.x; e < rb * (D / 8); e += kCW * 64) {
      const int i = e / (D / 8), q = e % (D / 8);
      *reinterpret_cast<uint4*>(sm.bas + i * kBRow + 8 * q) =
          *reinterpret_cast<const uint4*>(src + (int64_t)i * D + 8 * q);
    }
    __syncthreads();
    for (; t < s1; t += kCW) {
      TokenIn nxt = cur;
      if (t + kCW < s1) nxt = load_token(a, sl, lane, h, z, t + kCW);
      compress_token(a, sl, CWave{sm.bas, sm.xs[wv], sm.as[wv], sm.ech[wv], sm.ecode[wv]}, lane, z, t, cur);
      cur = nxt;
    }
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
