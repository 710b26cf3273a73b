// Online basis initialization (Sec. 3): a window's shared bases from a small
// randomized sketch of its prefill keys and values, per head and per Z.
// Y = Omega X, with X the window's prefill vectors of one head ((w T_b) x d)
// and Omega (r_b x (w T_b)) a caller-drawn random matrix; the basis is the
// Gram-Schmidt orthonormalization of Y's rows, rounded to fp16.
//
// Two launches: (1) split-K sketch partials, one workgroup per (4096-row
// chunk, head, Z), thread c owning channel c and accumulating r_b products in
// float64 (fp16 products are exact there); (2) per (head, Z), one wave sums
// the chunk partials in order and orthonormalizes the rows in float64,
// lanes owning channel pairs and wave shuffles forming the dot products.
#include "entry.h"
#include "internal.h"

namespace dwkv {
namespace {

constexpr int D = kHeadDim;
constexpr int kSkRows = 4096;            // sketch rows (tokens x layers) per workgroup

template <int RB>
__global__ __launch_bounds__(D) void sketch_partial_kernel(const SketchArgs a) {
  const int chunk = blockIdx.x, h = blockIdx.y, z = blockIdx.z, c = threadIdx.x;
  const int64_t N = (int64_t)a.w * a.n_tokens;
  const int64_t r0 = (int64_t)chunk * kSkRows, r1 = min(r0 + (int64_t)kSkRows, N);
  double acc[RB];
#pragma unroll
  for (int k = 0; k < RB; ++k) acc[k] = 0.0;
  for (int64_t r = r0; r < r1; ++r) {
    const int64_t l = r / a.n_tokens, t = r - l * a.n_tokens;
    const double xv = (double)half_bits_to_float(a.x[(((l * 2 + z) * a.n_tokens + t) * a.n_kv_heads + h) * D + c]);
    const uint16_t* om = a.omega + r * RB;             // the same row for every thread
#pragma unroll
    for (int k = 0; k < RB; ++k) acc[k] = __builtin_fma((double)half_bits_to_float(om[k]), xv, acc[k]);
  }
  double* out = a.part + (((int64_t)chunk * a.n_kv_heads + h) * 2 + z) * RB * D;
#pragma unroll
  for (int k = 0; k < RB; ++k) out[(int64_t)k * D + c] = acc[k];
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// grid (Hkv, 2), one wave: lane l owns channels 2l, 2l + 1
template <int RB>
__global__ __launch_bounds__(64) void sketch_orth_kernel(const SketchArgs a) {
  const int h = blockIdx.x, z = blockIdx.y, lane = threadIdx.x;
  const int c0 = 2 * lane;
  double* q = a.q + ((int64_t)h * 2 + z) * RB * D;      // orthonormal rows (float64)
  // Y rows: the chunk partials summed in chunk order
  double ymax = 0.0;
  for (int k = 0; k < RB; ++k) {
    double y0 = 0.0, y1 = 0.0;
    for (int ch = 0; ch < a.n_chunks; ++ch) {
      const double* p = a.part + (((int64_t)ch * a.n_kv_heads + h) * 2 + z) * RB * D + (int64_t)k * D + c0;
      y0 += p[0];
      y1 += p[1];
    }
    q[(int64_t)k * D + c0] = y0;
    q[(int64_t)k * D + c0 + 1] = y1;
    ymax = fmax(ymax, sqrt(wave_sum_d(y0 * y0 + y1 * y1)));
  }
  // the rows' own lanes rewrite them, so program order makes them visible
  const double floor_n = 1e-9 * ymax;
  uint16_t* bout = a.basis + ((int64_t)h * 2 + z) * RB * D;
  for (int i = 0; i < RB; ++i) {
    double v0 = q[(int64_t)i * D + c0], v1 = q[(int64_t)i * D + c0 + 1];
    for (int j = 0; j < i; ++j) {                       // modified Gram-Schmidt
      const double q0 = q[(int64_t)j * D + c0], q1 = q[(int64_t)j * D + c0 + 1];
      const double dot = wave_sum_d(v0 * q0 + v1 * q1);
      v0 -= dot * q0;
      v1 -= dot * q1;
    }
    const double n = sqrt(wave_sum_d(v0 * v0 + v1 * v1));
    if (n > floor_n && n > 0.0) { v0 /= n; v1 /= n; } else { v0 = 0.0; v1 = 0.0; }
    q[(int64_t)i * D + c0] = v0;
    q[(int64_t)i * D + c0 + 1] = v1;
    const uint32_t pk = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)(float)v0) |
                        ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)(float)v1) << 16);
    *reinterpret_cast<uint32_t*>(bout + (int64_t)i * D + c0) = pk;
  }
}

template <int RB>
hipError_t launch_sketch_rb(const SketchArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(sketch_partial_kernel<RB>, dim3(a.n_chunks, a.n_kv_heads, 2), dim3(D), 0, s, a);
  hipLaunchKernelGGL(sketch_orth_kernel<RB>, dim3(a.n_kv_heads, 2), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace

int sketch_chunks(int64_t rows) { return (int)((rows + kSkRows - 1) / kSkRows); }

hipError_t launch_sketch(const SketchArgs& a, hipStream_t s) {
  switch (a.rb) {
    case 16: return launch_sketch_rb<16>(a, s);
    case 32: return launch_sketch_rb<32>(a, s);
    case 48: return launch_sketch_rb<48>(a, s);
    case 64: return launch_sketch_rb<64>(a, s);
    case 80: return launch_sketch_rb<80>(a, s);
    case 96: return launch_sketch_rb<96>(a, s);
    case 112: return launch_sketch_rb<112>(a, s);
    case 128: return launch_sketch_rb<128>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace dwkv
