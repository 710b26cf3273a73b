// Router features from the decode (Sec. 3: the router scores a token by,
// among others, its accumulated attention mass and its maximum attention
// spike).  After a decode pass that stored every token's raw scores, this
// launch normalizes them with the merged softmax statistics of its sequence
// and query head, p = 2^(s - m*) / l*, and folds one layer's contribution into
// the window's feature table:
//   phi[t][0] += sum over the KV head's query heads of p
//   phi[t][1]  = max(phi[t][1], max over those heads of p)
// One workgroup per 256 packed tokens of one KV head; m* and l* of each
// sequence and query head are the merge's own (it merged the split partials
// just before and stored them).
#include "internal.h"

namespace dwkv {
namespace {

constexpr int kFT = 256;                 // tokens (threads) per workgroup

__device__ __forceinline__ int seq_at(const int32_t* cu, int batch, int64_t t) {
  int lo = 0, hi = batch;                // cu[lo] <= t < cu[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if ((int64_t)cu[mid] <= t) lo = mid; else hi = mid;
  }
  return lo;
}

template <int G>
__global__ __launch_bounds__(kFT) void features_kernel(const FeatArgs a) {
  __shared__ float mstar[G], linv[G];
  const int h = blockIdx.y, tid = threadIdx.x;
  const int64_t g0 = (int64_t)blockIdx.x * kFT;
  const int64_t gend = min(g0 + (int64_t)kFT, a.T);
  const int64_t t = g0 + tid;
  float s[G];
  if (t < gend) {
#pragma unroll
    for (int g = 0; g < G; ++g) s[g] = a.scores[((int64_t)h * a.T + t) * G + g];
  }
  for (int b = seq_at(a.cu, a.batch, g0); b < a.batch && (int64_t)a.cu[b] < gend; ++b) {
    const int64_t s0 = max(g0, (int64_t)a.cu[b]), s1 = min(gend, (int64_t)a.cu[b + 1]);
    if (s1 <= s0) continue;              // empty sequence (uniform)
    __syncthreads();                     // the previous sequence's statistics are read
    if (tid < G) {                       // the merge's statistics of (b, h, g)
      const float* ms = a.mstats + ((int64_t)b * a.n_q_heads + h * G + tid) * 2;
      mstar[tid] = ms[0];
      linv[tid] = 1.0f / ms[1];
    }
    __syncthreads();
    if (t >= s0 && t < s1) {
      float mass = 0.f, spike = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float p = exp2f(s[g] - mstar[g]) * linv[g];
        mass += p;
        spike = fmaxf(spike, p);
      }
      float* f = a.phi + ((int64_t)h * a.T + t) * 4;
      f[0] += mass;
      f[1] = fmaxf(f[1], spike);
    }
  }
}

// The probe-error feature: one thread per token of one probed KV head.  The
// error of (sequence, head) is the largest over the head's group members;
// `fresh` overwrites column 3, otherwise it keeps the maximum.
__global__ __launch_bounds__(kFT) void probe_feature_kernel(const ProbeFeatArgs a) {
  const int i = blockIdx.y;
  const int64_t t = (int64_t)blockIdx.x * kFT + threadIdx.x;
  if (t >= a.T) return;
  const int b = seq_at(a.cu, a.batch, t);
  const float* e = a.err + ((int64_t)b * a.n_heads + i) * a.G;
  float mx = e[0];
  for (int g = 1; g < a.G; ++g) mx = fmaxf(mx, e[g]);
  float* f = a.phi + ((int64_t)a.kv_heads[i] * a.T + t) * 4 + 3;
  *f = a.fresh ? mx : fmaxf(*f, mx);
}

}  // namespace

hipError_t launch_features(int g, const FeatArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  const dim3 grid((unsigned)((a.T + kFT - 1) / kFT), a.n_kv_heads);
  switch (g) {
    case 1: hipLaunchKernelGGL(features_kernel<1>, grid, dim3(kFT), 0, s, a); break;
    case 2: hipLaunchKernelGGL(features_kernel<2>, grid, dim3(kFT), 0, s, a); break;
    case 4: hipLaunchKernelGGL(features_kernel<4>, grid, dim3(kFT), 0, s, a); break;
    case 8: hipLaunchKernelGGL(features_kernel<8>, grid, dim3(kFT), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_probe_feature(const ProbeFeatArgs& a, hipStream_t s) {
  if (a.T <= 0 || a.n_heads <= 0) return hipSuccess;
  const dim3 grid((unsigned)((a.T + kFT - 1) / kFT), a.n_heads);
  hipLaunchKernelGGL(probe_feature_kernel, grid, dim3(kFT), 0, s, a);
  return hipGetLastError();
}

}  // namespace dwkv
