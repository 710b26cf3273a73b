// Router (Eq. 2) with its residual-offset scan (over the whole packed axis or a
// token range that continues an existing table), the residual-map test hook and
// the layout validator (gfx950).
#include "entry.h"
#include "internal.h"

namespace dwkv {
namespace {

constexpr int D = kHeadDim;
constexpr int kRT = 256;                                  // route block threads
constexpr int kPerThread = kRouteTokensPerBlock / kRT;   // 4 tokens per thread

// Router score, float32, left to right, each product and sum rounded on its own
// (no fused multiply-add), so it reproduces bit for bit on any IEEE machine.
__device__ __forceinline__ float router_score(const float4 u, const float4 f) {
#pragma clang fp contract(off)
  float z = u.x * f.x;
  z = z + u.y * f.y;
  z = z + u.z * f.z;
  z = z + u.w * f.w;
  return z;
}

__device__ __forceinline__ uint32_t block_sum(uint32_t v, uint32_t* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (lane == 0) red[wv] = v;
  __syncthreads();
  uint32_t t = 0;
  for (int i = 0; i < kRT / 64; ++i) t += red[i];
  return t;
}

// Exclusive prefix over the block's threads (kRT threads); returns the block total in *total.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* red, uint32_t* total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  uint32_t inc = v;
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t n = __shfl_up(inc, o);
    if (lane >= o) inc += n;
  }
  if (lane == 63) red[wv] = inc;
  __syncthreads();
  uint32_t before = 0, all = 0;
  for (int i = 0; i < kRT / 64; ++i) {
    if (i < wv) before += red[i];
    all += red[i];
  }
  *total = all;
  return before + inc - v;
}

// Level codes of this thread's tokens of block `blk`, written to a.code; the
// routed ranks go to rho[] (0 past the range).  Returns their sum.
__device__ __forceinline__ uint32_t route_block_tokens(const RouteArgs& a, int mh, int blk,
                                                       uint32_t (&rho)[kPerThread]) {
  const int m = mh / a.n_kv_heads;
  const float4 u = *reinterpret_cast<const float4*>(a.u + 4 * m);
  const int nth = a.n_levels - 1;
  float th[DWKV_MAX_LEVELS - 1];
#pragma unroll
  for (int j = 0; j < DWKV_MAX_LEVELS - 1; ++j) th[j] = j < nth ? a.theta[m * nth + j] : 0.f;
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int64_t t = a.t0 + (int64_t)blk * kRouteTokensPerBlock + threadIdx.x * kPerThread + i;
    rho[i] = 0u;
    if (t < a.t0 + a.n) {
      const float4 f = *reinterpret_cast<const float4*>(a.phi + ((int64_t)mh * a.T + t) * 4);
      const float z = router_score(u, f);
      int k = 0;
#pragma unroll
      for (int j = 0; j < DWKV_MAX_LEVELS - 1; ++j) k += (j < nth && z > th[j]) ? 1 : 0;
      a.code[(int64_t)mh * a.T + t] = (uint8_t)k;
      rho[i] = (uint32_t)a.levels[k];
      sum += rho[i];
    }
  }
  return sum;
}

// Offsets of this thread's tokens: off[t+1] = carry + (ranks of earlier tokens) + rho_t,
// with `carry` the offset of the block's first token.
__device__ __forceinline__ void route_write_offsets(const RouteArgs& a, int mh, int blk, uint32_t carry,
                                                    const uint32_t (&rho)[kPerThread], uint32_t* red) {
  uint32_t mine = 0;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) mine += rho[i];
  uint32_t total;
  uint32_t run = carry + block_exclusive_scan(mine, red, &total);
  uint32_t* off = a.off + (int64_t)mh * (a.T + 1);
  if (a.t0 == 0 && blk == 0 && threadIdx.x == 0) off[0] = 0u;
  const int64_t end = a.t0 + a.n;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int64_t t = a.t0 + (int64_t)blk * kRouteTokensPerBlock + threadIdx.x * kPerThread + i;
    run += rho[i];
    if (t < end) off[t + 1] = run;
  }
}

// A range of at most one block of tokens in one launch: codes, scan, offsets.  grid (M*Hkv)
__global__ __launch_bounds__(kRT) void route_small_kernel(const RouteArgs a) {
  __shared__ uint32_t red[kRT / 64];
  const int mh = blockIdx.x;
  uint32_t rho[kPerThread];
  route_block_tokens(a, mh, 0, rho);
  const uint32_t carry = a.t0 == 0 ? 0u : a.off[(int64_t)mh * (a.T + 1) + a.t0];
  route_write_offsets(a, mh, 0, carry, rho, red);
}

// Level codes and per-block rank sums.  grid (nblk, M*Hkv)
__global__ __launch_bounds__(kRT) void route_codes_kernel(const RouteArgs a) {
  __shared__ uint32_t red[kRT / 64];
  const int mh = blockIdx.y;
  uint32_t rho[kPerThread];
  const uint32_t sum = route_block_tokens(a, mh, blockIdx.x, rho);
  const uint32_t tot = block_sum(sum, red);
  if (threadIdx.x == 0) a.bsum[(int64_t)mh * a.nblk + blockIdx.x] = tot;
}

// Exclusive scan of the block sums of one (window, head).  grid (M*Hkv)
__global__ __launch_bounds__(kRT) void route_block_scan_kernel(const RouteArgs a) {
  __shared__ uint32_t red[kRT / 64];
  const int mh = blockIdx.x;
  uint32_t carry = 0;
  for (int b0 = 0; b0 < a.nblk; b0 += kRT) {
    const int b = b0 + threadIdx.x;
    const uint32_t v = b < a.nblk ? a.bsum[(int64_t)mh * a.nblk + b] : 0u;
    uint32_t total;
    const uint32_t ex = block_exclusive_scan(v, red, &total);
    if (b < a.nblk) a.bpre[(int64_t)mh * a.nblk + b] = carry + ex;
    carry += total;
    __syncthreads();
  }
}

// Offsets of a multi-block range from the codes and the scanned block sums.
__global__ __launch_bounds__(kRT) void route_offsets_kernel(const RouteArgs a) {
  __shared__ uint32_t red[kRT / 64];
  const int mh = blockIdx.y;
  const int64_t end = a.t0 + a.n;
  uint32_t rho[kPerThread];
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int64_t t = a.t0 + (int64_t)blockIdx.x * kRouteTokensPerBlock + threadIdx.x * kPerThread + i;
    rho[i] = t < end ? (uint32_t)a.levels[a.code[(int64_t)mh * a.T + t]] : 0u;
  }
  // carry-in: the offset of the range's first token (0 for a table that starts here)
  const uint32_t base = a.t0 == 0 ? 0u : a.off[(int64_t)mh * (a.T + 1) + a.t0];
  route_write_offsets(a, mh, blockIdx.x, base + a.bpre[(int64_t)mh * a.nblk + blockIdx.x], rho, red);
}

// Budget routing (two levels, Eq. 2 with tau chosen for a memory budget): the
// n = floor((E - N rho_min) / (rho_max - rho_min)) tokens of largest score z
// get level 1, ties to the lower token.  Keys are (order-preserving bits of z,
// then the complement of the token's index), all distinct; the n-th largest
// is found one byte at a time from the top (a 256-bin histogram of the
// candidates that match the bytes fixed so far), then codes and offsets are
// written in one ordered sweep.  grid (M*Hkv)
__global__ __launch_bounds__(kRT) void route_budget_kernel(const RouteArgs a) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t red[kRT / 64];
  __shared__ unsigned long long s_prefix;
  __shared__ int64_t s_rem;
  const int mh = blockIdx.x;
  const int m = mh / a.n_kv_heads;
  const int64_t N = a.n;
  unsigned long long* keys = a.keys + (int64_t)mh * a.T;
  const float4 u = *reinterpret_cast<const float4*>(a.u + 4 * m);
  for (int64_t i = threadIdx.x; i < N; i += kRT) {
    const int64_t t = a.t0 + i;
    const float4 f = *reinterpret_cast<const float4*>(a.phi + ((int64_t)mh * a.T + t) * 4);
    const float z = router_score(u, f) + 0.0f;           // -0 -> +0: equal scores tie
    const uint32_t b = __float_as_uint(z);
    const uint32_t ord = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
    keys[i] = ((unsigned long long)ord << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)i);
  }
  const int64_t rmin = a.levels[0], rmax = a.levels[1];
  int64_t n = rmax > rmin ? (a.entries[mh] - N * rmin) / (rmax - rmin) : 0;
  if (a.entries[mh] - N * rmin < 0) n = 0;
  n = min(max(n, (int64_t)0), N);
  unsigned long long thr = ~0ull;                        // n == 0: nothing reaches it
  if (n == N) {
    thr = 0;
  } else if (n > 0) {
    if (threadIdx.x == 0) { s_prefix = 0; s_rem = n; }
    unsigned long long mask = 0;
    for (int sh = 56; sh >= 0; sh -= 8) {
      __syncthreads();                                   // keys written / previous pass read
      hist[threadIdx.x] = 0u;                            // kRT == 256 bins
      __syncthreads();
      const unsigned long long prefix = s_prefix;
      for (int64_t i = threadIdx.x; i < N; i += kRT) {
        const unsigned long long k = keys[i];
        if ((k & mask) == prefix) atomicAdd(&hist[(k >> sh) & 255u], 1u);
      }
      __syncthreads();
      if (threadIdx.x == 0) {                            // the byte of the rem-th largest candidate
        int64_t rem = s_rem, above = 0;
        int d = 255;
        for (; d > 0; --d) {
          if (above + hist[d] >= rem) break;
          above += hist[d];
        }
        s_rem = rem - above;
        s_prefix = prefix | ((unsigned long long)d << sh);
      }
      mask |= 255ull << sh;
    }
    __syncthreads();
    thr = s_prefix;                                      // the n-th largest key
  }
  // codes and offsets, in token order, continuing the table from off[t0]
  uint32_t* off = a.off + (int64_t)mh * (a.T + 1);
  uint8_t* code = a.code + (int64_t)mh * a.T;
  uint32_t carry = a.t0 == 0 ? 0u : off[a.t0];
  __syncthreads();
  if (a.t0 == 0 && threadIdx.x == 0) off[0] = 0u;
  for (int64_t c0 = 0; c0 < N; c0 += kRouteTokensPerBlock) {
    uint32_t rho[kPerThread], mine = 0;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int64_t j = c0 + threadIdx.x * kPerThread + i;
      rho[i] = 0u;
      if (j < N) {
        const int k = keys[j] >= thr ? 1 : 0;
        code[a.t0 + j] = (uint8_t)k;
        rho[i] = (uint32_t)a.levels[k];
      }
      mine += rho[i];
    }
    uint32_t total;
    uint32_t run = carry + block_exclusive_scan(mine, red, &total);
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int64_t j = c0 + threadIdx.x * kPerThread + i;
      run += rho[i];
      if (j < N) off[a.t0 + j + 1] = run;
    }
    carry += total;
    __syncthreads();                                     // red[] is reused by the next chunk
  }
}

// One thread per token: dense g*R row of the token.
__global__ __launch_bounds__(256) void residual_map_kernel(const uint32_t* off, const uint8_t* idx,
                                                           const uint8_t* val, const uint16_t* scale,
                                                           int64_t t0, int64_t t1, int64_t slab_len,
                                                           float* dense) {
  const int64_t t = t0 + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= t1) return;
  float* row = dense + (t - t0) * D;
  for (int c = 0; c < D; ++c) row[c] = 0.f;
  const float s = half_bits_to_float(scale[t]);
  const int64_t e0 = off[t], e1 = off[t + 1];
  const int64_t end = min(min(e1, e0 + D), slab_len);   // bounded even for a corrupt table
  for (int64_t e = e0; e < end; ++e)
    row[idx[e] & (D - 1)] = s * (float)entry_code(val[e >> 1], e);
}

struct ValidateArgs {
  const uint8_t* code;
  const uint32_t* off;
  const uint8_t* idx;
  const uint8_t* val;
  unsigned long long* bad;
  int64_t T, res_stride;
  int32_t n_kv_heads, window, n_levels;
  int32_t levels[DWKV_MAX_LEVELS];
};

__device__ __forceinline__ void report(unsigned long long* bad, int64_t mh, int64_t T, int64_t t, int kind) {
  atomicMin(bad, (unsigned long long)(((mh * (T + 1) + t) << 3) | kind));
}

__global__ void fill_u64_kernel(unsigned long long* p, unsigned long long v) { *p = v; }

// grid (ceil((T+1)/256), M*Hkv)
__global__ __launch_bounds__(256) void validate_kernel(const ValidateArgs a) {
  const int64_t mh = blockIdx.y;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t > a.T) return;
  const uint32_t* off = a.off + mh * (a.T + 1);
  if (t == a.T) {              // global checks ride on the extra thread
    if (off[0] != 0u || (int64_t)off[a.T] + kResTailPad > a.res_stride) report(a.bad, mh, a.T, t, 7);
    return;
  }
  const uint32_t o0 = off[t], o1 = off[t + 1];
  const uint32_t k = a.code[mh * a.T + t];
  if (k >= (uint32_t)a.n_levels) { report(a.bad, mh, a.T, t, 2); return; }
  if (o1 < o0 || o1 - o0 != (uint32_t)a.levels[k]) { report(a.bad, mh, a.T, t, 1); return; }
  if ((int64_t)o1 > a.res_stride) { report(a.bad, mh, a.T, t, 7); return; }
  const int m = (int)(mh / a.n_kv_heads), h = (int)(mh % a.n_kv_heads);
  for (int li = 0; li < a.window; ++li) {
    const int l = m * a.window + li;
    for (int z = 0; z < 2; ++z) {
      const int64_t slab = ((int64_t)(l * 2 + z) * a.n_kv_heads + h);
      const uint8_t* ix = a.idx + slab * a.res_stride;
      const uint8_t* vl = a.val + slab * (a.res_stride / 2);
      uint32_t seen[4] = {0u, 0u, 0u, 0u};
      int prev_abs = 8, prev_c = -1;
      for (uint32_t e = o0; e < o1; ++e) {
        const int c = ix[e];
        if (c >= D) { report(a.bad, mh, a.T, t, 3); return; }
        if (seen[c >> 5] & (1u << (c & 31))) { report(a.bad, mh, a.T, t, 4); return; }
        seen[c >> 5] |= 1u << (c & 31);
        const int code = entry_code(vl[e >> 1], e);
        if (code == -8) { report(a.bad, mh, a.T, t, 5); return; }
        const int ab = code < 0 ? -code : code;
        if (ab > prev_abs || (ab == prev_abs && c < prev_c)) { report(a.bad, mh, a.T, t, 6); return; }
        prev_abs = ab;
        prev_c = c;
      }
    }
  }
}

}  // namespace

hipError_t launch_route(const RouteArgs& a, int n_mh, hipStream_t s) {
  if (a.nblk <= 1) {                     // one block per (window, head): a single launch
    hipLaunchKernelGGL(route_small_kernel, dim3(n_mh), dim3(kRT), 0, s, a);
  } else {
    hipLaunchKernelGGL(route_codes_kernel, dim3(a.nblk, n_mh), dim3(kRT), 0, s, a);
    hipLaunchKernelGGL(route_block_scan_kernel, dim3(n_mh), dim3(kRT), 0, s, a);
    hipLaunchKernelGGL(route_offsets_kernel, dim3(a.nblk, n_mh), dim3(kRT), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_route_budget(const RouteArgs& a, int n_mh, hipStream_t s) {
  hipLaunchKernelGGL(route_budget_kernel, dim3(n_mh), dim3(kRT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_residual_map(const uint32_t* off, const uint8_t* idx, const uint8_t* val,
                               const uint16_t* scale, int64_t t0, int64_t t1, int64_t slab_len,
                               float* dense, hipStream_t s) {
  const int64_t n = t1 - t0;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(residual_map_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, off,
                     idx, val, scale, t0, t1, slab_len, dense);
  return hipGetLastError();
}

hipError_t launch_validate(const dwkv_dims* d, const dwkv_cache* c, unsigned long long* bad,
                           hipStream_t s) {
  ValidateArgs a;
  a.code = c->rank_code;
  a.off = c->res_off;
  a.idx = c->res_idx;
  a.val = c->res_val;
  a.bad = bad;
  a.T = d->total_tokens;
  a.res_stride = d->res_stride;
  a.n_kv_heads = d->n_kv_heads;
  a.window = d->window;
  a.n_levels = d->n_levels;
  for (int i = 0; i < DWKV_MAX_LEVELS; ++i) a.levels[i] = d->levels[i];
  const int n_mh = (d->n_layers / d->window) * d->n_kv_heads;
  hipLaunchKernelGGL(fill_u64_kernel, dim3(1), dim3(1), 0, s, bad, ~0ull);
  hipLaunchKernelGGL(validate_kernel, dim3((unsigned)((a.T + 1 + 255) / 256), n_mh), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace dwkv
