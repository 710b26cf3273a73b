// Materialization of the rebuilt cache (Eq. 1 written out to HBM) on gfx950:
// K_hat = A^K B^K + g R^K and V_hat = A^V B^V + g R^V for every token and KV
// head of one layer, rounded once to fp16.  It exists for the unfused
// comparison path (rebuild, then dense attention over the rebuilt cache), the
// design the fused decode avoids.
//
// One workgroup of 2 waves takes 256 packed tokens (16 blocks of 16) of one
// (KV head, Z).  It stages the basis of each sequence the tokens belong to in
// LDS, transposed (channel-major, so an MFMA B fragment is one 8-byte read),
// and the waves take alternate blocks, each computing [16 tokens x 128 channels] on
// v_mfma_f32_16x16x16f16: coefficient rows as the A operand, basis columns as
// B, 8 output tiles of 16 channels.  The tile goes through LDS (fp32), the
// token's routed residual channels are added there by the token's lane, and
// the rows are rounded to fp16 and stored: keys row-major, values in the
// 16-token blocked layout (padding tokens of the last block zeroed).
#include "entry.h"
#include "internal.h"

namespace dwkv {
namespace {

constexpr int D = kHeadDim;
constexpr int kMW = 2;                   // waves per workgroup
constexpr int kMTok = 256;               // tokens per workgroup (16 blocks of 16; waves alternate)
constexpr int kMaxEnt = 16;              // entries of a token read in one batch (4 per lane of its column)

typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int seq_of(const int32_t* cu, int batch, int64_t t) {
  int lo = 0, hi = batch;                // cu[lo] <= t < cu[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if ((int64_t)cu[mid] <= t) lo = mid; else hi = mid;
  }
  return lo;
}

__device__ __forceinline__ uint32_t pack_half2(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)lo) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)hi) << 16);
}

template <int RB>
struct MSmem {
  static constexpr int BT = RB + 4;      // transposed basis row (halves); the pad spreads the
                                         // 16 lanes of a fragment read over distinct banks
  alignas(16) uint16_t bt[D * BT];       // bt[c][k] = B[k][c]
  alignas(16) float tile[kMW][16][D + 4];
};

// Inputs of one 16-token block a wave loads ahead of its arithmetic.
template <int RB>
struct MBlock {
  h4 af[RB / 16];                        // coefficient fragments of token w0 + r
  uint32_t e0, e1;                       // entry range of token w0 + r
  uint32_t sbits;                        // its gate-folded scale (fp16 bits)
  uint32_t chs[kMaxEnt / 4], cbs[kMaxEnt / 4];   // entries grp + 4u: channel byte, code byte
};

// First stage: coefficients, offsets and scale of block [w0, w0+16), rows
// [a0, a1) (zero outside).
template <int RB>
__device__ __forceinline__ void mat_load(MBlock<RB>& m, int64_t w0, int64_t a0, int64_t a1, int z, int lane,
                                         const uint16_t* ck, const uint16_t* cv, const uint32_t* off,
                                         const uint16_t* scale) {
  constexpr int NS = RB / 16;
  const int grp = lane >> 4, r = lane & 15;
  const int64_t t = w0 + r;
  const bool mine = t >= a0 && t < a1;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    uint2 w = make_uint2(0u, 0u);
    if (mine) {
      if (z == 0) {
        w = *reinterpret_cast<const uint2*>(ck + key_index(t, 16 * s + 4 * grp, RB));
      } else {                          // 4 channels of token t, 8 elements apart
        const uint16_t* p = cv + value_index(t, 16 * s + 4 * grp, RB);
        w.x = (uint32_t)p[0] | ((uint32_t)p[8] << 16);
        w.y = (uint32_t)p[16] | ((uint32_t)p[24] << 16);
      }
    }
    m.af[s] = __builtin_bit_cast(h4, w);
  }
  m.e0 = m.e1 = 0;
  m.sbits = 0;
  if (mine) {
    m.e0 = off[t];
    m.e1 = off[t + 1];
    m.sbits = scale[t];
  }
}

// Second stage: the block's residual entries (needs the offsets).  The four
// lanes of a token's column share its entries: lane group grp takes entries
// grp, grp + 4, ...
template <int RB>
__device__ __forceinline__ uint32_t mat_entries(MBlock<RB>& m, const MatArgs& a, const uint8_t* idx,
                                                const uint8_t* val, int lane) {
  const uint32_t grp = (uint32_t)lane >> 4;
  uint32_t rho = m.e1 > m.e0 ? min(m.e1 - m.e0, (uint32_t)D) : 0u;
  if (m.e0 + rho > (uint64_t)a.res_stride) rho = 0;    // a malformed table adds nothing
#pragma unroll
  for (int u = 0; u < kMaxEnt / 4; ++u) {
    const uint32_t j = grp + 4u * u;
    m.chs[u] = j < rho ? idx[m.e0 + j] : 0u;
    m.cbs[u] = j < rho ? val[(m.e0 + j) >> 1] : 0u;
  }
  return rho;
}

// One wave, one 16-token block [w0, w0+16): rows [a0, a1) of it belong to the
// sequence whose basis is in LDS; they are computed, completed with their
// residual channels and stored (other rows untouched).
template <int RB>
__device__ __forceinline__ void mat_block(const MatArgs& a, MSmem<RB>& sm, float (*tile)[D + 4], int64_t w0,
                                          int64_t a0, int64_t a1, int z, int lane, const MBlock<RB>& m,
                                          uint32_t rho, const uint8_t* idx, const uint8_t* val,
                                          uint16_t* kout, uint16_t* vout) {
  constexpr int NS = RB / 16;
  constexpr int BT = MSmem<RB>::BT;
  const int grp = lane >> 4, r = lane & 15;
  const uint32_t e0 = m.e0;
  const float gs = half_bits_to_float((uint16_t)m.sbits);
  wave_lds_sync();                     // the previous block's stores have read the tile
  // 8 output tiles of 16 channels
#pragma unroll
  for (int nt = 0; nt < D / 16; ++nt) {
    f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const h4 bf = *reinterpret_cast<const h4*>(&sm.bt[(16 * nt + r) * BT + 16 * s + 4 * grp]);
      acc = __builtin_amdgcn_mfma_f32_16x16x16f16(m.af[s], bf, acc, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) tile[4 * grp + j][16 * nt + r] = acc[j];
  }
  wave_lds_sync();
  // routed residual channels: the four lanes of a token's column add
  // g*s*code at its channels (distinct channels, so no two lanes meet)
  if (rho > 0) {
#pragma unroll
    for (int u = 0; u < kMaxEnt / 4; ++u) {
      const uint32_t j = (uint32_t)grp + 4u * u;
      if (j < rho) tile[r][m.chs[u] & (D - 1)] += gs * (float)entry_code(m.cbs[u], (int64_t)(e0 + j));
    }
    for (uint32_t j = kMaxEnt + grp; j < rho; j += 4) {   // ranks above 16
      const uint32_t e = e0 + j;
      tile[r][idx[e] & (D - 1)] += gs * (float)entry_code(val[e >> 1], (int64_t)e);
    }
  }
  wave_lds_sync();
  // store the rows of this sequence, rounded once to fp16
  if (z == 0) {
    const int tr = lane >> 2, q = lane & 3;          // token row, 32-channel quarter
    const int64_t tt = w0 + tr;
    if (tt >= a0 && tt < a1) {
      uint4* dst = reinterpret_cast<uint4*>(kout + tt * D + 32 * q);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float4 x0 = *reinterpret_cast<const float4*>(&tile[tr][32 * q + 8 * u]);
        const float4 x1 = *reinterpret_cast<const float4*>(&tile[tr][32 * q + 8 * u + 4]);
        dst[u] = make_uint4(pack_half2(x0.x, x0.y), pack_half2(x0.z, x0.w), pack_half2(x1.x, x1.y),
                            pack_half2(x1.z, x1.w));
      }
    }
  } else {
    const bool full = a0 == w0 && a1 == w0 + 16;
#pragma unroll
    for (int cc = 0; cc < 2; ++cc) {
      const int c = 2 * lane + cc;
      uint16_t* dst = vout + ((w0 >> 4) * D + c) * 16;
      if (full) {
        uint32_t pk[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) pk[u] = pack_half2(tile[2 * u][c], tile[2 * u + 1][c]);
        reinterpret_cast<uint4*>(dst)[0] = make_uint4(pk[0], pk[1], pk[2], pk[3]);
        reinterpret_cast<uint4*>(dst)[1] = make_uint4(pk[4], pk[5], pk[6], pk[7]);
      } else {
        for (int64_t tt = a0; tt < a1; ++tt)
          dst[tt - w0] = __builtin_bit_cast(uint16_t, (_Float16)tile[tt - w0][c]);
      }
    }
  }
}

// grid (ceil(T16 / 256), Hkv, 2)
template <int RB>
__global__ __launch_bounds__(kMW * 64) void materialize_kernel(const MatArgs a) {
  constexpr int BT = MSmem<RB>::BT;
  __shared__ MSmem<RB> sm;
  const int h = blockIdx.y, z = blockIdx.z;
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t T = a.T;
  const int64_t g0 = (int64_t)blockIdx.x * kMTok;         // a multiple of 16
  const int64_t gend = min(g0 + (int64_t)kMTok, T);
  const int64_t slab = (int64_t)z * a.n_kv_heads + h;
  const uint16_t* ck = a.coef_k + (int64_t)h * a.T16 * RB;
  const uint16_t* cv = a.coef_v + (int64_t)h * a.T16 * RB;
  const uint32_t* off = a.off + (int64_t)h * (T + 1);
  const uint8_t* idx = a.idx + slab * a.res_stride;
  const uint8_t* val = a.val + slab * (a.res_stride / 2);
  const uint16_t* scale = a.scale + slab * T;
  uint16_t* kout = a.k_out + (int64_t)h * T * D;
  uint16_t* vout = a.v_out + (int64_t)h * a.T16 * D;
  float (*tile)[D + 4] = sm.tile[wv];

  if (g0 < T) {
    for (int b = seq_of(a.cu, a.batch, g0); b < a.batch && (int64_t)a.cu[b] < gend; ++b) {
      const int64_t s0 = max(g0, (int64_t)a.cu[b]), s1 = min(gend, (int64_t)a.cu[b + 1]);
      if (s1 <= s0) continue;            // empty sequence (uniform)
      __syncthreads();                   // both waves are done with the previous basis
      const uint16_t* src = a.basis + (int64_t)b * a.basis_b_stride + (int64_t)(h * 2 + z) * RB * D;
      for (int e = threadIdx.x; e < RB * (D / 8); e += kMW * 64) {
        const int k = e / (D / 8), c8 = e % (D / 8);
        const uint4 w = *reinterpret_cast<const uint4*>(src + (int64_t)k * D + 8 * c8);
        const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int u = 0; u < 8; ++u)
          sm.bt[(8 * c8 + u) * BT + k] = (uint16_t)(ws[u >> 1] >> (16 * (u & 1)));
      }
      __syncthreads();
      // block i of the workgroup (16 tokens from g0 + 16 i) belongs to wave i % kMW;
      // the next block's inputs are loaded while this one computes
      const int64_t i0 = (s0 - g0) >> 4, i1 = (s1 - 1 - g0) >> 4;
      int64_t i = i0 + ((wv - i0) % kMW + kMW) % kMW;
      if (i <= i1) {
        MBlock<RB> cur, nxt;
        int64_t w0 = g0 + 16 * i;
        mat_load<RB>(cur, w0, max(s0, w0), min(s1, w0 + 16), z, lane, ck, cv, off, scale);
        uint32_t rho = mat_entries<RB>(cur, a, idx, val, lane);
        for (; i <= i1; i += kMW) {
          w0 = g0 + 16 * i;
          const int64_t wn = w0 + 16 * kMW;
          const bool more = i + kMW <= i1;
          if (more) mat_load<RB>(nxt, wn, max(s0, wn), min(s1, wn + 16), z, lane, ck, cv, off, scale);
          mat_block<RB>(a, sm, tile, w0, max(s0, w0), min(s1, w0 + 16), z, lane, cur, rho, idx, val, kout, vout);
          if (more) {
            cur = nxt;
            rho = mat_entries<RB>(cur, a, idx, val, lane);
          }
        }
      }
    }
  }
  // value padding of the last block: tokens [T, T16) are zero
  if (z == 1 && T < a.T16) {
    const int64_t wl = a.T16 - 16;
    if (wl >= g0 && wl < g0 + kMTok && ((wl - g0) >> 4) % kMW == wv) {
      for (int c = lane; c < D; c += 64) {
        uint16_t* dst = vout + ((wl >> 4) * D + c) * 16;
        for (int64_t tt = T; tt < wl + 16; ++tt) dst[tt - wl] = 0;
      }
    }
  }
}

template <int RB>
hipError_t launch_mat(const MatArgs& a, hipStream_t s) {
  const unsigned nb = (unsigned)((a.T16 + kMTok - 1) / kMTok);
  hipLaunchKernelGGL(materialize_kernel<RB>, dim3(nb, a.n_kv_heads, 2), dim3(kMW * 64), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_materialize(const MatArgs& a, hipStream_t s) {
  if (a.T16 <= 0) return hipSuccess;
  switch (a.rb) {
    case 16: return launch_mat<16>(a, s);
    case 32: return launch_mat<32>(a, s);
    case 48: return launch_mat<48>(a, s);
    case 64: return launch_mat<64>(a, s);
    case 80: return launch_mat<80>(a, s);
    case 96: return launch_mat<96>(a, s);
    case 112: return launch_mat<112>(a, s);
    case 128: return launch_mat<128>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace dwkv
