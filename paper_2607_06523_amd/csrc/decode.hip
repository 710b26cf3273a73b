// General split-K decode kernel (any r_b to 128, groups to 16) and the merge
// kernels; the split pass's device code is in split_dev.h.
#include "split_dev.h"

namespace dwkv {
namespace {

using namespace gsplit;

template <int RB, int G, bool RESID, bool IDENT>
__global__ __launch_bounds__(kThreads) void split_kernel(const SplitArgs a) {
  __shared__ Smem<RB, G, RESID> sm;
  split_body<RB, G, RESID, IDENT>(a, blockIdx.x, blockIdx.y, threadIdx.x, sm);
}

// An earlier probe position's two passes in one launch: workgroups
// [0, n_work * n_slots) of A.s run the factorized pass over the probed heads
// (in split_kernel's order), the rest the reference pass A.r (identity basis).
template <int RB, int G, bool RESID>
__global__ __launch_bounds__(kThreads) void pos_pair_kernel(const TLProbeArgs A) {
  using FS = Smem<RB, G, RESID>;
  using RS = Smem<D, G, false>;
  __shared__ alignas(16) unsigned char lds[sizeof(FS) > sizeof(RS) ? sizeof(FS) : sizeof(RS)];
  const int nf = A.s.n_work * A.s.n_slots;
  const int i = blockIdx.x;
  if (i < nf) {
    split_body<RB, G, RESID, false>(A.s, i % A.s.n_work, i / A.s.n_work, threadIdx.x, *reinterpret_cast<FS*>(lds));
    return;
  }
  const int k = i - nf;
  split_body<D, G, false, true>(A.r, k % A.r.n_work, k / A.r.n_work, threadIdx.x, *reinterpret_cast<RS*>(lds));
}

// One workgroup per (query head, sequence) merges that head's split partials
// in a fixed order: every partial's (m, l) and output slice are requested in
// one round of loads.  For a probed KV head it also merges the reference
// partials and writes Eq. 3's error.
constexpr int kMergeThreads = 256;
constexpr int kMergeGroups = kMergeThreads / (D / 4);     // split groups (8)
constexpr int kMergePerThread = 8;                        // splits per thread per round

// Merges the first ncols (<= 2d) columns of the rows row0 + s * row_step
// (s < ns) of partials with `stride` floats and (m, l) at m_off.  A thread
// owns columns 4*c4.. and d + 4*c4..; split group 0 returns them divided by
// the merged l (x: first slice, y: second slice).
struct Merged {
  f4 x, y;
};

template <int NT = kMergeThreads>
__device__ __forceinline__ Merged merge_rows(const float* part, int64_t row0, int64_t row_step, int ns,
                                             int stride, int m_off, int ncols, float* red_m, float* red_l,
                                             f4* red_o) {
  constexpr int kMergeGroups = NT / (D / 4);
  const int tid = threadIdx.x, c4 = tid % (D / 4), sg = tid / (D / 4);
  const bool two = D + 4 * c4 < ncols;
  const f4 z4 = f4{0.f, 0.f, 0.f, 0.f};
  f4 acc = z4, acc2 = z4;
  float mstar = -INFINITY, lsum = 0.f;
  for (int s0 = 0; s0 < ns; s0 += kMergeGroups * kMergePerThread) {
    // this round's splits: s0 + sg + kMergeGroups * i, all requested at once
    f4 ov[kMergePerThread], ov2[kMergePerThread];
    float mv[kMergePerThread], lv[kMergePerThread];
    // unconditional loads (split index clamped), selected afterwards, so every
    // request of the round is in flight before the first wait
#pragma unroll
    for (int i = 0; i < kMergePerThread; ++i) {
      const int s = min(s0 + sg + kMergeGroups * i, ns - 1);
      const float* p = part + (row0 + (int64_t)s * row_step) * stride;
      ov[i] = *reinterpret_cast<const f4*>(p + 4 * c4);
      ov2[i] = *reinterpret_cast<const f4*>(p + (two ? D : 0) + 4 * c4);
      mv[i] = p[m_off];
      lv[i] = p[m_off + 1];
    }
#pragma unroll
    for (int i = 0; i < kMergePerThread; ++i) {
      const bool ok = s0 + sg + kMergeGroups * i < ns;
      ov[i] = ok ? ov[i] : z4;
      ov2[i] = ok && two ? ov2[i] : z4;
      mv[i] = ok ? mv[i] : -INFINITY;
      lv[i] = ok ? lv[i] : 0.f;
    }
    // the round's maximum: per thread, then over the split groups through LDS
    float mr = mv[0];
#pragma unroll
    for (int i = 1; i < kMergePerThread; ++i) mr = fmaxf(mr, mv[i]);
    if (c4 == 0) red_m[sg] = mr;
    __syncthreads();
    mr = mstar;
#pragma unroll
    for (int q = 0; q < kMergeGroups; ++q) mr = fmaxf(mr, red_m[q]);
    __syncthreads();
    // rescale what the earlier rounds accumulated, then add this round's splits
    const float resc = mstar == -INFINITY ? 0.f : exp2f(mstar - mr);
    acc.x *= resc; acc.y *= resc; acc.z *= resc; acc.w *= resc;
    acc2.x *= resc; acc2.y *= resc; acc2.z *= resc; acc2.w *= resc;
    lsum *= resc;
#pragma unroll
    for (int i = 0; i < kMergePerThread; ++i) {
      if (mv[i] == -INFINITY) continue;
      const float w = exp2f(mv[i] - mr);
      acc.x += w * ov[i].x; acc.y += w * ov[i].y; acc.z += w * ov[i].z; acc.w += w * ov[i].w;
      acc2.x += w * ov2[i].x; acc2.y += w * ov2[i].y; acc2.z += w * ov2[i].z; acc2.w += w * ov2[i].w;
      lsum += w * lv[i];
    }
    mstar = mr;
  }
  // combine the split groups of each 4-channel slice (fixed order)
  Merged o{z4, z4};
  red_o[tid] = acc;
  if (c4 == 0) red_l[sg] = lsum;
  __syncthreads();
  float l = 0.f;
  if (sg == 0) {
    for (int q = 0; q < kMergeGroups; ++q) {
      const f4 u = red_o[q * (D / 4) + c4];
      o.x.x += u.x; o.x.y += u.y; o.x.z += u.z; o.x.w += u.w;
      l += red_l[q];
    }
  }
  __syncthreads();
  if (ncols > D) {
    red_o[tid] = acc2;
    __syncthreads();
    if (sg == 0) {
      for (int q = 0; q < kMergeGroups; ++q) {
        const f4 u = red_o[q * (D / 4) + c4];
        o.y.x += u.x; o.y.y += u.y; o.y.z += u.z; o.y.w += u.w;
      }
    }
    __syncthreads();
  }
  if (sg == 0) {
    const float inv = ns > 0 ? 1.0f / l : 0.f;
    o.x.x *= inv; o.x.y *= inv; o.x.z *= inv; o.x.w *= inv;
    o.y.x *= inv; o.y.y *= inv; o.y.z *= inv; o.y.w *= inv;
  }
  return o;
}

constexpr int kMergeMaxRB = 64;      // basis ranks of token-lane partials

__global__ __launch_bounds__(kMergeThreads) void merge_kernel(const MergeArgs a) {
  __shared__ float red_m[kMergeGroups], red_l[kMergeGroups];
  __shared__ f4 red_o[kMergeThreads];
  __shared__ float red2[2][kMergeThreads / 64];
  __shared__ alignas(16) uint16_t bvs[kMergeMaxRB][D];
  __shared__ float abar[kMergeMaxRB];
  const int hq = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  // the head counts pass through the statement so that nothing computed from
  // them is scheduled ahead of the one batch of argument loads it requests
  int nq = a.n_q_heads, nkv = a.n_kv_heads;
  asm volatile("" : "+s"(nq), "+s"(nkv) : "s"(a.part), "s"(a.out), "s"(a.basis), "s"(a.basis_b_stride), "s"(a.tl),
               "s"(a.rb), "s"(a.split), "s"(a.n_work), "s"(a.n_probe), "s"(a.wt.n_seq), "s"(a.wt.work[min(b, kKernargSeqs - 1)]),
               "s"(a.wt.work[min(b, kKernargSeqs - 1) + 1]));
  const int G = nq / nkv, h = hq / G, g = hq % G;
  int base, ns;
  seq_work_entry(a.wt, a.cu, a.split, b, base, ns);
  const int c4 = tid % (D / 4), sg = tid / (D / 4);
  const int64_t row0 = (int64_t)base * a.n_kv_heads * G + h * G + g;
  const int64_t row_step = (int64_t)a.n_kv_heads * G;
  f4 o;
  if (a.tl) {
    // token-lane partials: merge r and a~ together, then o = r + a~ B^V with
    // the k range split over the 8 thread groups
    typedef uint32_t u4v __attribute__((ext_vector_type(4)));
    const int nch = a.rb * D / 8;                   // 16-byte chunks of B^V (multiple of 256)
    const u4v* bv = reinterpret_cast<const u4v*>(a.basis + (int64_t)b * a.basis_b_stride +
                                                  ((int64_t)h * 2 + 1) * a.rb * D);
    u4v bvr[kMergeMaxRB * D / 8 / kMergeThreads];
#pragma unroll
    for (int n = 0; n < kMergeMaxRB * D / 8 / kMergeThreads; ++n) bvr[n] = bv[min(tid + n * kMergeThreads, nch - 1)];
    const Merged mg = merge_rows(a.part, ((int64_t)h * a.n_work + base) * G + g, G, ns, kPartStrideTL, kPartTLM,
                                 D + a.rb, red_m, red_l, red_o);
#pragma unroll
    for (int n = 0; n < kMergeMaxRB * D / 8 / kMergeThreads; ++n)
      if (tid + n * kMergeThreads < nch) reinterpret_cast<u4v*>(&bvs[0][0])[tid + n * kMergeThreads] = bvr[n];
    if (sg == 0 && 4 * c4 < a.rb) {
      abar[4 * c4] = mg.y.x; abar[4 * c4 + 1] = mg.y.y; abar[4 * c4 + 2] = mg.y.z; abar[4 * c4 + 3] = mg.y.w;
    }
    __syncthreads();
    const int kp = (a.rb + kMergeGroups - 1) / kMergeGroups;
    f4 pr = f4{0.f, 0.f, 0.f, 0.f};
    for (int k = sg * kp; k < min(a.rb, sg * kp + kp); ++k) {
      const uint2 w2 = *reinterpret_cast<const uint2*>(&bvs[k][4 * c4]);
      const float ak = abar[k];
      pr.x += ak * half_bits_to_float((uint16_t)(w2.x & 0xFFFF));
      pr.y += ak * half_bits_to_float((uint16_t)(w2.x >> 16));
      pr.z += ak * half_bits_to_float((uint16_t)(w2.y & 0xFFFF));
      pr.w += ak * half_bits_to_float((uint16_t)(w2.y >> 16));
    }
    red_o[tid] = pr;
    __syncthreads();
    o = mg.x;
    if (sg == 0) {
      for (int q = 0; q < kMergeGroups; ++q) {
        const f4 u = red_o[q * (D / 4) + c4];
        o.x += u.x; o.y += u.y; o.z += u.z; o.w += u.w;
      }
    }
    __syncthreads();
  } else {
    o = merge_rows(a.part, row0, row_step, ns, kPartStride, D, D, red_m, red_l, red_o).x;
  }
  if (sg == 0) reinterpret_cast<f4*>(a.out + ((int64_t)b * a.n_q_heads + hq) * D)[c4] = o;
  if (a.n_probe > 0) {
    const int sl = a.probe_slot_of_kv[h];
    if (sl >= 0) {
      int base_r, ns_r;                  // the probe pass has its own work split
      seq_work(a.ref_wt, a.cu, a.ref_split, b, base_r, ns_r);
      const f4 r = merge_rows(a.part_ref, (int64_t)base_r * a.n_probe * G + sl * G + g,
                                  (int64_t)a.n_probe * G, ns_r, kPartStride, D, D, red_m, red_l, red_o).x;
      const int64_t col = (int64_t)b * a.n_probe * G + sl * G + g;
      float d2 = 0.f, r2 = 0.f;
      if (sg == 0) {
        if (a.out_ref) reinterpret_cast<f4*>(a.out_ref + col * D)[c4] = r;
        const float dx = r.x - o.x, dy = r.y - o.y, dz = r.z - o.z, dw = r.w - o.w;
        d2 = dx * dx + dy * dy + dz * dz + dw * dw;
        r2 = r.x * r.x + r.y * r.y + r.z * r.z + r.w * r.w;
      }
      for (int o2 = 32; o2 > 0; o2 >>= 1) {
        d2 += __shfl_xor(d2, o2);
        r2 += __shfl_xor(r2, o2);
      }
      if ((tid & 63) == 0) {
        red2[0][tid >> 6] = d2;
        red2[1][tid >> 6] = r2;
      }
      __syncthreads();
      if (tid == 0) {
        float sd = 0.f, sr = 0.f;
        for (int i = 0; i < kMergeThreads / 64; ++i) { sd += red2[0][i]; sr += red2[1][i]; }
        if (a.acc) {
          a.acc[2 * col] = sd;
          a.acc[2 * col + 1] = sr;
        } else {
          a.err[col] = sqrtf(sd) / (sqrtf(sr) + a.eps);
        }
      }
    }
  }
}

// Eq. 3 over the earlier query positions: one workgroup per (probed query
// head, sequence).  For every position j = 1..n_pos-1 it merges the rebuilt
// and the reference partials of the sequence cut j tokens short (none when
// T_b <= j: the position adds nothing), adds their squared distance and the
// reference's squared norm to the current position's sums, and writes
// sqrt(sum d^2) / (sqrt(sum r^2) + eps).
__global__ __launch_bounds__(kMergeThreads) void probe_pos_merge_kernel(const MergeArgs a) {
  __shared__ float red_m[kMergeGroups], red_l[kMergeGroups];
  __shared__ f4 red_o[kMergeThreads];
  __shared__ float red2[2][kMergeThreads / 64];
  const int b = blockIdx.y, tid = threadIdx.x;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int sl = blockIdx.x / G, g = blockIdx.x % G;
  const int sg = tid / (D / 4);
  const int64_t col = (int64_t)b * a.n_probe * G + sl * G + g;
  const int len = a.cu[b + 1] - a.cu[b];
  float d2 = 0.f, r2 = 0.f;
  for (int j = 1; j < a.n_pos; ++j) {
    // work items of sequence b in the pass over sequences cut j tokens short
    int base = 0;
    for (int i = 0; i < b; ++i) base += (max(a.cu[i + 1] - a.cu[i] - j, 0) + a.ref_split - 1) / a.ref_split;
    const int ns = (max(len - j, 0) + a.ref_split - 1) / a.ref_split;
    const float* pm = a.part_pos + (int64_t)(j - 1) * 2 * a.pos_stride;
    const int64_t row0 = (int64_t)base * a.n_probe * G + sl * G + g, step = (int64_t)a.n_probe * G;
    const f4 o = merge_rows(pm, row0, step, ns, kPartStride, D, D, red_m, red_l, red_o).x;
    const f4 r = merge_rows(pm + a.pos_stride, row0, step, ns, kPartStride, D, D, red_m, red_l, red_o).x;
    if (sg == 0) {
      const float dx = r.x - o.x, dy = r.y - o.y, dz = r.z - o.z, dw = r.w - o.w;
      d2 += dx * dx + dy * dy + dz * dz + dw * dw;
      r2 += r.x * r.x + r.y * r.y + r.z * r.z + r.w * r.w;
    }
  }
  for (int o2 = 32; o2 > 0; o2 >>= 1) {
    d2 += __shfl_xor(d2, o2);
    r2 += __shfl_xor(r2, o2);
  }
  if ((tid & 63) == 0) {
    red2[0][tid >> 6] = d2;
    red2[1][tid >> 6] = r2;
  }
  __syncthreads();
  if (tid == 0) {
    float sd = a.acc[2 * col], sr = a.acc[2 * col + 1];
    for (int i = 0; i < kMergeThreads / 64; ++i) { sd += red2[0][i]; sr += red2[1][i]; }
    a.err[col] = sqrtf(sd) / (sqrtf(sr) + a.eps);
  }
}

template <int RB, int G, bool R, bool I>
hipError_t launch_t(const SplitArgs& a, int n_work, hipStream_t s) {
  hipLaunchKernelGGL((split_kernel<RB, G, R, I>), dim3(n_work, a.n_slots), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

template <int RB, bool R, bool I>
hipError_t launch_g(int g, const SplitArgs& a, int n_work, hipStream_t s) {
  switch (g) {
    case 1: return launch_t<RB, 1, R, I>(a, n_work, s);
    case 2: return launch_t<RB, 2, R, I>(a, n_work, s);
    case 4: return launch_t<RB, 4, R, I>(a, n_work, s);
    case 8: return launch_t<RB, 8, R, I>(a, n_work, s);
    case 16: return launch_t<RB, 16, R, I>(a, n_work, s);
  }
  return hipErrorInvalidValue;
}

template <bool R>
hipError_t launch_rb(int rb, int g, const SplitArgs& a, int n_work, hipStream_t s) {
  switch (rb) {
    case 16: return launch_g<16, R, false>(g, a, n_work, s);
    case 32: return launch_g<32, R, false>(g, a, n_work, s);
    case 48: return launch_g<48, R, false>(g, a, n_work, s);
    case 64: return launch_g<64, R, false>(g, a, n_work, s);
    case 80: return launch_g<80, R, false>(g, a, n_work, s);
    case 96: return launch_g<96, R, false>(g, a, n_work, s);
    case 112: return launch_g<112, R, false>(g, a, n_work, s);
    case 128: return launch_g<128, R, false>(g, a, n_work, s);
  }
  return hipErrorInvalidValue;
}

template <int RB, int G, bool R>
hipError_t launch_pp_t(const TLProbeArgs& a, hipStream_t s) {
  const int n = a.s.n_work * a.s.n_slots + a.r.n_work * a.r.n_slots;
  hipLaunchKernelGGL((pos_pair_kernel<RB, G, R>), dim3(n), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

template <int RB, bool R>
hipError_t launch_pp_g(int g, const TLProbeArgs& a, hipStream_t s) {
  switch (g) {
    case 1: return launch_pp_t<RB, 1, R>(a, s);
    case 2: return launch_pp_t<RB, 2, R>(a, s);
    case 4: return launch_pp_t<RB, 4, R>(a, s);
    case 8: return launch_pp_t<RB, 8, R>(a, s);
    case 16: return launch_pp_t<RB, 16, R>(a, s);
  }
  return hipErrorInvalidValue;
}

template <bool R>
hipError_t launch_pp_rb(int rb, int g, const TLProbeArgs& a, hipStream_t s) {
  switch (rb) {
    case 16: return launch_pp_g<16, R>(g, a, s);
    case 32: return launch_pp_g<32, R>(g, a, s);
    case 48: return launch_pp_g<48, R>(g, a, s);
    case 64: return launch_pp_g<64, R>(g, a, s);
    case 80: return launch_pp_g<80, R>(g, a, s);
    case 96: return launch_pp_g<96, R>(g, a, s);
    case 112: return launch_pp_g<112, R>(g, a, s);
    case 128: return launch_pp_g<128, R>(g, a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_probe_pos(int rb, int g, bool resid, const TLProbeArgs& a, hipStream_t s) {
  return resid ? launch_pp_rb<true>(rb, g, a, s) : launch_pp_rb<false>(rb, g, a, s);
}

hipError_t launch_split(int rb, int g, bool resid, bool ident, const SplitArgs& a, int n_work,
                        hipStream_t s) {
  if (ident) return rb == D ? launch_g<D, false, true>(g, a, n_work, s) : hipErrorInvalidValue;
  return resid ? launch_rb<true>(rb, g, a, n_work, s) : launch_rb<false>(rb, g, a, n_work, s);
}

hipError_t launch_merge(const MergeArgs& a, hipStream_t s) {
  if (a.part_pos) {
    const int g = a.n_q_heads / a.n_kv_heads;
    hipLaunchKernelGGL(probe_pos_merge_kernel, dim3(a.n_probe * g, a.batch), dim3(kMergeThreads), 0, s, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(merge_kernel, dim3(a.n_q_heads, a.batch), dim3(kMergeThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace dwkv
