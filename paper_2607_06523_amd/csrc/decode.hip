// Fused split-K decode attention over the cross-depth factorized KV cache, gfx950.
//
// Sec. 3 of the paper rebuilds the key/value of token t at layer l as
// X_hat = A^Z_{l,h,t} B^Z_{m,h} + g R^Z_{l,h,t} (Eq. 1) and fuses basis lookup,
// residual dequantisation and the attention product so no rebuilt K/V reaches
// HBM.  This kernel never rebuilds K/V at all.  Because Eq. 1 is linear,
//   q . K_hat_t = A^K_t (B^K q) + g s sum_e code_e q[c_e]
//   sum_t p_t V_hat_t = (sum_t p_t A^V_t) B^V + sum_t p_t g s sum_e code_e e_{c_e},
// so the query is projected once into basis space (q~ = B^K q), the coefficient
// rows stream through MFMA against q~ and against the probabilities, and the
// routed residual entries touch only the score of their token (keys) or one
// channel of a d-vector accumulator (values).
//
// Mapping (one workgroup = 4 waves = one chunk of `split` tokens of one
// sequence and one KV head; every wave streams its own 64-token tiles):
//  * scores  S[tok][g] = A^K[tok][:] . q~[:][g]: v_mfma_f32_16x16x16_f16 with
//    A^K rows as the A operand straight from HBM (lane = token % 16, k-slice by
//    lane/16) and q~ as the B operand held in registers for the whole split;
//    q~ is split into fp16 hi + lo parts (two MFMAs) so the scores carry
//    float32 accuracy; the G query heads of the group fill columns 0..G-1.
//  * the MFMA result layout (lane = head, 4 consecutive tokens per lane) is
//    exactly the A-operand layout of the value product, so probabilities feed
//    a~[g][:] += P[g][tok] A^V[tok][:] without a shuffle (again hi + lo);
//    A^V tiles are staged through LDS (rows padded 8 bytes, conflict-free
//    transposed reads).
//  * online softmax in exp2 units; running max over the tile via lane shuffles.
//  * residual entries: entry-parallel (one lane per entry), token found by
//    binary search over the tile's offsets; key entries add into an LDS score
//    buffer, value entries into an LDS d-vector per head (ds_add_f32).
//  * epilogue: the 4 waves merge their (m, l, a~, r) in LDS, project a~
//    through B^V and write one partial (o, m, l) per query head; a second
//    kernel merges the splits (and computes the Eq. 3 probe error).
#include "entry.h"
#include "internal.h"

namespace dwkv {
namespace {

typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int D = kHeadDim;

__device__ __forceinline__ f4 mfma16(h4 a, h4 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
}

// Order LDS traffic between lanes of one wave (LDS executes a wave's
// instructions in order; this keeps the compiler from moving accesses).
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ uint32_t dword_at(const uint4& v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

template <int RB>
struct Cfg {
  static constexpr int NBK = RB <= 64 ? 4 : 2;     // 16-token blocks per tile
  static constexpr int TT = NBK * 16;              // tokens per tile
  static constexpr int KH = RB / 4;                // halves of a row each lane holds
  static constexpr int NS = RB / 16;               // MFMA k-steps (K = 16)
  static constexpr int VQ = TT * RB / 512;         // 16-byte V chunks per lane per tile
  static constexpr int VROW = RB + 4;              // LDS row pitch in halves
  static_assert(RB % 16 == 0 && RB >= 16 && RB <= 128, "r_b");
  static_assert((TT * RB) % 512 == 0, "tile");
};

template <int RB, int G, bool RESID>
struct WaveSmem {
  static constexpr int TT = Cfg<RB>::TT;
  static constexpr int RG = RESID ? G : 1;
  static constexpr int RT = RESID ? TT : 1;
  static constexpr int RD = RESID ? D : 1;
  static constexpr int RE = RESID ? kEntChunk / 4 : 1;
  _Float16 v[TT][Cfg<RB>::VROW];       // A^V tile (also the epilogue's a~ staging)
  float resid[RT][RG];                 // key-residual score per token and head
  float p[RT][RG];                     // tile probabilities (for value residuals)
  float rsk[RT];                       // gate-folded residual scale, keys
  float rsv[RT];                       // ... values
  uint32_t off[RESID ? TT + 1 : 1];    // absolute entry offsets of the tile
  float racc[RG][RD];                  // value-residual accumulator
  uint32_t eidx[2][RE];                // staged channel bytes (keys, values)
  uint32_t eval[2][RE];                // staged code bytes
  static_assert(sizeof(v) >= sizeof(float) * G * RB, "a~ overlay");
};

template <int RB, int G, bool RESID>
struct Smem {
  alignas(16) float qs[D][G];          // q * sm_scale * log2(e)
  float qt[G][RB];                     // q~ = B^K q (scaled)
  float ep_m[kWaves][G];
  float ep_l[kWaves][G];
  float sw[kWaves][G];
  float mstar[G];
  float lstar[G];
  float acomb[G][RB];
  WaveSmem<RB, G, RESID> w[kWaves];
};

template <int RB>
struct Tile {
  uint2 a[Cfg<RB>::NBK][Cfg<RB>::NS];   // A^K fragments: 4 halves per k-step
  uint4 v[Cfg<RB>::VQ];                 // A^V tile chunks
  uint32_t oa, ob;                      // off[t0+lane], off[t0+lane+1] (clamped)
  uint32_t sk, sv;                      // residual scale bits of token t0+lane
};

template <int RB>
struct State {
  h4 qhi[Cfg<RB>::NS], qlo[Cfg<RB>::NS];
  f4 acc[Cfg<RB>::NS];                  // a~ in MFMA result layout
  float m, l, down;
};

struct Ctx {
  const uint16_t* ck;
  const uint16_t* cv;
  const uint32_t* off;
  const uint8_t* idx[2];
  const uint8_t* val[2];
  const uint16_t* sk;
  const uint16_t* sv;
  int64_t c0, c1, res_stride;
  int ntile;
};

template <int RB, bool RESID>
__device__ __forceinline__ void load_tile(Tile<RB>& r, const Ctx& x, int j, int lane) {
  using C = Cfg<RB>;
  const int64_t t0 = x.c0 + (int64_t)j * C::TT;
  const int nv = (int)min((int64_t)C::TT, x.c1 - t0);
  const int grp = lane >> 4, col = lane & 15;
#pragma unroll
  for (int bk = 0; bk < C::NBK; ++bk) {
    const int tok = min(16 * bk + col, nv - 1);
    const uint2* p = reinterpret_cast<const uint2*>(x.ck + (t0 + tok) * RB + C::KH * grp);
#pragma unroll
    for (int s = 0; s < C::NS; ++s) r.a[bk][s] = p[s];
  }
#pragma unroll
  for (int q = 0; q < C::VQ; ++q) {
    const int flat = (q * 64 + lane) * 8;
    const int row = min(flat / RB, nv - 1);
    r.v[q] = *reinterpret_cast<const uint4*>(x.cv + (t0 + row) * RB + flat % RB);
  }
  if constexpr (RESID) {
    r.oa = x.off[t0 + min(lane, nv)];
    r.ob = x.off[t0 + min(lane + 1, nv)];
    r.sk = x.sk[t0 + min(lane, nv - 1)];
    r.sv = x.sv[t0 + min(lane, nv - 1)];
  }
}

// Four dwords of residual storage starting at byte `pos` of a slab of `len`
// bytes (0 beyond the slab; such bytes belong to no entry of the tile).
__device__ __forceinline__ uint32_t load_dword_clamped(const uint8_t* base, int64_t pos, int64_t len) {
  return pos + 4 <= len ? *reinterpret_cast<const uint32_t*>(base + pos) : 0u;
}

template <int TT>
__device__ __forceinline__ int token_of_entry(const uint32_t* off, uint32_t e) {
  // largest t in [0, TT) with off[t] <= e  (off[0] <= e < off[TT])
  int lo = 0, hi = TT;
#pragma unroll
  for (int it = 0; it < 7; ++it) {
    if (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (off[mid] <= e) lo = mid; else hi = mid;
    }
  }
  return lo;
}

// One residual pass over the tile's entries [e0, e1) of slab z (0 keys, 1 values).
// The first 256-entry chunk is already staged in LDS at (ia, va); later chunks
// are fetched here.
template <int RB, int G, bool ISV>
__device__ __forceinline__ void resid_pass(WaveSmem<RB, G, true>& ws, const Ctx& x,
                                           const float (*qs)[G], uint32_t e0, uint32_t e1,
                                           uint32_t ia, uint32_t va, int lane) {
  constexpr int TT = Cfg<RB>::TT;
  constexpr int z = ISV ? 1 : 0;
  uint32_t beg = e0;
  for (;;) {
    const uint32_t end = min(e1, ia + (uint32_t)kEntChunk);
    for (uint32_t base = beg; base < end; base += 64) {
      const uint32_t e = base + lane;
      if (e < end) {
        const int t = token_of_entry<TT>(ws.off, e);
        const uint32_t c = reinterpret_cast<const uint8_t*>(ws.eidx[z])[e - ia] & (D - 1);
        const uint32_t vb = reinterpret_cast<const uint8_t*>(ws.eval[z])[(e >> 1) - va];
        const float code = (float)entry_code(vb, e);
        if constexpr (!ISV) {
          const float s = ws.rsk[t] * code;
#pragma unroll
          for (int g = 0; g < G; ++g) atomicAdd(&ws.resid[t][g], s * qs[c][g]);
        } else {
          const float s = ws.rsv[t] * code;
#pragma unroll
          for (int g = 0; g < G; ++g) atomicAdd(&ws.racc[g][c], ws.p[t][g] * s);
        }
      }
    }
    if (end >= e1) break;
    // next chunk (rare: a tile with more than ~250 routed entries)
    beg = end;
    ia = end;
    va = (end >> 1) & ~3u;
    wave_lds_fence();
    ws.eidx[z][lane] = load_dword_clamped(x.idx[z], (int64_t)ia + 4 * lane, x.res_stride);
    ws.eval[z][lane] = load_dword_clamped(x.val[z], (int64_t)va + 4 * lane, x.res_stride / 2);
    wave_lds_fence();
  }
}

template <int RB, int G, bool RESID>
__device__ __forceinline__ void step(State<RB>& st, Tile<RB>& cur, Tile<RB>& nxt, int j,
                                     const Ctx& x, Smem<RB, G, RESID>& sm,
                                     WaveSmem<RB, G, RESID>& ws, int lane) {
  using C = Cfg<RB>;
  constexpr int TT = C::TT, NBK = C::NBK, NS = C::NS;
  const int grp = lane >> 4, col = lane & 15;
  const int64_t t0 = x.c0 + (int64_t)j * TT;
  const int nv = (int)min((int64_t)TT, x.c1 - t0);

  // 1. residual entry range of the tile; first chunk fetched before the prefetch
  uint32_t e0 = 0, e1 = 0, ia = 0, va = 0;
  uint32_t ik = 0, iv = 0, vk = 0, vv = 0;
  if constexpr (RESID) {
    e0 = (uint32_t)__shfl((int)cur.oa, 0);
    e1 = (uint32_t)__shfl((int)cur.ob, 63);
    // a well-formed tile holds at most TT*d entries; the bound keeps a corrupt
    // offset table from running the passes long
    e1 = (e1 > e0 && e1 - e0 > (uint32_t)(TT * D)) ? e0 + TT * D : e1;
    ia = e0 & ~3u;
    va = (e0 >> 1) & ~3u;
    if (e1 > e0) {
      ik = load_dword_clamped(x.idx[0], (int64_t)ia + 4 * lane, x.res_stride);
      iv = load_dword_clamped(x.idx[1], (int64_t)ia + 4 * lane, x.res_stride);
      vk = load_dword_clamped(x.val[0], (int64_t)va + 4 * lane, x.res_stride / 2);
      vv = load_dword_clamped(x.val[1], (int64_t)va + 4 * lane, x.res_stride / 2);
    }
  }
  // 2. prefetch the wave's next tile
  if (j + kWaves < x.ntile) load_tile<RB, RESID>(nxt, x, j + kWaves, lane);

  // 3. stage the value tile (and the tile's residual metadata) in LDS
#pragma unroll
  for (int q = 0; q < C::VQ; ++q) {
    const int flat = (q * 64 + lane) * 8;
    uint2* dst = reinterpret_cast<uint2*>(&ws.v[flat / RB][flat % RB]);
    dst[0] = make_uint2(cur.v[q].x, cur.v[q].y);
    dst[1] = make_uint2(cur.v[q].z, cur.v[q].w);
  }
  if constexpr (RESID) {
    if (lane < TT) {
      ws.off[lane] = cur.oa;
      ws.rsk[lane] = half_bits_to_float((uint16_t)cur.sk);
      ws.rsv[lane] = half_bits_to_float((uint16_t)cur.sv);
    }
    if (lane == TT - 1) ws.off[TT] = cur.ob;
    for (int i = lane; i < TT * G; i += 64) (&ws.resid[0][0])[i] = 0.f;
    ws.eidx[0][lane] = ik;
    ws.eidx[1][lane] = iv;
    ws.eval[0][lane] = vk;
    ws.eval[1][lane] = vv;
  }
  wave_lds_fence();

  // 4. basis-space scores on MFMA (q~ hi + lo)
  f4 sacc[NBK];
#pragma unroll
  for (int bk = 0; bk < NBK; ++bk) {
    sacc[bk] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const h4 av = __builtin_bit_cast(h4, cur.a[bk][s]);
      sacc[bk] = mfma16(av, st.qhi[s], sacc[bk]);
      sacc[bk] = mfma16(av, st.qlo[s], sacc[bk]);
    }
  }

  // 5. key residual entries add q[c]*code*scale to their token's score
  if constexpr (RESID) {
    if (e1 > e0) resid_pass<RB, G, false>(ws, x, sm.qs, e0, e1, ia, va, lane);
    wave_lds_fence();
  }

  // 6. online softmax (exp2 units); this lane holds head `col`, tokens 16bk+4grp+i
  float sc[NBK][4];
  float mt = -INFINITY;
#pragma unroll
  for (int bk = 0; bk < NBK; ++bk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tok = 16 * bk + 4 * grp + i;
      float s = sacc[bk][i] * st.down;
      if constexpr (RESID) {
        if (col < G) s += ws.resid[tok][col];
      }
      s = tok < nv ? s : -INFINITY;
      sc[bk][i] = s;
      mt = fmaxf(mt, s);
    }
  }
  mt = fmaxf(mt, __shfl_xor(mt, 16));
  mt = fmaxf(mt, __shfl_xor(mt, 32));
  const float mn = fmaxf(st.m, mt);
  const float alpha = exp2_hw(st.m - mn);
  float psum = 0.f;
#pragma unroll
  for (int bk = 0; bk < NBK; ++bk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float p = col < G ? exp2_hw(sc[bk][i] - mn) : 0.f;
      sc[bk][i] = p;
      psum += p;
    }
  }
  st.l = st.l * alpha + psum;
  st.m = mn;

  // 7. rescale the basis-space value accumulator (rows g = 4grp+i)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float ai = __shfl(alpha, 4 * grp + i);
#pragma unroll
    for (int cb = 0; cb < NS; ++cb) st.acc[cb][i] *= ai;
  }

  if constexpr (RESID) {
    // 8. rescale the value-residual accumulator when a running max moved
    const bool moved = (col < G) && (alpha != 1.0f);
    if (__ballot(moved) != 0) {
#pragma unroll
      for (int it = 0; it < (G * D) / 64; ++it) {
        const int g = (it * 64) / D;
        const float ag = __shfl(alpha, g);
        (&ws.racc[0][0])[it * 64 + lane] *= ag;
      }
    }
    // 9. probabilities to LDS for the value entries
    if (col < G) {
#pragma unroll
      for (int bk = 0; bk < NBK; ++bk)
#pragma unroll
        for (int i = 0; i < 4; ++i) ws.p[16 * bk + 4 * grp + i][col] = sc[bk][i];
    }
  }

  // 10. a~ += P A^V on MFMA (P hi + lo); A^V read transposed from LDS
#pragma unroll
  for (int bk = 0; bk < NBK; ++bk) {
    h4 ph, pl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const _Float16 hh = (_Float16)sc[bk][i];
      ph[i] = hh;
      pl[i] = (_Float16)(sc[bk][i] - (float)hh);
    }
#pragma unroll
    for (int cb = 0; cb < NS; ++cb) {
      h4 vf;
#pragma unroll
      for (int i = 0; i < 4; ++i) vf[i] = ws.v[16 * bk + 4 * grp + i][16 * cb + col];
      st.acc[cb] = mfma16(ph, vf, st.acc[cb]);
      st.acc[cb] = mfma16(pl, vf, st.acc[cb]);
    }
  }

  // 11. value residual entries scatter p*code*scale into their channel
  if constexpr (RESID) {
    wave_lds_fence();
    if (e1 > e0) resid_pass<RB, G, true>(ws, x, sm.qs, e0, e1, ia, va, lane);
  }
  wave_lds_fence();
}

template <int RB, int G, bool RESID, bool IDENT>
__global__ __launch_bounds__(kThreads) void split_kernel(const SplitArgs a) {
  using C = Cfg<RB>;
  constexpr int NS = C::NS;
  __shared__ Smem<RB, G, RESID> sm;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int grp = lane >> 4, col = lane & 15;
  const int slot = blockIdx.y;
  const int kvh = a.kv_of_slot[slot];

  // work item -> (sequence, chunk)
  const int w = blockIdx.x;
  int b = 0, base = 0;
  for (; b < a.batch - 1; ++b) {
    const int tb = a.cu[b + 1] - a.cu[b];
    const int ns = (tb + a.split - 1) / a.split;
    if (w < base + ns) break;
    base += ns;
  }
  Ctx x;
  x.c0 = (int64_t)a.cu[b] + (int64_t)(w - base) * a.split;
  x.c1 = min(min((int64_t)a.cu[b + 1], x.c0 + a.split), a.T);
  x.c0 = min(x.c0, x.c1);
  x.ntile = (int)((x.c1 - x.c0 + C::TT - 1) / C::TT);
  x.res_stride = a.res_stride;
  x.ck = a.coef_k + (int64_t)slot * a.T * RB;
  x.cv = a.coef_v + (int64_t)slot * a.T * RB;
  if constexpr (RESID) {
    x.off = a.off + (int64_t)kvh * (a.T + 1);
    x.idx[0] = a.idx_k + (int64_t)kvh * a.res_stride;
    x.idx[1] = a.idx_v + (int64_t)kvh * a.res_stride;
    x.val[0] = a.val_k + (int64_t)kvh * (a.res_stride / 2);
    x.val[1] = a.val_v + (int64_t)kvh * (a.res_stride / 2);
    x.sk = a.scale_k + (int64_t)kvh * a.T;
    x.sv = a.scale_v + (int64_t)kvh * a.T;
  }
  const uint16_t* bk_rows = IDENT ? nullptr : a.basis + (int64_t)b * a.basis_b_stride + (int64_t)kvh * 2 * RB * D;
  const uint16_t* bv_rows = IDENT ? nullptr : bk_rows + RB * D;

  // the first tile's loads go out before the query projection
  Tile<RB> ta, tb;
  if (wv < x.ntile) load_tile<RB, RESID>(ta, x, wv, lane);

  // scaled query and q~ = B^K q
  for (int i = tid; i < G * D; i += kThreads) {
    const int g = i / D, c = i % D;
    const uint16_t bits = a.q[((int64_t)b * a.n_q_heads + kvh * G + g) * D + c];
    sm.qs[c][g] = (a.q_bf16 ? bf16_bits_to_float(bits) : half_bits_to_float(bits)) * a.qscale;
  }
  __syncthreads();
  if constexpr (!IDENT) {
    for (int it = tid; it < RB * 4; it += kThreads) {
      const int k = it >> 2, qq = it & 3;
      const uint16_t* row = bk_rows + k * D + qq * 32;
      float acc[G];
#pragma unroll
      for (int g = 0; g < G; ++g) acc[g] = 0.f;
#pragma unroll
      for (int c8 = 0; c8 < 32; c8 += 8) {
        const uint4 v = *reinterpret_cast<const uint4*>(row + c8);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t dw = dword_at(v, e >> 1);
          const float xv = half_bits_to_float((uint16_t)((e & 1) ? (dw >> 16) : (dw & 0xFFFF)));
#pragma unroll
          for (int g = 0; g < G; ++g) acc[g] += xv * sm.qs[qq * 32 + c8 + e][g];
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        acc[g] += __shfl_xor(acc[g], 1);
        acc[g] += __shfl_xor(acc[g], 2);
      }
      if (qq == 0) {
#pragma unroll
        for (int g = 0; g < G; ++g) sm.qt[g][k] = acc[g];
      }
    }
    __syncthreads();
  }

  // q~ as MFMA B operand (column = head), scaled by a power of two so its
  // largest entry sits just under 2^14, split into fp16 hi + lo
  State<RB> st;
  {
    int kexp = 0;
    if (col < G) {
      float mx = 0.f;
      for (int k = 0; k < RB; ++k) mx = fmaxf(mx, fabsf(IDENT ? sm.qs[k][col] : sm.qt[col][k]));
      if (mx > 0.f) {
        int e;
        frexpf(mx, &e);
        kexp = 14 - e;
      }
    }
    kexp = max(-100, min(100, kexp));
    const float up = ldexpf(1.0f, kexp);
    st.down = ldexpf(1.0f, -kexp);
#pragma unroll
    for (int s = 0; s < NS; ++s) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int k = C::KH * grp + 4 * s + i;
        const float v = col < G ? (IDENT ? sm.qs[k][col] : sm.qt[col][k]) * up : 0.f;
        const _Float16 hh = (_Float16)v;
        st.qhi[s][i] = hh;
        st.qlo[s][i] = (_Float16)(v - (float)hh);
      }
      st.acc[s] = f4{0.f, 0.f, 0.f, 0.f};
    }
  }
  st.m = -INFINITY;
  st.l = 0.f;
  auto& ws = sm.w[wv];
  if constexpr (RESID) {
    for (int i = lane; i < G * D; i += 64) (&ws.racc[0][0])[i] = 0.f;
  }

  // stream the wave's tiles (ping-pong register buffers)
  for (int j = wv; j < x.ntile; j += 2 * kWaves) {
    step<RB, G, RESID>(st, ta, tb, j, x, sm, ws, lane);
    if (j + kWaves >= x.ntile) break;
    step<RB, G, RESID>(st, tb, ta, j + kWaves, x, sm, ws, lane);
  }

  // epilogue: merge the 4 waves, project a~ through B^V, write the partial
  st.l += __shfl_xor(st.l, 16);
  st.l += __shfl_xor(st.l, 32);
  float* epa = reinterpret_cast<float*>(&ws.v[0][0]);        // [G][RB]
  if (grp == 0 && col < G) {
    sm.ep_m[wv][col] = st.m;
    sm.ep_l[wv][col] = st.l;
  }
#pragma unroll
  for (int cb = 0; cb < NS; ++cb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = 4 * grp + i;
      if (g < G) epa[g * RB + 16 * cb + col] = st.acc[cb][i];
    }
  __syncthreads();
  if (tid < G) {
    const int g = tid;
    float mx = -INFINITY;
    for (int v = 0; v < kWaves; ++v) mx = fmaxf(mx, sm.ep_m[v][g]);
    float l = 0.f;
    for (int v = 0; v < kWaves; ++v) {
      const float s = sm.ep_m[v][g] == -INFINITY ? 0.f : exp2f(sm.ep_m[v][g] - mx);
      sm.sw[v][g] = s;
      l += s * sm.ep_l[v][g];
    }
    sm.mstar[g] = mx;
    sm.lstar[g] = l;
  }
  __syncthreads();
  for (int i = tid; i < G * RB; i += kThreads) {
    const int g = i / RB, k = i % RB;
    float s = 0.f;
    for (int v = 0; v < kWaves; ++v) s += sm.sw[v][g] * reinterpret_cast<const float*>(&sm.w[v].v[0][0])[g * RB + k];
    sm.acomb[g][k] = s;
  }
  __syncthreads();
  for (int i = tid; i < G * D; i += kThreads) {
    const int g = i / D, c = i % D;
    float o;
    if constexpr (IDENT) {
      o = sm.acomb[g][c];
    } else {
      o = 0.f;
      for (int k = 0; k < RB; ++k) o += sm.acomb[g][k] * half_bits_to_float(bv_rows[k * D + c]);
    }
    if constexpr (RESID) {
      for (int v = 0; v < kWaves; ++v) o += sm.sw[v][g] * sm.w[v].racc[g][c];
    }
    float* dst = a.part + (((int64_t)w * a.n_slots + slot) * G + g) * kPartStride;
    dst[c] = o;
    if (c == 0) {
      dst[D] = sm.mstar[g];
      dst[D + 1] = sm.lstar[g];
    }
  }
}

// One workgroup per (query head, sequence): merges the split partials in a
// fixed order; with a probe, also merges the reference partials and writes
// Eq. 3's relative error.
__global__ __launch_bounds__(D) void merge_kernel(const MergeArgs a) {
  const int hq = blockIdx.x, b = blockIdx.y, c = threadIdx.x;
  const int G = a.n_q_heads / a.n_kv_heads, h = hq / G, g = hq % G;
  int base = 0;
  for (int i = 0; i < b; ++i) base += (a.cu[i + 1] - a.cu[i] + a.split - 1) / a.split;
  const int ns = (a.cu[b + 1] - a.cu[b] + a.split - 1) / a.split;

  auto merge = [&](const float* part, int n_slots, int s_slot) -> float {
    float mx = -INFINITY;
    for (int s = 0; s < ns; ++s)
      mx = fmaxf(mx, part[(((int64_t)(base + s) * n_slots + s_slot) * G + g) * kPartStride + D]);
    float l = 0.f, acc = 0.f;
    for (int s = 0; s < ns; ++s) {
      const float* p = part + (((int64_t)(base + s) * n_slots + s_slot) * G + g) * kPartStride;
      const float wgt = exp2f(p[D] - mx);
      l += wgt * p[D + 1];
      acc += wgt * p[c];
    }
    return ns > 0 ? acc / l : 0.f;
  };

  const float o = merge(a.part, a.n_kv_heads, h);
  a.out[((int64_t)b * a.n_q_heads + hq) * D + c] = o;
  if (a.n_probe > 0) {
    const int sl = a.probe_slot_of_kv[h];
    if (sl >= 0) {
      const float r = merge(a.part_ref, a.n_probe, sl);
      const int64_t col = (int64_t)b * a.n_probe * G + sl * G + g;
      if (a.out_ref) a.out_ref[col * D + c] = r;
      float d2 = (r - o) * (r - o), r2 = r * r;
      for (int o2 = 32; o2 > 0; o2 >>= 1) {
        d2 += __shfl_xor(d2, o2);
        r2 += __shfl_xor(r2, o2);
      }
      __shared__ float red[2][2];
      if ((c & 63) == 0) {
        red[c >> 6][0] = d2;
        red[c >> 6][1] = r2;
      }
      __syncthreads();
      if (c == 0) a.err[col] = sqrtf(red[0][0] + red[1][0]) / (sqrtf(red[0][1] + red[1][1]) + a.eps);
    }
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

}  // namespace

hipError_t launch_split(int rb, int g, bool resid, bool ident, const SplitArgs& a, int n_work,
                        hipStream_t s) {
  if (ident) return rb == D ? launch_g<D, false, true>(g, a, n_work, s) : hipErrorInvalidValue;
  return resid ? launch_rb<true>(rb, g, a, n_work, s) : launch_rb<false>(rb, g, a, n_work, s);
}

hipError_t launch_merge(const MergeArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(merge_kernel, dim3(a.n_q_heads, a.batch), dim3(D), 0, s, a);
  return hipGetLastError();
}

}  // namespace dwkv
