// Fused split-K decode attention over the cross-depth factorized KV cache, gfx950.
//
// Sec. 3 of the paper rebuilds the key/value of token t at layer l as
// X_hat = A^Z_{l,h,t} B^Z_{m,h} + g R^Z_{l,h,t} (Eq. 1) and fuses basis lookup,
// residual dequantisation and the attention product so no rebuilt K/V reaches
// HBM.  This kernel never rebuilds K/V at all.  Because Eq. 1 is linear,
//   q . K_hat_t = A^K_t (B^K q) + g s sum_e code_e q[c_e]
//   sum_t p_t V_hat_t = (sum_t p_t A^V_t) B^V + sum_t p_t g s sum_e code_e e_{c_e},
// so the query is projected once into basis space (q~ = B^K q), coefficient
// rows stream through MFMA against q~ and against the probabilities, and the
// routed residual entries touch only the score of their token (keys) or one
// channel of a d-vector accumulator (values).
//
// Mapping (one workgroup = 4 waves = one chunk of `split` tokens of one
// sequence and one KV head; each wave streams every 4th tile of 16*NBK tokens):
//  * scores S[tok][g] = A^K[tok][:] . q~[:][g] on v_mfma_f32_16x16x16_f16: key
//    coefficients are the A operand, loaded straight into registers (lane =
//    token % 16, 4 consecutive coefficients by lane / 16: one 8-byte load from
//    the key tiles, or from a dense cache's rows); q~ is the B operand, held
//    for the whole split as fp16 hi + lo parts (two MFMAs, float32-accurate
//    scores); the G query heads of the group fill columns 0..G-1.
//  * the MFMA result layout (lane = head, 4 consecutive tokens per lane) is the
//    A-operand layout of a~[g][:] += P[g][tok] A^V[tok][:], so probabilities feed
//    the value product with no shuffle; value coefficients are stored in
//    8-token blocks (a dense cache's values in 16-token blocks) with the token
//    index fastest, so the B operand (4 consecutive tokens of one channel per
//    lane) is one 8-byte load per lane, straight from HBM.
//  * fragments are single-buffered with early release: the next tile's key
//    fragments are requested right after this tile's score MFMAs, its value
//    fragments right after the value MFMAs; offsets run two tiles ahead and
//    residual entries one tile ahead.
//  * online softmax in exp2 units; running max via lane shuffles.
//  * residual entries: one lane per entry; token of an entry from an LDS map
//    written by the token lanes; key entries add into an LDS score buffer,
//    value entries into an LDS d-vector per head (ds_add_f32).
//  * epilogue: the 4 waves merge (m, l, a~, r) in LDS, project a~ through B^V
//    and write one partial (o, m, l) per query head; a merge kernel combines
//    the splits (and computes Eq. 3's error for probed heads).
#include <type_traits>

#include "entry.h"
#include "internal.h"

namespace dwkv {
namespace {

typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

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

// s_waitcnt immediate for gfx9: vmcnt(0), expcnt and lgkmcnt left at their maxima.
constexpr int kWaitVmcnt0 = 0x0F70;

__device__ __forceinline__ uint32_t dword_at(const uint4& v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

__device__ __forceinline__ int64_t clamp64(int64_t v, int64_t lo, int64_t hi) {
  return v < lo ? lo : (v > hi ? hi : v);
}

template <int RB>
struct Cfg {
  static constexpr int NBK = RB <= 64 ? 4 : 2;     // 16-token blocks per tile
  static constexpr int TT = NBK * 16;              // tokens per tile
  static constexpr int KH = RB / 4;                // key coefficients a lane holds per token
  static constexpr int NS = RB / 16;               // MFMA k-steps (K = 16)
  static_assert(RB % 16 == 0 && RB >= 16 && RB <= 128, "r_b");
};

// Value residuals accumulate in int64 fixed point (units of 2^(ex - kFxTopG),
// ex the wave's bound on the value scales: |p code s| 2^(kFxTopG - ex) < 2^45
// with p <= 1) wherever the workgroup's LDS still fits with 8-byte
// accumulators (every G <= 8; G = 16 up to r_b = 96), else in float.
constexpr int kFxTopG = 42;

template <int RB, int G>
constexpr bool kFixedResid = G <= 8 || RB <= 96;

template <int RB, int G, bool RESID>
struct alignas(16) WaveSmem {
  static constexpr int TT = Cfg<RB>::TT;
  static constexpr int RG = RESID ? G : 1;
  static constexpr int RT = RESID ? TT : 1;
  static constexpr int RD = RESID ? D : 1;
  static constexpr int RE = RESID ? kEntChunk : 8;
  using Acc = std::conditional_t<kFixedResid<RB, G>, long long, float>;
  float resid[RG][RT];                 // key-residual score per head and token
  float p[RT][RG];                     // tile probabilities (for value residuals)
  float rsv[RT];                       // gate-folded residual scale, values
  Acc racc[RG][RD];                    // value-residual accumulator
  int ex;                              // fixed point: the wave's scale bound, for the epilogue
  uint8_t eidx[2][RE];                 // staged channel bytes (keys, values)
  uint8_t eval[2][RE / 2];             // staged code bytes (2 entries per byte)
  uint8_t emap[RE];                    // tile token of each staged entry
};

template <int RB, int G, bool RESID>
struct Smem {
  alignas(16) float qs[D][G];          // q * sm_scale * log2(e)
  float qt[G][RB];                     // q~ = B^K q (scaled)
  alignas(16) uint16_t bvs[RB][D];     // B^V rows (fp16 bits) for the projection
  float ep_m[kWaves][G];
  float ep_l[kWaves][G];
  float ep_a[kWaves][G][RB];
  float sw[kWaves][G];
  float mstar[G];
  float lstar[G];
  float acomb[G][RB];
  int qmax[G];                         // bits of max |q~| per head
  WaveSmem<RB, G, RESID> w[kWaves];
};

// Registers holding one tile's coefficient fragments.
template <int RB>
struct Frags {
  uint2 k[Cfg<RB>::NBK][Cfg<RB>::NS];   // key fragments: 4 coefficients per k-step
  uint2 v[Cfg<RB>::NBK][Cfg<RB>::NS];   // value blocks: 4 tokens of one channel per step
};

struct Meta {
  uint32_t oa, ob;                      // entry range of this lane's token
  uint32_t sk, sv;                      // residual scale bits of this lane's token
};

struct Ent {
  uint32_t ik[2], iv[2];                // staged chunk: channel bytes, 8 per lane (keys, values)
  uint32_t vk, vv;                      // staged chunk: code bytes, 4 per lane (8 entries)
};

template <int RB>
struct State {
  h4 qhi[Cfg<RB>::NS], qlo[Cfg<RB>::NS];
  f4 acc[Cfg<RB>::NS];                  // a~ in MFMA result layout
  float m, l, down;
  int ex;                               // fixed point: bound on the value scales seen, |s_v| < 2^ex
};

// One value-residual term into its accumulator (fixed point or float).
template <typename Acc>
__device__ __forceinline__ void resid_add(Acc* r, float v, double scale) {
  if constexpr (sizeof(Acc) == 8) atomicAdd(reinterpret_cast<unsigned long long*>(r), to_fixed(v, scale));
  else atomicAdd(r, v);
}

struct Ctx {
  const uint16_t* ck;                   // key tiles of this slab (key_index); dense: rows [T][RB]
  const uint16_t* cv;                   // value blocks of this slab (value_index); dense: [NB][RB][16]
  const uint32_t* off;                  // [T+1]
  const uint8_t* idx[2];
  const uint8_t* val[2];
  const uint16_t* sk;
  const uint16_t* sv;
  int64_t c0, c1, tb;                   // chunk [c0, c1); tiles start at tb = c0 & ~15
  int64_t T, nblk;                      // packed tokens, value blocks per slab
  int64_t res_stride;
  int ntile;
};

template <int RB>
__device__ __forceinline__ int64_t tile_start(const Ctx& x, int j) {
  return x.tb + (int64_t)j * Cfg<RB>::TT;
}

// Key fragments (row = token, 4 coefficients per k-step).  From the coefficient
// tiles in the key_k order: lane group g reads a 16-byte piece of coefficient
// group 4 m + g for k-steps 2 m, 2 m + 1 (an odd last k-step: 8-byte halves),
// so every instruction reads whole tile rows, nontemporal.  For a dense cache
// (TILED false) rows [T][RB], coefficients KH g + 4 s + i.
template <int RB, bool TILED>
__device__ __forceinline__ void load_k(Frags<RB>& f, const Ctx& x, int j, int lane) {
  using C = Cfg<RB>;
  typedef uint32_t u4n __attribute__((ext_vector_type(4)));
  typedef uint32_t u2n __attribute__((ext_vector_type(2)));
  const int64_t t0 = tile_start<RB>(x, j);
  const int grp = lane >> 4, col = lane & 15;
#pragma unroll
  for (int bk = 0; bk < C::NBK; ++bk) {
    if constexpr (TILED) {
      const int64_t blk = min((t0 >> 4) + bk, x.nblk - 1);
      const uint16_t* tile = x.ck + blk * 16 * RB + col * 8;
#pragma unroll
      for (int s = 0; s + 1 < C::NS; s += 2) {
        const u4n w = __builtin_nontemporal_load(reinterpret_cast<const u4n*>(tile + (2 * s + grp) * 128));
        f.k[bk][s] = make_uint2(w.x, w.y);
        f.k[bk][s + 1] = make_uint2(w.z, w.w);
      }
      if constexpr (C::NS % 2 == 1) {
        const u2n w = __builtin_nontemporal_load(
            reinterpret_cast<const u2n*>(tile + (2 * (C::NS - 1) + (grp >> 1)) * 128 + 4 * (grp & 1)));
        f.k[bk][C::NS - 1] = make_uint2(w.x, w.y);
      }
    } else {
      const int64_t row = min(t0 + 16 * bk + col, x.T - 1);
#pragma unroll
      for (int s = 0; s < C::NS; ++s)
        f.k[bk][s] = *reinterpret_cast<const uint2*>(x.ck + row * RB + C::KH * grp + 4 * s);
    }
  }
}

// Value rows (4 consecutive tokens of one channel): from the coefficient
// blocks (value_index) or, for a dense cache, 16-token blocks [T16/16][RB][16].
template <int RB, bool TILED>
__device__ __forceinline__ void load_v(Frags<RB>& f, const Ctx& x, int j, int lane) {
  using C = Cfg<RB>;
  const int64_t b0 = tile_start<RB>(x, j) >> 4;
  const int grp = lane >> 4, col = lane & 15;
#pragma unroll
  for (int bk = 0; bk < C::NBK; ++bk) {
    const int64_t blk = min(b0 + bk, x.nblk - 1);
#pragma unroll
    for (int s = 0; s < C::NS; ++s) {
      const int c = col + 16 * s;
      if constexpr (TILED) {             // 16 channels x 16 bytes of two 8-token blocks: whole lines
        typedef uint32_t u2n __attribute__((ext_vector_type(2)));
        const u2n w = __builtin_nontemporal_load(
            reinterpret_cast<const u2n*>(x.cv + value_index(16 * blk + 4 * grp, c, RB)));
        f.v[bk][s] = make_uint2(w.x, w.y);
      } else {
        f.v[bk][s] = *reinterpret_cast<const uint2*>(x.cv + (blk * RB + c) * 16 + 4 * grp);
      }
    }
  }
}

// Entry range of tile j's lane token, clipped to the chunk (tokens outside the
// chunk own no entries).
template <int RB>
__device__ __forceinline__ void load_offsets(Meta& m, const Ctx& x, int j, int lane) {
  const int64_t t = tile_start<RB>(x, j) + lane;
  m.oa = x.off[clamp64(t, x.c0, x.c1)];
  m.ob = x.off[clamp64(t + 1, x.c0, x.c1)];
}

template <int RB>
__device__ __forceinline__ void load_scales(Meta& m, const Ctx& x, int j, int lane) {
  const int64_t t = clamp64(tile_start<RB>(x, j) + lane, x.c0, x.c1 - 1);
  m.sk = x.sk[t];
  m.sv = x.sv[t];
}

// The load is unconditional, its address clamped into the slab, so every wave
// issues the same sequence of vector loads whatever the data and the compiler
// can wait for each load by its exact position in the queue.  Bytes at or past
// the slab end are never used (a tile's entries end before it), so the value
// read for a clamped position does not matter.
__device__ __forceinline__ uint32_t load_dword_clamped(const uint8_t* base, int64_t pos, int64_t len) {
  return *reinterpret_cast<const uint32_t*>(base + min(pos, len - 4));
}

template <int TT>
__device__ __forceinline__ void tile_entry_range(const Meta& m, uint32_t& e0, uint32_t& e1) {
  e0 = (uint32_t)__shfl((int)m.oa, 0);
  e1 = (uint32_t)__shfl((int)m.ob, TT - 1);
  // a well-formed tile holds at most TT*d entries; the bound keeps a corrupt
  // offset table from running the loops long
  if (e1 < e0) e1 = e0;
  if (e1 - e0 > (uint32_t)(TT * D)) e1 = e0 + TT * D;
}

// The staged chunk of a tile starts at the 8-aligned entry at or below its
// first entry; it holds kEntChunk entries (channel bytes) and their codes.
__device__ __forceinline__ uint32_t chunk_base(uint32_t e0) { return e0 & ~7u; }

template <int TT>
__device__ __forceinline__ void load_entries(Ent& en, const Ctx& x, const Meta& m, int lane) {
  uint32_t e0, e1;
  tile_entry_range<TT>(m, e0, e1);
  const int64_t ia = chunk_base(e0), va = ia >> 1;
  en.ik[0] = load_dword_clamped(x.idx[0], ia + 4 * lane, x.res_stride);
  en.ik[1] = load_dword_clamped(x.idx[0], ia + 256 + 4 * lane, x.res_stride);
  en.iv[0] = load_dword_clamped(x.idx[1], ia + 4 * lane, x.res_stride);
  en.iv[1] = load_dword_clamped(x.idx[1], ia + 256 + 4 * lane, x.res_stride);
  en.vk = load_dword_clamped(x.val[0], va + 4 * lane, x.res_stride / 2);
  en.vv = load_dword_clamped(x.val[1], va + 4 * lane, x.res_stride / 2);
}

// Key residual, one lane per token: the lane walks its own entries (no
// atomics), adds code * q[c] per head, and records its index in the entry map
// the value pass reads.  `staged`: every entry lies in the LDS chunk; else the
// entries are read from HBM.
template <int RB, int G>
__device__ __forceinline__ void key_resid_tokens(WaveSmem<RB, G, true>& ws, const Ctx& x,
                                                 const float (*qs)[G], const Meta& m, uint32_t ia,
                                                 bool staged, int lane) {
  constexpr int TT = Cfg<RB>::TT;
  if (lane >= TT) return;
  float acc[G];
#pragma unroll
  for (int g = 0; g < G; ++g) acc[g] = 0.f;
  uint32_t e = m.oa;
  const uint32_t hi = m.ob;
  if (staged) {
    // four entries at a time while aligned (ranks that are multiples of 4 keep
    // every token's entries 4-aligned), then pairs (ranks are even)
    for (; e + 4 <= hi && ((e - ia) & 3) == 0; e += 4) {
      const uint32_t r = e - ia;
      const uint32_t cw = *reinterpret_cast<const uint32_t*>(&ws.eidx[0][r]);
      const uint32_t vw = *reinterpret_cast<const uint16_t*>(&ws.eval[0][r >> 1]);
      *reinterpret_cast<uint32_t*>(&ws.emap[r]) = 0x01010101u * (uint32_t)lane;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t c = (cw >> (8 * j)) & (D - 1);
        const float code = (float)int4_value(vw >> (4 * j));
        const float* q = qs[c];
#pragma unroll
        for (int g = 0; g < G; ++g) acc[g] += code * q[g];
      }
    }
    for (; e < hi; ++e) {
      const uint32_t r = e - ia;
      const uint32_t c = ws.eidx[0][r] & (D - 1);
      const float code = (float)entry_code(ws.eval[0][r >> 1], e);
      ws.emap[r] = (uint8_t)lane;
#pragma unroll
      for (int g = 0; g < G; ++g) acc[g] += code * qs[c][g];
    }
  } else {
    for (; e < hi; ++e) {
      const uint32_t c = x.idx[0][e] & (D - 1);
      const float code = (float)entry_code(x.val[0][e >> 1], e);
#pragma unroll
      for (int g = 0; g < G; ++g) acc[g] += code * qs[c][g];
    }
  }
  const float rs = half_bits_to_float((uint16_t)m.sk);
#pragma unroll
  for (int g = 0; g < G; ++g) ws.resid[g][lane] = acc[g] * rs;
}

// Value residual, one lane per entry: p * scale * code into its channel's
// accumulator (ds_add_f32; channels of different tokens may coincide).
template <int RB, int G>
__device__ __forceinline__ void value_resid_entries(WaveSmem<RB, G, true>& ws, uint32_t e0, uint32_t e1,
                                                    uint32_t ia, int lane, double scale) {
  for (uint32_t base = e0; base < e1; base += 64) {
    const uint32_t e = base + lane;
    if (e < e1) {
      const uint32_t r = e - ia;
      const int t = ws.emap[r];
      const uint32_t c = ws.eidx[1][r] & (D - 1);
      const float code = (float)entry_code(ws.eval[1][r >> 1], e);
      float pv[G];
#pragma unroll
      for (int g = 0; g < G; ++g) pv[g] = ws.p[t][g];
      const float s = ws.rsv[t] * code;
#pragma unroll
      for (int g = 0; g < G; ++g) resid_add(&ws.racc[g][c], pv[g] * s, scale);
    }
  }
}

// Value residual for a tile too large for the LDS chunk: one lane per token,
// entries read from HBM.
template <int RB, int G>
__device__ __forceinline__ void value_resid_tokens_global(WaveSmem<RB, G, true>& ws, const Ctx& x,
                                                          const Meta& m, int lane, double scale) {
  if (lane >= Cfg<RB>::TT) return;
  float pv[G];
#pragma unroll
  for (int g = 0; g < G; ++g) pv[g] = ws.p[lane][g];
  const float rs = half_bits_to_float((uint16_t)m.sv);
  for (uint32_t e = m.oa; e < m.ob; ++e) {
    const uint32_t c = x.idx[1][e] & (D - 1);
    const float s = rs * (float)entry_code(x.val[1][e >> 1], e);
#pragma unroll
    for (int g = 0; g < G; ++g) resid_add(&ws.racc[g][c], pv[g] * s, scale);
  }
}

template <int RB, int G, bool RESID, bool TILED>
__device__ __forceinline__ void step(State<RB>& st, Frags<RB>& fr, Meta& mc, Meta& mn, Meta& mnn,
                                     Ent& ec, Ent& en, int j, const Ctx& x, Smem<RB, G, RESID>& sm,
                                     WaveSmem<RB, G, RESID>& ws, int lane) {
  using C = Cfg<RB>;
  constexpr int TT = C::TT, NBK = C::NBK, NS = C::NS;
  const int grp = lane >> 4, col = lane & 15;
  const int64_t t0 = tile_start<RB>(x, j);
  const int jn = j + kWaves, jnn = j + 2 * kWaves;
  const bool has_next = jn < x.ntile;
  // past the wave's last tile the prefetches re-read a tile of this chunk
  // (cache resident, results unused) so the load sequence stays the same
  const int jn_l = has_next ? jn : j;
  const int jnn_l = jnn < x.ntile ? jnn : jn_l;

  // 1. stage this tile's residual entries; request the next tiles' metadata
  uint32_t e0 = 0, e1 = 0, ia = 0;
  bool staged = true;
  if constexpr (RESID) {
    tile_entry_range<TT>(mc, e0, e1);
    ia = chunk_base(e0);
    staged = e1 <= ia + (uint32_t)kEntChunk;
    if (lane < TT) ws.rsv[lane] = half_bits_to_float((uint16_t)mc.sv);
    reinterpret_cast<uint32_t*>(ws.eidx[0])[lane] = ec.ik[0];
    reinterpret_cast<uint32_t*>(ws.eidx[0])[lane + 64] = ec.ik[1];
    reinterpret_cast<uint32_t*>(ws.eidx[1])[lane] = ec.iv[0];
    reinterpret_cast<uint32_t*>(ws.eidx[1])[lane + 64] = ec.iv[1];
    reinterpret_cast<uint32_t*>(ws.eval[0])[lane] = ec.vk;
    reinterpret_cast<uint32_t*>(ws.eval[1])[lane] = ec.vv;
    load_offsets<RB>(mnn, x, jnn_l, lane);
    load_entries<TT>(en, x, mn, lane);
    load_scales<RB>(mn, x, jn_l, lane);
    wave_lds_fence();
  }

  // 2. basis-space scores on MFMA (q~ hi + lo); then the next key fragments
  f4 sacc[NBK];
#pragma unroll
  for (int bk = 0; bk < NBK; ++bk) {
    sacc[bk] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const h4 av = __builtin_bit_cast(h4, fr.k[bk][s]);
      sacc[bk] = mfma16(av, st.qhi[s], sacc[bk]);
      sacc[bk] = mfma16(av, st.qlo[s], sacc[bk]);
    }
  }
  load_k<RB, TILED>(fr, x, jn_l, lane);

  // 3. key residual entries add q[c]*code*scale to their token's score
  if constexpr (RESID) {
    key_resid_tokens<RB, G>(ws, x, sm.qs, mc, ia, staged, lane);
    wave_lds_fence();
  }

  // 4. online softmax (exp2 units); this lane holds head `col`, tokens 16bk+4grp+i
  float sc[NBK][4];
  float mt = -INFINITY;
#pragma unroll
  for (int bk = 0; bk < NBK; ++bk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tok = 16 * bk + 4 * grp + i;
      const int64_t t = t0 + tok;
      float s = sacc[bk][i] * st.down;
      if constexpr (RESID) {
        if (col < G) s += ws.resid[col][tok];
      }
      s = (t >= x.c0 && t < x.c1) ? s : -INFINITY;
      sc[bk][i] = s;
      mt = fmaxf(mt, s);
    }
  }
  mt = fmaxf(mt, __shfl_xor(mt, 16));
  mt = fmaxf(mt, __shfl_xor(mt, 32));
  const float mnew = fmaxf(st.m, mt);
  const float alpha = exp2_hw(st.m - mnew);
  float psum = 0.f;
#pragma unroll
  for (int bk = 0; bk < NBK; ++bk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float p = col < G ? exp2_hw(sc[bk][i] - mnew) : 0.f;
      sc[bk][i] = p;
      psum += p;
    }
  }
  st.l = st.l * alpha + psum;
  st.m = mnew;

  // 5. rescale the basis-space value accumulator (rows g = 4grp+i)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float ai = __shfl(alpha, 4 * grp + i);
#pragma unroll
    for (int cb = 0; cb < NS; ++cb) st.acc[cb][i] *= ai;
  }

  if constexpr (RESID) {
    // 6. rescale the value-residual accumulator when a running max moved
    const bool moved = (col < G) && (alpha != 1.0f);
    if (__ballot(moved) != 0) {
#pragma unroll
      for (int it = 0; it < (G * D) / 64; ++it) {
        const int g = (it * 64) / D;
        const float ag = __shfl(alpha, g);
        auto& r = (&ws.racc[0][0])[it * 64 + lane];
        if constexpr (kFixedResid<RB, G>) r = __double2ll_rn((double)r * (double)ag);
        else r *= ag;
      }
    }
    // 7. probabilities to LDS for the value entries
    if (col < G) {
#pragma unroll
      for (int bk = 0; bk < NBK; ++bk)
#pragma unroll
        for (int i = 0; i < 4; ++i) ws.p[16 * bk + 4 * grp + i][col] = sc[bk][i];
    }
  }

  // 8. a~ += P A^V on MFMA (P hi + lo); then the next value fragments
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
      const h4 vf = __builtin_bit_cast(h4, fr.v[bk][cb]);
      st.acc[cb] = mfma16(ph, vf, st.acc[cb]);
      st.acc[cb] = mfma16(pl, vf, st.acc[cb]);
    }
  }
  load_v<RB, TILED>(fr, x, jn_l, lane);

  // 9. value residual entries scatter p*code*scale into their channel
  if constexpr (RESID) {
    double scale = 0.0;
    if constexpr (kFixedResid<RB, G>) {
      // a value scale beyond the wave's bound shifts the accumulators down first
      const uint32_t eb = (mc.sv >> 10) & 31u;
      const int el = lane < TT ? (int)max(eb, 1u) - 14 : st.ex;
      if (__ballot(el > st.ex) != 0) {
        int emax = el;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) emax = max(emax, __shfl_xor(emax, o));
        const double f = ldexp(1.0, st.ex - emax);
        for (int i = lane; i < G * D; i += 64) {
          auto& r = (&ws.racc[0][0])[i];
          r = __double2ll_rn((double)r * f);
        }
        st.ex = emax;
      }
      scale = ldexp(1.0, kFxTopG - st.ex);
    }
    wave_lds_fence();
    if (e1 > e0) {
      if (staged) value_resid_entries<RB, G>(ws, e0, e1, ia, lane, scale);
      else value_resid_tokens_global<RB, G>(ws, x, mc, lane, scale);
    }
    wave_lds_fence();
    mc = mn;
    mn = mnn;
    ec = en;
  }
}

template <int RB, int G, bool RESID, bool IDENT>
__global__ __launch_bounds__(kThreads) void split_kernel(const SplitArgs a) {
  using C = Cfg<RB>;
  constexpr int NS = C::NS, TT = C::TT;
  __shared__ Smem<RB, G, RESID> sm;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int grp = lane >> 4, col = lane & 15;
  const int slot = blockIdx.y;
  const int kvh = a.kv_of_slot[slot];
  pin_split_args(a, kvh);
  if constexpr (IDENT) {
    if (a.zero && blockIdx.x == 0 && blockIdx.y == 0)
      for (int i = threadIdx.x; i < a.n_zero; i += kThreads) a.zero[i] = 0;
  }

  // work item -> (sequence, chunk)
  const int w = blockIdx.x;
  int b;
  Ctx x;
  work_item(a.wt, a.cu, a.batch, a.split, w, b, x.c0, x.c1, a.trim);
  x.c1 = min(x.c1, a.T);
  x.c0 = min(x.c0, x.c1);
  x.tb = x.c0 & ~(int64_t)15;
  x.ntile = (int)((x.c1 - x.tb + TT - 1) / TT);
  x.T = a.T;
  x.nblk = (a.T + 15) / 16;
  x.res_stride = a.res_stride;
  // the reference rows are stored per probed slot, the factorized cache per KV head
  const int64_t ch = IDENT ? slot : kvh;
  x.ck = a.coef_k + ch * (IDENT ? a.T : x.nblk * 16) * RB;
  x.cv = a.coef_v + ch * x.nblk * 16 * RB;
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

  // Requests in issue order (vector loads complete in order): the first
  // tile's offsets and scales; the query, B^K rows and B^V rows; the first
  // tile's coefficient fragments; last its residual entries, whose addresses
  // need the offsets.  Every load is unconditional (a wave with no tile reads
  // the chunk's last one and never uses it).
  constexpr int NIT = (RB * 4 + kThreads - 1) / kThreads;   // q~ work items per thread
  constexpr int QPT = (G * D + kThreads - 1) / kThreads;     // query elements per thread
  constexpr int BVQ = IDENT ? 1 : RB * D / 8 / kThreads;     // 16-byte B^V chunks per thread
  const int j0 = min(wv, x.ntile - 1);
  const int j1 = min(wv + kWaves, x.ntile - 1);
  Frags<RB> fr;
  Meta mc{}, mn{}, mnn{};
  Ent ec{}, en{};
  if constexpr (RESID) {
    load_offsets<RB>(mc, x, j0, lane);
    load_scales<RB>(mc, x, j0, lane);
    load_offsets<RB>(mn, x, j1, lane);
  }
  __builtin_amdgcn_sched_barrier(0);
  uint4 rv[NIT][4];
  uint16_t qraw[QPT];
#pragma unroll
  for (int n = 0; n < QPT; ++n) {
    const int i = min(tid + n * kThreads, G * D - 1);
    qraw[n] = a.q[((int64_t)b * a.n_q_heads + kvh * G + i / D) * D + i % D];
  }
  if constexpr (!IDENT) {
#pragma unroll
    for (int n = 0; n < NIT; ++n) {
      const int it = min(tid + n * kThreads, RB * 4 - 1);
      const uint4* row = reinterpret_cast<const uint4*>(bk_rows + (it >> 2) * D + (it & 3) * 32);
#pragma unroll
      for (int i = 0; i < 4; ++i) rv[n][i] = row[i];
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  load_k<RB, !IDENT>(fr, x, j0, lane);
  load_v<RB, !IDENT>(fr, x, j0, lane);
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (RESID) load_entries<TT>(ec, x, mc, lane);
  if (tid < G) sm.qmax[tid] = 0;
#pragma unroll
  for (int n = 0; n < QPT; ++n) {
    const int i = tid + n * kThreads;
    if (i < G * D)
      sm.qs[i % D][i / D] = (a.q_bf16 ? bf16_bits_to_float(qraw[n]) : half_bits_to_float(qraw[n])) * a.qscale;
  }
  __syncthreads();
  if constexpr (!IDENT) {
#pragma unroll
    for (int n = 0; n < NIT; ++n) {
      const int it = tid + n * kThreads;
      if (it >= RB * 4) continue;
      const int k = it >> 2, qq = it & 3;
      float acc[G];
#pragma unroll
      for (int g = 0; g < G; ++g) acc[g] = 0.f;
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        const uint32_t dw = dword_at(rv[n][e >> 3], (e >> 1) & 3);
        const float xv = half_bits_to_float((uint16_t)((e & 1) ? (dw >> 16) : (dw & 0xFFFF)));
#pragma unroll
        for (int g = 0; g < G; ++g) acc[g] += xv * sm.qs[qq * 32 + e][g];
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        acc[g] += __shfl_xor(acc[g], 1);
        acc[g] += __shfl_xor(acc[g], 2);
      }
      if (qq == 0) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
          sm.qt[g][k] = acc[g];
          atomicMax(&sm.qmax[g], __float_as_int(fabsf(acc[g])));
        }
      }
    }
  } else {
    for (int i = tid; i < G * D; i += kThreads) {
      const int g = i / D, c = i % D;
      atomicMax(&sm.qmax[g], __float_as_int(fabsf(sm.qs[c][g])));
    }
  }
  __syncthreads();

  // q~ as MFMA B operand (column = head), scaled by a power of two so its
  // largest entry sits just under 2^14, split into fp16 hi + lo
  State<RB> st;
  {
    int kexp = 0;
    if (col < G) {
      const float mx = __int_as_float(sm.qmax[col]);
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
        const int k = IDENT ? C::KH * grp + 4 * s + i : key_k<NS>(s, grp, i);
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
  st.ex = -14;
  auto& ws = sm.w[wv];
  if constexpr (RESID) {
    for (int i = lane; i < G * D; i += 64) (&ws.racc[0][0])[i] = 0;
  }

  // Every prologue load completes before the loop (the first iteration needs
  // the last of them at once), so the loop's own waits count only the loop's
  // loads and stay exact.
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);

  // stream the wave's tiles
  for (int j = wv; j < x.ntile; j += kWaves) step<RB, G, RESID, !IDENT>(st, fr, mc, mn, mnn, ec, en, j, x, sm, ws, lane);
  if constexpr (RESID) {
    if (lane == 0) ws.ex = st.ex;      // read by every thread after the epilogue's barrier
  }

  // epilogue: the 4 waves merge (B^V rows, needed only for the projection,
  // are requested while they do), project a~ through B^V, write the partial
  const int c_out = tid % D, par = tid / D;
  st.l += __shfl_xor(st.l, 16);
  st.l += __shfl_xor(st.l, 32);
  if (grp == 0 && col < G) {
    sm.ep_m[wv][col] = st.m;
    sm.ep_l[wv][col] = st.l;
  }
#pragma unroll
  for (int cb = 0; cb < NS; ++cb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = 4 * grp + i;
      if (g < G) sm.ep_a[wv][g][16 * cb + col] = st.acc[cb][i];
    }
  u4v bvr[BVQ];
  if constexpr (!IDENT) {
#pragma unroll
    for (int n = 0; n < BVQ; ++n) bvr[n] = reinterpret_cast<const u4v*>(bv_rows)[tid + n * kThreads];
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
  if constexpr (!IDENT) {
#pragma unroll
    for (int n = 0; n < BVQ; ++n) reinterpret_cast<u4v*>(&sm.bvs[0][0])[tid + n * kThreads] = bvr[n];
  }
  __syncthreads();
  for (int i = tid; i < G * RB; i += kThreads) {
    const int g = i / RB, k = i % RB;
    float s = 0.f;
    for (int v = 0; v < kWaves; ++v) s += sm.sw[v][g] * sm.ep_a[v][g][k];
    sm.acomb[g][k] = s;
  }
  __syncthreads();
  float* const part_ws = a.part;
  for (int g = par; g < G; g += kThreads / D) {
    float o;
    if constexpr (IDENT) {
      o = sm.acomb[g][c_out];
    } else {
      o = 0.f;
#pragma unroll 16
      for (int k = 0; k < RB; ++k) o += sm.acomb[g][k] * half_bits_to_float(sm.bvs[k][c_out]);
    }
    if constexpr (RESID) {
      for (int v = 0; v < kWaves; ++v) {
        if constexpr (kFixedResid<RB, G>)
          o += sm.sw[v][g] * (fixed_to_float(sm.w[v].racc[g][c_out]) * ldexpf(1.0f, sm.w[v].ex - kFxTopG));
        else
          o += sm.sw[v][g] * sm.w[v].racc[g][c_out];
      }
    }
    float* dst = part_ws + (((int64_t)w * a.n_slots + slot) * G + g) * kPartStride;
    dst[c_out] = o;
    if (c_out == 0) {
      dst[D] = sm.mstar[g];
      dst[D + 1] = sm.lstar[g];
    }
  }

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

}  // namespace

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
