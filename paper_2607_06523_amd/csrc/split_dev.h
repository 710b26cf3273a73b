#pragma once
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
// Mapping (one workgroup = NW waves, 4 in the general launch, = one chunk of
// `split` tokens of one sequence and one KV head; each wave streams every
// NW-th tile of 16*NBK tokens):
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
//    residual entries one tile ahead; a wave's last tile requests nothing.
//  * online softmax in exp2 units; running max via lane shuffles.
//  * residual entries: one lane per entry; token of an entry from an LDS map
//    written by the token lanes; key entries add into an LDS score buffer,
//    value entries into an LDS d-vector per head (ds_add_f32).
//  * epilogue: the 4 waves merge (m, l, a~, r) in LDS, project a~ through B^V
//    and write one partial (o, m, l) per query head; a merge kernel combines
//    the splits (and computes Eq. 3's error for probed heads).
//  * the wave count is a template argument: the probe's reference pass inside
//    the token-lane launch runs one item on that launch's 8 waves.
//
// The device code lives in this header so that the token-lane launch with a
// probe can run the reference pass (identity basis, dense fp16 rows) in its
// own grid: split_body takes the work item and slot as arguments.
#include <type_traits>

#include "entry.h"
#include "internal.h"

namespace dwkv {
namespace gsplit {

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

template <int RB, int G, bool RESID, int NW = kWaves>
struct Smem {
  alignas(16) float qs[D][G];          // q * sm_scale * log2(e)
  float qt[G][RB];                     // q~ = B^K q (scaled)
  alignas(16) uint16_t bvs[RB][D];     // B^V rows (fp16 bits) for the projection
  float ep_m[NW][G];
  float ep_l[NW][G];
  float ep_a[NW][G][RB];
  float sw[NW][G];
  float mstar[G];
  float lstar[G];
  float acomb[G][RB];
  int qmax[G];                         // bits of max |q~| per head
  WaveSmem<RB, G, RESID> w[NW];
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

// One tile of the wave; LAST: the wave's last tile, which requests nothing
// for later tiles (a request there would hold the epilogue until it lands).
template <int RB, int G, bool RESID, bool TILED, int NW, bool LAST>
__device__ __forceinline__ void step(State<RB>& st, Frags<RB>& fr, Meta& mc, Meta& mn, Meta& mnn,
                                     Ent& ec, Ent& en, int j, const Ctx& x, Smem<RB, G, RESID, NW>& sm,
                                     WaveSmem<RB, G, RESID>& ws, int lane) {
  using C = Cfg<RB>;
  constexpr int TT = C::TT, NBK = C::NBK, NS = C::NS;
  const int grp = lane >> 4, col = lane & 15;
  const int64_t t0 = tile_start<RB>(x, j);
  const int jn = j + NW, jnn = j + 2 * NW;
  // two tiles ahead of the wave's second-to-last tile the offset prefetch
  // re-reads a tile of this chunk (cache resident, results unused)
  const int jn_l = jn < x.ntile ? jn : j;
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
    if constexpr (!LAST) {
      load_offsets<RB>(mnn, x, jnn_l, lane);
      load_entries<TT>(en, x, mn, lane);
      load_scales<RB>(mn, x, jn_l, lane);
    }
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
  if constexpr (!LAST) load_k<RB, TILED>(fr, x, jn_l, lane);

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
  if constexpr (!LAST) load_v<RB, TILED>(fr, x, jn_l, lane);

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

// One work item (chunk w of a sequence, head slot `slot`) on the NW waves of
// the workgroup (thread index tid); wave v streams tiles v, v + NW, ...
template <int RB, int G, bool RESID, bool IDENT, int NW = kWaves>
__device__ __forceinline__ void split_body(const SplitArgs& a, int w, int slot, int tid,
                                           Smem<RB, G, RESID, NW>& sm) {
  constexpr int kThreads = 64 * NW;
  using C = Cfg<RB>;
  constexpr int NS = C::NS, TT = C::TT;
  const int lane = tid & 63, wv = tid >> 6;
  const int grp = lane >> 4, col = lane & 15;
  const int kvh = a.kv_of_slot[slot];
  pin_split_args(a, kvh);
  if constexpr (IDENT) {
    if (a.zero && w == 0 && slot == 0)
      for (int i = tid; i < a.n_zero; i += kThreads) a.zero[i] = 0;
  }

  // work item -> (sequence, chunk)
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
  const int j1 = min(wv + NW, x.ntile - 1);
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
  int j = wv;
  for (; j + NW < x.ntile; j += NW) step<RB, G, RESID, !IDENT, NW, false>(st, fr, mc, mn, mnn, ec, en, j, x, sm, ws, lane);
  if (j < x.ntile) step<RB, G, RESID, !IDENT, NW, true>(st, fr, mc, mn, mnn, ec, en, j, x, sm, ws, lane);
  if constexpr (RESID) {
    if (lane == 0) ws.ex = st.ex;      // read by every thread after the epilogue's barrier
  }

  // epilogue: the waves merge (B^V rows, needed only for the projection,
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
    for (int v = 0; v < NW; ++v) mx = fmaxf(mx, sm.ep_m[v][g]);
    float l = 0.f;
    for (int v = 0; v < NW; ++v) {
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
    for (int v = 0; v < NW; ++v) s += sm.sw[v][g] * sm.ep_a[v][g][k];
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
      for (int v = 0; v < NW; ++v) {
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

}  // namespace gsplit
}  // namespace dwkv
