// Token-lane split-K decode attention over the cross-depth factorized KV cache,
// gfx950, for query groups of 1, 2, 4 (ranks up to 16) or 8 heads (ranks up
// to 32) and basis ranks up to 64.
//
// Same arithmetic as the general kernel (Sec. 3, Eq. 1 used through its
// linearity: scores A^K_t (B^K q) plus the routed residual channels, values
// (sum_t p_t A^V_t) B^V plus the routed residual channels), organised so that
// every lane of a wave owns one token of a 64-token tile for the whole step:
//
//  * scores on v_mfma_f32_16x16x32_f16 (16x16x16 for an odd 16-deep rest of
//    r_b) with the coefficient rows as the B operand (column = token) and
//    q~ = B^K q as the A operand, its 4 head rows repeated in each of the 4
//    row groups.  The result of 16-token block bk then
//    holds the 4 head scores of token 16bk+c in lane c of every lane group, and
//    lane 16g+c keeps block g's copy: each lane ends up with its own token's
//    scores for all heads, in registers.
//  * key residual, one lane per token: the token's entries (a window of
//    channel bytes and int4 codes per lane, straight from HBM) add code*q[c]
//    to its scores (q from an LDS table) with no exchange between lanes.
//  * value residual, one lane per entry: token lanes publish p*scale and mark
//    their entries in an entry->token map; entry lanes add p*code*scale into
//    a per-wave accumulator of the value channels.  The accumulator is fixed
//    point in int64 (ds_add_u64): integer LDS atomics cost a few cycles per
//    instruction, float ones a few cycles per active lane.
//  * softmax with a lazily moved reference: the running reference of a head
//    moves only when a score exceeds it by more than 2^8, so probabilities stay
//    below 256 and the rescaling of the value accumulators is rare.
//  * values on v_mfma_f32_4x4x4f16 (16 blocks): a 4x4 transpose inside each
//    lane quad turns the probabilities into (head, 4 tokens) rows; each
//    instruction broadcasts one quad's rows to all blocks (CBSZ/ABID) and the
//    blocks cover 64 coefficient channels, read as 4 consecutive tokens of one
//    channel from the 8-token value blocks.  The accumulator holds, in lane c,
//    the basis-space value of channel c for the 4 heads.
//  * the epilogue combines the waves and writes the partial in basis space
//    (a~, the residual channels, m, l).  A second, wide launch merges them in
//    a fixed order and applies B^V: one workgroup per (KV head, query head,
//    16 output channels), so that every CU reads a small share.
#include <utility>

#include "compress_dev.h"
#include "entry.h"
#include "internal.h"
#include "split_dev.h"

namespace dwkv {
namespace {

typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));
typedef uint32_t u3v __attribute__((ext_vector_type(3)));
typedef uint32_t u2v __attribute__((ext_vector_type(2)));

constexpr int D = kHeadDim;
constexpr int TT = 64;                  // tokens per tile = lanes per wave
constexpr float kLazy = 8.0f;           // log2 headroom of the running reference
constexpr int kVB = 3;                  // value-entry batches of 64 loaded ahead per tile

// Sizes that follow the query-group size G: groups of up to 4 heads use 4
// head rows in the score product and read ranks up to 16; groups of 8 use 8
// head rows (two groups of 4 in the value product) and read ranks up to 32.
template <int G>
struct TGrp {
  static constexpr int HG = G > 4 ? 8 : 4;     // head rows (heads past G are zero)
  static constexpr int NHG = HG / 4;           // groups of 4 heads
  static constexpr int MR = G > 4 ? 32 : 16;   // residual entries per token the kernel reads
  static constexpr int KR = G > 4 ? 4 : 8;     // key-residual entries per LDS lookup round
  static constexpr int NR = MR / KR;           // lookup rounds for the largest rank
  static constexpr int EMAP = TT * MR;         // residual entries a tile can hold
  static constexpr int CW = MR / 4 + 1;        // channel-byte dwords of a lane's entry window
  static constexpr int VW = MR / 8 + 1;        // code dwords of the window
  static_assert(G == 1 || G == 2 || G == 4 || G == 8, "query group");
};
constexpr int kFxTop = 34;              // fixed-point fraction bits = kFxTop - scale exponent bound
constexpr int kWaitVmcnt0 = 0x0F70;     // s_waitcnt immediate: vmcnt(0) only
constexpr int kNT = 2;                  // buffer cache policy: nontemporal (whole lines read once)
constexpr int kTW = kTLWaves;           // waves per workgroup (one workgroup per CU)
constexpr int kTThreads = 64 * kTW;

template <int RB>
struct TCfg {
  static constexpr int NS = RB / 16;    // k-steps of the score product
  static constexpr int KH = RB / 4;     // coefficients of a row one lane holds
  static_assert(RB % 16 == 0 && RB >= 16 && RB <= 64, "basis rank");
};

template <int RB, int G, bool RESID>
struct alignas(16) TSmem {
  static constexpr int HG = TGrp<G>::HG;
  alignas(16) float qs[D][HG];          // q * sm_scale * log2(e), heads past G zero
  float qt[HG][RB];                     // q~ = B^K q (scaled)
  float ep_m[kTW][HG];
  float ep_l[kTW][HG];
  float ep_a[kTW][HG][RB];
  float qmaxw[4][HG];                   // per q~ wave: largest |q~| of each head
  // groups of 8 (and r_b 64 with int8 codes): the score product's q~
  // operands (hi, lo per k-step, the lane's fragment), re-read each tile
  // instead of held in registers
  static constexpr bool QLDS = HG == 8 || RB == 64;
  alignas(16) h4 qa[QLDS ? 2 : 1][QLDS ? TCfg<RB>::NS : 1][64];
  // Value residual, per wave.  Accumulators are fixed point in units of
  // 2^(ex - kFxTop) (ex: the wave's bound on the value scales): integer LDS
  // atomics run at one instruction per few cycles whatever the active lanes,
  // float LDS atomics at a few cycles per lane.  After its loop a wave
  // rewrites its accumulators as floats [HG][D] in the same storage.
  long long racc[kTW][RESID ? HG : 1][RESID ? D : 1];
  alignas(4) uint8_t emap[kTW][RESID ? TGrp<G>::EMAP : 4];  // token lane + 1 at each token's first entry
  alignas(16) float pw[kTW][RESID ? TT : 1][HG];  // p * value scale per token lane
};

template <int RB, bool C8>
struct TFrags {
  uint2 k[4][TCfg<RB>::NS];             // key fragments (tile order, key_k), block bk, k-step s
  uint2 v[16];                          // value channel `lane`, token quad q
};

// int8-blockwise coefficients: 4 codes per dword, and the lane's own token's
// block scales (block s covers coefficients [16 s, 16 s + 16))
template <int RB>
struct TFrags<RB, true> {
  uint32_t k[4][TCfg<RB>::NS];          // token 16 bk + col, coefficients 16 s + 4 grp + (0..3)
  uint32_t v[16];                       // channel `lane`, the 4 tokens of quad q
  uint32_t ks[TCfg<RB>::NS];            // key scale bits of block s, token `lane`
  uint32_t vs[TCfg<RB>::NS];            // value scale bits of block s, token `lane`
};

struct TMeta {
  uint32_t oa, ob;                      // entry range of this lane's token
  uint32_t sk, sv;                      // residual scale bits
};

template <int G>
struct TEnt {
  uint32_t ck[TGrp<G>::CW], vk[TGrp<G>::VW];  // key channel bytes / codes around this lane's oa
  uint32_t vc[kVB], vv[kVB];            // value entries e0 + 64b + lane: channel byte, code byte
};

template <int RB, int G, bool C8>
struct TState {
  static constexpr int HG = TGrp<G>::HG;
  static constexpr int NACC = C8 ? TCfg<RB>::NS : TGrp<G>::NHG;
  h4 qhi[TCfg<RB>::NS], qlo[TCfg<RB>::NS];
  f4 acc_h[NACC], acc_l[NACC];          // a~[head][channel lane] from p hi / p lo: one pair per group
                                        // of 4 heads (int8: one pair per coefficient block, each
                                        // valid in its block's lanes)
  float m[HG], l[HG], down[HG];
  int ex;                               // bound on the value scales seen: |s_v| < 2^ex
};

// Every stream is read through a raw buffer resource over its slab: offsets
// are 32-bit and a read past the slab returns zero, so no load needs a clamp
// for safety (the host keeps every slab below 2^31 bytes).
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;  // raw (untyped) buffer, gfx9 family

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kRsrcWord3);
}

struct TCtx {
  rsrc_t ck, cv;                        // coefficient slabs (bytes)
  rsrc_t off, sk, sv;                   // offsets and residual scales of the slab
  rsrc_t idx[2], val[2];                // residual channel bytes and code bytes (K, V)
  int32_t c0, c1, tb;                   // chunk [c0, c1); tiles start at tb = c0 & ~15
  int32_t ntile;
  float* sco;                           // raw scores of this slot [T][G] (score-storing pass only)
  rsrc_t cks, cvs;                      // int8 coefficients: block scales [NS][T] (fp16)
  int32_t T;
};

__device__ __forceinline__ f4 mfma16(h4 a, h4 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
}

// 16x16x32: same cost per instruction as 16x16x16 on gfx950, twice the depth.
// The operand k index of (lane group, element) only has to agree between A
// and B, so two 4-element quads of a lane form one 8-element operand.
__device__ __forceinline__ f4 mfma32(h4 a0, h4 a1, h4 b0, h4 b1, f4 c) {
  const h8 a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
  const h8 b = __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ int32_t tstart(const TCtx& x, int j) { return x.tb + j * TT; }

// signed 4-bit code in bits [4n, 4n+4) of w
__device__ __forceinline__ float code_at(uint32_t w, int n) {
  return (float)((int32_t)(w << (28 - 4 * n)) >> 28);
}

// Key tiles (16 tokens x 8 coefficients, key_index): for a pair of 16-deep
// k-steps lane group g reads coefficient group 4 m + g of its token, 16 bytes;
// for an odd last k-step lane groups 2 i and 2 i + 1 read the two halves of
// group 4 m + i.  Every instruction reads whole 256-byte tile rows.
template <int RB>
__device__ __forceinline__ void load_k(TFrags<RB, false>& f, const TCtx& x, int j, int lane) {
  using C = TCfg<RB>;
  const int grp = lane >> 4, col = lane & 15;
  const uint32_t blk0 = (uint32_t)tstart(x, j) >> 4;
#pragma unroll
  for (int bk = 0; bk < 4; ++bk) {
    const uint32_t tile = (blk0 + bk) * (RB / 8);
#pragma unroll
    for (int s = 0; s + 1 < C::NS; s += 2) {
      const uint32_t g8 = 2 * s + grp;
      const u4v w = __builtin_amdgcn_raw_buffer_load_b128(x.ck, ((tile + g8) * 128 + col * 8) * 2, 0, kNT);
      f.k[bk][s] = make_uint2(w.x, w.y);
      f.k[bk][s + 1] = make_uint2(w.z, w.w);
    }
    if constexpr (C::NS % 2 == 1) {
      const uint32_t g8 = 2 * (C::NS - 1) + (grp >> 1);
      const u2v w = __builtin_amdgcn_raw_buffer_load_b64(x.ck, ((tile + g8) * 128 + col * 8 + 4 * (grp & 1)) * 2, 0, kNT);
      f.k[bk][C::NS - 1] = make_uint2(w.x, w.y);
    }
  }
}

// Value blocks (8 tokens, value_index): lane c reads channel c's 8 tokens of
// each block, quads 2 u and 2 u + 1; one instruction reads a whole block.
// Lanes past r_b read nothing (their products are never used).
template <int RB>
__device__ __forceinline__ void load_v(TFrags<RB, false>& f, const TCtx& x, int j, int lane) {
  if (lane < RB) {
    const uint32_t base = ((uint32_t)(tstart(x, j) >> 3) * RB + lane) * 16;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const u4v w = __builtin_amdgcn_raw_buffer_load_b128(x.cv, base + u * RB * 16, 0, kNT);
      f.v[2 * u] = make_uint2(w.x, w.y);
      f.v[2 * u + 1] = make_uint2(w.z, w.w);
    }
  }
}

// 4 signed bytes to fp16, in the order (b0, b2, b1, b3): each byte, offset by
// 128, becomes the low byte of the fp16 number 1024 + byte, exact, then
// 1152 is subtracted.  Operands built from these take the same k order.
__device__ __forceinline__ h4 i8x4_to_h4(uint32_t w) {
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  const uint32_t u = w ^ 0x80808080u;
  const h2 lo = __builtin_bit_cast(h2, __builtin_amdgcn_perm(0x64646464u, u, 0x04020400u)) - h2{1152, 1152};
  const h2 hi = __builtin_bit_cast(h2, __builtin_amdgcn_perm(0x64646464u, u, 0x04030401u)) - h2{1152, 1152};
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3);
}

// int8 key tiles (16 tokens x 16 codes): k-step s of lane (grp, col) is codes
// 16 s + 4 grp .. + 4 of token col, so one instruction reads a whole 256-byte
// tile.  Value blocks: lane c reads channel c's 16 codes, lanes past r_b
// nothing.  Scales: one 2-byte load per lane and block.
template <int RB>
__device__ __forceinline__ void load_k8(TFrags<RB, true>& f, const TCtx& x, int j, int lane) {
  using C = TCfg<RB>;
  const int grp = lane >> 4, col = lane & 15;
  const uint32_t blk0 = (uint32_t)tstart(x, j) >> 4;
#pragma unroll
  for (int bk = 0; bk < 4; ++bk)
#pragma unroll
    for (int s = 0; s < C::NS; ++s)
      f.k[bk][s] = __builtin_amdgcn_raw_buffer_load_b32(x.ck, ((blk0 + bk) * C::NS + s) * 256 + col * 16 + 4 * grp, 0, kNT);
  const uint32_t t = (uint32_t)(tstart(x, j) + lane);
#pragma unroll
  for (int s = 0; s < C::NS; ++s)
    f.ks[s] = __builtin_amdgcn_raw_buffer_load_b16(x.cks, ((uint32_t)s * (uint32_t)x.T + t) * 2, 0, 0);
}

template <int RB>
__device__ __forceinline__ void load_v8(TFrags<RB, true>& f, const TCtx& x, int j, int lane) {
  using C = TCfg<RB>;
  if (lane < RB) {
    // 16 bytes per (16-token block, channel): the 16 tokens' codes of channel `lane`
    const uint32_t base = ((uint32_t)(tstart(x, j) >> 4) * RB + lane) * 16;
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      const u4v w = __builtin_amdgcn_raw_buffer_load_b128(x.cv, base + tb * RB * 16, 0, kNT);
      f.v[4 * tb] = w.x;
      f.v[4 * tb + 1] = w.y;
      f.v[4 * tb + 2] = w.z;
      f.v[4 * tb + 3] = w.w;
    }
  }
  const uint32_t t = (uint32_t)(tstart(x, j) + lane);
#pragma unroll
  for (int s = 0; s < C::NS; ++s)
    f.vs[s] = __builtin_amdgcn_raw_buffer_load_b16(x.cvs, ((uint32_t)s * (uint32_t)x.T + t) * 2, 0, 0);
}

template <int RB, bool C8>
__device__ __forceinline__ void load_coef(TFrags<RB, C8>& f, const TCtx& x, int j, int lane) {
  if constexpr (C8) {
    load_k8<RB>(f, x, j, lane);
    load_v8<RB>(f, x, j, lane);
  } else {
    load_k<RB>(f, x, j, lane);
    load_v<RB>(f, x, j, lane);
  }
}

// Tiles of wave w in a chunk of `ntile` 64-token tiles.  Waves w and w + 4
// share a SIMD, and the older one (w < 4) issues first, so the pair's tiles
// j = p + 4 i (p = w % 4, i = 0 .. m - 1) are split unevenly: the older wave
// takes every even i and, when the pair has an even count of at least four,
// also the last one; the younger wave takes the other odd i.  At 32 tiles per
// chunk that is 5 and 3 tiles.  The assignment is fixed, so each wave's
// summation order does not depend on timing.
static_assert(kTW == 8, "the tile schedule pairs waves w and w + 4");
struct TileSeq {
  int p, m, older, n;
  __device__ __forceinline__ int at(int k) const {
    if (!older) return p + 4 * (2 * k + 1);
    return k < (m + 1) / 2 ? p + 8 * k : p + 4 * (m - 1);
  }
};

__device__ __forceinline__ TileSeq tile_seq(int w, int ntile) {
  TileSeq t;
  t.p = w & 3;
  t.m = ntile > t.p ? (ntile - t.p + 3) / 4 : 0;
  t.older = w < 4;
  const int extra = (t.m >= 4 && (t.m & 1) == 0) ? 1 : 0;
  t.n = t.older ? (t.m + 1) / 2 + extra : t.m / 2 - extra;
  return t;
}

// Entry range of the lane's token, clipped to the chunk (tokens outside it own
// no entries).
__device__ __forceinline__ void load_offsets(TMeta& m, const TCtx& x, int j, int lane) {
  const int32_t t = tstart(x, j) + lane;
  m.oa = __builtin_amdgcn_raw_buffer_load_b32(x.off, (uint32_t)min(max(t, x.c0), x.c1) * 4, 0, 0);
  m.ob = __builtin_amdgcn_raw_buffer_load_b32(x.off, (uint32_t)min(max(t + 1, x.c0), x.c1) * 4, 0, 0);
}

// Scales of tokens outside the chunk are read but never used.
__device__ __forceinline__ void load_scales(TMeta& m, const TCtx& x, int j, int lane) {
  const uint32_t t = (uint32_t)(tstart(x, j) + lane);
  m.sk = __builtin_amdgcn_raw_buffer_load_b16(x.sk, t * 2, 0, 0);
  m.sv = __builtin_amdgcn_raw_buffer_load_b16(x.sv, t * 2, 0, 0);
}

// Key entries: the window around the lane's own entries, 4 CW channel bytes
// from oa rounded down to 4 and 4 VW code bytes from oa/2 rounded down to 4
// (MR entries; oa is even).  Value entries: the tile's first 64*kVB, one per
// lane and batch.  Bytes past the entries in use are never used.
template <int N>
__device__ __forceinline__ void load_words(uint32_t (&w)[N], rsrc_t r, uint32_t off) {
#pragma unroll
  for (int i = 0; i + 4 <= N; i += 4) {
    const u4v v = __builtin_amdgcn_raw_buffer_load_b128(r, off + 4 * i, 0, 0);
    w[i] = v.x; w[i + 1] = v.y; w[i + 2] = v.z; w[i + 3] = v.w;
  }
  constexpr int R = N % 4, B = N - R;
  if constexpr (R == 3) {
    const u3v v = __builtin_amdgcn_raw_buffer_load_b96(r, off + 4 * B, 0, 0);
    w[B] = v.x; w[B + 1] = v.y; w[B + 2] = v.z;
  } else if constexpr (R == 2) {
    const u2v v = __builtin_amdgcn_raw_buffer_load_b64(r, off + 4 * B, 0, 0);
    w[B] = v.x; w[B + 1] = v.y;
  } else if constexpr (R == 1) {
    w[B] = __builtin_amdgcn_raw_buffer_load_b32(r, off + 4 * B, 0, 0);
  }
}

template <int G>
__device__ __forceinline__ void load_entries(TEnt<G>& e, const TCtx& x, const TMeta& m, int lane) {
  const uint32_t a = m.oa & ~3u, ca = (m.oa >> 1) & ~3u;
  load_words(e.ck, x.idx[0], a);
  load_words(e.vk, x.val[0], ca);
  const uint32_t e0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)m.oa);
#pragma unroll
  for (int b = 0; b < kVB; ++b) {
    const uint32_t pos = e0 + 64 * b + lane;
    e.vc[b] = __builtin_amdgcn_raw_buffer_load_b8(x.idx[1], pos, 0, 0);
    e.vv[b] = __builtin_amdgcn_raw_buffer_load_b8(x.val[1], pos >> 1, 0, 0);
  }
}

// Order LDS traffic between lanes of one wave.
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Channel bytes of entries [4w, 4w+4) of the token and its MR codes, aligned.
template <int G>
struct Window {
  uint32_t ch[TGrp<G>::MR / 4];
  uint32_t cd[TGrp<G>::MR / 8];
};

template <int G>
__device__ __forceinline__ Window<G> align_window(const uint32_t* cw, const uint32_t* vw, uint32_t oa) {
  Window<G> w;
  const uint32_t sc = oa & 3u, sv = (oa >> 1) & 3u;
#pragma unroll
  for (int i = 0; i < TGrp<G>::MR / 4; ++i) w.ch[i] = __builtin_amdgcn_alignbyte(cw[i + 1], cw[i], sc);
#pragma unroll
  for (int i = 0; i < TGrp<G>::MR / 8; ++i) w.cd[i] = __builtin_amdgcn_alignbyte(vw[i + 1], vw[i], sv);
  return w;
}

// Whole-wave reductions without LDS: DPP inside each row of 16 (lane xor 1,
// xor 2, then the half-row and row mirrors), which leaves every lane of a
// row with the row's result, then the four rows' results read into scalar
// registers and combined in a fixed order.  Every lane returns the same bits.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));        // quad_perm(1,0,3,2)
  v = fmaxf(v, dpp_f<0x4E>(v));        // quad_perm(2,3,0,1)
  v = fmaxf(v, dpp_f<0x141>(v));       // row_half_mirror
  v = fmaxf(v, dpp_f<0x140>(v));       // row_mirror
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

// Inclusive running maximum over the lanes of a wave (non-negative values):
// DPP shifts within rows of 16, then row broadcasts across rows.
__device__ __forceinline__ int wave_incl_max(int v) {
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false));   // row_shr:1
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false));   // row_shr:2
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false));   // row_shr:4
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false));   // row_shr:8
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false));   // row_bcast:15
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false));   // row_bcast:31
  return v;
}

__device__ __forceinline__ int wave_imax(int v) {
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false));
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false));
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false));
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false));
  return max(max(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
             max(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}

__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  v += dpp_f<0x141>(v);
  v += dpp_f<0x140>(v);
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return (r0 + r1) + (r2 + r3);
}

// 4x4 transpose inside each lane quad: lane 4q+r holds row r (x[0..3]) on
// entry and column r on exit.
__device__ __forceinline__ void quad_transpose(float (&x)[4], int lane) {
  const bool b1 = (lane & 2) != 0, b0 = (lane & 1) != 0;
  float t[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)   // partner lane ^ 2
    t[i] = __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x[i]), 0x4E, 0xF, 0xF, false));
  if (b1) { x[0] = t[2]; x[1] = t[3]; } else { x[2] = t[0]; x[3] = t[1]; }
#pragma unroll
  for (int i = 0; i < 4; ++i)   // partner lane ^ 1
    t[i] = __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x[i]), 0xB1, 0xF, 0xF, false));
  if (b0) { x[0] = t[1]; x[2] = t[3]; } else { x[1] = t[0]; x[3] = t[2]; }
}

template <int Q>
__device__ __forceinline__ void pv_quad(f4& acc_h, f4& acc_l, h4 ph, h4 pl, uint2 v) {
  const h4 b = __builtin_bit_cast(h4, v);
  acc_h = __builtin_amdgcn_mfma_f32_4x4x4f16(ph, b, acc_h, 4, Q, 0);
  acc_l = __builtin_amdgcn_mfma_f32_4x4x4f16(pl, b, acc_l, 4, Q, 0);
}

template <int... Q>
__device__ __forceinline__ void pv_tile(f4& acc_h, f4& acc_l, h4 ph, h4 pl, const uint2 (&v)[16],
                                        std::integer_sequence<int, Q...>) {
  (pv_quad<Q>(acc_h, acc_l, ph, pl, v[Q]), ...);
}

template <int... Q>
__device__ __forceinline__ void pv_tile_h(f4& acc_h, f4& acc_l, h4 ph, h4 pl, const h4 (&v)[16],
                                          std::integer_sequence<int, Q...>) {
  ((acc_h = __builtin_amdgcn_mfma_f32_4x4x4f16(ph, v[Q], acc_h, 4, Q, 0),
    acc_l = __builtin_amdgcn_mfma_f32_4x4x4f16(pl, v[Q], acc_l, 4, Q, 0)), ...);
}

template <int RB, int G, bool RESID, bool SCORES, bool C8, bool LAST>
__device__ __forceinline__ void tstep(TState<RB, G, C8>& st, TFrags<RB, C8>& fr, TMeta& mc, TMeta& mn, TMeta& mnn,
                                      TEnt<G>& ec, TEnt<G>& en, int j, int jn, int jnn, const TCtx& x,
                                      TSmem<RB, G, RESID>& sm, int wv, int lane) {
  using C = TCfg<RB>;
  using Q = TGrp<G>;
  constexpr int NS = C::NS;
  constexpr int HG = Q::HG, NHG = Q::NHG, MR = Q::MR, KR = Q::KR, NR = Q::NR;
  const int grp = lane >> 4;
  const int32_t t0 = tstart(x, j);
  // two tiles ahead of the wave's second-to-last tile the offset prefetch
  // re-reads a tile of this chunk (cache resident, results unused)
  const int jn_l = jn < x.ntile ? jn : j;
  const int jnn_l = jnn < x.ntile ? jnn : jn_l;

  // 1. metadata of the next tiles, issued here, ahead of this tile's work (the
  // registers rotate at the end of the step and the copies wait for them).
  // The wave's last step requests nothing.
  if constexpr (RESID && !LAST) {
    load_offsets(mnn, x, jnn_l, lane);
    load_entries(en, x, mn, lane);
    load_scales(mn, x, jn_l, lane);
  }
  __builtin_amdgcn_sched_barrier(0);

  // 1b. residual work that does not need the scores, requested here so that
  // its LDS round trips overlap the score MFMAs: the key residual's first
  // query-table lookups, and the entry->token map of the value residual
  // (token lanes mark their first entry; a running maximum over the entry
  // lanes resolves it after the scores)
  uint32_t rank = 0, e0 = 0, n = 0;
  uint32_t cd[MR / 8] = {};
  Window<G> wk{};
  f4 qv0[KR][NHG];
  if constexpr (RESID) {
    rank = min(mc.ob - mc.oa, (uint32_t)MR);
    if (mc.ob < mc.oa) rank = 0;
    wk = align_window<G>(ec.ck, ec.vk, mc.oa);
    // codes past the token's rank read as zero: mask the packed code words
    // once (rank <= MR, 4 bits per entry)
    const uint32_t nb = 4u * rank;
#pragma unroll
    for (int k = 0; k < MR / 8; ++k) {
      const uint32_t lo = 32u * k;
      cd[k] = nb >= lo + 32u ? wk.cd[k] : (nb <= lo ? 0u : wk.cd[k] & ((1u << (nb - lo)) - 1u));
    }
#pragma unroll
    for (int u = 0; u < KR; ++u)
#pragma unroll
      for (int h = 0; h < NHG; ++h)
        qv0[u][h] = *reinterpret_cast<const f4*>(&sm.qs[(wk.ch[u >> 2] >> (8 * (u & 3))) & (D - 1)][4 * h]);
    e0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)mc.oa);
    const uint32_t e1 = (uint32_t)__builtin_amdgcn_readlane((int)mc.ob, 63);
    n = e1 > e0 ? min(e1 - e0, (uint32_t)Q::EMAP) : 0u;
    for (uint32_t i = 4 * lane; i < n; i += 256) *reinterpret_cast<uint32_t*>(&sm.emap[wv][i]) = 0u;
    if (rank > 0 && mc.oa - e0 < n) sm.emap[wv][mc.oa - e0] = (uint8_t)(lane + 1);
  }

  // the q~ operands: from registers, or for groups of 8 from the LDS table
  h4 qh[NS], ql[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    if constexpr (HG == 8 || (C8 && RB == 64)) {
      qh[k] = sm.qa[0][k][lane];
      ql[k] = sm.qa[1][k][lane];
    } else {
      qh[k] = st.qhi[k];
      ql[k] = st.qlo[k];
    }
  }

  // 2. scores: block bk lands in every lane group; lane group g keeps block g
  f4 sacc[4];
#pragma unroll
  for (int bk = 0; bk < 4; ++bk) sacc[bk] = f4{0.f, 0.f, 0.f, 0.f};
  if constexpr (C8) {
    // one 16-deep product per coefficient block, scaled by the lane's own
    // token's block scale (other blocks' lanes are discarded below)
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const float ksc = half_bits_to_float((uint16_t)fr.ks[s]);
#pragma unroll
      for (int bk = 0; bk < 4; ++bk) {
        const h4 kf = i8x4_to_h4(fr.k[bk][s]);
        f4 o = mfma16(qh[s], kf, f4{0.f, 0.f, 0.f, 0.f});
        o = mfma16(ql[s], kf, o);
#pragma unroll
        for (int i = 0; i < 4; ++i) sacc[bk][i] += o[i] * ksc;
      }
    }
    if constexpr (!LAST) load_k8<RB>(fr, x, jn_l, lane);
  } else {
#pragma unroll
    for (int s = 0; s + 1 < NS; s += 2)
#pragma unroll
      for (int bk = 0; bk < 4; ++bk) {
        const h4 k0 = __builtin_bit_cast(h4, fr.k[bk][s]), k1 = __builtin_bit_cast(h4, fr.k[bk][s + 1]);
        sacc[bk] = mfma32(qh[s], qh[s + 1], k0, k1, sacc[bk]);
        sacc[bk] = mfma32(ql[s], ql[s + 1], k0, k1, sacc[bk]);
      }
    if constexpr (NS % 2 == 1) {
#pragma unroll
      for (int bk = 0; bk < 4; ++bk) {
        const h4 kf = __builtin_bit_cast(h4, fr.k[bk][NS - 1]);
        sacc[bk] = mfma16(qh[NS - 1], kf, sacc[bk]);
        sacc[bk] = mfma16(ql[NS - 1], kf, sacc[bk]);
      }
    }
    if constexpr (!LAST) load_k<RB>(fr, x, jn_l, lane);
  }
  float sc[HG];
  if constexpr (HG == 4) {
#pragma unroll
    for (int i = 0; i < HG; ++i) {
      const float a01 = grp == 0 ? sacc[0][i] : sacc[1][i];
      const float a23 = grp == 2 ? sacc[2][i] : sacc[3][i];
      sc[i] = (grp < 2 ? a01 : a23) * st.down[i];
    }
  } else {
    // 8 head rows: lane group g holds heads 4 (g & 1) .. + 3 of every block;
    // its own token's other four heads are in the partner group g ^ 1's copy
    // of block g, fetched with one row swap (v_permlane16_swap)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a01 = grp == 0 ? sacc[0][i] : sacc[1][i];
      const float a23 = grp == 2 ? sacc[2][i] : sacc[3][i];
      const float own = grp < 2 ? a01 : a23;
      const float b01 = grp == 0 ? sacc[1][i] : sacc[0][i];
      const float b23 = grp == 2 ? sacc[3][i] : sacc[2][i];
      const uint32_t y = __builtin_bit_cast(uint32_t, grp < 2 ? b01 : b23);
      const auto r = __builtin_amdgcn_permlane16_swap(y, y, false, false);
      const float oth = __builtin_bit_cast(float, (grp & 1) ? r[0] : r[1]);
      sc[i] = ((grp & 1) ? oth : own) * st.down[i];
      sc[4 + i] = ((grp & 1) ? own : oth) * st.down[4 + i];
    }
  }

  // 3. key residual: this lane's entries add code * q[c] * scale
  int tk[kVB];                          // value residual: token lane + 1 of each preloaded entry
  int carry = 0;
  if constexpr (RESID) {
    float rk[HG];
#pragma unroll
    for (int i = 0; i < HG; ++i) rk[i] = 0.f;
    // entries 0 .. KR-1 from the lookups of step 1b, then further rounds of
    // KR while some token of the wave has more entries
#pragma unroll
    for (int u = 0; u < KR; ++u) {
      const float code = code_at(cd[u >> 3], u & 7);
#pragma unroll
      for (int i = 0; i < G; ++i) rk[i] += code * qv0[u][i >> 2][i & 3];
    }
#pragma unroll
    for (int r = 1; r < NR; ++r) {
      if (__ballot(rank > (uint32_t)(KR * r)) == 0) break;
      f4 qv[KR][NHG];
#pragma unroll
      for (int u = 0; u < KR; ++u) {
        const int e = KR * r + u;
#pragma unroll
        for (int h = 0; h < NHG; ++h)
          qv[u][h] = *reinterpret_cast<const f4*>(&sm.qs[(wk.ch[e >> 2] >> (8 * (e & 3))) & (D - 1)][4 * h]);
      }
#pragma unroll
      for (int u = 0; u < KR; ++u) {
        const int e = KR * r + u;
        const float code = code_at(cd[e >> 3], e & 7);
#pragma unroll
        for (int i = 0; i < G; ++i) rk[i] += code * qv[u][i >> 2][i & 3];
      }
    }
    const float rs = half_bits_to_float((uint16_t)mc.sk);
#pragma unroll
    for (int i = 0; i < G; ++i) sc[i] += rk[i] * rs;
    // the value residual's entry->token map: entry e's token is the last
    // token lane whose first entry is <= e
    wave_lds_fence();
#pragma unroll
    for (int bb = 0; bb < kVB; ++bb) tk[bb] = sm.emap[wv][64 * bb + lane];
#pragma unroll
    for (int bb = 0; bb < kVB; ++bb) {
      tk[bb] = 64u * bb + lane < n ? tk[bb] : 0;
      tk[bb] = max(wave_incl_max(tk[bb]), carry);
      carry = __builtin_amdgcn_readlane(tk[bb], 63);
    }
  }
  {
    const int32_t t = t0 + lane;
    const bool valid = t >= x.c0 && t < x.c1;
#pragma unroll
    for (int i = 0; i < HG; ++i) sc[i] = (valid && i < G) ? sc[i] : -INFINITY;
    if constexpr (SCORES) {             // the token's scores, for the attention-mass features
      if (valid) {
        float* dst = x.sco + (int64_t)t * G;
        if constexpr (G == 8) {
          *reinterpret_cast<f4*>(dst) = f4{sc[0], sc[1], sc[2], sc[3]};
          *reinterpret_cast<f4*>(dst + 4) = f4{sc[4], sc[5], sc[6], sc[7]};
        } else if constexpr (G == 4) *reinterpret_cast<f4*>(dst) = f4{sc[0], sc[1], sc[2], sc[3]};
        else if constexpr (G == 2) *reinterpret_cast<float2*>(dst) = make_float2(sc[0], sc[1]);
        else dst[0] = sc[0];
      }
    }
  }

  // 4. softmax against the lazily moved reference
  {
    bool need = false;
#pragma unroll
    for (int i = 0; i < G; ++i) need |= sc[i] > st.m[i] + kLazy;
    if (__ballot(need) != 0) {
      float alpha[HG];
#pragma unroll
      for (int i = 0; i < HG; ++i) {
        const float mnew = i < G ? fmaxf(st.m[i], wave_max(sc[i])) : st.m[i];
        alpha[i] = mnew == -INFINITY ? 1.0f : exp2f(st.m[i] - mnew);
        st.m[i] = mnew;
        st.l[i] *= alpha[i];
      }
      // accumulator pair b, element i holds head i (int8: one pair per
      // coefficient block) or head 4 b + i (one pair per group of 4 heads)
#pragma unroll
      for (int b = 0; b < TState<RB, G, C8>::NACC; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float al = alpha[C8 ? i : 4 * b + i];
          st.acc_h[b][i] *= al;
          st.acc_l[b][i] *= al;
        }
      if constexpr (RESID) {
#pragma unroll
        for (int i = 0; i < G; ++i) {
          long long* r = &sm.racc[wv][i][0];
          r[lane] = __double2ll_rn((double)r[lane] * (double)alpha[i]);
          r[lane + 64] = __double2ll_rn((double)r[lane + 64] * (double)alpha[i]);
        }
      }
    }
  }
  float p[HG];
#pragma unroll
  for (int i = 0; i < HG; ++i) {
    p[i] = sc[i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sc[i] - st.m[i]);
    st.l[i] += p[i];
  }

  // 5. a~ += P A^V: quad transpose, fp16 hi + lo, one 4x4x4 pair per quad
  if constexpr (C8) {
    // int8: the codes are exact fp16 operands; the value block scale of each
    // token goes into its probabilities, one pass per coefficient block
    h4 vb[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) vb[q] = i8x4_to_h4(fr.v[q]);
#pragma unroll
    for (int b = 0; b < NS; ++b) {
      const float vsc = half_bits_to_float((uint16_t)fr.vs[b]);
      float pt[4] = {p[0] * vsc, p[1] * vsc, p[2] * vsc, p[3] * vsc};
      quad_transpose(pt, lane);
      h4 ph, pl;
      constexpr int ord[4] = {0, 2, 1, 3};      // the k order of i8x4_to_h4
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const _Float16 hh = (_Float16)pt[ord[i]];
        ph[i] = hh;
        pl[i] = (_Float16)(pt[ord[i]] - (float)hh);
      }
      pv_tile_h(st.acc_h[b], st.acc_l[b], ph, pl, vb, std::make_integer_sequence<int, 16>{});
    }
    if constexpr (!LAST) load_v8<RB>(fr, x, jn_l, lane);
  } else {
#pragma unroll
    for (int hg = 0; hg < NHG; ++hg) {      // one pass per group of 4 heads
      float pt[4] = {p[4 * hg], p[4 * hg + 1], p[4 * hg + 2], p[4 * hg + 3]};
      quad_transpose(pt, lane);
      h4 ph, pl;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const _Float16 hh = (_Float16)pt[i];
        ph[i] = hh;
        pl[i] = (_Float16)(pt[i] - (float)hh);
      }
      pv_tile(st.acc_h[hg], st.acc_l[hg], ph, pl, fr.v, std::make_integer_sequence<int, 16>{});
    }
    if constexpr (!LAST) load_v<RB>(fr, x, jn_l, lane);
  }

  // 6. value residual, one lane per entry: p * code * scale into the channel
  // accumulators.  Token lanes publish p * scale; entry lanes read their
  // token's through the map built in step 3.
  if constexpr (RESID) {
    // keep |p * code * s_v| * 2^fx below 2^45 (2^8 * 2^3 * 2^ex): a larger
    // scale exponent shifts the accumulators down first
    {
      const uint32_t eb = (mc.sv >> 10) & 31u;
      const int el = (int)max(eb, 1u) - 14;
      if (__ballot(el > st.ex) != 0) {
        const int emax = wave_imax(el);
        const double f = ldexp(1.0, st.ex - emax);
#pragma unroll
        for (int i = 0; i < G; ++i) {
          long long* r = &sm.racc[wv][i][0];
          r[lane] = __double2ll_rn((double)r[lane] * f);
          r[lane + 64] = __double2ll_rn((double)r[lane + 64] * f);
        }
        st.ex = emax;
      }
    }
    const double scale = ldexp(1.0, kFxTop - st.ex);
    const float rs = half_bits_to_float((uint16_t)mc.sv);
#pragma unroll
    for (int hg = 0; hg < NHG; ++hg)
      *reinterpret_cast<f4*>(&sm.pw[wv][lane][4 * hg]) =
          f4{p[4 * hg] * rs, p[4 * hg + 1] * rs, p[4 * hg + 2] * rs, p[4 * hg + 3] * rs};
    wave_lds_fence();
    f4 wv4[kVB][NHG];
#pragma unroll
    for (int bb = 0; bb < kVB; ++bb)
#pragma unroll
      for (int hg = 0; hg < NHG; ++hg)
        wv4[bb][hg] = *reinterpret_cast<const f4*>(&sm.pw[wv][max(tk[bb] - 1, 0)][4 * hg]);
#pragma unroll
    for (int bb = 0; bb < kVB; ++bb) {
      const uint32_t e = 64u * bb + lane;
      if (e < n) {
        const uint32_t ea = e0 + e;
        const float code = (float)int4_value(ec.vv[bb] >> ((ea & 1u) * 4u));
        const uint32_t c = ec.vc[bb] & (D - 1);
#pragma unroll
        for (int i = 0; i < G; ++i)
          atomicAdd(reinterpret_cast<unsigned long long*>(&sm.racc[wv][i][c]),
                    to_fixed(wv4[bb][i >> 2][i & 3] * code, scale));
      }
    }
    // entries past the preloaded batches (tiles with more than 64 kVB): their
    // bytes are requested kXB batches at a time, one round trip per group
    constexpr int kXB = 4;
    for (uint32_t g0 = 64u * kVB; g0 < n; g0 += 64u * kXB) {
      uint32_t chv[kXB], cbv[kXB];
#pragma unroll
      for (int u = 0; u < kXB; ++u) {   // past the slab a buffer load reads zero
        const uint32_t ea = e0 + g0 + 64u * u + lane;
        chv[u] = __builtin_amdgcn_raw_buffer_load_b8(x.idx[1], ea, 0, 0);
        cbv[u] = __builtin_amdgcn_raw_buffer_load_b8(x.val[1], ea >> 1, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < kXB; ++u) {
        const uint32_t e = g0 + 64u * u + lane;
        if (g0 + 64u * u >= n) break;   // uniform
        int t = e < n ? sm.emap[wv][e] : 0;
        t = max(wave_incl_max(t), carry);
        carry = __builtin_amdgcn_readlane(t, 63);
        if (e < n) {
          const uint32_t ea = e0 + e;
          f4 w[NHG];
#pragma unroll
          for (int hg = 0; hg < NHG; ++hg) w[hg] = *reinterpret_cast<const f4*>(&sm.pw[wv][t - 1][4 * hg]);
          const float code = (float)int4_value(cbv[u] >> ((ea & 1u) * 4u));
          const uint32_t c = chv[u] & (D - 1);
#pragma unroll
          for (int i = 0; i < G; ++i)
            atomicAdd(reinterpret_cast<unsigned long long*>(&sm.racc[wv][i][c]),
                      to_fixed(w[i >> 2][i & 3] * code, scale));
        }
      }
    }
    mc = mn;
    mn = mnn;
    ec = en;
  }
}

constexpr int kSc1 = 16;                // buffer cache policy: device-coherent access

// Wide merge: one workgroup per (slot, head, CH output channels).  Each
// reads, from every partial of its (sequence, slot, head), its CH residual
// channels and all of a~ (plus m, l), merges them in a fixed order and writes
// o = r + a~ B^V for its channels.  Spreading one slot's merge over G * d/16
// workgroups keeps every CU's share of the partials small: the loads of one
// CU, not the bytes, bound a merge that a single workgroup does.
constexpr int kWmThreads = 256;
constexpr int kWmCh = 16;                       // channels of a probe reference chunk

constexpr int kPrG = kWmThreads / (kWmCh / 4);  // reference row groups of a probe chunk (64)
constexpr int kPrRPT = 4;                         // reference partials per thread per round
constexpr int kWmNCH = D / kWmCh;                 // output-channel chunks of a row

// Eq. 3 for a probed column (b, probed slot, group member) in the wide merge:
// its d/CH output chunks (the merge's own workgroups) and its 8 reference
// chunks of 16 channels (extra workgroups) each publish their channels and
// count themselves in; the last of the n_arrive to arrive reads both rows and
// writes err (or, with several positions, the sums to acc), then resets the
// counter.  Nothing waits.
__device__ __forceinline__ void wm_probe_arrive(const WideProbe& P, int64_t col, int64_t orow, const float* out,
                                                uint32_t n_arrive) {
  __shared__ uint32_t arrived;
  // the chunk's rows went out as device-coherent (agent-scope atomic) stores;
  // each wave waits for its own to complete before the count, so a reader
  // that sees the count reaches them with device-coherent loads
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  __syncthreads();
  if (threadIdx.x == 0) arrived = atomicAdd(&P.count[col], 1u);
  __syncthreads();
  if (arrived != n_arrive - 1u) return;
  if (threadIdx.x >= 64) return;
  const int lane = threadIdx.x;
  float d2 = 0.f, r2 = 0.f;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int c = lane + 64 * h;
    const float o = __hip_atomic_load(out + orow + c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const float r = __hip_atomic_load(P.oref + col * D + c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    d2 += (r - o) * (r - o);
    r2 += r * r;
  }
  d2 = wave_sum(d2);
  r2 = wave_sum(r2);
  if (lane == 0) {
    if (P.acc) {
      P.acc[2 * col] = d2;
      P.acc[2 * col + 1] = r2;
    } else {
      P.err[col] = sqrtf(d2) / (sqrtf(r2) + P.eps);
    }
    P.count[col] = 0;                   // ready for the next call
  }
}

// Reference chunk `idx` (probed slot, group member, channel chunk) of
// sequence b: the reference partials' channels [c0, c0 + 16) merged in a
// fixed order (64 row groups of 4 quads, each taking every 64th partial; then
// a butterfly over the wave's row groups and the 4 waves through LDS).
template <int G>
__device__ __forceinline__ void wm_probe_ref(const WMergeArgs& A, int idx, int b, uint32_t n_arrive) {
  __shared__ f4 wr[kWmThreads / 64][kWmCh / 4];
  __shared__ float wmx[kWmThreads / 64][kWmCh / 4], wlx[kWmThreads / 64][kWmCh / 4];
  const SplitArgs& a = A.s;
  const WideProbe& P = A.p;
  const int ch = idx % kWmNCH, g = (idx / kWmNCH) % G, sl = idx / (kWmNCH * G);
  const int c0 = ch * kWmCh;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  int base_r, ns_r;
  seq_work_entry(P.ref_wt, a.cu, P.ref_split, b, base_r, ns_r);
  const int pq = tid % (kWmCh / 4), prg = tid / (kWmCh / 4);
  const int64_t prs = (int64_t)P.n_probe * G * kPartStride;
  const float* pr0 = P.part_ref + (((int64_t)base_r * P.n_probe + sl) * G + g) * kPartStride;
  f4 racc = f4{0.f, 0.f, 0.f, 0.f};
  float rm = -INFINITY, rl = 0.f;
  for (int s0 = 0; s0 < ns_r; s0 += kPrG * kPrRPT) {
    f4 xv[kPrRPT];
    float2 ml[kPrRPT];
#pragma unroll
    for (int i = 0; i < kPrRPT; ++i) {
      const float* row = pr0 + (int64_t)min(s0 + prg + kPrG * i, ns_r - 1) * prs;
      xv[i] = *reinterpret_cast<const f4*>(row + c0 + 4 * pq);
      ml[i] = *reinterpret_cast<const float2*>(row + D);
    }
    float mv[kPrRPT];
    float mr = rm;
#pragma unroll
    for (int i = 0; i < kPrRPT; ++i) {
      mv[i] = s0 + prg + kPrG * i < ns_r ? ml[i].x : -INFINITY;
      mr = fmaxf(mr, mv[i]);
    }
    const float resc = rm == -INFINITY ? 0.f : exp2f(rm - mr);
    racc *= resc;
    rl *= resc;
#pragma unroll
    for (int i = 0; i < kPrRPT; ++i) {
      const float w = mv[i] == -INFINITY ? 0.f : exp2f(mv[i] - mr);
      racc += w * xv[i];
      rl += w * ml[i].y;
    }
    rm = mr;
  }
  // the wave's 16 row groups of each quad (lanes pq, pq + 4, ...)
#pragma unroll
  for (int o = 4; o < 64; o <<= 1) {
    const float m2 = __shfl_xor(rm, o), l2 = __shfl_xor(rl, o);
    const f4 a2 = f4{__shfl_xor(racc.x, o), __shfl_xor(racc.y, o), __shfl_xor(racc.z, o), __shfl_xor(racc.w, o)};
    const float mx = fmaxf(rm, m2);
    const float e1 = rm == -INFINITY ? 0.f : exp2f(rm - mx), e2 = m2 == -INFINITY ? 0.f : exp2f(m2 - mx);
    racc = e1 * racc + e2 * a2;
    rl = e1 * rl + e2 * l2;
    rm = mx;
  }
  if (lane < kWmCh / 4) {
    wr[wv][lane] = racc;
    wmx[wv][lane] = rm;
    wlx[wv][lane] = rl;
  }
  __syncthreads();
  const int64_t col = (int64_t)b * P.n_probe * G + sl * G + g;
  if (tid < kWmCh / 4) {
    float mx = -INFINITY;
#pragma unroll
    for (int v = 0; v < kWmThreads / 64; ++v) mx = fmaxf(mx, wmx[v][tid]);
    f4 r = f4{0.f, 0.f, 0.f, 0.f};
    float l = 0.f;
#pragma unroll
    for (int v = 0; v < kWmThreads / 64; ++v) {
      const float e = wmx[v][tid] == -INFINITY ? 0.f : exp2f(wmx[v][tid] - mx);
      r += e * wr[v][tid];
      l += e * wlx[v][tid];
    }
    r *= l > 0.f ? 1.0f / l : 0.f;
    float* dst = P.oref + col * D + c0 + 4 * tid;
    __hip_atomic_store(dst, r.x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(dst + 1, r.y, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(dst + 2, r.z, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(dst + 3, r.w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (P.out_ref) *reinterpret_cast<f4*>(P.out_ref + col * D + c0 + 4 * tid) = r;
  }
  const int64_t orow = ((int64_t)b * a.n_q_heads + P.kv_of_slot[sl] * G + g) * D;
  if (ns_r > 0) wm_probe_arrive(P, col, orow, a.out, n_arrive);   // an empty sequence: see wm_body
}

// CH output channels per workgroup: 16 (and Eq. 3 for probed heads), or 64
// for merges of a few partials per sequence (fewer, wider workgroups).
template <int RB, int G, int CH>
__global__ __launch_bounds__(kWmThreads) void tl_wmerge_kernel(const WMergeArgs A) {
  const SplitArgs& a = A.s;
  constexpr int QW = CH / 4 + RB / 4;        // quads per row: the r chunk, then a~
  constexpr int RG = kWmThreads / QW;           // row groups
  // partials per thread per round: at 32 channels one round covers 32
  // partials (a 64K sequence's chunks) at every r_b (4.0 us per launch
  // against 4.3 in two rounds); 64-channel columns merge at most kWideFew
  constexpr int RPT = CH >= 64 ? 2 : ((32 + RG - 1) / RG > 2 ? (32 + RG - 1) / RG : 2);
  constexpr int KG = kWmThreads / CH;        // k groups of the projection
  constexpr int KPG = (RB + KG - 1) / KG;       // basis rows per k group
  constexpr int NCH = D / CH;
  __shared__ f4 red[RG][QW];
  __shared__ float wm[RG], wl[RG];
  __shared__ alignas(16) float fin[4 * QW];
  __shared__ float red2[KG][CH];
  const int tid = threadIdx.x;
  if ((int)blockIdx.x >= a.n_slots * G * NCH) {     // a probed column's reference chunk
    wm_probe_ref<G>(A, blockIdx.x - a.n_slots * G * NCH, blockIdx.y, NCH + kWmNCH);
    return;
  }
  const int ch = blockIdx.x % NCH, g = (blockIdx.x / NCH) % G, slot = blockIdx.x / (NCH * G), b = blockIdx.y;
  const int c0 = ch * CH;
  const int kvh = a.kv_of_slot[slot];
  // every kernel argument the merge needs, loaded in one batch at entry
  asm volatile("" ::"s"(a.part), "s"(a.basis), "s"(a.basis_b_stride), "s"(a.out), "s"(a.n_q_heads), "s"(a.n_work),
               "s"(a.split), "s"(kvh), "s"(a.mstats));
  int base, ns;
  seq_work_entry(a.wt, a.cu, a.split, b, base, ns);
  // B^V rows [kg KPG, kg KPG + KPG) of channel c0 + tid % CH
  const int pc = tid % CH, kg = tid / CH;
  const uint16_t* bv = a.basis + (int64_t)b * a.basis_b_stride + ((int64_t)kvh * 2 + 1) * RB * D + c0 + pc;
  uint16_t bvr[KPG];
#pragma unroll
  for (int k = 0; k < KPG; ++k) bvr[k] = bv[(int64_t)min(kg * KPG + k, RB - 1) * D];
  // this thread's quad of every RG-th partial
  const int qi = tid % QW, rg = min(tid / QW, RG - 1);
  const bool active = tid < RG * QW;
  const int64_t rs = (int64_t)G * kPartStrideTL;
  const float* p0 = a.part + (((int64_t)slot * a.n_work + base) * G + g) * kPartStrideTL;
  const rsrc_t pr = make_rsrc(p0, (uint32_t)(max(ns, 1) * rs * 4));
  const uint32_t qoff = qi < CH / 4 ? (uint32_t)(c0 + 4 * qi) : (uint32_t)(D + 4 * (qi - CH / 4));
  f4 acc = f4{0.f, 0.f, 0.f, 0.f};
  float mstar = -INFINITY, lsum = 0.f;
  for (int s0 = 0; s0 < ns; s0 += RG * RPT) {
    u4v xv[RPT];
    u2v ml[RPT];
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const uint32_t s = (uint32_t)min(s0 + rg + RG * i, ns - 1);
      xv[i] = __builtin_amdgcn_raw_buffer_load_b128(pr, (uint32_t)((s * rs + qoff) * 4), 0, kSc1);
      ml[i] = __builtin_amdgcn_raw_buffer_load_b64(pr, (uint32_t)((s * rs + kPartTLM) * 4), 0, kSc1);
    }
    float mv[RPT];
    float mr = mstar;
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      mv[i] = s0 + rg + RG * i < ns ? __uint_as_float(ml[i].x) : -INFINITY;
      mr = fmaxf(mr, mv[i]);
    }
    const float resc = mstar == -INFINITY ? 0.f : exp2f(mstar - mr);
    acc *= resc;
    lsum *= resc;
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const float w = mv[i] == -INFINITY ? 0.f : exp2f(mv[i] - mr);
      acc += w * __builtin_bit_cast(f4, xv[i]);
      lsum += w * __uint_as_float(ml[i].y);
    }
    mstar = mr;
  }
  if (active) {
    red[rg][qi] = acc;
    if (qi == 0) {
      wm[rg] = mstar;
      wl[rg] = lsum;
    }
  }
  __syncthreads();
  if (tid < QW) {
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < RG; ++j) mx = fmaxf(mx, wm[j]);
    f4 o = f4{0.f, 0.f, 0.f, 0.f};
    float l = 0.f;
#pragma unroll
    for (int j = 0; j < RG; ++j) {
      const float e = wm[j] == -INFINITY ? 0.f : exp2f(wm[j] - mx);
      o += e * red[j][tid];
      l += e * wl[j];
    }
    o *= l > 0.f ? 1.0f / l : 0.f;
    *reinterpret_cast<f4*>(&fin[4 * tid]) = o;
    if (a.mstats && ch == 0 && tid == 0) {   // the merged statistics, for the attention features
      float* ms = a.mstats + ((int64_t)b * a.n_q_heads + kvh * G + g) * 2;
      ms[0] = mx;
      ms[1] = l;
    }
  }
  __syncthreads();
  {
    // fin: [r chunk (CH) | a~ (RB)]
    float o = 0.f;
#pragma unroll
    for (int k = 0; k < KPG; ++k)
      if (kg * KPG + k < RB) o += fin[CH + kg * KPG + k] * half_bits_to_float(bvr[k]);
    red2[kg][pc] = o;
  }
  __syncthreads();
  const int sl = A.p.n_probe > 0 ? A.p.slot_of_kv[kvh] : -1;
  const int64_t orow = ((int64_t)b * a.n_q_heads + kvh * G + g) * D;
  if (tid < CH) {
    float o = fin[tid];
#pragma unroll
    for (int j = 0; j < KG; ++j) o += red2[j][tid];
    if (sl >= 0)                        // device-coherent: read back by the column's Eq. 3
      __hip_atomic_store(a.out + orow + c0 + tid, o, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
      a.out[orow + c0 + tid] = o;
  }
  if (sl >= 0) {
    const int64_t col = (int64_t)b * A.p.n_probe * G + sl * G + g;
    if (ns > 0) {
      wm_probe_arrive(A.p, col, orow, a.out, NCH + kWmNCH);
    } else if (ch == 0 && tid == 0) {   // an empty sequence: e = 0 with no count (its counter may be stale)
      if (A.p.acc) {
        A.p.acc[2 * col] = 0.f;
        A.p.acc[2 * col + 1] = 0.f;
      } else {
        A.p.err[col] = 0.f;
      }
    }
  }
}

template <int RB, int G, bool RESID, bool SCORES, bool C8>
__device__ __forceinline__ void tl_body(const SplitArgs& a, TSmem<RB, G, RESID>& sm, int w, int slot) {
  using C = TCfg<RB>;
  constexpr int NS = C::NS;
  constexpr int HG = TGrp<G>::HG;
  static_assert(!C8 || HG == 4, "int8 coefficients: query groups of up to 4 heads");
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int grp = lane >> 4, col = lane & 15;
  const int kvh = a.kv_of_slot[slot];
  pin_split_args(a, kvh);

  // work item -> (sequence, chunk)
  int b;
  TCtx x;
  {
    int64_t c0, c1;
    work_item(a.wt, a.cu, a.batch, a.split, w, b, c0, c1, a.trim);
    c1 = min(c1, a.T);
    c0 = min(c0, c1);
    x.c0 = (int32_t)c0;
    x.c1 = (int32_t)c1;
  }
  x.tb = x.c0 & ~15;
  x.ntile = (x.c1 - x.tb + TT - 1) / TT;
  x.sco = SCORES ? a.scores + (int64_t)slot * a.T * G : nullptr;
  {
    const int64_t T = a.T, nblk = (T + 15) / 16, rs = a.res_stride;
    x.T = (int32_t)T;
    if constexpr (C8) {
      const uint8_t* ck8 = reinterpret_cast<const uint8_t*>(a.coef_k);
      const uint8_t* cv8 = reinterpret_cast<const uint8_t*>(a.coef_v);
      x.ck = make_rsrc(ck8 + (int64_t)slot * nblk * 16 * RB, (uint32_t)(nblk * 16 * RB));
      x.cv = make_rsrc(cv8 + (int64_t)slot * nblk * 16 * RB, (uint32_t)(nblk * 16 * RB));
      x.cks = make_rsrc(a.cscale_k + (int64_t)slot * C::NS * T, (uint32_t)(C::NS * T * 2));
      x.cvs = make_rsrc(a.cscale_v + (int64_t)slot * C::NS * T, (uint32_t)(C::NS * T * 2));
    } else {
      x.ck = make_rsrc(a.coef_k + (int64_t)slot * nblk * 16 * RB, (uint32_t)(nblk * 16 * RB * 2));
      x.cv = make_rsrc(a.coef_v + (int64_t)slot * nblk * 16 * RB, (uint32_t)(nblk * 16 * RB * 2));
    }
    if constexpr (RESID) {
      x.off = make_rsrc(a.off + (int64_t)kvh * (T + 1), (uint32_t)((T + 1) * 4));
      x.idx[0] = make_rsrc(a.idx_k + (int64_t)kvh * rs, (uint32_t)rs);
      x.idx[1] = make_rsrc(a.idx_v + (int64_t)kvh * rs, (uint32_t)rs);
      x.val[0] = make_rsrc(a.val_k + (int64_t)kvh * (rs / 2), (uint32_t)(rs / 2));
      x.val[1] = make_rsrc(a.val_v + (int64_t)kvh * (rs / 2), (uint32_t)(rs / 2));
      x.sk = make_rsrc(a.scale_k + (int64_t)kvh * T, (uint32_t)(T * 2));
      x.sv = make_rsrc(a.scale_v + (int64_t)kvh * T, (uint32_t)(T * 2));
    }
  }
  const uint16_t* bk_rows = a.basis + (int64_t)b * a.basis_b_stride + (int64_t)kvh * 2 * RB * D;

  // Requests in issue order (vector loads complete in order): the first
  // tile's offsets, alone, so that its residual entries can be requested as
  // soon as they return; the fragments of the q~ product (B^K rows, q); the
  // query for the LDS table; the first tile's scales and the second tile's
  // offsets; the residual entries.  Then the coefficient burst of the first
  // tile, which stalls a wave's instruction issue for a while: the waves that
  // do not compute q~ issue it at once, the others once q~ is written, so that
  // q~ is ready before the burst has landed.  One barrier publishes q~ and the
  // query table.  Every tile load is unconditional (a wave with no tile reads
  // the chunk's last one and never uses it).
  constexpr int QPT = (G * D + kTThreads - 1) / kTThreads;     // query elements per thread
  const TileSeq ts = tile_seq(wv, x.ntile);
  const int j0 = ts.n > 0 ? ts.at(0) : x.ntile - 1;
  const int j1 = ts.n > 1 ? ts.at(1) : j0;
  TFrags<RB, C8> fr{};                  // lanes past r_b never load values: keep them zero
  TMeta mc{}, mn{}, mnn{};
  TEnt<G> ec{}, en{};
  // q~ fragments, waves below NS only: wave w takes basis rows [16w, 16w+16)
  // on 16x16x32 MFMA, A = B^K rows (row = lane % 16, channels 32s + 8(lane/16)
  // + i), B = q (column = head lane % 16)
  u4v bkf[4], qf[4];
  if constexpr (RESID) load_offsets(mc, x, j0, lane);
  __builtin_amdgcn_sched_barrier(0);
  if (wv < NS) {
    const uint16_t* brow = bk_rows + (int64_t)(16 * wv + col) * D + 8 * grp;
    const uint16_t* qrow = a.q + ((int64_t)b * a.n_q_heads + kvh * G + min(col, G - 1)) * D + 8 * grp;
#pragma unroll
    for (int s = 0; s < 4; ++s) bkf[s] = *reinterpret_cast<const u4v*>(brow + 32 * s);
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = *reinterpret_cast<const u4v*>(qrow + 32 * s);
  }
  uint16_t qraw[QPT];
#pragma unroll
  for (int n = 0; n < QPT; ++n) {
    const int i = min(tid + n * kTThreads, G * D - 1);
    qraw[n] = a.q[((int64_t)b * a.n_q_heads + kvh * G + i / D) * D + i % D];
  }
  if constexpr (RESID) {
    load_scales(mc, x, j0, lane);
    load_offsets(mn, x, j1, lane);
  }
  __builtin_amdgcn_sched_barrier(0);
  // the waves that do not compute q~ request their first tile now, ahead of
  // the entries (which wait for the offsets)
  if (wv >= NS) load_coef<RB, C8>(fr, x, j0, lane);
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (RESID) load_entries(ec, x, mc, lane);
  __builtin_amdgcn_sched_barrier(0);
  // every entry of the query table once: the group's heads, zeros past G
#pragma unroll
  for (int n = 0; n < (D * HG + kTThreads - 1) / kTThreads; ++n) {
    const int i = tid + n * kTThreads;
    if (i >= D * HG) break;
    const int hh = i / D, c = i % D;
    float v = 0.f;
    if (hh < G && n < QPT) {
      const uint16_t bits = qraw[n < QPT ? n : 0];
      v = (a.q_bf16 ? bf16_bits_to_float(bits) : half_bits_to_float(bits)) * a.qscale;
    }
    sm.qs[c][hh] = v;
  }
  if (wv < NS) {
    // q * qscale for head col, scaled by a power of two so the head's largest
    // entry sits just under 2^14 and split into fp16 hi + lo
    float qv[4][8];
    float mq = 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint16_t bits = (uint16_t)(qf[s][i >> 1] >> (16 * (i & 1)));
        const float v = col < G ? (a.q_bf16 ? bf16_bits_to_float(bits) : half_bits_to_float(bits)) * a.qscale : 0.f;
        qv[s][i] = v;
        mq = fmaxf(mq, fabsf(v));
      }
    mq = fmaxf(mq, __shfl_xor(mq, 16));
    mq = fmaxf(mq, __shfl_xor(mq, 32));
    int eq = 0;
    if (mq > 0.f) {
      int e;
      frexpf(mq, &e);
      eq = max(-100, min(100, 14 - e));
    }
    const float upq = ldexpf(1.0f, eq);
    f4 dq = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      h8 qh, ql;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float v = qv[s][i] * upq;
        const _Float16 hh = (_Float16)v;
        qh[i] = hh;
        ql[i] = (_Float16)(v - (float)hh);
      }
      const h8 bkv = __builtin_bit_cast(h8, bkf[s]);
      dq = __builtin_amdgcn_mfma_f32_16x16x32_f16(bkv, qh, dq, 0, 0, 0);
      dq = __builtin_amdgcn_mfma_f32_16x16x32_f16(bkv, ql, dq, 0, 0, 0);
    }
    // lane (grp, col): q~[head col][row 16w + 4grp + i] = dq[i] / 2^eq
    if (col < G) {
      const float dn = ldexpf(1.0f, -eq);
      float am = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = dq[i] * dn;
        sm.qt[col][16 * wv + 4 * grp + i] = v;
        am = fmaxf(am, fabsf(v));
      }
      am = fmaxf(am, __shfl_xor(am, 16));
      am = fmaxf(am, __shfl_xor(am, 32));
      if (grp == 0) sm.qmaxw[wv][col] = am;
    }
    load_coef<RB, C8>(fr, x, j0, lane);
  }
  __syncthreads();

  // q~ as the A operand (row = head, repeated per 4 rows), scaled per head by
  // a power of two so its largest entry sits just under 2^14, split into fp16
  // hi + lo; the score of head i is scaled back by down[i]
  TState<RB, G, C8> st;
  {
    const int h = col & (HG - 1);
    float up = 1.0f;
#pragma unroll
    for (int i = 0; i < HG; ++i) {
      int kexp = 0;
      if (i < G) {
        float mx = 0.f;
#pragma unroll
        for (int w2 = 0; w2 < NS; ++w2) mx = fmaxf(mx, sm.qmaxw[w2][i]);
        if (mx > 0.f) {
          int e;
          frexpf(mx, &e);
          kexp = 14 - e;
        }
      }
      kexp = max(-100, min(100, kexp));
      st.down[i] = ldexpf(1.0f, -kexp);
      if (i == h) up = ldexpf(1.0f, kexp);
    }
#pragma unroll
    for (int s = 0; s < NS; ++s) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // fp16: the key tiles' order (key_k); int8: k-step s is coefficient
        // block s, in the byte order of i8x4_to_h4
        constexpr int ord[4] = {0, 2, 1, 3};
        const int k = C8 ? 16 * s + 4 * grp + ord[i] : key_k<NS>(s, grp, i);
        const float v = h < G ? sm.qt[h][k] * up : 0.f;
        const _Float16 hh = (_Float16)v;
        st.qhi[s][i] = hh;
        st.qlo[s][i] = (_Float16)(v - (float)hh);
      }
    }
    if constexpr (HG == 8 || (C8 && RB == 64)) {   // every wave writes the same bytes
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        sm.qa[0][s][lane] = st.qhi[s];
        sm.qa[1][s][lane] = st.qlo[s];
      }
      wave_lds_fence();
    }
#pragma unroll
    for (int b = 0; b < TState<RB, G, C8>::NACC; ++b) {
      st.acc_h[b] = f4{0.f, 0.f, 0.f, 0.f};
      st.acc_l[b] = f4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int i = 0; i < HG; ++i) {
      st.m[i] = -INFINITY;
      st.l[i] = 0.f;
    }
    st.ex = -14;
  }
  if constexpr (RESID) {
    for (int i = lane; i < HG * D; i += 64) (&sm.racc[wv][0][0])[i] = 0;
  }


  // the wave's tiles (tile_seq): a fixed assignment keeps the summation
  // order, and so the result, independent of timing.  The last tile of the
  // wave runs without the next tiles' loads.
  for (int k = 0; k + 1 < ts.n; ++k)
    tstep<RB, G, RESID, SCORES, C8, false>(st, fr, mc, mn, mnn, ec, en, ts.at(k), ts.at(k + 1),
                                           k + 2 < ts.n ? ts.at(k + 2) : x.ntile, x, sm, wv, lane);
  if (ts.n > 0)
    tstep<RB, G, RESID, SCORES, C8, true>(st, fr, mc, mn, mnn, ec, en, ts.at(ts.n - 1), x.ntile, x.ntile, x, sm,
                                          wv, lane);

  // epilogue: the waves combine; the partial keeps a~ in basis space (the
  // merge projects it through B^V once per sequence and head).  Each wave
  // first turns its fixed-point residual accumulators into floats in place
  // (its LDS operations run in order: every lane has read its integers before
  // the first float is written).
  if constexpr (RESID) {
    long long rv[G][2];
#pragma unroll
    for (int i = 0; i < G; ++i) {
      rv[i][0] = sm.racc[wv][i][lane];
      rv[i][1] = sm.racc[wv][i][lane + 64];
    }
    const float fs = ldexpf(1.0f, st.ex - kFxTop);
    float* rf = reinterpret_cast<float*>(&sm.racc[wv][0][0]);
#pragma unroll
    for (int i = 0; i < G; ++i) {
      rf[i * D + lane] = fixed_to_float(rv[i][0]) * fs;
      rf[i * D + lane + 64] = fixed_to_float(rv[i][1]) * fs;
    }
  }
#pragma unroll
  for (int i = 0; i < HG; ++i) st.l[i] = wave_sum(st.l[i]);
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < HG; ++i) {
      sm.ep_m[wv][i] = st.m[i];
      sm.ep_l[wv][i] = st.l[i];
    }
  }
  if (lane < RB) {
    if constexpr (C8) {                 // lane c keeps the pass of its coefficient block c / 16
      f4 ah = st.acc_h[0], al = st.acc_l[0];
#pragma unroll
      for (int b = 1; b < TState<RB, G, C8>::NACC; ++b)
        if ((lane >> 4) == b) { ah = st.acc_h[b]; al = st.acc_l[b]; }
#pragma unroll
      for (int i = 0; i < 4; ++i) sm.ep_a[wv][i][lane] = ah[i] + al[i];
    } else {                            // pair hg holds heads 4 hg .. 4 hg + 3
#pragma unroll
      for (int hg = 0; hg < TGrp<G>::NHG; ++hg)
#pragma unroll
        for (int i = 0; i < 4; ++i) sm.ep_a[wv][4 * hg + i][lane] = st.acc_h[hg][i] + st.acc_l[hg][i];
    }
  }
  __syncthreads();
  constexpr int ROW = D + RB;                 // r[d] then a~[r_b]
  constexpr int TPH = kTThreads / G;           // threads per head
  {
    const int g = tid / TPH;
    float mx = -INFINITY;
#pragma unroll
    for (int v = 0; v < kTW; ++v) mx = fmaxf(mx, sm.ep_m[v][g]);
    float sw[kTW], l = 0.f;
#pragma unroll
    for (int v = 0; v < kTW; ++v) {
      sw[v] = sm.ep_m[v][g] == -INFINITY ? 0.f : exp2f(sm.ep_m[v][g] - mx);
      l += sw[v] * sm.ep_l[v][g];
    }
    float* dst = a.part + (((int64_t)slot * a.n_work + w) * G + g) * kPartStrideTL;
    for (int c = tid % TPH; c < ROW; c += TPH) {
      float o = 0.f;
      if (c < D) {
        if constexpr (RESID) {
#pragma unroll
          for (int v = 0; v < kTW; ++v) o += sw[v] * reinterpret_cast<const float*>(&sm.racc[v][0][0])[g * D + c];
        }
      } else {
#pragma unroll
        for (int v = 0; v < kTW; ++v) o += sw[v] * sm.ep_a[v][g][c - D];
      }
      __hip_atomic_store(dst + c, o, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (tid % TPH == 0) {
      __hip_atomic_store(dst + kPartTLM, mx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(dst + kPartTLM + 1, l, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

template <int RB, int G, bool RESID, bool SCORES, bool C8>
__global__ __launch_bounds__(kTThreads) void tl_kernel(const SplitArgs a) {
  __shared__ TSmem<RB, G, RESID> sm;
  tl_body<RB, G, RESID, SCORES, C8>(a, sm, blockIdx.x, blockIdx.y);
}

// LDS of the append item, in the decode workgroup's storage: both bases of
// the sequence's window and head (K rows, then V rows), per Z the compress
// arrays, the rebuilt key, the value's residual g R and the heads' scores.
template <int RB>
struct alignas(16) ASmem {
  alignas(16) uint16_t bas[2][RB * cdev::kBRow];
  alignas(16) float xs[2][D];
  alignas(16) float as[2][RB];
  uint8_t ech[2][D];
  uint8_t ecode[2][D];
  float kh[D];
  float vr[D];
  float sc[8];
  int rho;
  uint16_t scale[2];
};

// The append item of sequence b and KV head `slot`: wave 0 compresses the new
// token t's key and wave 1 its value (the append/compress arithmetic, written
// to the cache), then the workgroup writes the token's own partial for every
// head of the group: score m = q . K_hat (log2 units, K_hat = A^K B^K + g R^K
// rebuilt from what was stored), l = 1, and the value in basis space:
// r = g R^V, a~ = A^V.  The merge takes it like any other partial.
template <int RB, int G>
__device__ __forceinline__ void tl_append(const TLAppendArgs& A, unsigned char* lds, int b, int64_t t, int slot,
                                          int w) {
  ASmem<RB>& sm = *reinterpret_cast<ASmem<RB>*>(lds);
  const SplitArgs& a = A.s;
  const CompressArgs& c = A.c;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int kvh = a.kv_of_slot[slot];
  const int Hk = c.n_kv_heads;
  const uint16_t* src = c.basis + (int64_t)b * c.basis_b_stride + (int64_t)kvh * 2 * RB * D;
  for (int e = tid; e < 2 * RB * (D / 8); e += kTThreads) {
    const int z = e / (RB * (D / 8)), r = e % (RB * (D / 8));
    const int i = r / (D / 8), q = r % (D / 8);
    *reinterpret_cast<uint4*>(&sm.bas[z][i * cdev::kBRow + 8 * q]) =
        *reinterpret_cast<const uint4*>(src + ((int64_t)z * RB + i) * D + 8 * q);
  }
  cdev::TokenIn in{};
  cdev::Slab sl{};
  if (wv < 2) {
    const int z = wv;
    const int64_t slab = (int64_t)z * Hk + kvh;
    sl.code = c.code + (int64_t)kvh * c.T;
    sl.off = c.off + (int64_t)kvh * (c.T + 1);
    sl.coef = (z == 0 ? c.coef_k : c.coef_v) + (int64_t)kvh * c.T16 * c.rb;
    sl.res_idx = c.res_idx + slab * c.res_stride;
    sl.res_val = c.res_val + slab * (c.res_stride / 2);
    sl.res_scale = c.res_scale + slab * c.T;
    const uint16_t* X = (z ? c.xv : c.xk) + ((int64_t)b * Hk + kvh) * D;
    in.xw = reinterpret_cast<const uint32_t*>(X)[lane];
    in.lvl = sl.code[t];
    in.e0 = sl.off[t];
    in.e1 = sl.off[t + 1];
    in.g = c.gate ? c.gate[(int64_t)(z * Hk + kvh) * c.gate_ld + b] : 1.0f;
  }
  __syncthreads();
  if (wv < 2) {
    const cdev::TokOut o =
        cdev::compress_token(c, sl, cdev::CWave{sm.bas[wv], sm.xs[wv], sm.as[wv], sm.ech[wv], sm.ecode[wv]}, lane,
                             wv, t, in);
    if (lane == 0) {
      sm.scale[wv] = o.scale;
      if (wv == 0) sm.rho = o.rho;
    }
  }
  __syncthreads();
  // the rebuilt key's basis term and a zero value residual, channel tid
  if (tid < D) {
    float k = 0.f;
    for (int i = 0; i < RB; ++i) k = __builtin_fmaf(sm.as[0][i], half_bits_to_float(sm.bas[0][i * cdev::kBRow + tid]), k);
    sm.kh[tid] = k;
    sm.vr[tid] = 0.f;
  }
  __syncthreads();
  // the residual entries (distinct channels within each of K and V)
  const int rho = sm.rho;
  if (tid < rho) {
    sm.kh[sm.ech[0][tid]] += half_bits_to_float(sm.scale[0]) * (float)int4_value(sm.ecode[0][tid]);
    sm.vr[sm.ech[1][tid]] = half_bits_to_float(sm.scale[1]) * (float)int4_value(sm.ecode[1][tid]);
  }
  __syncthreads();
  if (wv < G) {                          // wave g: the score of head g
    const uint16_t* qrow = a.q + ((int64_t)b * a.n_q_heads + kvh * G + wv) * D;
    const float q0 = a.q_bf16 ? bf16_bits_to_float(qrow[lane]) : half_bits_to_float(qrow[lane]);
    const float q1 = a.q_bf16 ? bf16_bits_to_float(qrow[lane + 64]) : half_bits_to_float(qrow[lane + 64]);
    const float sv = wave_sum(q0 * sm.kh[lane] + q1 * sm.kh[lane + 64]);
    if (lane == 0) sm.sc[wv] = sv * a.qscale;
  }
  __syncthreads();
  constexpr int ROW = D + RB;
  for (int e = tid; e < G * ROW; e += kTThreads) {
    const int g = e / ROW, cc = e % ROW;
    float* dst = a.part + (((int64_t)slot * a.n_work + w) * G + g) * kPartStrideTL;
    __hip_atomic_store(dst + cc, cc < D ? sm.vr[cc] : sm.as[1][cc - D], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (tid < G) {
    float* dst = a.part + (((int64_t)slot * a.n_work + w) * G + tid) * kPartStrideTL;
    __hip_atomic_store(dst + kPartTLM, sm.sc[tid], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(dst + kPartTLM + 1, 1.0f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// The decode that appends: the append item of a sequence is the last of its
// work items (its chunk is empty once the new token is trimmed off).
template <int RB, int G, bool RESID>
__global__ __launch_bounds__(kTThreads) void tl_append_kernel(const TLAppendArgs A) {
  constexpr size_t kT = sizeof(TSmem<RB, G, RESID>), kA = sizeof(ASmem<RB>);
  __shared__ alignas(16) unsigned char lds[kT > kA ? kT : kA];
  const SplitArgs& a = A.s;
  int b;
  int64_t c0, c1;
  work_item(a.wt, a.cu, a.batch, a.split, blockIdx.x, b, c0, c1, a.trim);
  if (c0 >= c1) {
    tl_append<RB, G>(A, lds, b, c1, blockIdx.y, blockIdx.x);
    return;
  }
  tl_body<RB, G, RESID, false, false>(a, *reinterpret_cast<TSmem<RB, G, RESID>*>(lds), blockIdx.x, blockIdx.y);
}

// The split-K pass with a probe's reference pass in the same grid: workgroups
// [0, n_work * n_slots) take the token-lane items in tl_kernel's order, the
// rest one reference item each (the general kernel's identity-basis body on
// this launch's kTW waves).  The dispatcher hands out workgroups in index
// order, so the reference items start on the compute units as their split-K
// items finish, with no second launch.
template <int RB, int G, bool RESID, bool C8>
__global__ __launch_bounds__(kTThreads) void tl_probe_kernel(const TLProbeArgs A) {
  using RS = gsplit::Smem<D, G, false, kTW>;
  constexpr size_t kT = sizeof(TSmem<RB, G, RESID>), kR = sizeof(RS);
  __shared__ alignas(16) unsigned char lds[kT > kR ? kT : kR];
  const int nt = A.s.n_work * A.s.n_slots;
  const int i = blockIdx.x;
  if (i < nt) {
    tl_body<RB, G, RESID, false, C8>(A.s, *reinterpret_cast<TSmem<RB, G, RESID>*>(lds), i % A.s.n_work,
                                     i / A.s.n_work);
    return;
  }
  const int k = i - nt;
  gsplit::split_body<D, G, false, true, kTW>(A.r, k % A.r.n_work, k / A.r.n_work, threadIdx.x,
                                             *reinterpret_cast<RS*>(lds));
}

template <int RB, int G, bool R, bool C8>
hipError_t launch_tlp_t(const TLProbeArgs& a, hipStream_t s) {
  const int nt = a.s.n_work * a.s.n_slots, nr = a.r.n_work * a.r.n_slots;
  hipLaunchKernelGGL((tl_probe_kernel<RB, G, R, C8>), dim3(nt + nr), dim3(kTThreads), 0, s, a);
  return hipGetLastError();
}

template <int RB, bool R, bool C8>
hipError_t launch_tlp_g(int g, const TLProbeArgs& a, hipStream_t s) {
  switch (g) {
    case 1: return launch_tlp_t<RB, 1, R, C8>(a, s);
    case 2: return launch_tlp_t<RB, 2, R, C8>(a, s);
    case 4: return launch_tlp_t<RB, 4, R, C8>(a, s);
    case 8:
      if constexpr (!C8) return launch_tlp_t<RB, 8, R, C8>(a, s);
      break;
  }
  return hipErrorInvalidValue;
}

template <bool R, bool C8>
hipError_t launch_tlp_rb(int rb, int g, const TLProbeArgs& a, hipStream_t s) {
  switch (rb) {
    case 16: return launch_tlp_g<16, R, C8>(g, a, s);
    case 32: return launch_tlp_g<32, R, C8>(g, a, s);
    case 48: return launch_tlp_g<48, R, C8>(g, a, s);
    case 64: return launch_tlp_g<64, R, C8>(g, a, s);
  }
  return hipErrorInvalidValue;
}

template <int RB, int G, bool R>
hipError_t launch_tla_t(const TLAppendArgs& a, int n_work, hipStream_t s) {
  hipLaunchKernelGGL((tl_append_kernel<RB, G, R>), dim3(n_work, a.s.n_slots), dim3(kTThreads), 0, s, a);
  return hipGetLastError();
}

template <int RB, bool R>
hipError_t launch_tla_g(int g, const TLAppendArgs& a, int n_work, hipStream_t s) {
  switch (g) {
    case 1: return launch_tla_t<RB, 1, R>(a, n_work, s);
    case 2: return launch_tla_t<RB, 2, R>(a, n_work, s);
    case 4: return launch_tla_t<RB, 4, R>(a, n_work, s);
    case 8: return launch_tla_t<RB, 8, R>(a, n_work, s);
  }
  return hipErrorInvalidValue;
}

template <bool R>
hipError_t launch_tla_rb(int rb, int g, const TLAppendArgs& a, int n_work, hipStream_t s) {
  switch (rb) {
    case 16: return launch_tla_g<16, R>(g, a, n_work, s);
    case 32: return launch_tla_g<32, R>(g, a, n_work, s);
    case 48: return launch_tla_g<48, R>(g, a, n_work, s);
    case 64: return launch_tla_g<64, R>(g, a, n_work, s);
  }
  return hipErrorInvalidValue;
}

template <int RB, int G, bool R, bool S, bool C8>
hipError_t launch_tl_t(const SplitArgs& a, int n_work, hipStream_t s) {
  hipLaunchKernelGGL((tl_kernel<RB, G, R, S, C8>), dim3(n_work, a.n_slots), dim3(kTThreads), 0, s, a);
  return hipGetLastError();
}

template <int RB, bool R, bool S, bool C8>
hipError_t launch_tl_g(int g, const SplitArgs& a, int n_work, hipStream_t s) {
  switch (g) {
    case 1: return launch_tl_t<RB, 1, R, S, C8>(a, n_work, s);
    case 2: return launch_tl_t<RB, 2, R, S, C8>(a, n_work, s);
    case 4: return launch_tl_t<RB, 4, R, S, C8>(a, n_work, s);
    case 8:
      if constexpr (!C8) return launch_tl_t<RB, 8, R, S, C8>(a, n_work, s);
      break;
  }
  return hipErrorInvalidValue;
}

template <bool R, bool S, bool C8>
hipError_t launch_tl_rb(int rb, int g, const SplitArgs& a, int n_work, hipStream_t s) {
  switch (rb) {
    case 16: return launch_tl_g<16, R, S, C8>(g, a, n_work, s);
    case 32: return launch_tl_g<32, R, S, C8>(g, a, n_work, s);
    case 48: return launch_tl_g<48, R, S, C8>(g, a, n_work, s);
    case 64: return launch_tl_g<64, R, S, C8>(g, a, n_work, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

template <int RB, int CH>
hipError_t launch_merge_tl_ch(int g, const WMergeArgs& a, hipStream_t s) {
  const dim3 grid((a.s.n_slots * (D / CH) + a.p.n_probe * kWmNCH) * g, a.s.batch);
  switch (g) {
    case 1: hipLaunchKernelGGL((tl_wmerge_kernel<RB, 1, CH>), grid, dim3(kWmThreads), 0, s, a); break;
    case 2: hipLaunchKernelGGL((tl_wmerge_kernel<RB, 2, CH>), grid, dim3(kWmThreads), 0, s, a); break;
    case 4: hipLaunchKernelGGL((tl_wmerge_kernel<RB, 4, CH>), grid, dim3(kWmThreads), 0, s, a); break;
    case 8: hipLaunchKernelGGL((tl_wmerge_kernel<RB, 8, CH>), grid, dim3(kWmThreads), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Channels per merge workgroup: 64 when every sequence has at most kWideFew
// partials (a few loads per workgroup, and four times fewer workgroups start
// sooner), else 32 (at 32 partials per sequence, 4.0 us per launch against
// 4.2 with 16 channels and 4.1 with 64).  A probe's reference chunks keep 16
// channels.
constexpr int kWideFew = 4;

template <int RB>
hipError_t launch_merge_tl_rb(int g, const WMergeArgs& a, hipStream_t s) {
  if (a.max_ns <= kWideFew) return launch_merge_tl_ch<RB, 64>(g, a, s);
  return launch_merge_tl_ch<RB, 32>(g, a, s);
}

bool token_lane_supported(int rb, int g, int max_level, int64_t tokens, int64_t res_stride) {
  // every slab must stay below 2^31 bytes for the 32-bit buffer offsets
  const int64_t lim = (int64_t)1 << 31;
  const bool group = ((g == 1 || g == 2 || g == 4) && max_level <= TGrp<4>::MR) ||
                     (g == 8 && max_level <= TGrp<8>::MR);
  return group && rb % 16 == 0 && rb >= 16 && rb <= 64 && (tokens + 64) * rb * 2 < lim && (tokens + 64) * 4 < lim &&
         res_stride < lim;
}

hipError_t launch_split_tl(int rb, int g, bool resid, const SplitArgs& a, int n_work, hipStream_t s) {
  return resid ? launch_tl_rb<true, false, false>(rb, g, a, n_work, s)
               : launch_tl_rb<false, false, false>(rb, g, a, n_work, s);
}

hipError_t launch_split_tl_append(int rb, int g, bool resid, const TLAppendArgs& a, int n_work, hipStream_t s) {
  return resid ? launch_tla_rb<true>(rb, g, a, n_work, s) : launch_tla_rb<false>(rb, g, a, n_work, s);
}

hipError_t launch_split_tl_probe(int rb, int g, bool resid, bool c8, const TLProbeArgs& a, hipStream_t s) {
  if (c8) return resid ? launch_tlp_rb<true, true>(rb, g, a, s) : launch_tlp_rb<false, true>(rb, g, a, s);
  return resid ? launch_tlp_rb<true, false>(rb, g, a, s) : launch_tlp_rb<false, false>(rb, g, a, s);
}

hipError_t launch_split_tl_scores(int rb, int g, bool resid, const SplitArgs& a, int n_work, hipStream_t s) {
  return resid ? launch_tl_rb<true, true, false>(rb, g, a, n_work, s)
               : launch_tl_rb<false, true, false>(rb, g, a, n_work, s);
}

hipError_t launch_split_tl_scores_c8(int rb, int g, bool resid, const SplitArgs& a, int n_work, hipStream_t s) {
  return resid ? launch_tl_rb<true, true, true>(rb, g, a, n_work, s)
               : launch_tl_rb<false, true, true>(rb, g, a, n_work, s);
}

hipError_t launch_split_tl_c8(int rb, int g, bool resid, const SplitArgs& a, int n_work, hipStream_t s) {
  return resid ? launch_tl_rb<true, false, true>(rb, g, a, n_work, s)
               : launch_tl_rb<false, false, true>(rb, g, a, n_work, s);
}

hipError_t launch_merge_tl(int rb, int g, const WMergeArgs& a, hipStream_t s) {
  switch (rb) {
    case 16: return launch_merge_tl_rb<16>(g, a, s);
    case 32: return launch_merge_tl_rb<32>(g, a, s);
    case 48: return launch_merge_tl_rb<48>(g, a, s);
    case 64: return launch_merge_tl_rb<64>(g, a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace dwkv
