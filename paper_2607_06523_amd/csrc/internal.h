// Private to the library: kernel argument blocks and launcher entry points.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dwkv.h"

namespace dwkv {

constexpr int kHeadDim = 128;       // d
constexpr int kWaves = 4;           // waves per decode workgroup
constexpr int kTLWaves = 8;         // waves per token-lane decode workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kPartStride = kHeadDim + 4;   // floats per partial: o[d], m, l, pad
// Token-lane partials keep the value in basis space: r[d] (residual part),
// a~[r_b] (r_b <= 64) at d, m at d+64, l at d+65; the merge projects a~
// through B^V once per sequence and head.
constexpr int kPartStrideTL = kHeadDim + 64 + 4;
constexpr int kPartTLM = kHeadDim + 64;
constexpr int kEntChunk = 512;      // residual entries of a tile staged in LDS
constexpr int kResTailPad = 512;    // spare entries required after the longest slab

constexpr int kKernargSeqs = 16;    // sequences whose work split travels in the kernel arguments

// Work items of a batch, resolved on the host when it has at most
// kKernargSeqs sequences (n_seq > 0): items [work[b], work[b+1]) cover
// sequence b, whose packed tokens are [tok[b], tok[b+1]).  With n_seq == 0
// the kernels walk the device cu_seqlens instead.
struct WorkTable {
  int32_t n_seq;
  int32_t work[kKernargSeqs + 1];
  int32_t tok[kKernargSeqs + 1];
};

// Value-residual sums in LDS are int64 fixed point: integer LDS atomics cost a
// few cycles per instruction whatever the active lanes (float ones a few per
// lane), and their sums do not depend on the order of the additions.
// Fixed point: round(v * scale) as a two's complement int64 for
// |v * scale| < 2^51 (adding 1.5 * 2^52 leaves the rounded integer in the low
// mantissa bits).
__device__ __forceinline__ unsigned long long to_fixed(float v, double scale) {
  const double magic = 6755399441055744.0;
  const double t = __builtin_fma((double)v, scale, magic);
  return (unsigned long long)(__double_as_longlong(t) - __double_as_longlong(magic));
}

// A fixed-point accumulator as float.  Below 2^53 in magnitude the two
// halves combine exactly in double and the result is rounded once (with terms
// below 2^45 this holds while a wave adds at most 256 of them to one
// accumulator); above it a second rounding can move the result by one ulp.
__device__ __forceinline__ float fixed_to_float(long long v) {
  const double hi = (double)(int32_t)(v >> 32), lo = (double)(uint32_t)(v & 0xFFFFFFFFll);
  return (float)__builtin_fma(hi, 4294967296.0, lo);
}

// fp16 coefficient layouts, element index inside one (layer, KV head) slab of
// T16 = T rounded up to 16 tokens (padding zero).  Keys: tiles of 16 tokens x
// 8 coefficients, [T16/16][rb/8][16][8]; values: 8-token blocks, [T16/8][rb][8].
// A wave reading a key tile's 16 tokens for 4 coefficient groups, or a value
// block for 64 channels, reads whole 128-byte lines with one instruction.
__host__ __device__ __forceinline__ int64_t key_index(int64_t t, int k, int rb) {
  return (((t >> 4) * (rb >> 3) + (k >> 3)) << 7) + ((t & 15) << 3) + (k & 7);
}
__host__ __device__ __forceinline__ int64_t value_index(int64_t t, int c, int rb) {
  return ((t >> 3) * rb + c) * 8 + (t & 7);
}

// Score-product k order over the key tiles: coefficient k held in element i
// of 16-deep k-step s by lane group g (of NS k-steps), so that a pair of
// k-steps reads one 16-byte tile row piece per lane and an odd last k-step
// two 8-byte halves; both operands of the product use it.
template <int NS>
__device__ __forceinline__ int key_k(int s, int g, int i) {
  return s < NS - (NS & 1) ? 32 * (s >> 1) + 8 * g + 4 * (s & 1) + i : 32 * (NS >> 1) + 4 * g + i;
}

// One split-K pass over a layer: grid = (work items, head slots).
struct SplitArgs {
  const uint16_t* coef_k;      // slot 0 key tiles (key_index; int8: rows [T][RB]); slot s adds s*T16*RB (int8 s*T*RB)
  const uint16_t* coef_v;      // slot 0 value blocks (value_index; int8: [T16/16][RB][16]); slot s adds s*T16*RB
  const uint16_t* basis;       // basis of window m, sequence 0: + (b*M*Hkv + h)*2*RB*d
  int64_t basis_b_stride;      // halves between sequences (M*Hkv*2*RB*d)
  const uint32_t* off;         // res_off of window m, head 0; head h adds h*(T+1)
  const uint8_t* idx_k;        // res_idx of (layer, K), head 0; head h adds h*res_stride
  const uint8_t* idx_v;
  const uint8_t* val_k;        // res_val of (layer, K), head 0; head h adds h*res_stride/2
  const uint8_t* val_v;
  const uint16_t* scale_k;     // res_scale of (layer, K), head 0; head h adds h*T
  const uint16_t* scale_v;
  const uint16_t* q;           // [B][Hq][d] fp16 or bf16 bits
  const int32_t* cu;           // [B+1] device
  float* part;                 // [work][n_slots][G][kPartStride]; token-lane: [n_slots][work][G][kPartStrideTL]
  float* out;                  // [B][Hq][d], written by the token-lane merge launch
  float* scores;               // [n_slots][T][G] raw scores in exp2 units (token-lane pass with scores only)
  const uint16_t* cscale_k;    // int8 coefficients: key block scales, slot 0 [r_b/16][T]; slot s adds s*(r_b/16)*T
  const uint16_t* cscale_v;    // value block scales, same layout
  int64_t T;
  int64_t res_stride;
  int32_t batch;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t n_slots;             // grid.y
  int32_t split;               // tokens per work item
  int32_t n_work;              // work items of the launch
  int32_t q_bf16;
  float qscale;                // sm_scale * log2(e)
  int32_t kv_of_slot[DWKV_MAX_PROBE_HEADS];
  WorkTable wt;
  float* mstats;               // token-lane merge: merged (m*, l*) per [B][Hq] when not null
  int32_t trim;                // tokens dropped from the end of every sequence (earlier probe positions)
  uint32_t* zero;              // reference pass: n_zero words its first workgroup clears (the wide
  int32_t n_zero;              // merge's probe counters), or null
};

// Eq. 3 in the token-lane wide merge: extra workgroups merge the reference
// partials of a probed column 16 channels at a time into oref; the last of
// the column's output and reference chunk workgroups (a counter) reads both
// rows and writes err (or, with several positions, the sums to acc).
struct WideProbe {
  const float* part_ref;       // reference partials [work][n_probe][G][kPartStride]
  float* err;                  // [B][n_probe*G]
  float* out_ref;              // [B][n_probe*G][d] or null
  float* acc;                  // [B][n_probe*G][2] (several positions) or null
  float* oref;                 // [B][n_probe*G][d] the reference rows (workspace)
  uint32_t* count;             // [B][n_probe*G] chunks done: zero before the merge, reset by the last
  int32_t n_probe;             // 0: no probe
  float eps;
  int32_t ref_split;
  WorkTable ref_wt;
  int32_t slot_of_kv[DWKV_MAX_PROBE_HEADS];   // probed slot of each KV head, -1 when not probed
  int32_t kv_of_slot[DWKV_MAX_PROBE_HEADS];   // KV head of each probed slot
};

struct WMergeArgs {
  SplitArgs s;
  WideProbe p;
  int32_t max_ns;              // most work items of any sequence (picks the workgroup width)
};

// Split merge (and Eq. 3 for probed heads): grid = (Hq, B).
struct MergeArgs {
  const float* part;           // decode partials [work][Hkv][G][kPartStride] (token-lane: [Hkv][work][G][kPartStrideTL])
  const float* part_ref;       // probe partials [work][n_probe][G][kPartStride] or null
  float* out;                  // [B][Hq][d]
  float* err;                  // [B][n_probe*G] or null
  float* out_ref;              // [B][n_probe*G][d] or null
  const int32_t* cu;
  int32_t batch;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t split;
  int32_t n_probe;
  float eps;
  int32_t probe_slot_of_kv[DWKV_MAX_PROBE_HEADS];   // -1 when the KV head is not probed
  WorkTable wt;
  int32_t tl;                  // main partials in the token-lane layout
  int32_t n_work;              // work items (token-lane layout)
  int32_t rb;
  const uint16_t* basis;       // basis of window m, sequence 0: + (b*M*Hkv + h)*2*RB*d (tl only)
  int64_t basis_b_stride;
  int32_t ref_split;           // the probe pass's chunk size and work split
  WorkTable ref_wt;
  // probe over several query positions: the current position's merge writes
  // (sum d^2, sum r^2) per probed column to acc [B][n_probe*G][2] instead of
  // err; the position merge (grid (n_probe * G, B)) adds the earlier
  // positions' sums and writes err.  Position j (1..n_pos-1) keeps its
  // rebuilt partials at part_pos + (j-1) * 2 * pos_stride and its reference
  // partials pos_stride floats further, both [work][n_probe][G][kPartStride]
  // over chunks of ref_split tokens of the sequences cut j tokens short.
  float* acc;
  const float* part_pos;
  int64_t pos_stride;
  int32_t n_pos;
};

// Makes the kernel-argument values the whole split kernel needs live in scalar
// registers at this point, so their loads are issued together at kernel entry
// rather than one after another behind the work-item decode.
__device__ __forceinline__ void pin_split_args(const SplitArgs& a, int kvh) {
  asm volatile("" ::"s"(a.coef_k), "s"(a.coef_v), "s"(a.basis), "s"(a.basis_b_stride), "s"(a.q), "s"(a.off), "s"(a.idx_k),
               "s"(a.idx_v), "s"(a.val_k), "s"(a.val_v), "s"(a.scale_k), "s"(a.scale_v), "s"(a.T),
               "s"(a.res_stride), "s"(a.split), "s"(kvh), "s"(a.wt.n_seq), "s"(a.wt.tok[0]), "s"(a.wt.tok[1]),
               "s"(a.n_q_heads), "s"(a.q_bf16), "s"(a.qscale), "s"(a.part), "s"(a.n_work));
}

// Sequence b and token chunk [c0, c1) of work item w.  With trim > 0 every
// sequence ends trim tokens early (a query of an earlier decode position sees
// that prefix); the work table then counts the trimmed lengths.
__device__ __forceinline__ void work_item(const WorkTable& wt, const int32_t* cu, int batch, int split,
                                          int w, int& b, int64_t& c0, int64_t& c1, int trim = 0) {
  if (__builtin_expect(wt.n_seq > 0, 1)) {
    // branch-free scan of the whole table: every read is at a fixed argument
    // offset, so they are all issued at once
    int bw = 0, t0 = wt.tok[0], t1 = wt.tok[1], w0 = 0;
    if (wt.n_seq > 1) {
#pragma unroll
      for (int i = 1; i < kKernargSeqs; ++i) {
        const bool here = i < wt.n_seq && w >= wt.work[i];
        bw = here ? i : bw;
        w0 = here ? wt.work[i] : w0;
        t0 = here ? wt.tok[i] : t0;
        t1 = here ? wt.tok[i + 1] : t1;
      }
    }
    b = bw;
    c0 = (int64_t)t0 + (int64_t)(w - w0) * split;
    c1 = t1 - trim;
  } else {
    int base = 0;
    for (b = 0; b < batch - 1; ++b) {
      const int ns = (max(cu[b + 1] - cu[b] - trim, 0) + split - 1) / split;
      if (w < base + ns) break;
      base += ns;
    }
    c0 = (int64_t)cu[b] + (int64_t)(w - base) * split;
    c1 = cu[b + 1] - trim;
  }
  c1 = c1 < c0 + split ? c1 : c0 + split;
  c0 = c0 < c1 ? c0 : c1;
}

// First work item and number of work items of sequence b.
__device__ __forceinline__ void seq_work(const WorkTable& wt, const int32_t* cu, int split, int b,
                                         int& base, int& ns) {
  if (wt.n_seq > 0) {
    base = wt.work[b];
    ns = wt.work[b + 1] - base;
  } else {
    base = 0;
    for (int i = 0; i < b; ++i) base += (cu[i + 1] - cu[i] + split - 1) / split;
    ns = (cu[b + 1] - cu[b] + split - 1) / split;
  }
}

// seq_work at a kernel's entry (b uniform): the table entries are read
// unconditionally, at an index kept inside the table, and held in scalar
// registers, so their loads join the kernel's first batch of argument loads
// instead of waiting behind the n_seq test.
__device__ __forceinline__ void seq_work_entry(const WorkTable& wt, const int32_t* cu, int split, int b,
                                               int& base, int& ns) {
  const int bi = min(b, kKernargSeqs - 1);
  const int wa = wt.work[bi], wb = wt.work[bi + 1];
  asm volatile("" ::"s"(wt.n_seq), "s"(wa), "s"(wb));
  if (wt.n_seq > 0) {
    base = wa;
    ns = wb - wa;
  } else {
    seq_work(wt, cu, split, b, base, ns);
  }
}

struct RouteArgs {
  const float* phi;            // [M][Hkv][T][4]
  const float* u;              // [M][4]
  const float* theta;          // [M][n_levels-1]
  uint8_t* code;               // [M][Hkv][T]
  uint32_t* off;               // [M][Hkv][T+1]
  uint32_t* bsum;              // [M*Hkv][nblk]
  uint32_t* bpre;              // [M*Hkv][nblk]
  int64_t T;                   // token stride of code / off / phi
  int64_t t0, n;               // routed range [t0, t0 + n); off[t0] holds the carry-in
  const int64_t* entries;      // budget routing: residual entries allowed per (window, head)
  unsigned long long* keys;    // budget routing: selection keys [M*Hkv][T]
  int32_t n_kv_heads;
  int32_t n_levels;
  int32_t nblk;
  int32_t levels[DWKV_MAX_LEVELS];
};

constexpr int kRouteTokensPerBlock = 1024;

// Append/compress of packed tokens [t0, t0 + n) of one layer.
struct CompressArgs {
  const uint16_t* basis;       // window m of sequence 0; sequence b adds b*basis_b_stride,
                               // head h and Z add (h*2 + z)*rb*d
  int64_t basis_b_stride;
  const uint8_t* code;         // rank_code of window m: [Hkv][T]
  const uint32_t* off;         // res_off of window m: [Hkv][T+1]
  const int32_t* cu;           // device cu_seqlens [batch+1]
  const uint16_t* xk;          // [n][Hkv][d] fp16
  const uint16_t* xv;
  const float* gate;           // null (g = 1), or gate of token k of (z, h) at
                               // [(z*Hkv + h)*gate_ld + gate_k0 + k] ([2][Hkv][n] by default)
  uint16_t* coef_k;            // layer's [Hkv] slabs of T16*rb (key_index); int8: bytes, 16x16 key tiles
  uint16_t* coef_v;            // layer's [Hkv] slabs of T16*rb (value_index); int8: bytes, [T16/16][rb][16]
  uint16_t* cscale_k;          // int8 coefficients: layer's [Hkv] slabs of (rb/16)*T block scales, else null
  uint16_t* cscale_v;
  uint8_t* res_idx;            // layer's [2][Hkv][res_stride]
  uint8_t* res_val;            // layer's [2][Hkv][res_stride/2]
  uint16_t* res_scale;         // layer's [2][Hkv][T]
  int64_t T, T16, t0, n, res_stride;
  int32_t batch, n_kv_heads, rb, n_levels;
  int32_t c8;                  // write the 8-bit blockwise coefficient form
  int64_t gate_ld, gate_k0;
  int32_t levels[DWKV_MAX_LEVELS];
};

hipError_t launch_split(int rb, int g, bool resid, bool ident, const SplitArgs& a, int n_work,
                        hipStream_t s);
// Token-lane variant of the split pass (query groups of 1, 2 or 4 heads, basis
// ranks 16..64, at most 16 residual entries per token); same partials.
bool token_lane_supported(int rb, int g, int max_level, int64_t tokens, int64_t res_stride);
hipError_t launch_split_tl(int rb, int g, bool resid, const SplitArgs& a, int n_work, hipStream_t s);
// The same pass that also stores every token's raw scores (a.scores), for the
// attention-mass features.
hipError_t launch_split_tl_scores(int rb, int g, bool resid, const SplitArgs& a, int n_work, hipStream_t s);
// The pass over int8-blockwise coefficients (coef_k / coef_v point at int8
// codes, cscale_k / cscale_v at their fp16 block scales).
hipError_t launch_split_tl_c8(int rb, int g, bool resid, const SplitArgs& a, int n_work, hipStream_t s);
hipError_t launch_split_tl_scores_c8(int rb, int g, bool resid, const SplitArgs& a, int n_work, hipStream_t s);
// Token-lane merge: reads a.part, writes a.out (one workgroup per slot, head
// and 16 output channels).
hipError_t launch_merge_tl(int rb, int g, const WMergeArgs& a, hipStream_t s);
hipError_t launch_merge(const MergeArgs& a, hipStream_t s);
hipError_t launch_route(const RouteArgs& a, int n_mh, hipStream_t s);
// Two-level routing under a budget: a.entries [M*Hkv] (device), keys scratch
// a.keys [M*Hkv][T]; one workgroup per (window, head).
hipError_t launch_route_budget(const RouteArgs& a, int n_mh, hipStream_t s);
hipError_t launch_compress(const CompressArgs& a, hipStream_t s);

// Decode of one layer that first appends the new token of every sequence (its
// last): the split pass covers each sequence's tokens but the last (trim 1),
// and one more work item per non-empty sequence -- the last of its range --
// compresses the new token's key and value (as the append/compress kernel
// does, written to the cache) and writes the token's own partial (score
// against the rebuilt key; the rebuilt value in basis space).  c carries the
// compress arguments; x rows are [B][Hkv][d] and gate [2][Hkv][B]
// (gate_ld = B).
struct TLAppendArgs {
  SplitArgs s;
  CompressArgs c;
};
hipError_t launch_split_tl_append(int rb, int g, bool resid, const TLAppendArgs& a, int n_work, hipStream_t s);

// The token-lane split-K pass and a probe's reference pass (the general
// kernel's identity-basis path over the dense rows, kHeadDim ranks) in one
// launch: s as for launch_split_tl, r as for the reference launch_split call.
struct TLProbeArgs {
  SplitArgs s;
  SplitArgs r;
};
hipError_t launch_split_tl_probe(int rb, int g, bool resid, bool c8, const TLProbeArgs& a, hipStream_t s);
// An earlier probe position: the general kernel's factorized pass over the
// probed heads (s, r_b rb) and its reference pass (r) in one launch.
hipError_t launch_probe_pos(int rb, int g, bool resid, const TLProbeArgs& a, hipStream_t s);

// Materialization of one layer's rebuilt keys and values (Eq. 1) as fp16.
struct MatArgs {
  const uint16_t* basis;       // window m, sequence 0; sequence b adds b*basis_b_stride, (h, z) add (h*2+z)*rb*d
  int64_t basis_b_stride;
  const uint16_t* coef_k;      // layer's [Hkv] slabs of T16*rb (key_index)
  const uint16_t* coef_v;      // layer's [Hkv] slabs of T16*rb (value_index)
  const uint32_t* off;         // window's [Hkv][T+1]
  const uint8_t* idx;          // layer's [2][Hkv][res_stride]
  const uint8_t* val;          // layer's [2][Hkv][res_stride/2]
  const uint16_t* scale;       // layer's [2][Hkv][T]
  const int32_t* cu;           // device cu_seqlens
  uint16_t* k_out;             // [Hkv][T][d]
  uint16_t* v_out;             // [Hkv][T16/16][d][16]
  int64_t T, T16, res_stride;
  int32_t batch, n_kv_heads, rb;
};
hipError_t launch_materialize(const MatArgs& a, hipStream_t s);

// HBM read stream: kStreamBlocks blocks; block b writes sink[b].
constexpr int kStreamBlocks = 2048;
hipError_t launch_stream_read(const void* buf, uint64_t n16, uint32_t* sink, hipStream_t s);

// Attention-mass features of one decode (token-lane partials and stored scores).
struct FeatArgs {
  const float* mstats;         // merged softmax statistics (m*, l*) per [B][Hq], from the merge
  const float* scores;         // [Hkv][T][G] raw scores (exp2 units)
  float* phi;                  // the window's features [Hkv][T][4] (columns 0, 1 updated)
  const int32_t* cu;           // device cu_seqlens
  int64_t T;
  int32_t batch, n_kv_heads, n_q_heads;
};
hipError_t launch_features(int g, const FeatArgs& a, hipStream_t s);

// The probe-error router feature (column 3 of a window's phi) from one
// probed layer's Eq. 3 errors.
struct ProbeFeatArgs {
  const float* err;            // [B][n_heads * G]
  float* phi;                  // the window's features [Hkv][T][4]
  const int32_t* cu;           // device cu_seqlens
  int64_t T;
  int32_t batch, n_heads, G, fresh;
  int32_t kv_heads[DWKV_MAX_PROBE_HEADS];
};
hipError_t launch_probe_feature(const ProbeFeatArgs& a, hipStream_t s);

// Randomized-sketch basis initialization of one (sequence, window).
struct SketchArgs {
  const uint16_t* x;           // fp16 [w][2][n_tokens][Hkv][d] prefill keys (Z = 0) and values (Z = 1)
  const uint16_t* omega;       // fp16 [w * n_tokens][rb] sketch matrix, row l * n_tokens + t
  double* part;                // [n_chunks][Hkv][2][rb][d] sketch partials
  double* q;                   // [Hkv][2][rb][d] orthonormal rows
  uint16_t* basis;             // the (sequence, window)'s basis [Hkv][2][rb][d], written
  int64_t n_tokens;
  int32_t w, n_kv_heads, rb, n_chunks;
};
int sketch_chunks(int64_t rows);
hipError_t launch_sketch(const SketchArgs& a, hipStream_t s);
hipError_t launch_residual_map(const uint32_t* off, const uint8_t* idx, const uint8_t* val,
                               const uint16_t* scale, int64_t t0, int64_t t1, int64_t slab_len,
                               float* dense, hipStream_t s);
hipError_t launch_validate(const dwkv_dims* dims, const dwkv_cache* c, unsigned long long* bad,
                           hipStream_t s);

}  // namespace dwkv
