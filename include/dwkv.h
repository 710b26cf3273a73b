/*
 * dwkv.h -- C ABI of the MI355X (gfx950) decode path over a cross-depth
 * factorized KV cache (DepthWeave-KV, Sec. 3 of the paper).
 *
 * The cache stores, for every depth window m (a run of `window` consecutive
 * layers) and KV head h, shared channel bases B^K_{m,h}, B^V_{m,h} (r_b x d),
 * and for every layer l, token t: a coefficient row A^Z_{l,h,t} (1 x r_b) and
 * a routed residual of rho_{m,h,t} channels, each an int4 code, with one
 * gate-folded scale g*s per (l, Z, h, t).  The key/value of token t is, by
 * Eq. 1,  X_hat = A B + g R.  The decode entry point never materialises
 * X_hat: it projects the query into basis space once, streams the
 * coefficients and residual entries, and runs softmax attention on chip.
 *
 * Conventions for every entry point
 *  - Pointers are DEVICE pointers unless the name ends in `_host`.  The decode
 *    calls read and write them with 16-byte vector accesses: every device
 *    pointer they take (cache arrays, q, out, workspace) must be 16-byte
 *    aligned (hipMalloc and torch allocations are; so is any whole-row slice
 *    of them), else they return DWKV_E_ALIGN.
 *  - All buffers are owned by the caller; the library allocates nothing and
 *    keeps no global mutable state, so calls on different streams do not
 *    interfere (calls sharing one workspace must be ordered by the caller).
 *    The one exception is dwkv_decode_noalloc, whose static scratch array is
 *    shared by its calls on one GPU.
 *  - Argument errors are detected on the host before anything is enqueued and
 *    returned synchronously; DWKV_E_HIP reports a failed HIP call or launch.
 *  - Kernels run asynchronously on `stream` (a hipStream_t; NULL = the null
 *    stream).  Decode trusts the layout; dwkv_validate is the checked path.
 *  - No exception crosses the ABI.
 */
#ifndef DWKV_H
#define DWKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DWKV_ABI_VERSION 4
#define DWKV_MAX_LEVELS 8
#define DWKV_MAX_PROBE_HEADS 64
#define DWKV_MAX_PROBE_POS 8      /* recent query positions one probe evaluates */

typedef enum dwkv_status {
  DWKV_OK = 0,
  DWKV_E_NULL = 1,        /* a required pointer is NULL                           */
  DWKV_E_DIMS = 2,        /* sizes inconsistent with each other                   */
  DWKV_E_UNSUPPORTED = 3, /* consistent but not built: head_dim != 128,
                             G = Hq/Hkv not in {1,2,4,8,16}, r_b not a multiple of
                             16 in [16,128], more than 8 levels, 32-bit offset
                             overflow possible; int8 coefficients in a decode
                             off the token-lane path for groups of up to 4
                             (r_b <= 64, levels <= 16), with a probe over
                             several positions, or in dwkv_materialize            */
  DWKV_E_WORKSPACE = 4,   /* workspace smaller than the *_workspace_bytes value    */
  DWKV_E_LAYOUT = 5,      /* dwkv_validate found a malformed cache                 */
  DWKV_E_HIP = 6,         /* a HIP runtime call or kernel launch failed            */
  DWKV_E_ALIGN = 7,       /* a decode device pointer is not 16-byte aligned         */
  DWKV_E_SCRATCH = 8      /* dwkv_decode_noalloc: the call needs more scratch than
                             dwkv_static_scratch_bytes()                           */
} dwkv_status;

typedef enum dwkv_qtype { DWKV_F16 = 0, DWKV_BF16 = 1 } dwkv_qtype;

/* Shape of one factorized cache (all sequences packed along the token axis). */
typedef struct dwkv_dims {
  int32_t batch;          /* B sequences                                          */
  int32_t n_layers;       /* L layers held; L % window == 0                        */
  int32_t window;         /* w: layers per depth window (non-overlapping, m = l/w) */
  int32_t n_kv_heads;     /* Hkv                                                   */
  int32_t n_q_heads;      /* Hq; query head hq reads KV head hq / (Hq/Hkv)         */
  int32_t head_dim;       /* d (must be 128)                                       */
  int32_t basis_rank;     /* r_b                                                   */
  int32_t n_levels;       /* routed residual-rank levels, 1..8                     */
  int32_t levels[DWKV_MAX_LEVELS]; /* ascending, even, 0 <= level <= d             */
  const int32_t* cu_seqlens_host;  /* [B+1] packed token starts, host copy         */
  const int32_t* cu_seqlens;       /* the same [B+1], device copy                  */
  int64_t total_tokens;   /* T = cu_seqlens_host[B]                                */
  int64_t res_stride;     /* residual entries per (layer, Z, head) slab; a multiple
                             of 256 and >= the largest slab total + 512            */
  int32_t split_tokens;   /* tokens per workgroup chunk; 0 = automatic, otherwise a
                             multiple of 64                                        */
  int32_t coef_format;    /* DWKV_COEF_F16 or DWKV_COEF_I8 (see dwkv_cache)        */
} dwkv_dims;

/* Coefficient storage.  DWKV_COEF_F16: fp16 rows.  DWKV_COEF_I8: the paper's
 * 8-bit blockwise form (Sec. 3): per token, each block of 16 coefficients
 * [16 s, 16 s + 16) is an fp16 scale times int8 codes in [-127, 127],
 * A_i = scale_{t, i/16} * code_i. */
typedef enum dwkv_coef_format { DWKV_COEF_F16 = 0, DWKV_COEF_I8 = 1 } dwkv_coef_format;

/* Compressed cache (Eq. 1 factors).  M = L / window, Z = 0 keys, Z = 1 values. */
typedef struct dwkv_cache {
  const void*     basis;     /* fp16 [B][M][Hkv][2][r_b][d]: rows of B^Z_{m,h} per sequence */
  const void*     coef_k;    /* fp16 [L][Hkv][T16/16][r_b/8][16][8]: key coefficients
                                A^K_{l,h,t} in tiles of 16 tokens x 8 coefficients,
                                coefficient index fastest: token t, coefficient i at
                                [t/16][i/8][t%16][i%8]; T16 = T rounded up to 16       */
  const void*     coef_v;    /* fp16 [L][Hkv][T16/8][r_b][8]: value coefficients A^V_{l,h,t}
                                in 8-token blocks, token index fastest: token t,
                                coefficient i at [t/8][i][t%8].  In both, the padding
                                tokens past T must be finite (zero).  These layouts let
                                each wave load of the decode read whole 128-byte lines. */
  const uint8_t*  rank_code; /* [M][Hkv][T] level index k of each token (rho = levels[k])  */
  const uint32_t* res_off;   /* [M][Hkv][T+1] exclusive running sum of rho over the packed
                                tokens: token t's entries are [res_off[t], res_off[t+1])   */
  const uint8_t*  res_idx;   /* [L][2][Hkv][res_stride] channel index (< d) of each entry  */
  const uint8_t*  res_val;   /* [L][2][Hkv][res_stride/2] int4 two's-complement codes;
                                entry e in byte e/2, low nibble when e is even; -8 invalid */
  const void*     res_scale; /* fp16 [L][2][Hkv][T] gate-folded residual scale g*s         */
  const void*     coef_k_scale; /* DWKV_COEF_I8 only (else ignored): fp16 [L][Hkv][r_b/16][T]
                                block scales of the key coefficients; coef_k then holds int8
                                codes in tiles of 16 tokens x 16 codes,
                                [L][Hkv][T16/16][r_b/16][16][16]: token t, code i at
                                [t/16][i/16][t%16][i%16] (padding tokens zero)            */
  const void*     coef_v_scale; /* DWKV_COEF_I8 only: fp16 [L][Hkv][r_b/16][T] value block
                                scales; coef_v then holds int8 codes in 16-token blocks
                                [L][Hkv][T16/16][r_b][16], token fastest                    */
} dwkv_cache;

/* Attention-output probe (Eq. 3) against a dense higher-fidelity cache. */
typedef struct dwkv_probe {
  int32_t n_heads;             /* probed KV heads, 1..min(Hkv, 64)                     */
  const int32_t* kv_heads_host;/* [n_heads] distinct KV head ids                       */
  const void* k_ref;           /* fp16 [n_heads][T][d] reference keys (packed tokens)  */
  const void* v_ref;           /* fp16 [n_heads][T16/16][d][16] reference values in
                                  16-token blocks, token index fastest: token t, channel
                                  c at [t/16][c][t%16] (finite padding)                */
  float eps;                   /* Eq. 3 epsilon (e.g. 1e-6)                            */
  float* err;                  /* out fp32 [B][n_heads*G]: probed head i, group member g
                                  at column i*G+g                                      */
  float* out_ref;              /* optional out fp32 [B][n_heads*G][d]: attention over the
                                  reference cache of the current position's query; may
                                  be NULL                                              */
  /* Several recent query positions (Sec. 3 evaluates a subset of heads and
   * recent positions twice).  The query j steps back (j = 1..n_pos-1) attends
   * to the first T_b - j tokens of its sequence in this cache and in the
   * reference (nothing when T_b <= j), and err becomes, per column,
   *   sqrt(sum_j ||O_ref_j - O_j||^2) / (sqrt(sum_j ||O_ref_j||^2) + eps)
   * with the norms over the positions j = 0..n_pos-1 and d together. */
  int32_t n_pos;               /* positions, 1..DWKV_MAX_PROBE_POS; 0 reads as 1       */
  const void* q_prev;          /* n_pos > 1: [n_pos-1][B][Hq][d] in the decode's q_type,
                                  slice j-1 the query of the position j steps back
                                  (16-byte aligned); ignored when n_pos <= 1           */
} dwkv_probe;

int32_t dwkv_abi_version(void);
const char* dwkv_status_str(dwkv_status s);

/* Tokens per workgroup chunk the decode will use for these dims (the automatic
 * choice when dims->split_tokens is 0), or -1 when the dims are invalid. */
int32_t dwkv_split_tokens(const dwkv_dims* dims);

/* Which split-K kernel dwkv_decode runs for these dims: 1 the token-lane
 * kernel (query groups of 1, 2 or 4 heads with ranks up to 16, or 8 heads with
 * ranks up to 32; r_b up to 64), 0 the general kernel, -1 invalid dims. */
int32_t dwkv_decode_kernel(const dwkv_dims* dims);

/* Bytes of device workspace dwkv_decode needs (0 when dims are invalid).
 * probe may be NULL. */
size_t dwkv_workspace_bytes(const dwkv_dims* dims, const dwkv_probe* probe);

/* Kernel launches one dwkv_decode call enqueues for these dims (2: the
 * split-K pass and the merge; with a probe the merge also evaluates Eq. 3 and
 * the reference pass is added -- inside the split-K launch on the token-lane
 * kernel (still 2), as a launch of its own on the general kernel (3) -- and a
 * probe over n_pos > 1 positions adds
 * one launch -- the factorized and the reference pass on the probed heads --
 * for every earlier position that still sees a token of some sequence, and
 * one merge), or -1 when the dims or probe are invalid.  probe may be NULL. */
int32_t dwkv_decode_launches(const dwkv_dims* dims, const dwkv_probe* probe);

/* Per-layer decode attention over the factorized cache (Eq. 1 folded into the
 * attention, Sec. 3 fused data path): for every sequence b and query head hq,
 *   out[b][hq] = softmax_t(sm_scale * q[b][hq] . K_hat_t) V_hat_t
 * over the T_b cached tokens of sequence b (no mask; the decode token is
 * already appended), K_hat/V_hat as in Eq. 1 for layer `layer` (0-based index
 * into the layers held).  An empty sequence (T_b = 0) yields zeros.
 *   q:        [B][Hq][d] in q_type (fp16 or bf16), read-only
 *   sm_scale: softmax scale; <= 0 selects 1/sqrt(d)
 *   out:      fp32 [B][Hq][d], written
 *   probe:    NULL, or Eq. 3 error for the listed KV heads (see dwkv_probe)
 *   workspace:>= dwkv_workspace_bytes(dims, probe) bytes of device memory;
 *             contents need no initialisation and are clobbered; calls
 *             sharing it must be ordered (same stream).
 * Launches the split-K kernel(s) (with a probe, the reference pass too) and
 * the merge kernel(s) (dwkv_decode_launches gives the count).
 * Returns DWKV_OK once enqueued. */
dwkv_status dwkv_decode(const dwkv_dims* dims, const dwkv_cache* cache, int32_t layer,
                        const void* q, int32_t q_type, float sm_scale, float* out,
                        const dwkv_probe* probe, void* workspace, size_t ws_bytes,
                        void* stream);

/* dwkv_decode in two ordered steps on one stream, same arguments and
 * semantics: dwkv_decode_partials launches the split-K pass(es), writing one
 * partial per (work item, KV head, group member) into the workspace;
 * dwkv_decode_merge merges them into `out` (and, with a probe, writes err /
 * out_ref).  Both calls take the same dims, cache, layer and probe pointer;
 * the merge reads the cache's bases (it may finish the value product).
 * The outputs equal dwkv_decode's bit for bit. */
dwkv_status dwkv_decode_partials(const dwkv_dims* dims, const dwkv_cache* cache, int32_t layer,
                                 const void* q, int32_t q_type, float sm_scale,
                                 const dwkv_probe* probe, void* workspace, size_t ws_bytes,
                                 void* stream);
dwkv_status dwkv_decode_merge(const dwkv_dims* dims, const dwkv_cache* cache, int32_t layer,
                              float* out, const dwkv_probe* probe, void* workspace,
                              size_t ws_bytes, void* stream);

/* For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): dwkv_decode with the same
 * arguments and results, minus the workspace.  Its split partials live in a
 * library-owned static device array of dwkv_static_scratch_bytes() bytes
 * (DWKV_STATIC_SCRATCH_BYTES, 16 MiB), one copy per GPU the library runs on,
 * held until the process ends; its address on a device is looked up (without
 * allocating) on the first call made with that device current.  The call
 * itself allocates nothing and calls no allocating routine; the caller still
 * passes q, out and the cache.  It returns DWKV_E_SCRATCH, enqueuing nothing,
 * when the dims (and probe) need more than the array holds, i.e. when
 * dwkv_workspace_bytes(dims, probe) > dwkv_static_scratch_bytes().  Every call
 * on one GPU shares that GPU's array and leaves its partials there: calls that
 * overlap on one GPU (different streams, or threads without ordering) race and
 * must be serialised by the caller.  The decode needs no initial contents in
 * the array, so nothing is cleared between calls.  This is the one piece of
 * global state in the library (the per-device address table is guarded by a
 * mutex). */
#define DWKV_STATIC_SCRATCH_BYTES (16u << 20)
size_t dwkv_static_scratch_bytes(void);
dwkv_status dwkv_decode_noalloc(const dwkv_dims* dims, const dwkv_cache* cache, int32_t layer,
                                const void* q, int32_t q_type, float sm_scale, float* out,
                                const dwkv_probe* probe, void* stream);

/* Bytes of device workspace dwkv_route needs (0 when dims are invalid). */
size_t dwkv_route_workspace_bytes(const dwkv_dims* dims);

/* Token-conditional depth router (Eq. 2, multi-level reading) and the residual
 * offsets it implies.  For every window m, KV head h and packed token t:
 *   z = ((u0*phi0 + u1*phi1) + u2*phi2) + u3*phi3   (float32, each op rounded)
 *   k = #{ j < n_levels-1 : z > theta[m][j] }      (strict: ties keep the lower level)
 *   rank_code[m][h][t] = k,   rho = levels[k]
 *   res_off[m][h][0] = 0,     res_off[m][h][t+1] = res_off[m][h][t] + rho
 * theta holds logits of the gate thresholds tau (theta = log(tau/(1-tau))), so
 * z > theta is sigma(z) > tau.
 *   phi:   fp32 [M][Hkv][T][4] router features
 *   u:     fp32 [M][4] router weights (shared by the layers of a window)
 *   theta: fp32 [M][n_levels-1] ascending thresholds on z
 *   rank_code: out uint8 [M][Hkv][T];  res_off: out uint32 [M][Hkv][T+1]
 * Bit-exact by construction.  Returns DWKV_E_UNSUPPORTED when
 * T * levels[n_levels-1] could exceed 2^32-1. */
dwkv_status dwkv_route(const dwkv_dims* dims, const float* phi, const float* u,
                       const float* theta, uint8_t* rank_code, uint32_t* res_off,
                       void* workspace, size_t ws_bytes, void* stream);

/* dwkv_route for packed tokens [t0, t1) only, continuing an existing table:
 * writes rank_code[m][h][t] for those tokens and
 *   res_off[m][h][t+1] = res_off[m][h][t] + rho
 * starting from the res_off[m][h][t0] already in the table (when t0 == 0,
 * res_off[m][h][0] is set to 0 first).  Appending a decode token to the end of
 * the packed layout is the range [T-1, T).  Same arguments, layout and
 * workspace size (dwkv_route_workspace_bytes) as dwkv_route;
 * 0 <= t0 <= t1 <= T, else DWKV_E_DIMS.  Bit-exact by construction. */
dwkv_status dwkv_route_range(const dwkv_dims* dims, const float* phi, const float* u,
                             const float* theta, int64_t t0, int64_t t1, uint8_t* rank_code,
                             uint32_t* res_off, void* workspace, size_t ws_bytes, void* stream);

/* Bytes of device workspace dwkv_route_budget needs (0 when dims are invalid). */
size_t dwkv_route_budget_workspace_bytes(const dwkv_dims* dims);

/* Budget-driven routing (Sec. 3: the threshold tau_m is chosen to satisfy the
 * current memory budget), for the two-level form of Eq. 2 (n_levels == 2,
 * else DWKV_E_UNSUPPORTED).  For every window m and KV head h, over packed
 * tokens [t0, t1) (N of them), with z the router score of dwkv_route:
 *   n = floor((E - N levels[0]) / (levels[1] - levels[0])), clamped to [0, N]
 *   the n tokens of largest z get rank code 1, the others 0; equal scores go
 *   to the lower token (the n-th largest score is the effective tau)
 * and res_off continues from res_off[m][h][t0] as in dwkv_route_range.
 *   entries: DEVICE int64 [M][Hkv], E, the residual entries allowed over the
 *            range for (m, h) (8-byte aligned)
 *   phi, u, rank_code, res_off: as dwkv_route (phi and u 16-byte aligned)
 *   workspace: >= dwkv_route_budget_workspace_bytes(dims), no initial contents
 * phi must be finite (a NaN score has no defined place).  Bit-exact by
 * construction.  One launch, one workgroup per (window, head). */
dwkv_status dwkv_route_budget(const dwkv_dims* dims, const float* phi, const float* u, const int64_t* entries,
                              int64_t t0, int64_t t1, uint8_t* rank_code, uint32_t* res_off, void* workspace,
                              size_t ws_bytes, void* stream);

/* Append/compress (Sec. 3: coefficients by projection onto the window's
 * current basis, residuals 4-bit quantized at the routed rank, the gate of
 * Eq. 1 folded into the scale).  For packed tokens [t0, t1) of layer `layer`,
 * every KV head h and both Z, from the dense vector x (1 x d, fp16):
 *   A_i   = fp16(sum_j x_j B_ij)                      (B = B^Z of the token's
 *                                                      sequence, window, head)
 *   r_c   = x_c - sum_i A_i B_ic
 *   kept  = the rho channels of largest |r_c|, ties to the lower channel,
 *           rho = levels[rank_code[m][h][t]]
 *   S     = max_c |r_c| / 7;  code_c = round-half-even(r_c / S) in [-7, 7]
 *           (0 when S == 0)
 *   res_scale = fp16(g * S) (0 for a rank-0 token); entries stored at
 *           [res_off[t], res_off[t+1]) ordered by descending |code|, then
 *           ascending channel.
 * With dims->coef_format == DWKV_COEF_I8 the coefficient rows are written in
 * the 8-bit blockwise form instead (Sec. 3): per token and block of 16
 * coefficients [16 s, 16 s + 16), from the float32 projection A (not rounded
 * to fp16),
 *   S_s   = fp16(max_i |A_i| / 127),  code_i = round-half-even(A_i / S_s)
 *           clamped to [-127, 127] (0 when S_s == 0)
 * into coef_k / coef_v (int8 tiles) and coef_k_scale / coef_v_scale (the
 * layouts dwkv_cache states), and the residual is taken against the rebuilt
 * rows code_i * S_s; in the basis term of the residual each product is then
 * rounded to float32 before it is added.
 * Arithmetic: float32, every product and sum rounded on its own; each sum runs
 * left to right over its contracted index (j = 0..d-1 for A_i, i = 0..r_b-1
 * for the basis term), starting from its first product; A is rounded to fp16
 * before the residual; S and r_c / S are correctly rounded divisions.  The
 * integer results are therefore exact functions of the inputs.
 *   x_k, x_v: fp16 [t1-t0][Hkv][d] dense keys / values of the tokens
 *             (keys post positional encoding, as the decode expects)
 *   gate:     NULL (g = 1) or fp32 [2][Hkv][t1-t0], g in [0, 1]
 * WRITES through the cache's pointers (coef_k, coef_v, res_idx, res_val,
 * res_scale of `layer`, only at the range's tokens and entries; coef_v padding
 * is untouched); reads basis, rank_code and res_off, which must already hold
 * the tokens' routing (dwkv_route / dwkv_route_range).  A token whose rank code
 * or offsets are inconsistent gets its coefficients and scale 0 but no entries
 * (dwkv_validate reports it).  basis, coef_k, coef_v, x_k, x_v must be 16-byte
 * aligned, res_idx and res_scale 2-byte, gate 4-byte (else DWKV_E_ALIGN).
 * One launch; the library allocates nothing. */
dwkv_status dwkv_compress(const dwkv_dims* dims, const dwkv_cache* cache, int32_t layer,
                          const void* x_k, const void* x_v, const float* gate, int64_t t0,
                          int64_t t1, void* stream);

/* One decode step of layer `layer` that appends first: the new token of
 * every non-empty sequence b is its last packed token t_b = cu[b+1] - 1 (its
 * slot and routing already in the cache, as dwkv_compress requires);
 *   dwkv_compress of t_b from x_k[b], x_v[b] (and gate), then
 *   dwkv_decode of the layer (no probe),
 * with the same stored factors (bit for bit those of dwkv_compress) and the
 * same output semantics (the new token attended in its compressed form, Eq. 1).
 * For query groups and ranks the token-lane kernel serves, fp16 coefficients
 * and at most 16 sequences, it is one split-K launch plus the merge: the
 * split items cover each sequence's tokens but its last, and one more
 * workgroup per sequence and KV head compresses the new token, writes it to
 * the cache and contributes its own term to the merge (its score against the
 * key rebuilt from the stored factors, its value in basis space), so no
 * workgroup reads what another writes.  Otherwise the append/compress kernel
 * runs once per sequence, then the decode.  The output then differs from
 * dwkv_compress + dwkv_decode only in float32 rounding order.
 *   q, q_type, sm_scale, out: as in dwkv_decode
 *   x_k, x_v: fp16 [B][Hkv][d] the new token's key / value of each sequence
 *             (rows of empty sequences unused), 16-byte aligned
 *   gate:     NULL (g = 1) or fp32 [2][Hkv][B], 4-byte aligned
 *   workspace:>= dwkv_decode_append_workspace_bytes(dims) bytes of device
 *             memory, no initial contents, clobbered
 * WRITES the cache as dwkv_compress does.  Returns DWKV_OK once enqueued. */
size_t dwkv_decode_append_workspace_bytes(const dwkv_dims* dims);
/* Kernel launches of one dwkv_decode_append call: 2 on the one-launch path,
 * else the number of non-empty sequences plus 2; -1 for invalid dims. */
int32_t dwkv_decode_append_launches(const dwkv_dims* dims);
dwkv_status dwkv_decode_append(const dwkv_dims* dims, const dwkv_cache* cache, int32_t layer,
                               const void* q, int32_t q_type, float sm_scale, float* out,
                               const void* x_k, const void* x_v, const float* gate,
                               void* workspace, size_t ws_bytes, void* stream);

/* Dense residual term g*R of Eq. 1 for packed tokens [t0, t1) of slab
 * (layer, z, kv_head): dense[t-t0][c] = res_scale * code for every stored entry
 * of token t at channel c, zero elsewhere; fp32 [t1-t0][d] (may be NULL when
 * t1 == t0).  Decodes entries
 * with the same device routines the decode kernel uses (a test hook). */
dwkv_status dwkv_residual_map(const dwkv_dims* dims, const dwkv_cache* cache, int32_t layer,
                              int32_t z, int32_t kv_head, int64_t t0, int64_t t1,
                              float* dense, void* stream);

/* Bytes of device workspace dwkv_decode_features needs (0 when the dims are
 * invalid or the shape is not on the token-lane path: dwkv_decode_kernel
 * returns 0). */
size_t dwkv_features_workspace_bytes(const dwkv_dims* dims);

/* dwkv_decode (no probe), plus the attention features the router reads
 * (Sec. 3: accumulated attention mass, maximum attention spike).  With p the
 * softmax probability of token t for query head hq at this layer:
 *   phi[m][h][t][0] += sum over the query heads hq of KV head h of p
 *   phi[m][h][t][1]  = max(phi[m][h][t][1], max over those heads of p)
 * for every packed token t of every sequence, m = layer / window; columns 2
 * and 3 are untouched.  Calling it for every layer of a window and every
 * decode step accumulates the features over both.
 *   phi: fp32 [M][Hkv][T][4] (the layout dwkv_route reads), read and written
 *   workspace: >= dwkv_features_workspace_bytes(dims) bytes, no initial contents
 * `out` equals dwkv_decode's bit for bit.  Three launches (split-K pass that
 * also stores the scores, merge, features).  DWKV_E_UNSUPPORTED off the
 * token-lane path (fp16 coefficients, or int8 for groups of up to 4). */
dwkv_status dwkv_decode_features(const dwkv_dims* dims, const dwkv_cache* cache, int32_t layer,
                                 const void* q, int32_t q_type, float sm_scale, float* out, float* phi,
                                 void* workspace, size_t ws_bytes, void* stream);

/* The fourth router feature (Sec. 3: the attention-output reconstruction
 * error from the previous probe interval, Eq. 3).  Eq. 3 yields one error per
 * sequence and query head; the router scores tokens.  For every probed KV
 * head h = kv_heads_host[i] and sequence b, with e the largest of
 * err[b][i*G .. i*G + G-1] (over h's query heads):
 *   phi[m][h][t][3] = fresh ? e : max(phi[m][h][t][3], e)
 * for every packed token t of b, m = layer / window.  Call it once per probed
 * layer of an interval, the first time with fresh = 1, so that the column
 * holds the largest error over the window's probed layers; heads not probed
 * keep their value, and columns 0-2 are untouched.
 *   err:  device fp32 [B][n_heads * G], as dwkv_decode writes it for a probe
 *         with the same kv_heads_host
 *   phi:  device fp32 [M][Hkv][T][4], read and written
 * One launch.  Argument errors (n_heads outside 1..min(Hkv, 64), repeated or
 * out-of-range heads, layer out of range) return before anything is enqueued. */
dwkv_status dwkv_probe_feature(const dwkv_dims* dims, int32_t layer, int32_t n_heads,
                               const int32_t* kv_heads_host, const float* err, int32_t fresh,
                               float* phi, void* stream);

/* Bytes of device workspace dwkv_sketch_basis needs for a prefill of
 * n_tokens tokens (0 when invalid). */
size_t dwkv_sketch_workspace_bytes(const dwkv_dims* dims, int64_t n_tokens);

/* Online basis initialization (Sec. 3: a small randomized low-rank sketch of
 * the window's cached keys and values after prefill, per head, K and V apart).
 * For sequence `seq`, window `window`, every KV head h and Z:
 *   X     = the window's prefill vectors of head h, rows (layer l, token t),
 *           ((w n_tokens) x d)
 *   Y     = Omega X   (r_b x d, float64 sums of exact fp16 products)
 *   basis = Gram-Schmidt orthonormalization of Y's rows in order (float64),
 *           rounded to fp16; a row whose remaining norm is below 1e-9 of the
 *           largest row norm of Y (a rank-deficient sketch) becomes zero
 *   x:     fp16 [w][2][n_tokens][Hkv][d]  (Z = 0 keys, post positional
 *          encoding, Z = 1 values)
 *   omega: fp16 [w * n_tokens][r_b], row l * n_tokens + t: the random sketch
 *          matrix (transposed), drawn by the caller and shared by heads and Z
 * WRITES cache->basis[seq][window] (all heads, both Z); nothing else.  Two
 * launches.  All pointers 16-byte aligned. */
dwkv_status dwkv_sketch_basis(const dwkv_dims* dims, const dwkv_cache* cache, int32_t window, int32_t seq,
                              const void* x, const void* omega, int64_t n_tokens, void* workspace,
                              size_t ws_bytes, void* stream);

/* Probe-feedback threshold control (Sec. 3): when a window's probe error
 * (Eq. 3) exceeds its tolerance the router lowers the window's threshold;
 * after several probe intervals below tolerance it raises it.  The paper
 * gives no constants; they are the caller's. */
typedef struct dwkv_controller {
  float tol;              /* tolerance on the window's probe error               */
  float step_down;        /* logit step down of every threshold on e > tol (>= 0) */
  float step_up;          /* logit step up after `patience` intervals (>= 0)     */
  int32_t patience;       /* consecutive intervals at or below tol before a step up (>= 1) */
  float theta_min;        /* clamp of every threshold (theta_min <= theta_max)   */
  float theta_max;
} dwkv_controller;

/* One probe interval for n_windows windows, on HOST arrays:
 *   err_host:   [n_windows] the window's probe error (the largest Eq. 3 error
 *               over its probed layers, heads and sequences); NaN counts as
 *               above tolerance
 *   theta_host: [n_windows][n_thresholds] router thresholds on z (logits of
 *               tau, as dwkv_route reads them), updated in place: every
 *               threshold of a window moves by the same step (float32), then
 *               is clamped to [theta_min, theta_max], so their order is kept
 *   below_host: [n_windows] consecutive intervals at or below tol, updated;
 *               reset to 0 on every step
 * Synchronous host code; DWKV_E_DIMS for bad counts or constants. */
dwkv_status dwkv_controller_update(const dwkv_controller* ctl, int32_t n_windows, int32_t n_thresholds,
                                   const float* err_host, float* theta_host, int32_t* below_host);

/* Probe schedule (Sec. 3: every p decode steps a small subset of heads and
 * recent query positions is evaluated twice).  The paper fixes neither the
 * subset nor p; the schedule here rotates it: decode step `step` (0-based,
 * counted from the first decode step after prefill) probes when
 * step % period == 0, and the k-th probe (k = step / period) takes the KV
 * heads (k * n_heads + i) % n_kv_heads, i < n_heads, so every head is probed
 * in every ceil(n_kv_heads / n_heads) consecutive probes, over
 * min(n_pos, step + 1) recent positions (the decode steps so far).
 *   heads_host: [n_heads] written on a probe step (for dwkv_probe.kv_heads_host)
 *   n_pos_host: written, the positions to probe (0 on other steps)
 * Returns n_heads on a probe step, 0 on other steps, -1 for bad arguments
 * (period < 1, n_heads outside 1..min(n_kv_heads, 64), n_pos outside 1..8,
 * step < 0, null pointers).  Host code. */
int32_t dwkv_probe_schedule(int64_t step, int32_t period, int32_t n_heads, int32_t n_kv_heads, int32_t n_pos,
                            int32_t* heads_host, int32_t* n_pos_host);

/* Comparison paths (the fused decode's alternatives: the paper's "full KV"
 * baseline and its "w/o fused kernel" ablation, Table 1 and Table 2).
 *
 * dwkv_materialize: Eq. 1 written out for every packed token and KV head of
 * layer `layer`: K_hat = A^K B^K + g R^K, V_hat = A^V B^V + g R^V, summed in
 * float32 and rounded once to fp16.
 *   k_out: fp16 [Hkv][T][d] (row-major, packed tokens), written
 *   v_out: fp16 [Hkv][T16/16][d][16] (16-token blocks, token index fastest,
 *          the layout of dwkv_probe.v_ref), written; padding tokens zeroed
 * Reads the cache as dwkv_decode does (residual entries past res_stride or a
 * rank above d are not added).  basis, coef_k, coef_v, k_out and v_out must be
 * 16-byte aligned, res_scale 2-byte (else DWKV_E_ALIGN).  One launch. */
dwkv_status dwkv_materialize(const dwkv_dims* dims, const dwkv_cache* cache, int32_t layer,
                             void* k_out, void* v_out, void* stream);

/* Bytes of device workspace dwkv_dense_decode needs (0 when dims are invalid). */
size_t dwkv_dense_workspace_bytes(const dwkv_dims* dims);

/* Decode attention over a dense fp16 cache (no factorization): for every
 * sequence b and query head hq, out[b][hq] = softmax_t(sm_scale q.K_t) V_t
 * over the T_b packed tokens of sequence b, KV head hq / (Hq/Hkv).
 *   k: fp16 [Hkv][T][d];  v: fp16 [Hkv][T16/16][d][16] (blocked as above)
 *   q, q_type, sm_scale, out: as in dwkv_decode
 *   workspace: >= dwkv_dense_workspace_bytes(dims) bytes, no initial contents
 * Uses dims for the shape only (cu_seqlens, heads, T, split_tokens); the
 * cache fields of dims must still be valid.  Every pointer 16-byte aligned.
 * Two launches (split-K pass, merge). */
dwkv_status dwkv_dense_decode(const dwkv_dims* dims, const void* k, const void* v, const void* q,
                              int32_t q_type, float sm_scale, float* out, void* workspace,
                              size_t ws_bytes, void* stream);

/* Number of sink words dwkv_hbm_read writes (its block count). */
int32_t dwkv_hbm_read_blocks(void);

/* HBM read stream, for measurement; it implements no operation of the paper.
 * It reads `bytes` bytes of device memory once, each wave load covering 1 KB
 * of consecutive bytes with the nontemporal hint.  Timed on a buffer well
 * beyond the last-level caches, it gives the practical read-bandwidth
 * ceiling that the decode's achieved bandwidth is set against, next to the
 * published 8 TB/s (the paper's speed figures are tokens/s, Sec. 4).
 *   buf: device, 16-byte aligned; bytes: a multiple of 16 (0 allowed)
 *   sink: device uint32 [sink_words], 4-byte aligned, sink_words >=
 *     dwkv_hbm_read_blocks(); block b writes sink[b] = the xor of the 32-bit
 *     words it read, so the xor of sink[0 .. blocks) is the xor of every
 *     32-bit word of buf (0 for an empty buffer).  Words past the block
 *     count are not touched.
 * Errors: DWKV_E_NULL (sink, or buf with bytes > 0), DWKV_E_DIMS (bytes not
 * a multiple of 16), DWKV_E_WORKSPACE (sink too small), DWKV_E_ALIGN.  One
 * launch. */
dwkv_status dwkv_hbm_read(const void* buf, size_t bytes, uint32_t* sink, int32_t sink_words, void* stream);

/* Bytes of device workspace dwkv_validate needs. */
size_t dwkv_validate_workspace_bytes(void);

/* Checks the layout (synchronous; blocks on `stream`): for every window, head
 * and token, res_off[t+1]-res_off[t] == levels[rank_code[t]] and rank_code <
 * n_levels; res_off[0] == 0 and res_off[T] + 512 <= res_stride; for every
 * layer and Z, each token's channel indices are < d and distinct, no code is
 * -8, and entries are ordered by descending |code|, then ascending channel.
 * Returns DWKV_OK or DWKV_E_LAYOUT; *bad_index (if not NULL) receives a code
 * locating the first failure found (-1 when none). */
dwkv_status dwkv_validate(const dwkv_dims* dims, const dwkv_cache* cache, int64_t* bad_index,
                          void* workspace, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* DWKV_H */
