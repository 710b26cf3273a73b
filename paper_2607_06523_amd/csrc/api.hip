// C ABI of the library: argument checks, split planning, launches.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>

#include "internal.h"

using namespace dwkv;

namespace {

constexpr int kTargetWorkgroups = 512;   // ~2 decode workgroups per compute unit
constexpr int kSplitQuantum = 256;       // automatic chunks are multiples of this
constexpr int kSplitMax = 8192;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool is_pow2_group(int g) { return g == 1 || g == 2 || g == 4 || g == 8 || g == 16; }

int max_level(const dwkv_dims* d) {
  int mx = 0;
  for (int i = 0; i < d->n_levels; ++i) mx = d->levels[i] > mx ? d->levels[i] : mx;
  return mx;
}

// Shape checks shared by every entry point.
dwkv_status check_dims(const dwkv_dims* d) {
  if (!d) return DWKV_E_NULL;
  if (d->batch < 1 || d->n_layers < 1 || d->window < 1 || d->n_kv_heads < 1 || d->n_q_heads < 1 ||
      d->n_levels < 1 || d->total_tokens < 0 || d->split_tokens < 0)
    return DWKV_E_DIMS;
  if (d->n_layers % d->window != 0 || d->n_q_heads % d->n_kv_heads != 0) return DWKV_E_DIMS;
  if (d->n_levels > DWKV_MAX_LEVELS) return DWKV_E_UNSUPPORTED;
  if (d->head_dim != kHeadDim) return DWKV_E_UNSUPPORTED;
  if (!is_pow2_group(d->n_q_heads / d->n_kv_heads)) return DWKV_E_UNSUPPORTED;
  if (d->n_kv_heads > DWKV_MAX_PROBE_HEADS) return DWKV_E_UNSUPPORTED;
  if (d->basis_rank < 16 || d->basis_rank > 128 || d->basis_rank % 16 != 0) return DWKV_E_UNSUPPORTED;
  for (int i = 0; i < d->n_levels; ++i) {
    const int lv = d->levels[i];
    if (lv < 0 || lv > d->head_dim || (lv & 1)) return DWKV_E_DIMS;
    if (i > 0 && lv <= d->levels[i - 1]) return DWKV_E_DIMS;
  }
  if (!d->cu_seqlens_host || !d->cu_seqlens) return DWKV_E_NULL;
  if (d->cu_seqlens_host[0] != 0) return DWKV_E_DIMS;
  for (int b = 0; b < d->batch; ++b)
    if (d->cu_seqlens_host[b + 1] < d->cu_seqlens_host[b]) return DWKV_E_DIMS;
  if ((int64_t)d->cu_seqlens_host[d->batch] != d->total_tokens) return DWKV_E_DIMS;
  if (d->res_stride < kResTailPad || d->res_stride % 256 != 0) return DWKV_E_DIMS;
  if (d->split_tokens % 64 != 0) return DWKV_E_DIMS;
  if (d->coef_format != DWKV_COEF_F16 && d->coef_format != DWKV_COEF_I8) return DWKV_E_DIMS;
  // offsets, plus a few chunks of slack, must stay inside 32 bits
  if ((double)d->total_tokens * (double)max_level(d) + 65536.0 > 4294967295.0) return DWKV_E_UNSUPPORTED;
  return DWKV_OK;
}

// The token-lane split kernel serves query groups of up to 4 heads with
// basis ranks up to 64 and ranks up to 16, as long as one (KV head, query
// head)'s partials of a sequence span less than 2^31 bytes (its merge reads
// them through 32-bit offsets); the general kernel serves the rest.
bool uses_token_lane(const dwkv_dims* d) {
  const int g = d->n_q_heads / d->n_kv_heads;
  const int64_t min_split = d->split_tokens > 0 ? d->split_tokens : kSplitQuantum;
  int64_t longest = 0;
  for (int b = 0; b < d->batch; ++b)
    longest = std::max<int64_t>(longest, d->cu_seqlens_host[b + 1] - d->cu_seqlens_host[b]);
  const int64_t chunks = (longest + min_split - 1) / min_split;
  return token_lane_supported(d->basis_rank, g, max_level(d), d->total_tokens, d->res_stride) &&
         chunks * g * kPartStrideTL * (int64_t)sizeof(float) < ((int64_t)1 << 31);
}

int64_t count_work(const dwkv_dims* d, int split, int trim = 0);

int plan_split(const dwkv_dims* d) {
  if (d->split_tokens > 0) return d->split_tokens;
  const int64_t work = d->total_tokens * d->n_kv_heads;
  // one workgroup per CU for the token-lane kernel (8 waves), two for the general one (4 waves)
  const int64_t target = uses_token_lane(d) ? kTargetWorkgroups / 2 : kTargetWorkgroups;
  int64_t c = (work + target - 1) / target;
  c = (c + kSplitQuantum - 1) / kSplitQuantum * kSplitQuantum;
  if (c < kSplitQuantum) c = kSplitQuantum;
  // every sequence rounds its chunks up: grow the chunk until the workgroups
  // of all sequences fit one round of the target
  while (c < kSplitMax && count_work(d, (int)c) * d->n_kv_heads > target) c += kSplitQuantum;
  if (c > kSplitMax) c = kSplitMax;
  return (int)c;
}

// Chunk size of the general split kernel alone (the dense decode): about two
// workgroups per compute unit.
int plan_split_general(const dwkv_dims* d) {
  if (d->split_tokens > 0) return d->split_tokens;
  const int64_t work = d->total_tokens * d->n_kv_heads;
  int64_t c = (work + kTargetWorkgroups - 1) / kTargetWorkgroups;
  c = (c + kSplitQuantum - 1) / kSplitQuantum * kSplitQuantum;
  if (c < kSplitQuantum) c = kSplitQuantum;
  if (c > kSplitMax) c = kSplitMax;
  return (int)c;
}

// Chunk size of the probe's dense reference pass over n_heads probed KV
// heads: about kTargetWorkgroups / 2 workgroups for the pass, so that one
// probed head is not streamed by a handful of workgroups, while its merge
// still reads few partials.  An explicit split_tokens applies here too.
int plan_split_ref(const dwkv_dims* d, int n_heads) {
  if (d->split_tokens > 0) return d->split_tokens;
  const int64_t work = d->total_tokens * n_heads, target = kTargetWorkgroups / 2;
  int64_t c = (work + target - 1) / target;
  c = (c + kSplitQuantum - 1) / kSplitQuantum * kSplitQuantum;
  if (c < kSplitQuantum) c = kSplitQuantum;
  if (c > kSplitMax) c = kSplitMax;
  return (int)c;
}

// Work items of a pass over chunks of `split` tokens, every sequence cut
// `trim` tokens short.
int64_t count_work(const dwkv_dims* d, int split, int trim) {
  int64_t n = 0;
  for (int b = 0; b < d->batch; ++b) {
    const int64_t tb = std::max<int64_t>(d->cu_seqlens_host[b + 1] - d->cu_seqlens_host[b] - trim, 0);
    n += (tb + split - 1) / split;
  }
  return n;
}

int probe_positions(const dwkv_probe* p) { return p && p->n_pos > 1 ? p->n_pos : 1; }

// The probe's reference pass runs inside the split-K launch on the token-lane
// path (one grid of n_work * n_kv_heads split-K workgroups plus one workgroup
// per reference item).
bool fused_probe(const dwkv_dims* d, const dwkv_probe* p) {
  if (!p || !uses_token_lane(d)) return false;
  const int64_t nt = count_work(d, plan_split(d)) * d->n_kv_heads;
  const int64_t nr = count_work(d, plan_split_ref(d, p->n_heads)) * p->n_heads;
  return nr > 0 && nt + nr <= 0x7fffffff;
}

// Most work items of any one sequence (chunks of `split`, cut `trim` tokens
// short, plus `extra` items per non-empty sequence).
int32_t max_items(const dwkv_dims* d, int split, int trim = 0, int extra = 0) {
  int64_t n = 0;
  for (int b = 0; b < d->batch; ++b) {
    const int64_t len = d->cu_seqlens_host[b + 1] - d->cu_seqlens_host[b];
    const int64_t tb = std::max<int64_t>(len - trim, 0);
    n = std::max<int64_t>(n, (tb + split - 1) / split + (len > 0 ? extra : 0));
  }
  return (int32_t)std::min<int64_t>(n, 0x7fffffff);
}

dwkv_status check_probe(const dwkv_dims* d, const dwkv_probe* p) {
  if (!p) return DWKV_OK;
  if (p->n_heads < 1 || p->n_heads > d->n_kv_heads || p->n_heads > DWKV_MAX_PROBE_HEADS) return DWKV_E_DIMS;
  if (!p->kv_heads_host || !p->k_ref || !p->v_ref || !p->err) return DWKV_E_NULL;
  if (!aligned16(p->k_ref) || !aligned16(p->v_ref) || !aligned16(p->out_ref)) return DWKV_E_ALIGN;
  bool seen[DWKV_MAX_PROBE_HEADS] = {};
  for (int i = 0; i < p->n_heads; ++i) {
    const int h = p->kv_heads_host[i];
    if (h < 0 || h >= d->n_kv_heads || seen[h]) return DWKV_E_DIMS;
    seen[h] = true;
  }
  if (!(p->eps >= 0.f)) return DWKV_E_DIMS;
  if (p->n_pos < 0 || p->n_pos > DWKV_MAX_PROBE_POS) return DWKV_E_DIMS;
  if (p->n_pos > 1) {
    if (!p->q_prev) return DWKV_E_NULL;
    if (!aligned16(p->q_prev)) return DWKV_E_ALIGN;
  }
  return DWKV_OK;
}

// Workspace: the partials of the decode pass, then those of the probe pass;
// with several probe positions, for each earlier position its rebuilt and
// reference partials (pos_bytes each), then the Eq. 3 sums of the current one.
struct WsLayout {
  size_t main_bytes, ref_bytes, pos_bytes, acc_off, chunk_off, count_off, total;
};


WsLayout ws_layout(const dwkv_dims* d, const dwkv_probe* p) {
  const int split = plan_split(d);
  const int64_t nw = count_work(d, split);
  const int g = d->n_q_heads / d->n_kv_heads;
  const int stride = uses_token_lane(d) ? kPartStrideTL : kPartStride;
  WsLayout w;
  w.main_bytes = align_up((size_t)nw * d->n_kv_heads * g * stride * sizeof(float), 256);
  const int64_t nw_ref = p ? count_work(d, plan_split_ref(d, p->n_heads)) : 0;
  w.ref_bytes = p ? align_up((size_t)nw_ref * p->n_heads * g * kPartStride * sizeof(float), 256) : 0;
  const int np = probe_positions(p);
  w.pos_bytes = np > 1 ? w.ref_bytes : 0;
  w.acc_off = w.main_bytes + w.ref_bytes + (size_t)(np - 1) * 2 * w.pos_bytes;
  const size_t acc_bytes = np > 1 ? align_up((size_t)d->batch * p->n_heads * g * 2 * sizeof(float), 256) : 0;
  // the wide merge's reference rows of the probed columns, and its counters
  const size_t cols = p ? (size_t)d->batch * p->n_heads * g : 0;
  w.chunk_off = w.acc_off + acc_bytes;
  w.count_off = w.chunk_off + align_up(cols * kHeadDim * sizeof(float), 256);
  w.total = w.count_off + align_up(cols * sizeof(uint32_t), 256);
  if (w.total == 0) w.total = 256;
  return w;
}

dwkv_status hip_status(hipError_t e) { return e == hipSuccess ? DWKV_OK : DWKV_E_HIP; }

WorkTable work_table(const dwkv_dims* d, int split, int trim = 0) {
  WorkTable t;
  std::memset(&t, 0, sizeof(t));
  if (d->batch > kKernargSeqs) return t;
  t.n_seq = d->batch;
  for (int b = 0; b <= d->batch; ++b) t.tok[b] = d->cu_seqlens_host[b];
  for (int b = 0; b < d->batch; ++b) {
    const int64_t len = std::max<int64_t>(d->cu_seqlens_host[b + 1] - d->cu_seqlens_host[b] - trim, 0);
    t.work[b + 1] = t.work[b] + (int32_t)((len + split - 1) / split);
  }
  return t;
}

}  // namespace

extern "C" {

int32_t dwkv_abi_version(void) { return DWKV_ABI_VERSION; }

const char* dwkv_status_str(dwkv_status s) {
  switch (s) {
    case DWKV_OK: return "ok";
    case DWKV_E_NULL: return "null pointer";
    case DWKV_E_DIMS: return "inconsistent dimensions";
    case DWKV_E_UNSUPPORTED: return "unsupported shape";
    case DWKV_E_WORKSPACE: return "workspace too small";
    case DWKV_E_LAYOUT: return "malformed cache layout";
    case DWKV_E_HIP: return "HIP runtime error";
    case DWKV_E_ALIGN: return "device pointer not 16-byte aligned";
    case DWKV_E_SCRATCH: return "needs more than the library's static scratch";
  }
  return "unknown status";
}

int32_t dwkv_split_tokens(const dwkv_dims* dims) {
  if (check_dims(dims) != DWKV_OK) return -1;
  return plan_split(dims);
}

int32_t dwkv_decode_kernel(const dwkv_dims* dims) {
  if (check_dims(dims) != DWKV_OK) return -1;
  return uses_token_lane(dims) ? 1 : 0;
}

size_t dwkv_workspace_bytes(const dwkv_dims* dims, const dwkv_probe* probe) {
  if (check_dims(dims) != DWKV_OK || check_probe(dims, probe) != DWKV_OK) return 0;
  return ws_layout(dims, probe).total;
}

int32_t dwkv_decode_launches(const dwkv_dims* dims, const dwkv_probe* probe) {
  if (check_dims(dims) != DWKV_OK || check_probe(dims, probe) != DWKV_OK) return -1;
  if (!probe) return 2;
  int32_t n = fused_probe(dims, probe) ? 2 : 3;
  const int np = probe_positions(probe), split = plan_split_ref(dims, probe->n_heads);
  for (int j = 1; j < np; ++j)
    if (count_work(dims, split, j) > 0) n += 1;
  return np > 1 ? n + 1 : n;
}

}  // extern "C"

namespace {

dwkv_status check_decode_common(const dwkv_dims* d, const dwkv_probe* probe, void* workspace,
                                size_t ws_bytes) {
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  if (!workspace) return DWKV_E_NULL;
  if (!aligned16(workspace)) return DWKV_E_ALIGN;
  if ((st = check_probe(d, probe)) != DWKV_OK) return st;
  if (ws_bytes < ws_layout(d, probe).total) return DWKV_E_WORKSPACE;
  return DWKV_OK;
}

// Arguments of the layer's split-K pass over the whole cache (work split and
// partial layout left to the caller); checks the cache pointers.
dwkv_status split_args(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, const void* q, int32_t q_type,
                       float sm_scale, void* workspace, SplitArgs& a) {
  if (!c || !q) return DWKV_E_NULL;
  if (!c->basis || !c->coef_k || !c->coef_v || !c->res_off || !c->res_idx || !c->res_val ||
      !c->res_scale)
    return DWKV_E_NULL;
  if (layer < 0 || layer >= d->n_layers) return DWKV_E_DIMS;
  if (q_type != DWKV_F16 && q_type != DWKV_BF16) return DWKV_E_DIMS;
  const bool c8 = d->coef_format == DWKV_COEF_I8;
  if (c8) {
    if (!c->coef_k_scale || !c->coef_v_scale) return DWKV_E_NULL;
    if ((reinterpret_cast<uintptr_t>(c->coef_k_scale) | reinterpret_cast<uintptr_t>(c->coef_v_scale)) & 1u)
      return DWKV_E_ALIGN;
  }
  const void* const ptrs[] = {q, c->basis, c->coef_k, c->coef_v, c->res_off, c->res_idx, c->res_val, c->res_scale};
  for (const void* p : ptrs)
    if (!aligned16(p)) return DWKV_E_ALIGN;
  const int RB = d->basis_rank;
  const int64_t T = d->total_tokens;
  const int64_t T16 = (T + 15) / 16 * 16;
  const int64_t Hk = d->n_kv_heads;
  const int M = d->n_layers / d->window;
  const int m = layer / d->window;
  if (!(sm_scale > 0.f)) sm_scale = 1.0f / std::sqrt((float)kHeadDim);
  const uint16_t* scale = static_cast<const uint16_t*>(c->res_scale);
  std::memset(&a, 0, sizeof(a));
  if (c8) {                     // int8 codes: one byte per coefficient
    a.coef_k = reinterpret_cast<const uint16_t*>(static_cast<const uint8_t*>(c->coef_k) + (int64_t)layer * Hk * T16 * RB);
    a.coef_v = reinterpret_cast<const uint16_t*>(static_cast<const uint8_t*>(c->coef_v) + (int64_t)layer * Hk * T16 * RB);
    a.cscale_k = static_cast<const uint16_t*>(c->coef_k_scale) + (int64_t)layer * Hk * (RB / 16) * T;
    a.cscale_v = static_cast<const uint16_t*>(c->coef_v_scale) + (int64_t)layer * Hk * (RB / 16) * T;
  } else {
    a.coef_k = static_cast<const uint16_t*>(c->coef_k) + (int64_t)layer * Hk * T16 * RB;
    a.coef_v = static_cast<const uint16_t*>(c->coef_v) + (int64_t)layer * Hk * T16 * RB;
  }
  a.basis = static_cast<const uint16_t*>(c->basis) + (int64_t)m * Hk * 2 * RB * kHeadDim;
  a.basis_b_stride = (int64_t)M * Hk * 2 * RB * kHeadDim;
  a.off = c->res_off + (int64_t)m * Hk * (T + 1);
  a.idx_k = c->res_idx + ((int64_t)layer * 2 + 0) * Hk * d->res_stride;
  a.idx_v = c->res_idx + ((int64_t)layer * 2 + 1) * Hk * d->res_stride;
  a.val_k = c->res_val + ((int64_t)layer * 2 + 0) * Hk * (d->res_stride / 2);
  a.val_v = c->res_val + ((int64_t)layer * 2 + 1) * Hk * (d->res_stride / 2);
  a.scale_k = scale + ((int64_t)layer * 2 + 0) * Hk * T;
  a.scale_v = scale + ((int64_t)layer * 2 + 1) * Hk * T;
  a.q = static_cast<const uint16_t*>(q);
  a.cu = d->cu_seqlens;
  a.part = static_cast<float*>(workspace);
  a.T = T;
  a.res_stride = d->res_stride;
  a.batch = d->batch;
  a.n_q_heads = d->n_q_heads;
  a.n_kv_heads = d->n_kv_heads;
  a.n_slots = d->n_kv_heads;
  a.q_bf16 = q_type == DWKV_BF16;
  a.qscale = sm_scale * 1.4426950408889634f;
  for (int h = 0; h < d->n_kv_heads; ++h) a.kv_of_slot[h] = h;
  return DWKV_OK;
}

// Split-K pass(es): partial (o, m, l) per (work item, head slot, group member).
// On the token-lane path the probe's reference pass of the current position
// shares the split-K launch (launch_split_tl_probe).
dwkv_status partials_phase(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, const void* q,
                           int32_t q_type, float sm_scale, const dwkv_probe* probe, void* workspace,
                           hipStream_t s, float* scores = nullptr) {
  if (!c || !q) return DWKV_E_NULL;
  const bool c8 = d->coef_format == DWKV_COEF_I8;
  // int8 coefficients: the token-lane kernel for groups of up to 4; a probe of
  // the current position only (the earlier positions run the general kernel)
  if (c8 && (!uses_token_lane(d) || d->n_q_heads / d->n_kv_heads > 4 || probe_positions(probe) > 1))
    return DWKV_E_UNSUPPORTED;
  SplitArgs a;
  dwkv_status st = split_args(d, c, layer, q, q_type, sm_scale, workspace, a);
  if (st != DWKV_OK) return st;
  const WsLayout wl = ws_layout(d, probe);
  const int G = d->n_q_heads / d->n_kv_heads;
  const int RB = d->basis_rank;
  const int split = plan_split(d);
  const int64_t nw = count_work(d, split);
  if (nw > 0x7fffffff) return DWKV_E_UNSUPPORTED;
  if (nw == 0) return DWKV_OK;
  char* ws = static_cast<char*>(workspace);
  a.split = split;
  a.n_work = (int32_t)nw;
  a.wt = work_table(d, split);
  a.scores = scores;
  // the probe's reference pass (identity basis over the dense rows); its
  // first workgroup clears the wide merge's probe counters
  SplitArgs r;
  if (probe) {
    r = a;
    r.scores = nullptr;
    r.coef_k = static_cast<const uint16_t*>(probe->k_ref);
    r.coef_v = static_cast<const uint16_t*>(probe->v_ref);
    r.part = reinterpret_cast<float*>(ws + wl.main_bytes);
    r.n_slots = probe->n_heads;
    for (int i = 0; i < probe->n_heads; ++i) r.kv_of_slot[i] = probe->kv_heads_host[i];
    r.split = plan_split_ref(d, probe->n_heads);
    r.n_work = (int32_t)count_work(d, r.split);
    r.wt = work_table(d, r.split);
    r.zero = reinterpret_cast<uint32_t*>(ws + wl.count_off);
    r.n_zero = d->batch * probe->n_heads * G;
  }
  hipError_t e;
  if (probe && !scores && fused_probe(d, probe)) {
    e = launch_split_tl_probe(RB, G, max_level(d) > 0, c8, TLProbeArgs{a, r}, s);
  } else {
    e = c8 ? (scores ? launch_split_tl_scores_c8(RB, G, max_level(d) > 0, a, (int)nw, s)
                     : launch_split_tl_c8(RB, G, max_level(d) > 0, a, (int)nw, s))
           : uses_token_lane(d)
               ? (scores ? launch_split_tl_scores(RB, G, max_level(d) > 0, a, (int)nw, s)
                         : launch_split_tl(RB, G, max_level(d) > 0, a, (int)nw, s))
               : launch_split(RB, G, max_level(d) > 0, false, a, (int)nw, s);
    if (e == hipSuccess && probe) e = launch_split(kHeadDim, G, false, true, r, r.n_work, s);
  }
  if (e != hipSuccess) return DWKV_E_HIP;
  if (probe) {
    r.zero = nullptr;
    r.n_zero = 0;
    // earlier positions: the query j steps back over the sequences cut j
    // tokens short, on the factorized cache (general kernel, probed heads
    // only) and on the reference, both passes in one launch
    for (int j = 1; j < probe_positions(probe); ++j) {
      const int64_t nwj = count_work(d, r.split, j);
      if (nwj == 0) continue;
      char* pos = ws + wl.main_bytes + wl.ref_bytes + (size_t)(j - 1) * 2 * wl.pos_bytes;
      SplitArgs f = a;
      f.q = static_cast<const uint16_t*>(probe->q_prev) + (int64_t)(j - 1) * d->batch * d->n_q_heads * kHeadDim;
      f.n_slots = probe->n_heads;
      for (int i = 0; i < probe->n_heads; ++i) f.kv_of_slot[i] = probe->kv_heads_host[i];
      f.split = r.split;
      f.n_work = (int32_t)nwj;
      f.wt = work_table(d, r.split, j);
      f.trim = j;
      f.part = reinterpret_cast<float*>(pos);
      SplitArgs fr = r;
      fr.q = f.q;
      fr.n_work = f.n_work;
      fr.wt = f.wt;
      fr.trim = j;
      fr.part = reinterpret_cast<float*>(pos + wl.pos_bytes);
      if (launch_probe_pos(RB, G, max_level(d) > 0, TLProbeArgs{f, fr}, s) != hipSuccess) return DWKV_E_HIP;
    }
  }
  return DWKV_OK;
}

// Merge pass: output rows (and Eq. 3 for probed heads); also writes the zero
// outputs of empty sequences.
dwkv_status merge_phase(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, float* out,
                        const dwkv_probe* probe, void* workspace, hipStream_t s, float* mstats = nullptr) {
  if (!out || !c || !c->basis) return DWKV_E_NULL;
  if (layer < 0 || layer >= d->n_layers) return DWKV_E_DIMS;
  if (!aligned16(out) || !aligned16(c->basis)) return DWKV_E_ALIGN;
  const WsLayout wl = ws_layout(d, probe);
  char* ws = static_cast<char*>(workspace);
  const bool tl = uses_token_lane(d);
  if (tl) {
    SplitArgs a;
    std::memset(&a, 0, sizeof(a));
    const int64_t Hk = d->n_kv_heads, M = d->n_layers / d->window, m = layer / d->window;
    a.basis = static_cast<const uint16_t*>(c->basis) + m * Hk * 2 * d->basis_rank * kHeadDim;
    a.basis_b_stride = M * Hk * 2 * d->basis_rank * kHeadDim;
    a.cu = d->cu_seqlens;
    a.part = reinterpret_cast<float*>(ws);
    a.out = out;
    a.batch = d->batch;
    a.n_q_heads = d->n_q_heads;
    a.n_kv_heads = d->n_kv_heads;
    a.n_slots = d->n_kv_heads;
    a.split = plan_split(d);
    a.n_work = (int32_t)count_work(d, a.split);
    for (int h = 0; h < d->n_kv_heads; ++h) a.kv_of_slot[h] = h;
    a.wt = work_table(d, a.split);
    a.mstats = mstats;
    WMergeArgs wm;
    std::memset(&wm, 0, sizeof(wm));
    wm.s = a;
    wm.max_ns = max_items(d, a.split);
    for (int h = 0; h < DWKV_MAX_PROBE_HEADS; ++h) wm.p.slot_of_kv[h] = -1;
    if (probe) {                       // Eq. 3 in the same launch
      WideProbe& P = wm.p;
      P.part_ref = reinterpret_cast<const float*>(ws + wl.main_bytes);
      P.err = probe->err;
      P.out_ref = probe->out_ref;
      P.acc = probe_positions(probe) > 1 ? reinterpret_cast<float*>(ws + wl.acc_off) : nullptr;
      P.oref = reinterpret_cast<float*>(ws + wl.chunk_off);
      P.count = reinterpret_cast<uint32_t*>(ws + wl.count_off);
      P.n_probe = probe->n_heads;
      P.eps = probe->eps;
      P.ref_split = plan_split_ref(d, probe->n_heads);
      P.ref_wt = work_table(d, P.ref_split);
      for (int i = 0; i < probe->n_heads; ++i) {
        P.slot_of_kv[probe->kv_heads_host[i]] = i;
        P.kv_of_slot[i] = probe->kv_heads_host[i];
      }
    }
    const hipError_t e = launch_merge_tl(d->basis_rank, d->n_q_heads / d->n_kv_heads, wm, s);
    if (e != hipSuccess || probe_positions(probe) == 1) return hip_status(e);
  }
  MergeArgs mg;
  std::memset(&mg, 0, sizeof(mg));
  mg.part = reinterpret_cast<const float*>(ws);
  mg.part_ref = probe ? reinterpret_cast<const float*>(ws + wl.main_bytes) : nullptr;
  mg.out = out;
  mg.err = probe ? probe->err : nullptr;
  mg.out_ref = probe ? probe->out_ref : nullptr;
  mg.cu = d->cu_seqlens;
  mg.batch = d->batch;
  mg.n_q_heads = d->n_q_heads;
  mg.n_kv_heads = d->n_kv_heads;
  mg.split = plan_split(d);
  mg.wt = work_table(d, mg.split);
  mg.tl = uses_token_lane(d);
  mg.n_work = (int32_t)count_work(d, mg.split);
  mg.rb = d->basis_rank;
  {
    const int64_t Hk = d->n_kv_heads, M = d->n_layers / d->window, m = layer / d->window;
    mg.basis = static_cast<const uint16_t*>(c->basis) + m * Hk * 2 * d->basis_rank * kHeadDim;
    mg.basis_b_stride = M * Hk * 2 * d->basis_rank * kHeadDim;
  }
  mg.n_probe = probe ? probe->n_heads : 0;
  mg.eps = probe ? probe->eps : 0.f;
  mg.ref_split = probe ? plan_split_ref(d, probe->n_heads) : mg.split;
  mg.ref_wt = work_table(d, mg.ref_split);
  for (int h = 0; h < DWKV_MAX_PROBE_HEADS; ++h) mg.probe_slot_of_kv[h] = -1;
  if (probe)
    for (int i = 0; i < probe->n_heads; ++i) {
      mg.probe_slot_of_kv[probe->kv_heads_host[i]] = i;
    }
  const int np = probe_positions(probe);
  if (np > 1) mg.acc = reinterpret_cast<float*>(ws + wl.acc_off);
  if (!tl) {                           // outputs and the current position's Eq. 3
    const hipError_t e = launch_merge(mg, s);
    if (e != hipSuccess || np == 1) return hip_status(e);
  }
  // the earlier positions' sums, then err
  mg.part_pos = reinterpret_cast<const float*>(ws + wl.main_bytes + wl.ref_bytes);
  mg.pos_stride = (int64_t)(wl.pos_bytes / sizeof(float));
  mg.n_pos = np;
  return hip_status(launch_merge(mg, s));
}

}  // namespace

extern "C" {

dwkv_status dwkv_decode(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, const void* q,
                        int32_t q_type, float sm_scale, float* out, const dwkv_probe* probe,
                        void* workspace, size_t ws_bytes, void* stream) {
  dwkv_status st = check_decode_common(d, probe, workspace, ws_bytes);
  if (st != DWKV_OK) return st;
  if (!out) return DWKV_E_NULL;
  if (!aligned16(out)) return DWKV_E_ALIGN;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if ((st = partials_phase(d, c, layer, q, q_type, sm_scale, probe, workspace, s)) != DWKV_OK) return st;
  return merge_phase(d, c, layer, out, probe, workspace, s);
}

dwkv_status dwkv_decode_partials(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, const void* q,
                                 int32_t q_type, float sm_scale, const dwkv_probe* probe, void* workspace,
                                 size_t ws_bytes, void* stream) {
  dwkv_status st = check_decode_common(d, probe, workspace, ws_bytes);
  if (st != DWKV_OK) return st;
  return partials_phase(d, c, layer, q, q_type, sm_scale, probe, workspace,
                        reinterpret_cast<hipStream_t>(stream));
}

dwkv_status dwkv_decode_merge(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, float* out,
                              const dwkv_probe* probe, void* workspace, size_t ws_bytes, void* stream) {
  dwkv_status st = check_decode_common(d, probe, workspace, ws_bytes);
  if (st != DWKV_OK) return st;
  return merge_phase(d, c, layer, out, probe, workspace, reinterpret_cast<hipStream_t>(stream));
}

}  // extern "C"

// The allocation-free decode keeps its split partials in this file-scope
// array: one copy per GPU the library runs on, held until the process ends.
// Host code never uses the array's name as an address (on the host it is a
// stand-in, not device memory): each device's address is looked up once with
// hipGetSymbolAddress, with that device current, and kept below.
namespace {
constexpr size_t kStaticScratchBytes = (size_t)DWKV_STATIC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
void* g_scratch_ptr[kMaxDevices] = {};
std::mutex g_scratch_mu;
}  // namespace

__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
// Address of the current device's copy of `scratch`, looked up on the first
// call on that device; null when the lookup fails.
void* static_scratch_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}
}  // namespace

extern "C" {

size_t dwkv_static_scratch_bytes(void) { return kStaticScratchBytes; }

dwkv_status dwkv_decode_noalloc(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, const void* q,
                                int32_t q_type, float sm_scale, float* out, const dwkv_probe* probe,
                                void* stream) {
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  if ((st = check_probe(d, probe)) != DWKV_OK) return st;
  if (!out) return DWKV_E_NULL;
  if (!aligned16(out)) return DWKV_E_ALIGN;
  if (ws_layout(d, probe).total > kStaticScratchBytes) return DWKV_E_SCRATCH;
  void* ws = static_scratch_ptr();
  if (!ws) return DWKV_E_HIP;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if ((st = partials_phase(d, c, layer, q, q_type, sm_scale, probe, ws, s)) != DWKV_OK) return st;
  return merge_phase(d, c, layer, out, probe, ws, s);
}

size_t dwkv_route_workspace_bytes(const dwkv_dims* d) {
  if (check_dims(d) != DWKV_OK) return 0;
  const int64_t nblk = (d->total_tokens + kRouteTokensPerBlock - 1) / kRouteTokensPerBlock;
  const int64_t n_mh = (int64_t)(d->n_layers / d->window) * d->n_kv_heads;
  const size_t b = align_up((size_t)(nblk > 0 ? nblk : 1) * n_mh * sizeof(uint32_t), 256);
  return 2 * b;
}

dwkv_status dwkv_route_range(const dwkv_dims* d, const float* phi, const float* u, const float* theta,
                             int64_t t0, int64_t t1, uint8_t* rank_code, uint32_t* res_off,
                             void* workspace, size_t ws_bytes, void* stream) {
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  if (t0 < 0 || t1 < t0 || t1 > d->total_tokens) return DWKV_E_DIMS;
  if (!u || !res_off || !workspace || !rank_code) return DWKV_E_NULL;
  if (t1 > t0 && !phi) return DWKV_E_NULL;
  if (d->n_levels > 1 && !theta) return DWKV_E_NULL;
  const size_t need = dwkv_route_workspace_bytes(d);
  if (ws_bytes < need) return DWKV_E_WORKSPACE;
  const int64_t n = t1 - t0;
  if (n == 0 && t0 > 0) return DWKV_OK;           // nothing to route, no offset to reset
  const int64_t nblk = (n + kRouteTokensPerBlock - 1) / kRouteTokensPerBlock;
  const int n_mh = (d->n_layers / d->window) * d->n_kv_heads;
  if (nblk > 0x7fffffff) return DWKV_E_UNSUPPORTED;
  RouteArgs a;
  std::memset(&a, 0, sizeof(a));
  a.phi = phi;
  a.u = u;
  a.theta = theta;
  a.code = rank_code;
  a.off = res_off;
  a.bsum = static_cast<uint32_t*>(workspace);
  a.bpre = reinterpret_cast<uint32_t*>(static_cast<char*>(workspace) + need / 2);
  a.T = d->total_tokens;
  a.t0 = t0;
  a.n = n;
  a.n_kv_heads = d->n_kv_heads;
  a.n_levels = d->n_levels;
  a.nblk = (int)nblk;
  for (int i = 0; i < DWKV_MAX_LEVELS; ++i) a.levels[i] = i < d->n_levels ? d->levels[i] : 0;
  return hip_status(launch_route(a, n_mh, reinterpret_cast<hipStream_t>(stream)));
}

dwkv_status dwkv_route(const dwkv_dims* d, const float* phi, const float* u, const float* theta,
                       uint8_t* rank_code, uint32_t* res_off, void* workspace, size_t ws_bytes,
                       void* stream) {
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  return dwkv_route_range(d, phi, u, theta, 0, d->total_tokens, rank_code, res_off, workspace,
                          ws_bytes, stream);
}

size_t dwkv_route_budget_workspace_bytes(const dwkv_dims* d) {
  if (check_dims(d) != DWKV_OK) return 0;
  const size_t n = (size_t)(d->n_layers / d->window) * d->n_kv_heads * (size_t)d->total_tokens * 8;
  return n > 0 ? align_up(n, 256) : 256;
}

dwkv_status dwkv_route_budget(const dwkv_dims* d, const float* phi, const float* u, const int64_t* entries,
                              int64_t t0, int64_t t1, uint8_t* rank_code, uint32_t* res_off, void* workspace,
                              size_t ws_bytes, void* stream) {
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  if (d->n_levels != 2) return DWKV_E_UNSUPPORTED;
  if (t0 < 0 || t1 < t0 || t1 > d->total_tokens) return DWKV_E_DIMS;
  if (!u || !entries || !rank_code || !res_off || !workspace) return DWKV_E_NULL;
  if (t1 > t0 && !phi) return DWKV_E_NULL;
  if (!aligned16(phi) || !aligned16(u) || !aligned16(workspace) || (reinterpret_cast<uintptr_t>(entries) & 7u))
    return DWKV_E_ALIGN;
  if (ws_bytes < dwkv_route_budget_workspace_bytes(d)) return DWKV_E_WORKSPACE;
  if (t1 == t0 && t0 > 0) return DWKV_OK;
  RouteArgs a;
  std::memset(&a, 0, sizeof(a));
  a.phi = phi;
  a.u = u;
  a.code = rank_code;
  a.off = res_off;
  a.entries = entries;
  a.keys = static_cast<unsigned long long*>(workspace);
  a.T = d->total_tokens;
  a.t0 = t0;
  a.n = t1 - t0;
  a.n_kv_heads = d->n_kv_heads;
  a.n_levels = d->n_levels;
  for (int i = 0; i < DWKV_MAX_LEVELS; ++i) a.levels[i] = i < d->n_levels ? d->levels[i] : 0;
  const int n_mh = (d->n_layers / d->window) * d->n_kv_heads;
  return hip_status(launch_route_budget(a, n_mh, reinterpret_cast<hipStream_t>(stream)));
}

}  // extern "C"

namespace {

// Arguments of the append/compress kernel for layer `layer`, every field but
// the token range (t0, n, gate_ld, gate_k0); checks the cache and inputs.
dwkv_status compress_args(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, const void* x_k,
                          const void* x_v, const float* gate, CompressArgs& a) {
  const bool c8 = d->coef_format == DWKV_COEF_I8;
  if (!c || !c->basis || !c->coef_k || !c->coef_v || !c->rank_code || !c->res_off || !c->res_idx ||
      !c->res_val || !c->res_scale)
    return DWKV_E_NULL;
  if (c8 && (!c->coef_k_scale || !c->coef_v_scale)) return DWKV_E_NULL;
  if (c8 && ((reinterpret_cast<uintptr_t>(c->coef_k_scale) | reinterpret_cast<uintptr_t>(c->coef_v_scale)) & 1u))
    return DWKV_E_ALIGN;
  if (layer < 0 || layer >= d->n_layers) return DWKV_E_DIMS;
  if (!x_k || !x_v) return DWKV_E_NULL;
  const void* const ptrs[] = {c->basis, c->coef_k, c->coef_v, x_k, x_v};
  for (const void* p : ptrs)
    if (!aligned16(p)) return DWKV_E_ALIGN;
  if ((reinterpret_cast<uintptr_t>(c->res_idx) & 1u) || (reinterpret_cast<uintptr_t>(c->res_scale) & 1u) ||
      (reinterpret_cast<uintptr_t>(gate) & 3u))
    return DWKV_E_ALIGN;
  const int64_t T = d->total_tokens, Hk = d->n_kv_heads, rb = d->basis_rank;
  const int64_t T16 = (T + 15) / 16 * 16;
  const int M = d->n_layers / d->window, m = layer / d->window;
  std::memset(&a, 0, sizeof(a));
  a.basis = static_cast<const uint16_t*>(c->basis) + (int64_t)m * Hk * 2 * rb * kHeadDim;
  a.basis_b_stride = (int64_t)M * Hk * 2 * rb * kHeadDim;
  a.code = c->rank_code + (int64_t)m * Hk * T;
  a.off = c->res_off + (int64_t)m * Hk * (T + 1);
  a.cu = d->cu_seqlens;
  a.xk = static_cast<const uint16_t*>(x_k);
  a.xv = static_cast<const uint16_t*>(x_v);
  a.gate = gate;
  // the cache's arrays are written in place (the pointers are const only for decode)
  if (c8) {                     // int8 codes: one byte per coefficient; fp16 block scales
    a.coef_k = reinterpret_cast<uint16_t*>(const_cast<uint8_t*>(static_cast<const uint8_t*>(c->coef_k)) +
                                           (int64_t)layer * Hk * T16 * rb);
    a.coef_v = reinterpret_cast<uint16_t*>(const_cast<uint8_t*>(static_cast<const uint8_t*>(c->coef_v)) +
                                           (int64_t)layer * Hk * T16 * rb);
    a.cscale_k = const_cast<uint16_t*>(static_cast<const uint16_t*>(c->coef_k_scale)) + (int64_t)layer * Hk * (rb / 16) * T;
    a.cscale_v = const_cast<uint16_t*>(static_cast<const uint16_t*>(c->coef_v_scale)) + (int64_t)layer * Hk * (rb / 16) * T;
    a.c8 = 1;
  } else {
    a.coef_k = const_cast<uint16_t*>(static_cast<const uint16_t*>(c->coef_k)) + (int64_t)layer * Hk * T16 * rb;
    a.coef_v = const_cast<uint16_t*>(static_cast<const uint16_t*>(c->coef_v)) + (int64_t)layer * Hk * T16 * rb;
  }
  a.res_idx = const_cast<uint8_t*>(c->res_idx) + (int64_t)layer * 2 * Hk * d->res_stride;
  a.res_val = const_cast<uint8_t*>(c->res_val) + (int64_t)layer * 2 * Hk * (d->res_stride / 2);
  a.res_scale = const_cast<uint16_t*>(static_cast<const uint16_t*>(c->res_scale)) + (int64_t)layer * 2 * Hk * T;
  a.T = T;
  a.T16 = T16;
  a.res_stride = d->res_stride;
  a.batch = d->batch;
  a.n_kv_heads = d->n_kv_heads;
  a.rb = d->basis_rank;
  a.n_levels = d->n_levels;
  for (int i = 0; i < DWKV_MAX_LEVELS; ++i) a.levels[i] = i < d->n_levels ? d->levels[i] : 0;
  return DWKV_OK;
}

// The decode that appends runs in one split launch when the token-lane kernel
// serves the dims with fp16 coefficients and the batch's work split travels
// in the kernel arguments; otherwise it is the append/compress kernel, once
// per sequence, then the plain decode.
bool append_fused(const dwkv_dims* d) {
  return uses_token_lane(d) && d->coef_format != DWKV_COEF_I8 && d->batch <= kKernargSeqs;
}

int64_t nonempty_seqs(const dwkv_dims* d) {
  int64_t n = 0;
  for (int b = 0; b < d->batch; ++b) n += d->cu_seqlens_host[b + 1] > d->cu_seqlens_host[b];
  return n;
}

// Work items of the fused decode: each sequence's tokens but the last in
// chunks of `split`, then its append item.
int64_t count_work_append(const dwkv_dims* d, int split) {
  return count_work(d, split, 1) + nonempty_seqs(d);
}

// Chunk size of the fused decode: the token-lane kernel's one workgroup per
// CU, with room for the append items beside the split items when they are
// few (at most 32; more of them run once workgroups finish, as a separate
// launch would); chunks in multiples of 64 tokens.
int plan_split_append(const dwkv_dims* d) {
  if (d->split_tokens > 0) return d->split_tokens;
  const int64_t Hk = d->n_kv_heads, napp = nonempty_seqs(d) * Hk, target = kTargetWorkgroups / 2;
  const int64_t budget = napp <= 32 ? target - napp : target;
  const int64_t work = std::max<int64_t>(d->total_tokens - nonempty_seqs(d), 1) * Hk;
  int64_t c = (work + budget - 1) / budget;
  c = std::max<int64_t>((c + 63) / 64 * 64, 64);
  while (c < kSplitMax && count_work(d, (int)c, 1) * Hk > budget) c += 64;
  return (int)std::min<int64_t>(c, kSplitMax);
}

WorkTable work_table_append(const dwkv_dims* d, int split) {
  WorkTable t = work_table(d, split, 1);
  int acc = 0;                            // plus one append item per non-empty sequence
  for (int b = 0; b < t.n_seq; ++b) {
    const int64_t len = d->cu_seqlens_host[b + 1] - d->cu_seqlens_host[b];
    acc += len > 0 ? (int32_t)((len - 1 + split - 1) / split) + 1 : 0;
    t.work[b + 1] = acc;
  }
  return t;
}

size_t append_ws_bytes(const dwkv_dims* d) {
  if (!append_fused(d)) return ws_layout(d, nullptr).total;
  const int g = d->n_q_heads / d->n_kv_heads;
  const int64_t nw = count_work_append(d, plan_split_append(d));
  return std::max<size_t>(align_up((size_t)nw * d->n_kv_heads * g * kPartStrideTL * sizeof(float), 256), 256);
}

}  // namespace

extern "C" {

dwkv_status dwkv_compress(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, const void* x_k,
                          const void* x_v, const float* gate, int64_t t0, int64_t t1, void* stream) {
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  if (t0 < 0 || t1 < t0 || t1 > d->total_tokens) return DWKV_E_DIMS;
  CompressArgs a;
  if ((st = compress_args(d, c, layer, x_k, x_v, gate, a)) != DWKV_OK) {
    // an empty range needs no inputs
    if (t1 == t0 && st == DWKV_E_NULL && c && c->basis && c->coef_k && c->coef_v && c->rank_code &&
        c->res_off && c->res_idx && c->res_val && c->res_scale && layer >= 0 && layer < d->n_layers)
      return DWKV_OK;
    return st;
  }
  if (t1 == t0) return DWKV_OK;
  a.t0 = t0;
  a.n = t1 - t0;
  a.gate_ld = a.n;
  return hip_status(launch_compress(a, reinterpret_cast<hipStream_t>(stream)));
}

size_t dwkv_decode_append_workspace_bytes(const dwkv_dims* dims) {
  if (check_dims(dims) != DWKV_OK) return 0;
  return append_ws_bytes(dims);
}

int32_t dwkv_decode_append_launches(const dwkv_dims* dims) {
  if (check_dims(dims) != DWKV_OK) return -1;
  return append_fused(dims) ? 2 : (int32_t)nonempty_seqs(dims) + 2;
}

dwkv_status dwkv_decode_append(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, const void* q,
                               int32_t q_type, float sm_scale, float* out, const void* x_k, const void* x_v,
                               const float* gate, void* workspace, size_t ws_bytes, void* stream) {
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  if (!workspace || !q || !out) return DWKV_E_NULL;
  if (!aligned16(workspace) || !aligned16(q) || !aligned16(out)) return DWKV_E_ALIGN;
  if (q_type != DWKV_F16 && q_type != DWKV_BF16) return DWKV_E_DIMS;
  if (ws_bytes < append_ws_bytes(d)) return DWKV_E_WORKSPACE;
  CompressArgs ca;
  if ((st = compress_args(d, c, layer, x_k, x_v, gate, ca)) != DWKV_OK) return st;
  ca.gate_ld = d->batch;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (!append_fused(d)) {
    // the append/compress kernel on each sequence's last token, then the decode
    for (int b = 0; b < d->batch; ++b) {
      const int64_t t1 = d->cu_seqlens_host[b + 1];
      if (t1 == d->cu_seqlens_host[b]) continue;
      CompressArgs one = ca;
      one.t0 = t1 - 1;
      one.n = 1;
      one.xk = ca.xk + (int64_t)b * d->n_kv_heads * kHeadDim;
      one.xv = ca.xv + (int64_t)b * d->n_kv_heads * kHeadDim;
      one.gate_k0 = b;
      if (launch_compress(one, s) != hipSuccess) return DWKV_E_HIP;
    }
    if ((st = partials_phase(d, c, layer, q, q_type, sm_scale, nullptr, workspace, s)) != DWKV_OK) return st;
    return merge_phase(d, c, layer, out, nullptr, workspace, s);
  }
  // one split launch: the split items over every sequence but its last token,
  // and per sequence and KV head the append item; then the wide merge
  const int split = plan_split_append(d);
  const int64_t nw = count_work_append(d, split);
  if (nw == 0) return merge_phase(d, c, layer, out, nullptr, workspace, s);   // zero outputs only
  TLAppendArgs A;
  std::memset(&A, 0, sizeof(A));
  A.c = ca;
  const WorkTable wt = work_table_append(d, split);
  if ((st = split_args(d, c, layer, q, q_type, sm_scale, workspace, A.s)) != DWKV_OK) return st;
  A.s.split = split;
  A.s.n_work = (int32_t)nw;
  A.s.wt = wt;
  A.s.trim = 1;
  const int G = d->n_q_heads / d->n_kv_heads;
  if (launch_split_tl_append(d->basis_rank, G, max_level(d) > 0, A, (int)nw, s) != hipSuccess) return DWKV_E_HIP;
  WMergeArgs m;
  std::memset(&m, 0, sizeof(m));
  m.s = A.s;
  m.max_ns = max_items(d, split, 1, 1);
  m.s.out = out;
  m.s.mstats = nullptr;
  for (int h = 0; h < DWKV_MAX_PROBE_HEADS; ++h) m.p.slot_of_kv[h] = -1;
  return hip_status(launch_merge_tl(d->basis_rank, G, m, s));
}

dwkv_status dwkv_residual_map(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, int32_t z,
                              int32_t kv_head, int64_t t0, int64_t t1, float* dense, void* stream) {
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  if (!c || !c->res_off || !c->res_idx || !c->res_val || !c->res_scale) return DWKV_E_NULL;
  if (!dense && t1 > t0) return DWKV_E_NULL;          // an empty range writes nothing
  if (layer < 0 || layer >= d->n_layers || z < 0 || z > 1 || kv_head < 0 || kv_head >= d->n_kv_heads)
    return DWKV_E_DIMS;
  if (t0 < 0 || t1 < t0 || t1 > d->total_tokens) return DWKV_E_DIMS;
  const int64_t T = d->total_tokens, Hk = d->n_kv_heads;
  const int m = layer / d->window;
  const int64_t slab = ((int64_t)layer * 2 + z) * Hk + kv_head;
  return hip_status(launch_residual_map(
      c->res_off + ((int64_t)m * Hk + kv_head) * (T + 1), c->res_idx + slab * d->res_stride,
      c->res_val + slab * (d->res_stride / 2), static_cast<const uint16_t*>(c->res_scale) + slab * T,
      t0, t1, d->res_stride, dense, reinterpret_cast<hipStream_t>(stream)));
}

size_t dwkv_sketch_workspace_bytes(const dwkv_dims* d, int64_t n_tokens) {
  if (check_dims(d) != DWKV_OK || n_tokens < 1) return 0;
  const size_t row = (size_t)d->n_kv_heads * 2 * d->basis_rank * kHeadDim * sizeof(double);
  return align_up((size_t)sketch_chunks((int64_t)d->window * n_tokens) * row, 256) + align_up(row, 256);
}

dwkv_status dwkv_sketch_basis(const dwkv_dims* d, const dwkv_cache* c, int32_t window, int32_t seq,
                              const void* x, const void* omega, int64_t n_tokens, void* workspace,
                              size_t ws_bytes, void* stream) {
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  if (!c || !c->basis || !x || !omega || !workspace) return DWKV_E_NULL;
  const int M = d->n_layers / d->window;
  if (window < 0 || window >= M || seq < 0 || seq >= d->batch || n_tokens < 1) return DWKV_E_DIMS;
  if ((double)d->window * (double)n_tokens > 2147483647.0) return DWKV_E_UNSUPPORTED;
  if (!aligned16(c->basis) || !aligned16(x) || !aligned16(omega) || !aligned16(workspace)) return DWKV_E_ALIGN;
  if (ws_bytes < dwkv_sketch_workspace_bytes(d, n_tokens)) return DWKV_E_WORKSPACE;
  const int64_t rb = d->basis_rank, Hk = d->n_kv_heads;
  SketchArgs a;
  std::memset(&a, 0, sizeof(a));
  a.x = static_cast<const uint16_t*>(x);
  a.omega = static_cast<const uint16_t*>(omega);
  a.n_chunks = sketch_chunks((int64_t)d->window * n_tokens);
  a.part = static_cast<double*>(workspace);
  a.q = reinterpret_cast<double*>(static_cast<char*>(workspace) +
                                  align_up((size_t)a.n_chunks * Hk * 2 * rb * kHeadDim * sizeof(double), 256));
  // the cache's bases are written in place (the pointer is const only for decode)
  a.basis = const_cast<uint16_t*>(static_cast<const uint16_t*>(c->basis)) +
            (((int64_t)seq * M + window) * Hk) * 2 * rb * kHeadDim;
  a.n_tokens = n_tokens;
  a.w = d->window;
  a.n_kv_heads = d->n_kv_heads;
  a.rb = d->basis_rank;
  return hip_status(launch_sketch(a, reinterpret_cast<hipStream_t>(stream)));
}

dwkv_status dwkv_materialize(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, void* k_out,
                             void* v_out, void* stream) {
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  if (d->coef_format != DWKV_COEF_F16) return DWKV_E_UNSUPPORTED;
  if (!c || !c->basis || !c->coef_k || !c->coef_v || !c->res_off || !c->res_idx || !c->res_val ||
      !c->res_scale || !k_out || !v_out)
    return DWKV_E_NULL;
  if (layer < 0 || layer >= d->n_layers) return DWKV_E_DIMS;
  const void* const ptrs[] = {c->basis, c->coef_k, c->coef_v, k_out, v_out};
  for (const void* p : ptrs)
    if (!aligned16(p)) return DWKV_E_ALIGN;
  if (reinterpret_cast<uintptr_t>(c->res_scale) & 1u) return DWKV_E_ALIGN;
  const int64_t T = d->total_tokens, Hk = d->n_kv_heads, rb = d->basis_rank;
  const int M = d->n_layers / d->window, m = layer / d->window;
  MatArgs a;
  std::memset(&a, 0, sizeof(a));
  a.basis = static_cast<const uint16_t*>(c->basis) + (int64_t)m * Hk * 2 * rb * kHeadDim;
  a.basis_b_stride = (int64_t)M * Hk * 2 * rb * kHeadDim;
  a.T = T;
  a.T16 = (T + 15) / 16 * 16;
  a.coef_k = static_cast<const uint16_t*>(c->coef_k) + (int64_t)layer * Hk * a.T16 * rb;
  a.coef_v = static_cast<const uint16_t*>(c->coef_v) + (int64_t)layer * Hk * a.T16 * rb;
  a.off = c->res_off + (int64_t)m * Hk * (T + 1);
  a.idx = c->res_idx + (int64_t)layer * 2 * Hk * d->res_stride;
  a.val = c->res_val + (int64_t)layer * 2 * Hk * (d->res_stride / 2);
  a.scale = static_cast<const uint16_t*>(c->res_scale) + (int64_t)layer * 2 * Hk * T;
  a.cu = d->cu_seqlens;
  a.k_out = static_cast<uint16_t*>(k_out);
  a.v_out = static_cast<uint16_t*>(v_out);
  a.res_stride = d->res_stride;
  a.batch = d->batch;
  a.n_kv_heads = d->n_kv_heads;
  a.rb = d->basis_rank;
  return hip_status(launch_materialize(a, reinterpret_cast<hipStream_t>(stream)));
}

int32_t dwkv_hbm_read_blocks(void) { return kStreamBlocks; }

dwkv_status dwkv_hbm_read(const void* buf, size_t bytes, uint32_t* sink, int32_t sink_words, void* stream) {
  if (!sink || (bytes > 0 && !buf)) return DWKV_E_NULL;
  if (bytes % 16 != 0) return DWKV_E_DIMS;
  if (sink_words < kStreamBlocks) return DWKV_E_WORKSPACE;
  if (!aligned16(buf) || (reinterpret_cast<uintptr_t>(sink) & 3u)) return DWKV_E_ALIGN;
  return hip_status(launch_stream_read(buf, (uint64_t)(bytes / 16), sink, reinterpret_cast<hipStream_t>(stream)));
}

size_t dwkv_dense_workspace_bytes(const dwkv_dims* d) {
  if (check_dims(d) != DWKV_OK) return 0;
  const int split = plan_split_general(d);
  const int64_t nw = count_work(d, split);
  const size_t n = align_up((size_t)nw * d->n_kv_heads * (d->n_q_heads / d->n_kv_heads) * kPartStride *
                                sizeof(float), 256);
  return n > 0 ? n : 256;
}

dwkv_status dwkv_dense_decode(const dwkv_dims* d, const void* k, const void* v, const void* q,
                              int32_t q_type, float sm_scale, float* out, void* workspace,
                              size_t ws_bytes, void* stream) {
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  if (!k || !v || !q || !out || !workspace) return DWKV_E_NULL;
  if (q_type != DWKV_F16 && q_type != DWKV_BF16) return DWKV_E_DIMS;
  const void* const ptrs[] = {k, v, q, out, workspace};
  for (const void* p : ptrs)
    if (!aligned16(p)) return DWKV_E_ALIGN;
  if (ws_bytes < dwkv_dense_workspace_bytes(d)) return DWKV_E_WORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int split = plan_split_general(d);
  const int64_t nw = count_work(d, split);
  if (nw > 0x7fffffff) return DWKV_E_UNSUPPORTED;
  if (!(sm_scale > 0.f)) sm_scale = 1.0f / std::sqrt((float)kHeadDim);
  if (nw > 0) {
    SplitArgs a;
    std::memset(&a, 0, sizeof(a));
    a.coef_k = static_cast<const uint16_t*>(k);
    a.coef_v = static_cast<const uint16_t*>(v);
    a.q = static_cast<const uint16_t*>(q);
    a.cu = d->cu_seqlens;
    a.part = static_cast<float*>(workspace);
    a.T = d->total_tokens;
    a.batch = d->batch;
    a.n_q_heads = d->n_q_heads;
    a.n_kv_heads = d->n_kv_heads;
    a.n_slots = d->n_kv_heads;
    a.split = split;
    a.n_work = (int32_t)nw;
    a.q_bf16 = q_type == DWKV_BF16;
    a.qscale = sm_scale * 1.4426950408889634f;
    for (int h = 0; h < d->n_kv_heads; ++h) a.kv_of_slot[h] = h;
    a.wt = work_table(d, split);
    if (launch_split(kHeadDim, d->n_q_heads / d->n_kv_heads, false, true, a, (int)nw, s) != hipSuccess)
      return DWKV_E_HIP;
  }
  MergeArgs mg;
  std::memset(&mg, 0, sizeof(mg));
  mg.part = static_cast<const float*>(workspace);
  mg.out = out;
  mg.cu = d->cu_seqlens;
  mg.batch = d->batch;
  mg.n_q_heads = d->n_q_heads;
  mg.n_kv_heads = d->n_kv_heads;
  mg.split = split;
  mg.wt = work_table(d, split);
  mg.tl = 0;
  mg.n_work = (int32_t)nw;
  mg.rb = kHeadDim;
  for (int h = 0; h < DWKV_MAX_PROBE_HEADS; ++h) mg.probe_slot_of_kv[h] = -1;
  return hip_status(launch_merge(mg, s));
}

dwkv_status dwkv_probe_feature(const dwkv_dims* d, int32_t layer, int32_t n_heads, const int32_t* kv_heads_host,
                               const float* err, int32_t fresh, float* phi, void* stream) {
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  if (layer < 0 || layer >= d->n_layers) return DWKV_E_DIMS;
  if (n_heads < 1 || n_heads > d->n_kv_heads || n_heads > DWKV_MAX_PROBE_HEADS) return DWKV_E_DIMS;
  if (!kv_heads_host || !err || !phi) return DWKV_E_NULL;
  if (!aligned16(phi) || (reinterpret_cast<uintptr_t>(err) & 3u)) return DWKV_E_ALIGN;
  ProbeFeatArgs a;
  std::memset(&a, 0, sizeof(a));
  bool seen[DWKV_MAX_PROBE_HEADS] = {};
  for (int i = 0; i < n_heads; ++i) {
    const int h = kv_heads_host[i];
    if (h < 0 || h >= d->n_kv_heads || seen[h]) return DWKV_E_DIMS;
    seen[h] = true;
    a.kv_heads[i] = h;
  }
  a.err = err;
  a.phi = phi + (int64_t)(layer / d->window) * d->n_kv_heads * d->total_tokens * 4;
  a.cu = d->cu_seqlens;
  a.T = d->total_tokens;
  a.batch = d->batch;
  a.n_heads = n_heads;
  a.G = d->n_q_heads / d->n_kv_heads;
  a.fresh = fresh ? 1 : 0;
  return hip_status(launch_probe_feature(a, reinterpret_cast<hipStream_t>(stream)));
}

size_t dwkv_features_workspace_bytes(const dwkv_dims* d) {
  if (check_dims(d) != DWKV_OK || !uses_token_lane(d)) return 0;
  const size_t sc = align_up((size_t)d->n_q_heads * (size_t)d->total_tokens * sizeof(float), 256);
  const size_t ms = align_up((size_t)d->batch * d->n_q_heads * 2 * sizeof(float), 256);
  return ws_layout(d, nullptr).total + sc + ms;
}

dwkv_status dwkv_decode_features(const dwkv_dims* d, const dwkv_cache* c, int32_t layer, const void* q,
                                 int32_t q_type, float sm_scale, float* out, float* phi, void* workspace,
                                 size_t ws_bytes, void* stream) {
  dwkv_status st = check_decode_common(d, nullptr, workspace, ws_bytes);
  if (st != DWKV_OK) return st;
  if (!uses_token_lane(d)) return DWKV_E_UNSUPPORTED;
  if (!out || !phi) return DWKV_E_NULL;
  if (!aligned16(out) || !aligned16(phi)) return DWKV_E_ALIGN;
  if (ws_bytes < dwkv_features_workspace_bytes(d)) return DWKV_E_WORKSPACE;
  if (layer < 0 || layer >= d->n_layers) return DWKV_E_DIMS;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  float* scores = reinterpret_cast<float*>(ws + ws_layout(d, nullptr).total);
  float* mstats = reinterpret_cast<float*>(
      ws + ws_layout(d, nullptr).total + align_up((size_t)d->n_q_heads * (size_t)d->total_tokens * sizeof(float), 256));
  if ((st = partials_phase(d, c, layer, q, q_type, sm_scale, nullptr, workspace, s, scores)) != DWKV_OK) return st;
  if ((st = merge_phase(d, c, layer, out, nullptr, workspace, s, mstats)) != DWKV_OK) return st;
  FeatArgs f;
  std::memset(&f, 0, sizeof(f));
  f.mstats = mstats;
  f.scores = scores;
  f.phi = phi + (int64_t)(layer / d->window) * d->n_kv_heads * d->total_tokens * 4;
  f.cu = d->cu_seqlens;
  f.T = d->total_tokens;
  f.batch = d->batch;
  f.n_kv_heads = d->n_kv_heads;
  f.n_q_heads = d->n_q_heads;
  return hip_status(launch_features(d->n_q_heads / d->n_kv_heads, f, s));
}

dwkv_status dwkv_controller_update(const dwkv_controller* ctl, int32_t n_windows, int32_t n_thresholds,
                                   const float* err_host, float* theta_host, int32_t* below_host) {
  if (!ctl || !err_host || !below_host || (n_thresholds > 0 && !theta_host)) return DWKV_E_NULL;
  if (n_windows < 0 || n_thresholds < 0 || ctl->patience < 1 || !(ctl->step_down >= 0.f) ||
      !(ctl->step_up >= 0.f) || !(ctl->theta_min <= ctl->theta_max))
    return DWKV_E_DIMS;
  for (int32_t m = 0; m < n_windows; ++m) {
    const float e = err_host[m];
    float step = 0.f;
    if (!(e <= ctl->tol)) {                       // above tolerance, or not a number
      step = -ctl->step_down;
      below_host[m] = 0;
    } else if (++below_host[m] >= ctl->patience) {
      step = ctl->step_up;
      below_host[m] = 0;
    }
    if (step != 0.f)
      for (int32_t j = 0; j < n_thresholds; ++j) {
        float& th = theta_host[(int64_t)m * n_thresholds + j];
        th = std::min(std::max(th + step, ctl->theta_min), ctl->theta_max);
      }
  }
  return DWKV_OK;
}

int32_t dwkv_probe_schedule(int64_t step, int32_t period, int32_t n_heads, int32_t n_kv_heads, int32_t n_pos,
                            int32_t* heads_host, int32_t* n_pos_host) {
  if (step < 0 || period < 1 || n_kv_heads < 1 || n_heads < 1 || n_heads > n_kv_heads ||
      n_heads > DWKV_MAX_PROBE_HEADS || n_pos < 1 || n_pos > DWKV_MAX_PROBE_POS || !heads_host || !n_pos_host)
    return -1;
  *n_pos_host = 0;
  if (step % period != 0) return 0;
  const int64_t k = step / period;
  for (int32_t i = 0; i < n_heads; ++i) heads_host[i] = (int32_t)((k % n_kv_heads * n_heads + i) % n_kv_heads);
  *n_pos_host = (int32_t)std::min<int64_t>(n_pos, step + 1);
  return n_heads;
}

size_t dwkv_validate_workspace_bytes(void) { return 256; }

dwkv_status dwkv_validate(const dwkv_dims* d, const dwkv_cache* c, int64_t* bad_index, void* workspace,
                          size_t ws_bytes, void* stream) {
  if (bad_index) *bad_index = -1;
  dwkv_status st = check_dims(d);
  if (st != DWKV_OK) return st;
  if (!c || !c->rank_code || !c->res_off || !c->res_idx || !c->res_val || !workspace) return DWKV_E_NULL;
  if (ws_bytes < dwkv_validate_workspace_bytes()) return DWKV_E_WORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  unsigned long long* bad = static_cast<unsigned long long*>(workspace);
  if (launch_validate(d, c, bad, s) != hipSuccess) return DWKV_E_HIP;
  unsigned long long host = 0;
  if (hipMemcpyAsync(&host, bad, sizeof(host), hipMemcpyDeviceToHost, s) != hipSuccess) return DWKV_E_HIP;
  if (hipStreamSynchronize(s) != hipSuccess) return DWKV_E_HIP;
  if (host == ~0ull) return DWKV_OK;
  if (bad_index) *bad_index = (int64_t)host;
  return DWKV_E_LAYOUT;
}

}  // extern "C"
