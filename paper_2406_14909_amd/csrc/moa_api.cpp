// Host side of the C ABI: plan construction, argument validation, error
// reporting and dispatch to the HIP kernel launchers.  Compiled with
// -ffp-contract=off so the elastic rule is evaluated exactly as written.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <numeric>
#include <string>

#include "moa_internal.h"

namespace moa {

static thread_local std::string g_last_error;

moa_status_t fail(moa_status_t st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

moa_status_t ok() { return MOA_OK; }


// Workspace: decode partials, fp32 [workers + batch * hkv][group][head_dim + 4]
// (acc[head_dim], running max m, running sum l, padding), for the largest
// worker count a launch uses.
static size_t decode_workspace_bytes(const moa_plan_s& p, int32_t batch) {
  const size_t rows = static_cast<size_t>(kMaxDecodeWorkers) + static_cast<size_t>(batch) * p.desc.num_kv_heads;
  return rows * sizeof(float) * static_cast<size_t>(p.group) * (p.desc.head_dim + kDecodePartPad);
}

// Decode arguments shared by both decode entry points; seg_len[g] is head g's
// virtual segment per sequence (its fill, or its capacity with per-sequence
// positions).
static moa_status_t decode_args(const moa_plan_s& p, const char* who, const void* q, const void* k_cache,
                                const void* v_cache, void* o, int32_t batch, void* workspace,
                                const int64_t* seg_len, DecodeArgs* a) {
  const moa_desc_t& d = p.desc;
  memset(a, 0, sizeof(*a));
  a->q = q; a->kc = k_cache; a->vc = v_cache; a->o = o;
  a->part = static_cast<float*>(workspace);
  a->rows_total = p.offset[d.num_kv_heads];
  a->batch = batch;
  a->hq = d.num_q_heads;
  a->hkv = d.num_kv_heads;
  a->scale_log2 = p.scale * 1.4426950408889634f;
  a->seg_start[0] = 0;
  for (int h = 0; h < d.num_kv_heads; ++h) {
    a->seg_start[h + 1] = a->seg_start[h] + seg_len[h];
    a->capacity[h] = p.capacity[h];
    a->offset[h] = p.offset[h];
  }
  a->seq_keys = a->seg_start[d.num_kv_heads];
  if (a->seq_keys <= 0 || static_cast<double>(a->seq_keys) * batch >= 9007199254740992.0 ||
      static_cast<int64_t>(batch) * d.num_kv_heads >= (int64_t(1) << 31))
    return fail(MOA_ERR_UNSUPPORTED, std::string(who) + ": batch x cache slots too large for one launch");
  a->total = a->seq_keys * batch;
  return ok();
}

// Elastic rule alpha + beta * N (paper Sec. 3.2, Eq. 2), floored.  Default:
// the value is the band, clipped to [1, N].  MOA_SPAN_INCLUDES_SINKS: it is the
// whole span S (sinks + band, Appendix "Attention Span"), clipped to [0, N],
// and the band is S - s, at least 1.
static int64_t rule_window(double alpha, double beta, int64_t n, int32_t num_sink, uint32_t flags) {
  const double nd = static_cast<double>(n);
  volatile double prod = beta * nd;   // separate rounding: no fused multiply-add
  const double x = alpha + prod;
  if (flags & MOA_SPAN_INCLUDES_SINKS) {
    int64_t span;
    if (!(x >= 0.0)) span = 0;
    else if (x >= nd) span = n;
    else span = static_cast<int64_t>(floor(x));
    return std::max<int64_t>(span - num_sink, 1);
  }
  if (!(x >= 1.0)) return 1;
  if (x >= nd) return n;
  return static_cast<int64_t>(floor(x));
}

static bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

static bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

static size_t elem_size(const moa_plan_s& p) { return p.desc.dtype == MOA_BF16 ? 2 : 4; }

// Decode writes o and `ws_need` bytes of the workspace; true when either
// overlaps another argument (or the other written buffer).
static bool decode_overlap(const moa_plan_s& p, const void* q, const void* kc, const void* vc, const void* o,
                           int32_t batch, const void* ws, size_t ws_need) {
  const size_t es = elem_size(p);
  const size_t ob = es * static_cast<size_t>(batch) * p.desc.num_q_heads * p.desc.head_dim;
  const size_t cb = es * static_cast<size_t>(batch) * static_cast<size_t>(p.offset[p.desc.num_kv_heads]) *
                    p.desc.head_dim;
  return overlaps(o, ob, q, ob) || overlaps(o, ob, kc, cb) || overlaps(o, ob, vc, cb) ||
         overlaps(o, ob, ws, ws_need) || overlaps(ws, ws_need, q, ob) || overlaps(ws, ws_need, kc, cb) ||
         overlaps(ws, ws_need, vc, cb);
}

}  // namespace moa

using namespace moa;

extern "C" {

const char* moa_last_error(void) { return g_last_error.c_str(); }

moa_status_t moa_plan(const moa_desc_t* desc, const double* alpha, const double* beta,
                      moa_plan_t** out) {
  if (!desc || !alpha || !beta || !out) return fail(MOA_ERR_INVALID_ARG, "moa_plan: null argument");
  *out = nullptr;
  const moa_desc_t d = *desc;
  if (d.num_kv_heads < 1 || d.num_kv_heads > MOA_MAX_KV_HEADS)
    return fail(MOA_ERR_INVALID_ARG, "moa_plan: num_kv_heads must be in [1, MOA_MAX_KV_HEADS]");
  if (d.num_q_heads < 1 || d.num_q_heads > MOA_MAX_Q_HEADS)
    return fail(MOA_ERR_INVALID_ARG, "moa_plan: num_q_heads must be in [1, MOA_MAX_Q_HEADS]");
  if (d.num_q_heads % d.num_kv_heads != 0)
    return fail(MOA_ERR_INVALID_ARG, "moa_plan: num_q_heads must be a multiple of num_kv_heads");
  const int group = d.num_q_heads / d.num_kv_heads;
  if (group != 1 && group != 2 && group != 4 && group != 8)
    return fail(MOA_ERR_UNSUPPORTED, "moa_plan: query group size must be 1, 2, 4 or 8");
  if (d.head_dim != 64 && d.head_dim != 128)
    return fail(MOA_ERR_UNSUPPORTED, "moa_plan: head_dim must be 64 or 128");
  if (d.num_sink < 0 || d.num_sink >= (1 << 30))
    return fail(MOA_ERR_INVALID_ARG, "moa_plan: num_sink must be in [0, 2^30)");
  if (d.n < 1 || d.n >= (int64_t(1) << 30))
    return fail(MOA_ERR_INVALID_ARG, "moa_plan: n must be in [1, 2^30)");
  if (d.dtype != MOA_F32 && d.dtype != MOA_BF16)
    return fail(MOA_ERR_INVALID_ARG, "moa_plan: dtype must be MOA_F32 or MOA_BF16");
  if (!isfinite(d.softmax_scale) || d.softmax_scale < 0.0f)
    return fail(MOA_ERR_INVALID_ARG, "moa_plan: softmax_scale must be finite and >= 0");
  if ((d.flags & ~(MOA_SPAN_INCLUDES_SINKS | MOA_BLOCK_BAND)) != 0 || d.reserved != 0)
    return fail(MOA_ERR_INVALID_ARG, "moa_plan: unknown flags or nonzero reserved field");
  for (int h = 0; h < d.num_kv_heads; ++h)
    if (!isfinite(alpha[h]) || !isfinite(beta[h]))
      return fail(MOA_ERR_INVALID_ARG, "moa_plan: alpha and beta must be finite");

  moa_plan_s* p = new (std::nothrow) moa_plan_s();
  if (!p) return fail(MOA_ERR_INVALID_ARG, "moa_plan: out of host memory");
  p->desc = d;
  p->group = group;
  p->scale = d.softmax_scale > 0.0f ? d.softmax_scale : static_cast<float>(1.0 / sqrt(double(d.head_dim)));
  const int hkv = d.num_kv_heads;
  p->window.resize(hkv);
  p->capacity.resize(hkv);
  p->offset.assign(hkv + 1, 0);
  for (int h = 0; h < hkv; ++h) {
    const int64_t w = rule_window(alpha[h], beta[h], d.n, d.num_sink, d.flags);
    p->window[h] = static_cast<int32_t>(w);
    p->capacity[h] = static_cast<int32_t>(w + d.num_sink);
    p->offset[h + 1] = p->offset[h] + p->capacity[h];
  }
  p->kv_order.resize(hkv);
  std::iota(p->kv_order.begin(), p->kv_order.end(), 0);
  std::stable_sort(p->kv_order.begin(), p->kv_order.end(),
                   [&](int16_t a, int16_t b) { return p->window[a] > p->window[b]; });
  *out = p;
  return ok();
}

moa_status_t moa_plan_tables(const moa_plan_t* plan, int32_t* window, int32_t* capacity,
                             int64_t* offset) {
  if (!plan) return fail(MOA_ERR_INVALID_ARG, "moa_plan_tables: null plan");
  const int hkv = plan->desc.num_kv_heads;
  if (window) memcpy(window, plan->window.data(), sizeof(int32_t) * hkv);
  if (capacity) memcpy(capacity, plan->capacity.data(), sizeof(int32_t) * hkv);
  if (offset) memcpy(offset, plan->offset.data(), sizeof(int64_t) * (hkv + 1));
  return ok();
}

void moa_plan_free(moa_plan_t* plan) { delete plan; }

moa_status_t moa_prefill(const moa_plan_t* plan, const void* q, const void* k, const void* v,
                         void* o, int32_t batch, int64_t n_tokens, void* hip_stream) {
  if (!plan) return fail(MOA_ERR_INVALID_ARG, "moa_prefill: null plan");
  if (!q || !k || !v || !o) return fail(MOA_ERR_INVALID_ARG, "moa_prefill: null tensor pointer");
  if (batch < 1) return fail(MOA_ERR_INVALID_ARG, "moa_prefill: batch must be >= 1");
  if (n_tokens < 1 || n_tokens >= (int64_t(1) << 30))
    return fail(MOA_ERR_INVALID_ARG, "moa_prefill: n_tokens must be in [1, 2^30)");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
    return fail(MOA_ERR_INVALID_ARG, "moa_prefill: tensors must be 16-byte aligned");
  const moa_desc_t& d = plan->desc;
  const size_t es = elem_size(*plan);
  const size_t qbytes = es * batch * n_tokens * d.num_q_heads * d.head_dim;
  const size_t kbytes = es * batch * n_tokens * d.num_kv_heads * d.head_dim;
  if (overlaps(o, qbytes, q, qbytes) || overlaps(o, qbytes, k, kbytes) || overlaps(o, qbytes, v, kbytes))
    return fail(MOA_ERR_INVALID_ARG, "moa_prefill: output overlaps an input");
  const int64_t tiles = (n_tokens + kPrefillRows - 1) / kPrefillRows;
  // A unit spans at least kPrefillUnitBlocks work-groups (query tiles x group),
  // and at least kPrefillChunk query tiles.
  const int64_t qchunk = std::min<int64_t>(std::max<int64_t>(kPrefillChunk, kPrefillUnitBlocks / plan->group), tiles);
  const int64_t n_chunks = (tiles + qchunk - 1) / qchunk;
  const int64_t n_units = int64_t(d.num_kv_heads) * batch * n_chunks;
  const int64_t blocks = (n_units + kNumXcd - 1) / kNumXcd * kNumXcd * plan->group * qchunk;
  if (blocks >= (int64_t(1) << 31))
    return fail(MOA_ERR_UNSUPPORTED, "moa_prefill: too many work-groups for one launch");

  PrefillArgs a;
  memset(&a, 0, sizeof(a));
  a.q = q; a.k = k; a.v = v; a.o = o;
  a.n = n_tokens;
  a.batch = batch;
  a.hq = d.num_q_heads;
  a.hkv = d.num_kv_heads;
  a.group = plan->group;
  a.num_sink = d.num_sink;
  a.n_qtiles = static_cast<int32_t>(tiles);
  a.qchunk = static_cast<int32_t>(qchunk);
  a.n_chunks = static_cast<int32_t>(n_chunks);
  a.n_units = static_cast<int32_t>(n_units);
  a.scale_log2 = plan->scale * 1.4426950408889634f;
  a.band_shift = (d.flags & MOA_BLOCK_BAND) ? 6 : 0;
  static_assert(MOA_BAND_BLOCK == 64, "band_shift is log2(MOA_BAND_BLOCK)");
  // Keys and values larger than the last-level cache are re-read from HBM by
  // the band sweeps of different query tiles unless those sweeps run in step.
  a.rotate = 2 * static_cast<int64_t>(kbytes) > kLastLevelCacheBytes ? 1 : 0;
  for (int h = 0; h < d.num_kv_heads; ++h) {
    // Band length in tokens, or in blocks of MOA_BAND_BLOCK tokens (rounded up).
    a.window[h] = (d.flags & MOA_BLOCK_BAND) ? (plan->window[h] + MOA_BAND_BLOCK - 1) / MOA_BAND_BLOCK
                                             : plan->window[h];
    a.kv_order[h] = plan->kv_order[h];
  }
  const int err = launch_prefill(a, d.dtype, d.head_dim, hip_stream);
  if (err) return fail(MOA_ERR_HIP, "moa_prefill: kernel launch failed (hipError " + std::to_string(err) + ")");
  return ok();
}

moa_status_t moa_kv_append(const moa_plan_t* plan, void* k_cache, void* v_cache,
                           int32_t* pos_cache, const void* k_new, const void* v_new,
                           int32_t batch, int64_t start_pos, int64_t n_new, void* hip_stream) {
  if (!plan) return fail(MOA_ERR_INVALID_ARG, "moa_kv_append: null plan");
  if (!k_cache || !v_cache || !pos_cache || !k_new || !v_new)
    return fail(MOA_ERR_INVALID_ARG, "moa_kv_append: null tensor pointer");
  if (batch < 1 || batch > 65535) return fail(MOA_ERR_INVALID_ARG, "moa_kv_append: batch must be in [1, 65535]");
  if (start_pos < 0 || n_new < 1 || start_pos + n_new >= (int64_t(1) << 31))
    return fail(MOA_ERR_INVALID_ARG, "moa_kv_append: need start_pos >= 0, n_new >= 1, start_pos + n_new < 2^31");
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(k_new) || !aligned16(v_new) ||
      (reinterpret_cast<uintptr_t>(pos_cache) & 3u))
    return fail(MOA_ERR_INVALID_ARG, "moa_kv_append: tensors must be 16-byte aligned (pos_cache 4-byte)");
  const moa_desc_t& d = plan->desc;
  AppendArgs a;
  memset(&a, 0, sizeof(a));
  a.kc = k_cache; a.vc = v_cache; a.pos = pos_cache; a.kn = k_new; a.vn = v_new;
  a.rows_total = plan->offset[d.num_kv_heads];
  a.start = start_pos;
  a.end = start_pos + n_new;
  a.batch = batch;
  a.hkv = d.num_kv_heads;
  a.num_sink = d.num_sink;
  a.cand_start[0] = 0;
  const int64_t s = d.num_sink;
  for (int h = 0; h < d.num_kv_heads; ++h) {
    // Final occupants: sink positions in [start, min(end, s)) and the last
    // w_h positions >= s, i.e. [max(start, s, end - w_h), end).
    const int64_t w = plan->window[h];
    const int64_t n_sink = std::max<int64_t>(0, std::min<int64_t>(a.end, s) - start_pos);
    const int64_t lo = std::max<int64_t>(std::max<int64_t>(start_pos, s), a.end - w);
    const int64_t n_band = std::max<int64_t>(0, a.end - lo);
    a.cand_start[h + 1] = a.cand_start[h] + static_cast<int32_t>(n_sink + n_band);
    a.window[h] = plan->window[h];
    a.offset[h] = plan->offset[h];
  }
  a.rows_per_seq = a.cand_start[d.num_kv_heads];
  if (static_cast<int64_t>(a.rows_per_seq) * batch * 64 >= (int64_t(1) << 31))
    return fail(MOA_ERR_UNSUPPORTED, "moa_kv_append: too many rows for one launch");
  const int err = launch_kv_append(a, d.dtype, d.head_dim, hip_stream);
  if (err) return fail(MOA_ERR_HIP, "moa_kv_append: kernel launch failed (hipError " + std::to_string(err) + ")");
  return ok();
}

moa_status_t moa_kv_append_ragged(const moa_plan_t* plan, void* k_cache, void* v_cache,
                                  int32_t* pos_cache, const void* k_new, const void* v_new,
                                  const int32_t* positions, int32_t batch, void* hip_stream) {
  if (!plan) return fail(MOA_ERR_INVALID_ARG, "moa_kv_append_ragged: null plan");
  if (!k_cache || !v_cache || !pos_cache || !k_new || !v_new || !positions)
    return fail(MOA_ERR_INVALID_ARG, "moa_kv_append_ragged: null pointer");
  if (batch < 1 || batch > 65535)
    return fail(MOA_ERR_INVALID_ARG, "moa_kv_append_ragged: batch must be in [1, 65535]");
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(k_new) || !aligned16(v_new) ||
      (reinterpret_cast<uintptr_t>(pos_cache) & 3u) || (reinterpret_cast<uintptr_t>(positions) & 3u))
    return fail(MOA_ERR_INVALID_ARG, "moa_kv_append_ragged: misaligned pointer");
  const moa_desc_t& d = plan->desc;
  AppendArgs a;
  memset(&a, 0, sizeof(a));
  a.kc = k_cache; a.vc = v_cache; a.pos = pos_cache; a.kn = k_new; a.vn = v_new;
  a.positions = positions;
  a.rows_total = plan->offset[d.num_kv_heads];
  a.batch = batch;
  a.hkv = d.num_kv_heads;
  a.num_sink = d.num_sink;
  for (int h = 0; h <= d.num_kv_heads; ++h) a.cand_start[h] = h;    // one token per head
  for (int h = 0; h < d.num_kv_heads; ++h) {
    a.window[h] = plan->window[h];
    a.offset[h] = plan->offset[h];
  }
  a.rows_per_seq = d.num_kv_heads;
  const int err = launch_kv_append(a, d.dtype, d.head_dim, hip_stream);
  if (err) return fail(MOA_ERR_HIP, "moa_kv_append_ragged: kernel launch failed (hipError " + std::to_string(err) + ")");
  return ok();
}

size_t moa_decode_workspace_bytes(const moa_plan_t* plan, int32_t batch) {
  if (!plan || batch < 1) return 0;
  return decode_workspace_bytes(*plan, batch);
}

moa_status_t moa_decode(const moa_plan_t* plan, const void* q, const void* k_cache,
                        const void* v_cache, void* o, int32_t batch, int64_t pos,
                        void* workspace, size_t ws_bytes, void* hip_stream) {
  if (!plan) return fail(MOA_ERR_INVALID_ARG, "moa_decode: null plan");
  if (!q || !k_cache || !v_cache || !o) return fail(MOA_ERR_INVALID_ARG, "moa_decode: null tensor pointer");
  if (batch < 1) return fail(MOA_ERR_INVALID_ARG, "moa_decode: batch must be >= 1");
  if (pos < 0 || pos >= (int64_t(1) << 31) - 1)
    return fail(MOA_ERR_INVALID_ARG, "moa_decode: pos must be in [0, 2^31 - 1)");
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(o))
    return fail(MOA_ERR_INVALID_ARG, "moa_decode: tensors must be 16-byte aligned");
  const size_t need = decode_workspace_bytes(*plan, batch);
  if (!workspace || ws_bytes < need)
    return fail(MOA_ERR_WORKSPACE, "moa_decode: workspace missing or smaller than moa_decode_workspace_bytes (" +
                                       std::to_string(need) + " bytes)");
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(MOA_ERR_WORKSPACE, "moa_decode: workspace must be 256-byte aligned");
  if (decode_overlap(*plan, q, k_cache, v_cache, o, batch, workspace, need))
    return fail(MOA_ERR_INVALID_ARG, "moa_decode: o or the workspace overlaps another argument");
  const moa_desc_t& d = plan->desc;
  int64_t seg_len[MOA_MAX_KV_HEADS];
  for (int h = 0; h < d.num_kv_heads; ++h) seg_len[h] = std::min<int64_t>(pos + 1, plan->capacity[h]);
  DecodeArgs a;
  const moa_status_t st = decode_args(*plan, "moa_decode", q, k_cache, v_cache, o, batch, workspace, seg_len, &a);
  if (st != MOA_OK) return st;
  const int err = launch_decode(a, d.dtype, d.head_dim, plan->group, hip_stream);
  if (err) return fail(MOA_ERR_HIP, "moa_decode: kernel launch failed (hipError " + std::to_string(err) + ")");
  return ok();
}

moa_status_t moa_decode_noalloc(const moa_plan_t* plan, const void* q, const void* k_cache,
                                const void* v_cache, void* o, int32_t batch, int64_t pos, void* hip_stream) {
  if (!plan) return fail(MOA_ERR_INVALID_ARG, "moa_decode_noalloc: null plan");
  if (!q || !k_cache || !v_cache || !o) return fail(MOA_ERR_INVALID_ARG, "moa_decode_noalloc: null tensor pointer");
  if (batch < 1) return fail(MOA_ERR_INVALID_ARG, "moa_decode_noalloc: batch must be >= 1");
  if (pos < 0 || pos >= (int64_t(1) << 31) - 1)
    return fail(MOA_ERR_INVALID_ARG, "moa_decode_noalloc: pos must be in [0, 2^31 - 1)");
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(o))
    return fail(MOA_ERR_INVALID_ARG, "moa_decode_noalloc: tensors must be 16-byte aligned");
  const size_t need = decode_workspace_bytes(*plan, batch);
  if (need > kDecodeScratchBytes)
    return fail(MOA_ERR_WORKSPACE, "moa_decode_noalloc: this plan and batch need " + std::to_string(need) +
                                       " bytes of decode workspace, more than the library's " +
                                       std::to_string(kDecodeScratchBytes) + " (MOA_DECODE_SCRATCH_BYTES); "
                                       "use moa_decode with a caller-owned workspace");
  void* ws = nullptr;
  const int serr = decode_scratch(&ws);
  if (serr) return fail(MOA_ERR_HIP, "moa_decode_noalloc: hipGetSymbolAddress of the decode workspace failed (hipError " +
                                         std::to_string(serr) + ")");
  if (decode_overlap(*plan, q, k_cache, v_cache, o, batch, ws, need))
    return fail(MOA_ERR_INVALID_ARG, "moa_decode_noalloc: o overlaps another argument");
  const moa_desc_t& d = plan->desc;
  int64_t seg_len[MOA_MAX_KV_HEADS];
  for (int h = 0; h < d.num_kv_heads; ++h) seg_len[h] = std::min<int64_t>(pos + 1, plan->capacity[h]);
  DecodeArgs a;
  const moa_status_t st = decode_args(*plan, "moa_decode_noalloc", q, k_cache, v_cache, o, batch, ws, seg_len, &a);
  if (st != MOA_OK) return st;
  const int err = launch_decode(a, d.dtype, d.head_dim, plan->group, hip_stream);
  if (err) return fail(MOA_ERR_HIP, "moa_decode_noalloc: kernel launch failed (hipError " + std::to_string(err) + ")");
  return ok();
}

moa_status_t moa_decode_ragged(const moa_plan_t* plan, const void* q, const void* k_cache,
                               const void* v_cache, void* o, const int32_t* positions, int32_t batch,
                               void* workspace, size_t ws_bytes, void* hip_stream) {
  if (!plan) return fail(MOA_ERR_INVALID_ARG, "moa_decode_ragged: null plan");
  if (!q || !k_cache || !v_cache || !o || !positions)
    return fail(MOA_ERR_INVALID_ARG, "moa_decode_ragged: null pointer");
  if (batch < 1) return fail(MOA_ERR_INVALID_ARG, "moa_decode_ragged: batch must be >= 1");
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(o) ||
      (reinterpret_cast<uintptr_t>(positions) & 3u))
    return fail(MOA_ERR_INVALID_ARG, "moa_decode_ragged: misaligned pointer");
  const size_t need = decode_workspace_bytes(*plan, batch);
  if (!workspace || ws_bytes < need)
    return fail(MOA_ERR_WORKSPACE, "moa_decode_ragged: workspace missing or smaller than moa_decode_workspace_bytes (" +
                                       std::to_string(need) + " bytes)");
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(MOA_ERR_WORKSPACE, "moa_decode_ragged: workspace must be 256-byte aligned");
  if (decode_overlap(*plan, q, k_cache, v_cache, o, batch, workspace, need))
    return fail(MOA_ERR_INVALID_ARG, "moa_decode_ragged: o or the workspace overlaps another argument");
  const moa_desc_t& d = plan->desc;
  int64_t seg_len[MOA_MAX_KV_HEADS];
  for (int h = 0; h < d.num_kv_heads; ++h) seg_len[h] = plan->capacity[h];
  DecodeArgs a;
  const moa_status_t st =
      decode_args(*plan, "moa_decode_ragged", q, k_cache, v_cache, o, batch, workspace, seg_len, &a);
  if (st != MOA_OK) return st;
  a.positions = positions;
  const int err = launch_decode(a, d.dtype, d.head_dim, plan->group, hip_stream);
  if (err) return fail(MOA_ERR_HIP, "moa_decode_ragged: kernel launch failed (hipError " + std::to_string(err) + ")");
  return ok();
}

moa_status_t moa_influence(const moa_desc_t* desc, const void* q, const void* k, const void* v,
                           const void* dout, float* ebar, int32_t batch, int64_t n, void* hip_stream) {
  if (!desc || !q || !k || !v || !dout || !ebar) return fail(MOA_ERR_INVALID_ARG, "moa_influence: null pointer");
  const moa_desc_t& d = *desc;
  if (d.num_kv_heads < 1 || d.num_kv_heads > MOA_MAX_KV_HEADS || d.num_q_heads < 1 ||
      d.num_q_heads > MOA_MAX_Q_HEADS || d.num_q_heads % d.num_kv_heads != 0)
    return fail(MOA_ERR_INVALID_ARG, "moa_influence: bad head counts");
  if (d.head_dim != 64 && d.head_dim != 128)
    return fail(MOA_ERR_UNSUPPORTED, "moa_influence: head_dim must be 64 or 128");
  if (d.dtype != MOA_BF16) return fail(MOA_ERR_UNSUPPORTED, "moa_influence: dtype must be MOA_BF16");
  if (!isfinite(d.softmax_scale) || d.softmax_scale < 0.0f)
    return fail(MOA_ERR_INVALID_ARG, "moa_influence: softmax_scale must be finite and >= 0");
  if (batch < 1 || n < 1) return fail(MOA_ERR_INVALID_ARG, "moa_influence: batch and n must be >= 1");
  if (n > kMaxInfluenceN) return fail(MOA_ERR_UNSUPPORTED, "moa_influence: n must be <= 65536");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(dout) ||
      (reinterpret_cast<uintptr_t>(ebar) & 3u))
    return fail(MOA_ERR_INVALID_ARG, "moa_influence: misaligned pointer");
  const int64_t nb = (n + kInfluenceBlock - 1) / kInfluenceBlock;
  const size_t ebar_bytes = sizeof(float) * static_cast<size_t>(d.num_q_heads) * nb * nb;
  const size_t qb = 2 * static_cast<size_t>(batch) * n * d.num_q_heads * d.head_dim;
  const size_t kb = 2 * static_cast<size_t>(batch) * n * d.num_kv_heads * d.head_dim;
  if (overlaps(ebar, ebar_bytes, q, qb) || overlaps(ebar, ebar_bytes, k, kb) || overlaps(ebar, ebar_bytes, v, kb) ||
      overlaps(ebar, ebar_bytes, dout, qb))
    return fail(MOA_ERR_INVALID_ARG, "moa_influence: ebar overlaps an input");
  InfluenceArgs a;
  memset(&a, 0, sizeof(a));
  a.q = q; a.k = k; a.v = v; a.dout = dout; a.ebar = ebar;
  a.n = static_cast<int32_t>(n);
  a.batch = batch;
  a.hq = d.num_q_heads;
  a.hkv = d.num_kv_heads;
  a.group = d.num_q_heads / d.num_kv_heads;
  a.n_tiles = static_cast<int32_t>((n + 127) / 128);
  a.nb = static_cast<int32_t>(nb);
  const float scale = d.softmax_scale > 0.0f ? d.softmax_scale : static_cast<float>(1.0 / sqrt(double(d.head_dim)));
  a.scale_log2 = scale * 1.4426950408889634f;
  const int err = launch_influence(a, d.head_dim, hip_stream);
  if (err) return fail(MOA_ERR_HIP, "moa_influence: kernel launch failed (hipError " + std::to_string(err) + ")");
  return ok();
}

moa_status_t moa_rule_loss(const float* ebar, int32_t num_heads, int64_t n, int32_t num_sink, uint32_t flags,
                           const double* alpha, const double* beta, int32_t num_rules, double* dl,
                           double* density, void* hip_stream) {
  if (!ebar || !alpha || !beta || !dl || !density) return fail(MOA_ERR_INVALID_ARG, "moa_rule_loss: null pointer");
  if (num_heads < 1 || num_rules < 1 || num_rules > kMaxRules)
    return fail(MOA_ERR_INVALID_ARG, "moa_rule_loss: need num_heads >= 1 and 1 <= num_rules <= 64");
  if (n < 1 || n > kMaxInfluenceN) return fail(MOA_ERR_INVALID_ARG, "moa_rule_loss: n must be in [1, 65536]");
  if (num_sink < 0 || num_sink >= (1 << 30)) return fail(MOA_ERR_INVALID_ARG, "moa_rule_loss: bad num_sink");
  if ((flags & ~(MOA_SPAN_INCLUDES_SINKS | MOA_BLOCK_BAND)) != 0)
    return fail(MOA_ERR_INVALID_ARG, "moa_rule_loss: unknown flags");
  if ((reinterpret_cast<uintptr_t>(ebar) & 3u) || (reinterpret_cast<uintptr_t>(dl) & 7u) ||
      (reinterpret_cast<uintptr_t>(density) & 7u))
    return fail(MOA_ERR_INVALID_ARG, "moa_rule_loss: misaligned pointer");
  for (int r = 0; r < num_rules; ++r)
    if (!isfinite(alpha[r]) || !isfinite(beta[r]))
      return fail(MOA_ERR_INVALID_ARG, "moa_rule_loss: alpha and beta must be finite");
  const int64_t nb = (n + kInfluenceBlock - 1) / kInfluenceBlock;
  const size_t ebar_bytes = sizeof(float) * static_cast<size_t>(num_heads) * nb * nb;
  const size_t dl_bytes = sizeof(double) * static_cast<size_t>(num_heads) * num_rules;
  if (overlaps(dl, dl_bytes, ebar, ebar_bytes) || overlaps(density, sizeof(double) * num_rules, ebar, ebar_bytes) ||
      overlaps(density, sizeof(double) * num_rules, dl, dl_bytes))
    return fail(MOA_ERR_INVALID_ARG, "moa_rule_loss: output overlaps another buffer");
  RuleLossArgs a;
  memset(&a, 0, sizeof(a));
  a.ebar = ebar; a.dl = dl; a.density = density;
  a.num_heads = num_heads;
  a.n = static_cast<int32_t>(n);
  a.nb = static_cast<int32_t>(nb);
  a.num_rules = num_rules;
  a.num_sink = num_sink;
  a.band_shift = (flags & MOA_BLOCK_BAND) ? 6 : 0;
  for (int r = 0; r < num_rules; ++r) {
    const int64_t w = rule_window(alpha[r], beta[r], n, num_sink, flags);
    a.window[r] = static_cast<int32_t>((flags & MOA_BLOCK_BAND) ? (w + MOA_BAND_BLOCK - 1) / MOA_BAND_BLOCK : w);
    // the token-exact cache holds the sinks and the last w tokens (at most n)
    a.kv_len[r] = static_cast<int32_t>(std::min<int64_t>(int64_t(num_sink) + w, n));
  }
  const int err = launch_rule_loss(a, hip_stream);
  if (err) return fail(MOA_ERR_HIP, "moa_rule_loss: kernel launch failed (hipError " + std::to_string(err) + ")");
  return ok();
}

}  // extern "C"
