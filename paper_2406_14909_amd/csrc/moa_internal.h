// Internal declarations shared by the host entry points and the HIP kernels.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "moa.h"

// ---------------------------------------------------------------------------
// Plan: host-only tables of one attention layer.
// ---------------------------------------------------------------------------
struct moa_plan_s {
  moa_desc_t desc;
  int32_t group;                   // num_q_heads / num_kv_heads
  float scale;                     // resolved softmax scale
  std::vector<int32_t> window;     // [H_kv]
  std::vector<int32_t> capacity;   // [H_kv]
  std::vector<int64_t> offset;     // [H_kv + 1]
  std::vector<int16_t> kv_order;   // [H_kv] KV heads, widest window first
};

namespace moa {

// Error reporting (thread-local message behind moa_last_error).
moa_status_t fail(moa_status_t st, const std::string& msg);
moa_status_t ok();

// ---------------------------------------------------------------------------
// Kernel argument blocks (passed by value; the per-head tables ride along).
// ---------------------------------------------------------------------------
struct PrefillArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  int64_t n;                 // tokens per sequence
  int32_t batch;
  int32_t hq;
  int32_t hkv;
  int32_t group;
  int32_t num_sink;
  int32_t n_qtiles;          // ceil(n / query rows per block)
  int32_t qchunk;            // query tiles per dispatch unit
  int32_t n_chunks;          // ceil(n_qtiles / qchunk)
  int32_t n_units;           // hkv * batch * n_chunks
  float scale_log2;          // softmax scale * log2(e)
  int32_t band_shift;        // the band of row i starts at ((i >> shift) - window + 1) << shift
  int32_t rotate;            // visit each unit's band tiles in step (keys and values exceed the last-level cache)
  int32_t window[MOA_MAX_KV_HEADS];   // band length in units of 2^band_shift tokens
  int16_t kv_order[MOA_MAX_KV_HEADS];
};

struct AppendArgs {
  void* kc;
  void* vc;
  int32_t* pos;
  const void* kn;
  const void* vn;
  int64_t rows_total;        // cache rows per sequence
  int64_t start;
  int64_t end;               // start + n_new
  int32_t batch;
  int32_t hkv;
  int32_t num_sink;
  int32_t rows_per_seq;      // slots written per sequence
  const int32_t* positions;  // per-sequence positions of a one-token append (device), or null
  int32_t cand_start[MOA_MAX_KV_HEADS + 1];
  int32_t window[MOA_MAX_KV_HEADS];
  int64_t offset[MOA_MAX_KV_HEADS];
};

// Decode work split: the filled cache slots of every (sequence, KV head) pair,
// laid end to end in (sequence, head) order, form one virtual key range of
// `total` keys, cut into `workers` near-equal pieces (one per wave):
// worker w covers [start(w), start(w + 1)) with
// start(w) = w * per_worker + (w * rem) / workers.  Head g of a sequence owns
// virtual keys [seg_start[g], seg_start[g + 1]) of that sequence's range.
struct DecodeArgs {
  const void* q;
  const void* kc;
  const void* vc;
  void* o;
  float* part;               // [workers + batch * hkv][group][head_dim + 4] partials
  const int32_t* positions;  // per-sequence positions (device), or null: one position for all
  int64_t rows_total;        // cache rows per sequence
  int64_t total;             // virtual keys = batch * seq_keys
  int64_t seq_keys;          // virtual keys per sequence (= seg_start[hkv])
  int64_t per_worker;        // total / workers (set by the launcher)
  int32_t rem;               // total % workers (set by the launcher)
  int32_t workers;           // set by the launcher
  int32_t batch;
  int32_t hq;
  int32_t hkv;
  float scale_log2;
  int64_t seg_start[MOA_MAX_KV_HEADS + 1];
  int32_t capacity[MOA_MAX_KV_HEADS];
  int64_t offset[MOA_MAX_KV_HEADS];
};

// Attention-influence profile of dense causal attention (one launch).
struct InfluenceArgs {
  const void* q;             // [batch, n, hq, D]
  const void* k;             // [batch, n, hkv, D]
  const void* v;             // [batch, n, hkv, D]
  const void* dout;          // [batch, n, hq, D]
  float* ebar;               // [hq, nb, nb]
  int32_t n;
  int32_t batch;
  int32_t hq;
  int32_t hkv;
  int32_t group;
  int32_t n_tiles;           // ceil(n / 128) query-row tiles per head
  int32_t nb;                // ceil(n / 64) blocks
  float scale_log2;          // softmax scale * log2(e)
};

// Rule-loss table of a set of candidate rules (one launch).
constexpr int kMaxRules = 64;
struct RuleLossArgs {
  const float* ebar;         // [num_heads, nb, nb] block-averaged influence
  double* dl;                // [num_heads, num_rules]
  double* density;           // [num_rules]
  int32_t num_heads;
  int32_t n;
  int32_t nb;
  int32_t num_rules;
  int32_t num_sink;
  int32_t band_shift;        // 0: token band; 6: band in 64-token blocks
  int32_t window[kMaxRules]; // per rule: band length in units of 2^band_shift tokens
  int32_t kv_len[kMaxRules]; // per rule: tokens its cache holds at length n, min(s + w, n)
};

// Kernel launchers (return hipError_t as int; 0 = success).
int launch_prefill(const PrefillArgs& a, int dtype, int head_dim, void* stream);
int launch_kv_append(const AppendArgs& a, int dtype, int head_dim, void* stream);
int launch_decode(DecodeArgs a, int dtype, int head_dim, int group, void* stream);
int launch_influence(const InfluenceArgs& a, int head_dim, void* stream);
int launch_rule_loss(const RuleLossArgs& a, void* stream);
// Device address of the library-owned decode workspace on the current device
// (resolved once per device); returns a hipError_t as int.
int decode_scratch(void** out);

constexpr int kPrefillRows = 128;   // query rows per prefill work-group
constexpr int kPrefillChunk = 16;   // minimum query tiles per prefill dispatch unit
constexpr int kPrefillUnitBlocks = 64;  // minimum work-groups per prefill dispatch unit
constexpr int kNumXcd = 8;          // accelerator dies; work-groups go round-robin over them
constexpr int64_t kLastLevelCacheBytes = int64_t(256) << 20;   // MI355X Infinity Cache
constexpr int kMaxDecodeWorkers = 8192;  // decode workers (waves) per launch, at most
constexpr int kDecodeMinKeys = 256;      // virtual keys per decode worker, at least
constexpr int kDecodePartPad = 4;        // partial row: head_dim sums, m, l, 2 pad floats
constexpr size_t kDecodeScratchBytes = MOA_DECODE_SCRATCH_BYTES;   // library-owned decode workspace per GPU
constexpr int kInfluenceBlock = 64;      // profiling block (tokens)
constexpr int kMaxInfluenceN = 65536;    // longest profiled sequence (block sums stay in LDS)

}  // namespace moa
