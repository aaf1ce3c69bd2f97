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
  int32_t decode_chunk;            // cache slots per decode work item
  std::vector<int32_t> window;     // [H_kv]
  std::vector<int32_t> capacity;   // [H_kv]
  std::vector<int64_t> offset;     // [H_kv + 1]
  std::vector<int16_t> kv_order;   // [H_kv] KV heads, widest window first
};

namespace moa {

// Error reporting (thread-local message behind moa_last_error).
moa_status_t fail(moa_status_t st, const std::string& msg);
moa_status_t ok();

// Decode split-K geometry for one position (host side).
struct DecodeGeometry {
  int32_t fill[MOA_MAX_KV_HEADS];
  int32_t item_start[MOA_MAX_KV_HEADS + 1];
  int32_t items_per_seq;
};
void decode_geometry(const moa_plan_s& p, int64_t pos, DecodeGeometry* g);

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
  int32_t window[MOA_MAX_KV_HEADS];
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

struct DecodeArgs {
  const void* q;
  const void* kc;
  const void* vc;
  void* o;
  float* part;               // [items][group][D + 2] split-K partials
  int64_t rows_total;        // cache rows per sequence
  int32_t batch;
  int32_t hq;
  int32_t hkv;
  int32_t chunk;             // slots per work item
  int32_t items_per_seq;     // work items per sequence (ragged: at full caches)
  float scale_log2;
  const int32_t* positions;  // per-sequence positions (device), or null: one position for all
  int32_t fill[MOA_MAX_KV_HEADS];
  int32_t item_start[MOA_MAX_KV_HEADS + 1];
  int32_t capacity[MOA_MAX_KV_HEADS];
  int64_t offset[MOA_MAX_KV_HEADS];
};

// Kernel launchers (return hipError_t as int; 0 = success).
int launch_prefill(const PrefillArgs& a, int dtype, int head_dim, void* stream);
int launch_kv_append(const AppendArgs& a, int dtype, int head_dim, void* stream);
int launch_decode(const DecodeArgs& a, int dtype, int head_dim, int group, void* stream);

constexpr int kPrefillRows = 128;   // query rows per prefill work-group
constexpr int kPrefillChunk = 16;   // minimum query tiles per prefill dispatch unit
constexpr int kPrefillUnitBlocks = 64;  // minimum work-groups per prefill dispatch unit
constexpr int kNumXcd = 8;          // accelerator dies; work-groups go round-robin over them
constexpr int kDecodeChunk = 512;   // cache slots per decode work item (minimum)
constexpr int kMaxMergeChunks = 256;  // split-K chunks per cache the merge kernel stages in LDS

}  // namespace moa
