// Static per-head KV cache append with in-place replacement of the oldest
// non-sink entry (paper Appendix "Efficiency Experiment Setup": each head's
// cache is as long as its span, and a new token overwrites the entry that has
// left it).  Slot of position p: p if p < s, else s + ((p - s) mod w_g).
//
// Only each slot's final occupant among the appended positions is written,
// so a bulk (prefill) append touches at most C_g rows per head and equals
// the same tokens appended one at a time.  The copy is a bit copy: the
// kernel never interprets the elements.
//
// Grid: x = candidate rows of one (sequence, head), y = KV head, z = sequence.
// Each row (D elements = ROW_BYTES) is moved by LPR lanes with 16-byte loads.
#include "moa_device.h"

namespace moa {

template <int ROW_BYTES>
__global__ void __launch_bounds__(256) kv_append_kernel(AppendArgs a) {
  constexpr int LPR = ROW_BYTES / 16;
  const int g = blockIdx.y;
  const int b = blockIdx.z;
  const int n_cand = a.cand_start[g + 1] - a.cand_start[g];
  const int64_t ci = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / LPR;
  const int col = threadIdx.x % LPR;
  if (ci >= n_cand) return;
  const int64_t s = a.num_sink;
  const int64_t w = a.window[g];
  int64_t p, nrow;
  if (a.positions != nullptr) {                   // one token per sequence, own position
    p = a.positions[b];
    if (p < 0) return;                            // inactive sequence
    nrow = int64_t(b) * a.hkv + g;
  } else {
    const int64_t n_sink = max(int64_t(0), min(a.end, s) - a.start);
    if (ci < n_sink) {
      p = a.start + ci;
    } else {
      const int64_t lo = max(max(a.start, s), a.end - w);
      p = lo + (ci - n_sink);
    }
    nrow = (int64_t(b) * (a.end - a.start) + (p - a.start)) * a.hkv + g;
  }
  const int64_t slot = p < s ? p : s + (p - s) % w;
  const int64_t crow = int64_t(b) * a.rows_total + a.offset[g] + slot;
  const u32x4* ksrc = reinterpret_cast<const u32x4*>(static_cast<const char*>(a.kn) + nrow * ROW_BYTES) + col;
  const u32x4* vsrc = reinterpret_cast<const u32x4*>(static_cast<const char*>(a.vn) + nrow * ROW_BYTES) + col;
  u32x4* kdst = reinterpret_cast<u32x4*>(static_cast<char*>(a.kc) + crow * ROW_BYTES) + col;
  u32x4* vdst = reinterpret_cast<u32x4*>(static_cast<char*>(a.vc) + crow * ROW_BYTES) + col;
  const u32x4 kx = *ksrc;
  const u32x4 vx = *vsrc;
  *kdst = kx;
  *vdst = vx;
  if (col == 0) a.pos[crow] = static_cast<int32_t>(p);
}

template <int ROW_BYTES>
static int launch_append_t(const AppendArgs& a, void* stream) {
  constexpr int LPR = ROW_BYTES / 16;
  int max_cand = 0;
  for (int g = 0; g < a.hkv; ++g) max_cand = max(max_cand, a.cand_start[g + 1] - a.cand_start[g]);
  if (max_cand == 0) return 0;
  const int threads = (int64_t(max_cand) * LPR >= 256) ? 256 : 64;
  const int64_t gx = (int64_t(max_cand) * LPR + threads - 1) / threads;
  dim3 grid(static_cast<unsigned>(gx), static_cast<unsigned>(a.hkv), static_cast<unsigned>(a.batch));
  AppendArgs copy = a;
  void* args[] = {&copy};
  return static_cast<int>(hipLaunchKernel(reinterpret_cast<const void*>(&kv_append_kernel<ROW_BYTES>), grid,
                                          dim3(threads), args, 0, static_cast<hipStream_t>(stream)));
}

int launch_kv_append(const AppendArgs& a, int dtype, int head_dim, void* stream) {
  const int row_bytes = head_dim * (dtype == MOA_BF16 ? 2 : 4);
  switch (row_bytes) {
    case 128: return launch_append_t<128>(a, stream);
    case 256: return launch_append_t<256>(a, stream);
    case 512: return launch_append_t<512>(a, stream);
    default: return static_cast<int>(hipErrorInvalidValue);
  }
}

}  // namespace moa
