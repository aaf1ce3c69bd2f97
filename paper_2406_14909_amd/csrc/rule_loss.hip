// Rule-loss table (paper Sec. 3.3, Eq. 4): the accuracy loss of giving head h
// rule r at length N is the head's block-averaged attention influence summed
// over the causal pairs the rule masks,
//     dl[h][r] = sum over blocks (I, J) of masked_r(I, J) * ebar[h][I][J],
// where masked_r(I, J) counts the pairs (i, j) of the 64 x 64 block with
// j <= i, j >= s and j < band_start_r(i) (every token of a block carries the
// block's mean).  masked_r depends on the rule and the block only, in closed
// form: with the block band the band start is constant over the block's rows;
// with the token band it moves by one per row, and the row sum is an
// arithmetic series clipped to [0, block width].  Also writes each rule's
// density (paper Sec. 4 "Setups": in-memory KV-cache length over sequence
// length during decoding), kv_len / n, with kv_len = min(s + w, n) the tokens
// the rule's token-exact cache holds once n tokens have been seen.
//
// One work-group per head; lane r of every wave handles rule r; the 4 waves
// take interleaved block rows and meet in LDS.  Sums are fp64.
#include "moa_device.h"

namespace moa {

namespace {

constexpr int kWaves = 4;
constexpr int kBlock = kInfluenceBlock;

// sum_{x = 0}^{t} clamp(x, 0, m) for 0 <= m <= 64 and |t| < 2^20
__device__ __forceinline__ int clamp_prefix(int t, int m) {
  if (t < 0) return 0;
  if (t <= m) return t * (t + 1) / 2;
  return m * (m + 1) / 2 + (t - m) * m;
}

// Causal pairs of block (I, J) hidden by a rule (band length w in units of
// 2^bsh tokens, s sinks) at length n <= 65536 (at most 64 x 64).
__device__ __forceinline__ int masked_in_block(int I, int J, int n, int s, int w, int bsh) {
  const int r0 = I * kBlock, r1 = min(n, r0 + kBlock);
  const int c0 = J * kBlock, c1 = min(n, c0 + kBlock);
  const int lo = max(c0, s);                       // sinks are never masked
  if (c1 <= lo) return 0;
  if (bsh != 0) {
    const int bs = ((r0 >> bsh) - min(w, (r0 >> bsh) + 2) + 1) * (1 << bsh);   // same start for every row
    return (r1 - r0) * max(0, min(c1, bs) - lo);
  }
  // row i masks [lo, min(c1, i - w + 1)): clamp(i + 1 - w - lo, 0, c1 - lo)
  const int a = 1 - min(w, r1 + 1) - lo, m = c1 - lo;
  return clamp_prefix(r1 - 1 + a, m) - clamp_prefix(r0 - 1 + a, m);
}

// Per block row I, the blocks a rule masks completely form one range
// [ja, jb] (ja: first block past the sinks; jb: last block below the band
// start of the row block's first row), so their sum is rows(I) times a
// difference of the row's prefix sums of cols(J) * ebar[I][J].  At most three
// blocks are masked in part: the block holding the sink edge and, with the
// token band, the two blocks the band edge sweeps across; those use the
// closed-form count.  Each wave takes every fourth block row: its lanes load
// the row, scan it (fp64) into the wave's LDS strip, then act as rules.
// DPP move of an fp64 value (both halves with the same control); lanes with
// no source, or in rows outside row_mask, receive 0.
template <int ctrl, int row_mask>
__device__ __forceinline__ double dpp_f64(double x) {
  const uint64_t u = __builtin_bit_cast(uint64_t, x);
  const int lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(u & 0xffffffffu), ctrl, row_mask, 0xF, true);
  const int hi = __builtin_amdgcn_update_dpp(0, static_cast<int>(u >> 32), ctrl, row_mask, 0xF, true);
  return __builtin_bit_cast(double, (uint64_t(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo));
}

// Inclusive prefix sum over the 64 lanes: shifts by 1, 2, 4, 8 within each
// row of 16 lanes, then row_bcast:15 (row totals into rows 1 and 3) and
// row_bcast:31 (the first half's total into rows 2 and 3).
__device__ __forceinline__ double wave_inclusive_scan(double v) {
  v += dpp_f64<0x111, 0xF>(v);
  v += dpp_f64<0x112, 0xF>(v);
  v += dpp_f64<0x114, 0xF>(v);
  v += dpp_f64<0x118, 0xF>(v);
  v += dpp_f64<0x142, 0xA>(v);
  v += dpp_f64<0x143, 0xC>(v);
  return v;
}

__device__ __forceinline__ double lane63(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(u & 0xffffffffu), 63);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(u >> 32), 63);
  return __builtin_bit_cast(double, (uint64_t(hi) << 32) | lo);
}

template <int kChunks>   // 64-block chunks per row (covers nb <= 64 * kChunks)
__global__ void __launch_bounds__(kWaves * 64) rule_loss_kernel(RuleLossArgs a) {
  __shared__ double s_pre[kWaves][kChunks * 64];     // prefix sums of one row per wave
  __shared__ float s_raw[kWaves][kChunks * 64];      // the row itself
  __shared__ double s_dl[kWaves][kMaxRules];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int h = static_cast<int>(blockIdx.x);
  const int nb = a.nb, n = a.n, s = a.num_sink;
  const bool rule_ok = lane < a.num_rules;
  const int w = rule_ok ? a.window[lane] : 1;
  const float* e = a.ebar + int64_t(h) * nb * nb;
  double* pre = s_pre[wave];
  float* raw = s_raw[wave];
  const int ja = (s + kBlock - 1) / kBlock;                  // first block with no sink column
  const int js = (s % kBlock) ? s / kBlock : -1;             // block holding the sink edge, if any
  double acc = 0.0;

  // The wave's rows I = wave + kWaves * k are processed in groups of kDepth;
  // the next group is loaded into registers (lane holds J = 64 c + lane)
  // while the current one is scanned and used, so kDepth rows are in flight.
  constexpr int kDepth = kChunks >= 8 ? 2 : 16 / kChunks;
  auto row_of = [&](int k) { return wave + kWaves * k; };
  auto load_group = [&](int grp, float (&x)[kDepth][kChunks]) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      const int I = row_of(grp * kDepth + d);
#pragma unroll
      for (int c = 0; c < kChunks; ++c) {
        const int J = c * 64 + lane;
        x[d][c] = (I < nb && J <= I) ? e[int64_t(I) * nb + J] : 0.0f;
      }
    }
  };
  auto process_row = [&](int I, const float (&x)[kChunks]) {
    // prefix sums over J <= I of cols(J) * ebar[I][J]
    double carry = 0.0;
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      if (c * 64 > I) break;
      const int J = c * 64 + lane;
      double v = static_cast<double>(x[c]) * static_cast<double>(min(kBlock, n - J * kBlock));
      v = wave_inclusive_scan(v) + carry;
      if (J <= I) {
        pre[J] = v;
        raw[J] = x[c];
      }
      carry = lane63(v);
    }
    if (!rule_ok) return;
    const int r0 = I * kBlock;
    const int rows = min(kBlock, n - r0);
    // last completely masked block of this row block (band start of its first
    // row; windows beyond the row cannot mask anything)
    const int wc = min(w, (r0 >> a.band_shift) + 2);
    const int bs0 = ((r0 >> a.band_shift) - wc + 1) * (1 << a.band_shift);
    const int jb = min((bs0 >= 0 ? bs0 / kBlock : -((-bs0 + kBlock - 1) / kBlock)) - 1, I);
    if (jb >= ja) {
      const double lo = ja > 0 ? pre[ja - 1] : 0.0;
      acc += static_cast<double>(rows) * (pre[jb] - lo);
    }
    // blocks masked in part: the block holding the sink edge, and with the
    // token band the two blocks the band start sweeps across this row block
    const int cand[3] = {js, a.band_shift ? -1 : jb + 1, a.band_shift ? -1 : jb + 2};
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      const int J = cand[c];
      if (J < 0 || J > I || (J >= ja && J <= jb)) continue;
      if (c > 0 && J == js) continue;
      const int cnt = masked_in_block(I, J, n, s, w, a.band_shift);
      acc += static_cast<double>(cnt) * static_cast<double>(raw[J]);
    }
  };
  float cur[kDepth][kChunks], nxt[kDepth][kChunks];
  load_group(0, cur);
  for (int grp = 0; row_of(grp * kDepth) < nb; ++grp) {
    load_group(grp + 1, nxt);
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      const int I = row_of(grp * kDepth + d);
      if (I < nb) process_row(I, cur[d]);
    }
#pragma unroll
    for (int d = 0; d < kDepth; ++d)
#pragma unroll
      for (int c = 0; c < kChunks; ++c) cur[d][c] = nxt[d][c];
  }
  s_dl[wave][lane] = acc;
  __syncthreads();
  if (wave != 0 || !rule_ok) return;
  double dl = 0.0;
#pragma unroll
  for (int v = 0; v < kWaves; ++v) dl += s_dl[v][lane];
  a.dl[int64_t(h) * a.num_rules + lane] = dl;
  if (h == 0) a.density[lane] = static_cast<double>(a.kv_len[lane]) / static_cast<double>(n);
}

}  // namespace

int launch_rule_loss(const RuleLossArgs& a, void* stream) {
  RuleLossArgs copy = a;
  void* args[] = {&copy};
  const void* kernel;
  const int chunks = (a.nb + 63) / 64;
  if (chunks <= 1) kernel = reinterpret_cast<const void*>(&rule_loss_kernel<1>);
  else if (chunks <= 2) kernel = reinterpret_cast<const void*>(&rule_loss_kernel<2>);
  else if (chunks <= 4) kernel = reinterpret_cast<const void*>(&rule_loss_kernel<4>);
  else if (chunks <= 8) kernel = reinterpret_cast<const void*>(&rule_loss_kernel<8>);
  else if (chunks <= 16) kernel = reinterpret_cast<const void*>(&rule_loss_kernel<16>);
  else return static_cast<int>(hipErrorInvalidValue);
  return static_cast<int>(hipLaunchKernel(kernel, dim3(static_cast<unsigned>(a.num_heads)), dim3(kWaves * 64), args,
                                          0, static_cast<hipStream_t>(stream)));
}

}  // namespace moa
