// Decode attention over per-head static KV caches of different lengths
// (paper Appendix "Efficiency Experiment Setup": one new query per sequence
// against caches whose length differs across heads).
//
// After the token at position t is appended, the filled slots of KV head g
// are exactly the keys visible to t (sinks + the last w_g positions), so no
// mask is applied: o = softmax(scale * q K^T) V over slots [0, fill_g),
// fill_g = min(t + 1, s + w_g).  Slot order does not matter.
//
// Work split.  The caches differ in length by orders of magnitude across
// heads, so the work is not cut per cache: all filled slots of the batch,
// laid end to end in (sequence, KV head) order, form one virtual key range
// that is cut into equal pieces, one per work-group ("worker"), with as many
// workers as the chip holds resident work-groups.  A worker walks its piece
// cache by cache; its 4 waves take interleaved rows (or tiles) of each cache
// and keep an online softmax (base 2, running max m, running sum l,
// unnormalised output acc) for all G query heads of the KV head, so each K/V
// byte is read from HBM once; the waves' states are merged through LDS at the
// end of each cache.  A cache that lies inside one worker's piece is
// normalised and written straight to o; otherwise every worker touching it
// writes a partial (acc, m, l) at slot (worker + cache index), which is unique
// because workers and caches are both ordered along the same range, and a
// second kernel merges the partials.  The kernel boundary makes the partials
// visible across the chip's L2 slices without any in-kernel cache maintenance.
//
// Inner loops.  With G query heads per KV head the work per cache row is
// G dot products and G axpys of length head_dim.  For one head (and for
// fp32) the row is spread over 16-byte lanes and reduced with DPP.  For bf16
// groups (G >= 2) the same work is a small dense contraction and runs on the
// matrix cores (CDNA4 16x16x32 bf16 MFMA, G padded to 16 columns):
//   S^T = K Q^T    A = 16 keys x 32 dims, B = Q^T kept in registers; lane l
//                  then holds keys 4*(l/16) .. +3 of query head l % 16.  The K
//                  tile is read from the cache in whole rows (4 rows of 256
//                  bytes per load at head_dim 128; operand-layout loads, 16
//                  rows x 64 bytes each, stream about 13 % slower) and passes
//                  through the wave's LDS buffer, which then takes the V tile.
//   O^T += V^T P^T B = P^T straight from the score registers (bf16), A = V^T
//                  from a per-wave LDS copy of the V tile read with the
//                  transposing LDS read; the key order inside each 32-key
//                  step is permuted identically on both operands.
#include <algorithm>
#include <atomic>
#include <mutex>

#include "moa_device.h"

namespace moa {

// Library-owned decode workspace for callers that cannot allocate
// (moa_decode_noalloc): kDecodeScratchBytes of fp32 split-K partials, one copy
// per GPU the library runs on, held until the process ends.  Host code never
// passes the array's name to a kernel (on the host it is only a stand-in for
// the symbol): decode_scratch() resolves each device's own address once with
// hipGetSymbolAddress and kernels get that address.
__device__ __align__(256) float scratch[kDecodeScratchBytes / sizeof(float)];

int decode_scratch(void** out) {
  static std::mutex mu;
  static void* addr[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return static_cast<int>(e);
  if (dev < 0 || dev >= 64) return static_cast<int>(hipErrorInvalidDevice);
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return static_cast<int>(e);
    if (p == nullptr) return static_cast<int>(hipErrorInvalidSymbol);
    addr[dev] = p;
  }
  *out = addr[dev];
  return 0;
}

namespace {

constexpr int kWaves = 4;          // waves per worker (work-group)
// Keys per wave tile in the matrix-core loop: 32 (8 KB of LDS per wave, about
// 160 VGPRs at group 4 and 226 at group 8).  At group 8 the earlier 64-key
// tiles (2 work-groups per compute unit) measured 2.8 % slower than 32-key
// tiles once K no longer came in operand layout from HBM.
template <int G>
constexpr int mma_keys() { return 32; }
// Caches split over at most fast_parts<G>() workers merge in one pass: 32 for
// GQA groups (their caches span up to about 24 workers), 16 otherwise.
template <int G>
constexpr int fast_parts() { return G >= 4 ? 32 : 16; }

__device__ __forceinline__ int64_t worker_start(const DecodeArgs& a, int w) {
  return int64_t(w) * a.per_worker + (int64_t(w) * a.rem) / a.workers;
}

// The worker whose piece holds virtual key x (estimate, then exact correction).
__device__ int worker_of(const DecodeArgs& a, int64_t x) {
  int w = static_cast<int>(static_cast<double>(x) * static_cast<double>(a.workers) /
                           static_cast<double>(a.total));
  w = max(0, min(w, a.workers - 1));
  while (w + 1 < a.workers && worker_start(a, w + 1) <= x) ++w;
  while (w > 0 && worker_start(a, w) > x) --w;
  return w;
}

// Filled slots of KV head g in sequence b; 0 for an idle sequence (negative
// position).  Without per-sequence positions the virtual segment is the fill.
__device__ __forceinline__ int cache_fill(const DecodeArgs& a, int b, int g) {
  if (a.positions == nullptr) return static_cast<int>(a.seg_start[g + 1] - a.seg_start[g]);
  const int p = a.positions[b];
  return p < 0 ? 0 : static_cast<int>(min(int64_t(p) + 1, int64_t(a.capacity[g])));
}

// Calls seg(b, g, lo, hi, whole) for each cache that worker w's piece touches:
// virtual slots [lo, hi) of KV head g of sequence b; `whole` when the piece
// covers the cache's entire virtual segment.  Work-group uniform.
template <class Seg>
__device__ __forceinline__ void for_each_segment(const DecodeArgs& a, int w, Seg&& seg) {
  int64_t x = worker_start(a, w);
  const int64_t x_end = worker_start(a, w + 1);
  if (x >= x_end) return;
  int b = static_cast<int>(x / a.seq_keys);
  int64_t r = x - int64_t(b) * a.seq_keys;
  int g = 0;
  while (a.seg_start[g + 1] <= r) ++g;
  while (x < x_end) {
    const int64_t s0 = a.seg_start[g];
    const int len = static_cast<int>(a.seg_start[g + 1] - s0);
    const int lo = static_cast<int>(r - s0);
    const int hi = static_cast<int>(min(int64_t(len), int64_t(lo) + (x_end - x)));
    seg(b, g, lo, hi, lo == 0 && hi == len);
    x += hi - lo;
    r += hi - lo;
    if (hi == len && ++g == a.hkv) {
      g = 0;
      ++b;
      r = 0;
    }
  }
}

// Merges the kWaves per-wave states of one cache held in LDS (acc[w][h][d],
// ml[w][h] = (m, l)) and writes either o (whole cache) or the worker's
// partial.  All threads of the work-group call it after a barrier.
template <typename T, int D, int G>
__device__ __forceinline__ void merge_waves_and_store(const DecodeArgs& a, const float* s_acc, const float* s_ml,
                                                      int w, int b, int g, bool whole) {
  constexpr int PS = D + kDecodePartPad;
  for (int idx = threadIdx.x; idx < G * D; idx += kWaves * 64) {
    const int h = idx / D, d = idx % D;
    float mx = kNegBig;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) mx = fmaxf(mx, s_ml[(v * G + h) * 2]);
    float lsum = 0.0f, asum = 0.0f;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) {
      const float f = fast_exp2(s_ml[(v * G + h) * 2] - mx);
      lsum += s_ml[(v * G + h) * 2 + 1] * f;
      asum += s_acc[(v * G + h) * D + d] * f;
    }
    if (whole) {
      static_cast<T*>(a.o)[(int64_t(b) * a.hq + g * G + h) * D + d] = static_cast<T>(asum / lsum);
    } else {
      float* pp = a.part + ((int64_t(w) + b * a.hkv + g) * G + h) * PS;
      pp[d] = asum;
      if (d == 0) {
        pp[D] = mx;
        pp[D + 1] = lsum;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Vector-ALU worker: LPR lanes cover one cache row with 16-byte loads; the
// work-group reads kWaves * RPW consecutive rows per load step, U steps in
// flight; per-lane-group online softmax, merged across the wave, then across
// the waves.
// ---------------------------------------------------------------------------
template <typename T, int D, int G>
__global__ void __launch_bounds__(kWaves * 64) decode_valu_kernel(DecodeArgs a) {
  constexpr int EPL = Vec16<T>::N;    // elements per lane
  constexpr int LPR = D / EPL;        // lanes per cache row
  constexpr int RPW = 64 / LPR;       // rows per wave per load step
  constexpr int U = 8;                // load steps in flight per iteration
  constexpr int STEP = kWaves * RPW;  // rows per work-group per load step

  __shared__ float s_acc[kWaves * G * D];
  __shared__ float s_ml[kWaves * G * 2];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int w = static_cast<int>(blockIdx.x);
  const int rsub = lane / LPR;
  const int col = lane % LPR;

  for_each_segment(a, w, [&](int b, int g, int lo, int hi, bool whole) {
    const int fill = cache_fill(a, b, g);
    if (fill == 0) return;                          // idle sequence
    hi = min(hi, fill);
    const int64_t row0 = int64_t(b) * a.rows_total + a.offset[g];
    const T* kbase = static_cast<const T*>(a.kc) + row0 * D + col * EPL;
    const T* vbase = static_cast<const T*>(a.vc) + row0 * D + col * EPL;

    float qf[G][EPL];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const Vec16<T> qv =
          load16(static_cast<const T*>(a.q) + (int64_t(b) * a.hq + g * G + h) * D + col * EPL);
#pragma unroll
      for (int e = 0; e < EPL; ++e) qf[h][e] = qv.get(e) * a.scale_log2;
    }
    float m[G], l[G], acc[G][EPL];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      m[h] = kNegBig;
      l[h] = 0.0f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[h][e] = 0.0f;
    }

    for (int base = lo + wave * RPW; base < hi; base += STEP * U) {
      const int r0 = base + rsub;
      Vec16<T> kv[U], vv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = r0 + u * STEP;
        if (r < hi) {
          kv[u] = load16_stream(kbase + int64_t(r) * D);
          vv[u] = load16_stream(vbase + int64_t(r) * D);
        } else {
          kv[u] = zero16<T>();
          vv[u] = zero16<T>();
        }
      }
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float sc[U];
        float mb = kNegBig;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          float d = 0.0f;
#pragma unroll
          for (int e = 0; e < EPL; ++e) d += qf[h][e] * kv[u].get(e);
          d = group_sum<LPR>(d);
          sc[u] = (r0 + u * STEP < hi) ? d : -INFINITY;
          mb = fmaxf(mb, sc[u]);
        }
        const float mn = fmaxf(m[h], mb);
        const float alpha = fast_exp2(m[h] - mn);
        m[h] = mn;
        l[h] *= alpha;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[h][e] *= alpha;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const float p = fast_exp2(sc[u] - mn);
          l[h] += p;
#pragma unroll
          for (int e = 0; e < EPL; ++e) acc[h][e] += p * vv[u].get(e);
        }
      }
    }

    // Merge the RPW lane groups of the wave (lanes with equal `col`).
#pragma unroll
    for (int off = LPR; off < 64; off *= 2) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float m2 = __shfl_xor(m[h], off, 64);
        const float l2 = __shfl_xor(l[h], off, 64);
        const float mn = fmaxf(m[h], m2);
        const float f1 = fast_exp2(m[h] - mn), f2 = fast_exp2(m2 - mn);
        l[h] = l[h] * f1 + l2 * f2;
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
          const float a2 = __shfl_xor(acc[h][e], off, 64);
          acc[h][e] = acc[h][e] * f1 + a2 * f2;
        }
        m[h] = mn;
      }
    }
    if (rsub == 0) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
#pragma unroll
        for (int e = 0; e < EPL; ++e) s_acc[(wave * G + h) * D + col * EPL + e] = acc[h][e];
        if (col == 0) {
          s_ml[(wave * G + h) * 2] = m[h];
          s_ml[(wave * G + h) * 2 + 1] = l[h];
        }
      }
    }
    __syncthreads();
    merge_waves_and_store<T, D, G>(a, s_acc, s_ml, w, b, g, whole);
    __syncthreads();                                // LDS is reused by the next cache
  });
}

// ---------------------------------------------------------------------------
// Matrix-core worker (bf16, G query heads per KV head).
// ---------------------------------------------------------------------------
__device__ __forceinline__ f32x4 mma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
#else
  (void)a;
  (void)b;
  return c;
#endif
}

typedef short i16x4 __attribute__((ext_vector_type(4)));

// Transposing LDS read of four bf16: within each 16-lane group, lane 4a+b
// receives element b of the 8-byte reads issued by lanes 4e+a (e = 0..3), as
// its element e.
__device__ __forceinline__ bf16x4 read_tr(const char* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  const i16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(const_cast<char*>(p)));
  return __builtin_bit_cast(bf16x4, r);
#else
  (void)p;
  return bf16x4{};
#endif
}

// acc + a + b with a, b in bf16 (v_dot2_f32_bf16 against (1, 1)).
__device__ __forceinline__ float dot2_ones(bf16 a, bf16 b, float acc) {
  typedef bf16 bf16x2 __attribute__((ext_vector_type(2)));
#if defined(__HIP_DEVICE_COMPILE__)
  const bf16x2 ab = {a, b};
  const bf16x2 ones = {bf16(1.0f), bf16(1.0f)};
  return __builtin_amdgcn_fdot2_f32_bf16(ab, ones, acc, false);
#else
  return acc + float(a) + float(b);
#endif
}

template <int D, int KEYS>
struct MmaTile {
  static constexpr int KT = KEYS;
  static constexpr int KS = D / 32;           // S steps over the head dimension
  static constexpr int DT = D / 16;           // 16-row output tiles of O^T
  static constexpr int RB = D * 2;            // bytes per cache row
  static constexpr int CPR = RB / 16;         // 16-byte chunks per row
  static constexpr int VLD = KT * CPR / 64;   // 16-byte V loads per lane per tile
  // V rows in LDS: 32-byte block c of row r sits at block c ^ swz(r), so the
  // 8 rows read by half a wave in one transposing read hit 64 distinct banks.
  __device__ __forceinline__ static int swz(int r) { return D == 128 ? (r & 7) : ((r >> 1) & 3); }
};

template <int D, int G>
__global__ void __launch_bounds__(kWaves * 64, mma_keys<G>() == 32 ? 3 : 2) decode_mma_kernel(DecodeArgs a) {
  using TL = MmaTile<D, mma_keys<G>()>;
  constexpr int KT = TL::KT, KS = TL::KS, DT = TL::DT, RB = TL::RB, CPR = TL::CPR, VLD = TL::VLD;
  constexpr int NST = KT / 16, NKS = KT / 32;   // 16-key score tiles, 32-key PV steps per wave tile
  static_assert(KT % 32 == 0, "whole 32-key steps");
  static_assert(G >= 1 && G <= 16, "query heads per KV head");
  static_assert(kWaves * (G * D + 2 * G) * 4 <= kWaves * KT * RB, "merge state fits the V buffers");

  // Per-wave V tiles; between caches the same memory holds the waves' states.
  __shared__ __attribute__((aligned(1024))) char sV[kWaves][KT * RB];
  float* s_acc = reinterpret_cast<float*>(&sV[0][0]);
  float* s_ml = s_acc + kWaves * G * D;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int w = static_cast<int>(blockIdx.x);
  const int n = lane & 15;        // query head column (MFMA N index)
  const int q4 = lane >> 4;       // 16-lane group
  char* vs = &sV[wave][0];

  // Transposing V reads (tile independent): lane 16*q4 + 4e + a reads row
  // 4*q4 + e (+ 16 for the upper half of a 32-key step, + 32 per step),
  // columns 16*dt + 4a .. +3.
  auto swk = [](int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); };
  int rd_off[DT];
  {
    const int vr = 4 * q4 + ((lane >> 2) & 3);
    const int a4 = lane & 3;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) rd_off[dt] = vr * RB + ((dt ^ TL::swz(vr)) << 5) + 8 * a4;
  }

  for_each_segment(a, w, [&](int b, int g, int lo, int hi, bool whole) {
    const int fill = cache_fill(a, b, g);
    if (fill == 0) return;                          // idle sequence
    hi = min(hi, fill);
    const int64_t row0 = int64_t(b) * a.rows_total + a.offset[g];
    const bf16* kb = static_cast<const bf16*>(a.kc) + row0 * D;
    const bf16* vb = static_cast<const bf16*>(a.vc) + row0 * D;

    // B = Q^T: lane holds query head n, dims 32*kk + 8*q4 .. +7 (zero past G).
    bf16x8 qop[KS];
    if (n < G) {
      const bf16* qp = static_cast<const bf16*>(a.q) + (int64_t(b) * a.hq + g * G + n) * D + 8 * q4;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) qop[kk] = *reinterpret_cast<const bf16x8*>(qp + 32 * kk);
    } else {
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) qop[kk] = bf16x8{};
    }

    f32x4 oacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    float m_run = kNegBig, l_run = 0.0f;
    const float c2 = a.scale_log2;

    for (int t0 = lo + wave * KT; t0 < hi; t0 += kWaves * KT) {
      // A = K rows t0 + 16*st + n, dims 32*kk + 8*q4 .. +7.  Rows past hi
      // re-read row hi - 1: every load is unconditional (no branch per load);
      // their scores are masked to -inf below, so their weights, and with
      // them the re-read V rows, contribute exactly 0.
      const int last = hi - 1;
      // K and V tiles in whole rows, 16-byte chunks: chunk u*64 + lane is
      // row m / CPR, chunk m % CPR (4 whole 256-byte rows per load at D = 128).
      bf16x8 kr[VLD], vr[VLD];
#pragma unroll
      for (int u = 0; u < VLD; ++u) {
        const int m = u * 64 + lane;
        const int key = min(t0 + m / CPR, last);
        kr[u] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(kb + int64_t(key) * D + (m % CPR) * 8));
      }
#pragma unroll
      for (int u = 0; u < VLD; ++u) {
        const int m = u * 64 + lane;
        const int key = min(t0 + m / CPR, last);
        vr[u] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(vb + int64_t(key) * D + (m % CPR) * 8));
      }
      // K passes through this wave's LDS buffer into the A-operand layout:
      // chunk c of row r sits at chunk position c ^ swk(r), so the 16 rows read
      // by a 16-lane group in one operand load hit distinct banks.
#pragma unroll
      for (int u = 0; u < VLD; ++u) {
        const int m = u * 64 + lane;
        const int r = m / CPR, c = m % CPR;
        *reinterpret_cast<bf16x8*>(vs + r * RB + ((c ^ swk(r)) << 4)) = kr[u];
      }
      bf16x8 kop[NST][KS];
#pragma unroll
      for (int st = 0; st < NST; ++st) {
        const int r = 16 * st + n;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
          kop[st][kk] = *reinterpret_cast<const bf16x8*>(vs + r * RB + (((4 * kk + q4) ^ swk(r)) << 4));
      }

      f32x4 s[NST];
#pragma unroll
      for (int st = 0; st < NST; ++st) {
        s[st] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) s[st] = mma16(kop[st][kk], qop[kk], s[st]);
      }
      if (t0 + KT > hi) {
#pragma unroll
        for (int st = 0; st < NST; ++st)
#pragma unroll
          for (int i = 0; i < 4; ++i) s[st][i] = (t0 + 16 * st + 4 * q4 + i < hi) ? s[st][i] : -INFINITY;
      }
      float tmax = -INFINITY;
#pragma unroll
      for (int st = 0; st < NST; ++st)
#pragma unroll
        for (int i = 0; i < 4; ++i) tmax = fmaxf(tmax, s[st][i]);
      tmax = max_xor<16>(tmax);
      tmax = max_xor<32>(tmax);
      const float m_new = fmaxf(m_run, tmax * c2);
      const float alpha = fast_exp2(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;

      // P^T operands of the 32-key steps: step ks takes score tiles
      // 2ks (keys 4*q4 + i) and 2ks + 1 (keys 16 + 4*q4 + i).
      bf16x8 pop[NKS];
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pop[ks][i] = static_cast<bf16>(fast_exp2(__builtin_fmaf(s[2 * ks][i], c2, -m_new)));
          pop[ks][4 + i] = static_cast<bf16>(fast_exp2(__builtin_fmaf(s[2 * ks + 1][i], c2, -m_new)));
        }
#pragma unroll
        for (int i = 0; i < 8; i += 2) l_run = dot2_ones(pop[ks][i], pop[ks][i + 1], l_run);
      }

      // V tile into this wave's LDS buffer (swizzled), then A = V^T fragments.
#pragma unroll
      for (int u = 0; u < VLD; ++u) {
        const int m = u * 64 + lane;
        const int r = m / CPR, c = m % CPR;
        *reinterpret_cast<bf16x8*>(vs + r * RB + (((c >> 1) ^ TL::swz(r)) << 5) + ((c & 1) << 4)) = vr[u];
      }
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const bf16x4 v0 = read_tr(vs + rd_off[dt] + (32 * ks) * RB);
          const bf16x4 v1 = read_tr(vs + rd_off[dt] + (32 * ks + 16) * RB);
          const bf16x8 va = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
          oacc[dt] = mma16(va, pop[ks], oacc[dt]);
        }
      }
    }

    // Row sums of the four 16-lane groups; the running max is already shared.
    l_run = sum_xor<16>(l_run);
    l_run = sum_xor<32>(l_run);
    __syncthreads();                                // every wave is done with its V tile
    if (n < G) {
      // Lane holds O^T rows 16*dt + 4*q4 + i of query head n.
      float* sa = s_acc + (wave * G + n) * D + 4 * q4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) *reinterpret_cast<f32x4*>(sa + 16 * dt) = oacc[dt];
      if (q4 == 0) {
        s_ml[(wave * G + n) * 2] = m_run;
        s_ml[(wave * G + n) * 2 + 1] = l_run;
      }
    }
    __syncthreads();
    merge_waves_and_store<bf16, D, G>(a, s_acc, s_ml, w, b, g, whole);
    __syncthreads();                                // LDS is reused by the next cache
  });
}

// ---------------------------------------------------------------------------
// Merge of the partials of every cache split over several workers:
// o = sum_p 2^(m_p - M) acc_p / sum_p 2^(m_p - M) l_p, M = max_p m_p.
// One work-group per (sequence, KV head, slice of at most 2 query heads): a
// whole group of 8 heads per work-group left a GQA merge to only B * H_kv
// work-groups, each reading all the partials of every head.  The partials of
// workers w0..w1 sit at consecutive slots w0 + cache .. w1 + cache.  Thread
// groups of TPR threads (one float4 of each of the slice's head rows) take
// every PG-th partial, so PG partial rows are read at once; the groups' sums
// meet in LDS.
// ---------------------------------------------------------------------------
template <int G>
constexpr int merge_heads() { return G <= 2 ? G : 2; }   // query heads per merge work-group

template <typename T, int D, int G>
__global__ void __launch_bounds__(256) decode_combine_kernel(DecodeArgs a) {
  constexpr int PS = D + kDecodePartPad;
  constexpr int V4 = D / 4;                  // float4 per head row
  constexpr int HS = merge_heads<G>();       // query heads per work-group
  constexpr int TPR = HS * V4;               // threads per partial (the slice's heads)
  constexpr int PG = 256 / TPR;              // partials read at once
  constexpr int CH = 256;                    // partials whose weights are staged at a time
  static_assert(TPR <= 256 && 256 % TPR == 0, "thread mapping");
  __shared__ float s_w[HS][CH];
  __shared__ float s_m[HS], s_inv[HS];
  __shared__ f32x4 s_red[256];
  const int bg = static_cast<int>(blockIdx.x) / (G / HS);
  const int h0 = (static_cast<int>(blockIdx.x) - bg * (G / HS)) * HS;   // first head of the slice
  const int b = bg / a.hkv, g = bg - b * a.hkv;
  if (cache_fill(a, b, g) == 0) return;
  const int64_t base = int64_t(b) * a.seq_keys + a.seg_start[g];
  const int64_t len = a.seg_start[g + 1] - a.seg_start[g];
  const int w0 = worker_of(a, base), w1 = worker_of(a, base + len - 1);
  if (w0 == w1) return;                       // written directly by its worker
  const int np = w1 - w0 + 1;
  const float* part0 = a.part + (int64_t(w0) + bg) * G * PS;
  auto at = [&](int p, int h) { return part0 + (int64_t(p) * G + h0 + h) * PS; };

  constexpr int kFastParts = fast_parts<G>();
  if (np <= kFastParts) {
    // Few partials (the common case): every thread of the first TPR loads
    // (m, l, its float4 of acc) of all of them at once and merges in one pass.
    if (threadIdx.x >= TPR) return;
    const int h = threadIdx.x / V4, d4 = threadIdx.x % V4;
    float mp[kFastParts], lp[kFastParts];
    f32x4 xp[kFastParts];
#pragma unroll
    for (int p = 0; p < kFastParts; ++p) {
      if (p < np) {
        const float* q = at(p, h);
        mp[p] = q[D];
        lp[p] = q[D + 1];
        xp[p] = *reinterpret_cast<const f32x4*>(q + 4 * d4);
      } else {
        mp[p] = kNegBig;
        lp[p] = 0.0f;
        xp[p] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      }
    }
    float mx = kNegBig;
#pragma unroll
    for (int p = 0; p < kFastParts; ++p) mx = fmaxf(mx, mp[p]);
    float ls = 0.0f;
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int p = 0; p < kFastParts; ++p) {
      const float wgt = fast_exp2(mp[p] - mx);
      ls += wgt * lp[p];
      acc += xp[p] * wgt;
    }
    acc *= 1.0f / ls;
    T* op = static_cast<T*>(a.o) + (int64_t(b) * a.hq + g * G + h0 + h) * D + 4 * d4;
#pragma unroll
    for (int e = 0; e < 4; ++e) op[e] = static_cast<T>(acc[e]);
    return;
  }

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int h = wave; h < HS; h += 4) {
    float mx = kNegBig;
    for (int p = lane; p < np; p += 64) mx = fmaxf(mx, at(p, h)[D]);
#pragma unroll
    for (int off = 32; off >= 1; off /= 2) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    float ls = 0.0f;
    for (int p = lane; p < np; p += 64) ls += fast_exp2(at(p, h)[D] - mx) * at(p, h)[D + 1];
#pragma unroll
    for (int off = 32; off >= 1; off /= 2) ls += __shfl_xor(ls, off, 64);
    if (lane == 0) {
      s_m[h] = mx;
      s_inv[h] = 1.0f / ls;
    }
  }
  __syncthreads();

  const int pg = threadIdx.x / TPR, j = threadIdx.x % TPR;
  const int h = j / V4, d4 = j % V4;
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int p0 = 0; p0 < np; p0 += CH) {
    const int nc = min(CH, np - p0);
    for (int t = threadIdx.x; t < HS * CH; t += 256) {
      const int hh = t / CH, c = t % CH;
      s_w[hh][c] = c < nc ? fast_exp2(at(p0 + c, hh)[D] - s_m[hh]) : 0.0f;
    }
    __syncthreads();
    const float* pp = at(p0, h) + 4 * d4;
    const int64_t stride = int64_t(G) * PS;
    int c = pg;
    for (; c + 3 * PG < nc; c += 4 * PG) {
      const f32x4 x0 = *reinterpret_cast<const f32x4*>(pp + (c + 0 * PG) * stride);
      const f32x4 x1 = *reinterpret_cast<const f32x4*>(pp + (c + 1 * PG) * stride);
      const f32x4 x2 = *reinterpret_cast<const f32x4*>(pp + (c + 2 * PG) * stride);
      const f32x4 x3 = *reinterpret_cast<const f32x4*>(pp + (c + 3 * PG) * stride);
      acc += x0 * s_w[h][c + 0 * PG] + x1 * s_w[h][c + 1 * PG];
      acc += x2 * s_w[h][c + 2 * PG] + x3 * s_w[h][c + 3 * PG];
    }
    for (; c < nc; c += PG) acc += *reinterpret_cast<const f32x4*>(pp + c * stride) * s_w[h][c];
    __syncthreads();
  }
  s_red[threadIdx.x] = acc;
  __syncthreads();
  if (pg != 0) return;
#pragma unroll
  for (int k = 1; k < PG; ++k) acc += s_red[k * TPR + j];
  acc *= s_inv[h];
  T* op = static_cast<T*>(a.o) + (int64_t(b) * a.hq + g * G + h0 + h) * D + 4 * d4;
#pragma unroll
  for (int e = 0; e < 4; ++e) op[e] = static_cast<T>(acc[e]);
}

// Resident work-groups of `kernel` on the current device: compute units x
// resident work-groups per unit (cached per device; host threads may launch
// concurrently, and they all store the same value).
int resident_groups(const void* kernel, std::atomic<int>* cache) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  const int known = cache[dev].load(std::memory_order_relaxed);
  if (known > 0) return known;
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) cus = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kWaves * 64, 0) != hipSuccess) per_cu = 1;
  const int groups = std::max(1, cus) * std::max(1, per_cu);
  cache[dev].store(groups, std::memory_order_relaxed);
  return groups;
}

template <typename T, int D, int G>
int launch_t(DecodeArgs a, void* stream) {
  constexpr bool kMma = sizeof(T) == 2 && G >= 2;
  const void* kernel;
  if constexpr (kMma) kernel = reinterpret_cast<const void*>(&decode_mma_kernel<D, G>);
  else kernel = reinterpret_cast<const void*>(&decode_valu_kernel<T, D, G>);
  static std::atomic<int> group_cache[64];
  int64_t workers = resident_groups(kernel, group_cache);
  workers = std::min<int64_t>(workers, (a.total + kDecodeMinKeys - 1) / kDecodeMinKeys);
  workers = std::max<int64_t>(1, std::min<int64_t>(workers, kMaxDecodeWorkers));
  a.workers = static_cast<int32_t>(workers);
  a.per_worker = a.total / workers;
  a.rem = static_cast<int32_t>(a.total % workers);
  void* args[] = {&a};
  hipError_t e = hipLaunchKernel(kernel, dim3(static_cast<unsigned>(workers)), dim3(kWaves * 64), args, 0,
                                 static_cast<hipStream_t>(stream));
  if (e != hipSuccess || workers == 1) return static_cast<int>(e);   // one worker: every cache is whole
  e = hipLaunchKernel(reinterpret_cast<const void*>(&decode_combine_kernel<T, D, G>),
                      dim3(static_cast<unsigned>(a.batch * a.hkv * (G / merge_heads<G>()))), dim3(256), args, 0,
                      static_cast<hipStream_t>(stream));
  return static_cast<int>(e);
}

template <typename T, int D>
int launch_g(const DecodeArgs& a, int group, void* stream) {
  switch (group) {
    case 1: return launch_t<T, D, 1>(a, stream);
    case 2: return launch_t<T, D, 2>(a, stream);
    case 4: return launch_t<T, D, 4>(a, stream);
    case 8: return launch_t<T, D, 8>(a, stream);
    default: return static_cast<int>(hipErrorInvalidValue);
  }
}

}  // namespace

int launch_decode(DecodeArgs a, int dtype, int head_dim, int group, void* stream) {
  if (dtype == MOA_BF16) {
    if (head_dim == 128) return launch_g<bf16, 128>(a, group, stream);
    if (head_dim == 64) return launch_g<bf16, 64>(a, group, stream);
  } else {
    if (head_dim == 128) return launch_g<float, 128>(a, group, stream);
    if (head_dim == 64) return launch_g<float, 64>(a, group, stream);
  }
  return static_cast<int>(hipErrorInvalidValue);
}

}  // namespace moa
