// Decode attention over per-head static KV caches of different lengths
// (paper Appendix "Efficiency Experiment Setup": one new query per sequence
// against caches whose length differs across heads).
//
// After the token at position t is appended, the filled slots of KV head g
// are exactly the keys visible to t (sinks + the last w_g positions), so no
// mask is applied: o = softmax(scale * q K^T) V over slots [0, fill_g),
// fill_g = min(t + 1, s + w_g).  Slot order does not matter.
//
// Split-K: every (sequence, KV head) cache is cut into chunks of `chunk`
// slots; one work-group handles one chunk for all G query heads of the KV
// head, so each K/V byte is read from HBM once.  Work-groups stream K/V with
// 16-byte loads (LPR lanes cover one row), keep an online softmax per lane
// group (base-2 exponent, scale folded into q), merge lane groups and waves,
// and either write o directly (single chunk) or a partial (m, l, acc).  A
// second, small kernel merges the partials of multi-chunk caches; the kernel
// boundary makes the partials visible across the chip's L2 slices without
// any in-kernel cache maintenance.
#include "moa_device.h"

namespace moa {

namespace {

constexpr int kWaves = 4;

template <typename T, int D, int G>
__global__ void __launch_bounds__(256) decode_kernel(DecodeArgs a) {
  constexpr int EPL = Vec16<T>::N;    // elements per lane
  constexpr int LPR = D / EPL;        // lanes per cache row
  constexpr int RPW = 64 / LPR;       // rows per wave per load step
  constexpr int U = 8;                // load steps in flight per iteration
  constexpr int STEP = kWaves * RPW;  // rows per block per load step

  __shared__ float s_acc[kWaves][G][D];
  __shared__ float s_ml[kWaves][G][2];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int rsub = lane / LPR;
  const int col = lane % LPR;

  const int b = blockIdx.x / a.items_per_seq;
  const int item = blockIdx.x - b * a.items_per_seq;
  const ItemGeometry geo = locate_item(a, b, item);
  if (geo.g < 0) return;                          // past this sequence's items
  const int g = geo.g;
  const int c = geo.c;
  const int nchunk = geo.nchunk;
  const int lo = c * a.chunk;
  const int hi = min(lo + a.chunk, geo.fill);

  const int64_t row0 = int64_t(b) * a.rows_total + a.offset[g];
  const T* kbase = static_cast<const T*>(a.kc) + row0 * D + col * EPL;
  const T* vbase = static_cast<const T*>(a.vc) + row0 * D + col * EPL;

  float qf[G][EPL];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const T* qp = static_cast<const T*>(a.q) + (int64_t(b) * a.hq + g * G + h) * D + col * EPL;
    const Vec16<T> qv = load16(qp);
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
        kv[u] = load16(kbase + int64_t(r) * D);
        vv[u] = load16(vbase + int64_t(r) * D);
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

  // Merge the RPW lane groups of this wave (lanes with equal `col`).
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
      for (int e = 0; e < EPL; ++e) s_acc[wave][h][col * EPL + e] = acc[h][e];
      if (col == 0) {
        s_ml[wave][h][0] = m[h];
        s_ml[wave][h][1] = l[h];
      }
    }
  }
  __syncthreads();

  // Merge waves: each thread owns (h, d) outputs.
  const int64_t item_global = int64_t(b) * a.items_per_seq + item;
  for (int idx = threadIdx.x; idx < G * D; idx += blockDim.x) {
    const int h = idx / D, d = idx % D;
    float mx = kNegBig;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) mx = fmaxf(mx, s_ml[w][h][0]);
    float lsum = 0.0f, asum = 0.0f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float f = fast_exp2(s_ml[w][h][0] - mx);
      lsum += s_ml[w][h][1] * f;
      asum += s_acc[w][h][d] * f;
    }
    if (nchunk == 1) {
      T* op = static_cast<T*>(a.o) + (int64_t(b) * a.hq + g * G + h) * D + d;
      *op = static_cast<T>(asum / lsum);
    } else {
      float* pp = a.part + (item_global * G + h) * (D + 2);
      pp[d] = asum;
      if (d == 0) {
        pp[D] = mx;
        pp[D + 1] = lsum;
      }
    }
  }
}

// Merges the split-K partials of every (sequence, KV head) with more than one
// chunk: o = sum_c w_c acc_c with w_c = 2^(m_c - M) / sum_c' 2^(m_c' - M) l_c',
// M = max_c m_c.  The per-chunk (m, l) are staged in LDS once (the plan keeps
// every cache within kMaxMergeChunks chunks); the weighted sum over chunks
// then issues independent, coalesced loads per output.

template <typename T, int D, int G>
__global__ void __launch_bounds__(256) decode_combine_kernel(DecodeArgs a) {
  __shared__ float s_w[G][kMaxMergeChunks];
  __shared__ float s_inv[G];
  const int b = blockIdx.x / a.hkv;
  const int g = blockIdx.x - b * a.hkv;
  int nchunk, first_item;
  if (a.positions == nullptr) {
    nchunk = a.item_start[g + 1] - a.item_start[g];
    first_item = a.item_start[g];
  } else {
    const int pos = a.positions[b];
    first_item = 0;
    for (int h = 0; h < g; ++h) {
      const int f = min(pos + 1, a.capacity[h]);
      first_item += f > 0 ? (f + a.chunk - 1) / a.chunk : 0;
    }
    const int f = min(pos + 1, a.capacity[g]);
    nchunk = f > 0 ? (f + a.chunk - 1) / a.chunk : 0;
  }
  if (nchunk <= 1) return;
  const int64_t first = int64_t(b) * a.items_per_seq + first_item;
  // 1) raw running maxima into LDS
  for (int t = threadIdx.x; t < G * nchunk; t += blockDim.x) {
    const int h = t / nchunk, c = t % nchunk;
    s_w[h][c] = a.part[((first + c) * G + h) * (D + 2) + D];
  }
  __syncthreads();
  // 2) one wave per query head: weights 2^(m_c - M) and 1 / sum_c 2^(m_c - M) l_c
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int h = wave; h < G; h += blockDim.x / 64) {
    float mx = kNegBig;
    for (int c = lane; c < nchunk; c += 64) mx = fmaxf(mx, s_w[h][c]);
#pragma unroll
    for (int off = 32; off >= 1; off /= 2) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    float lsum = 0.0f;
    for (int c = lane; c < nchunk; c += 64) {
      const float f = fast_exp2(s_w[h][c] - mx);
      s_w[h][c] = f;
      lsum += f * a.part[((first + c) * G + h) * (D + 2) + D + 1];
    }
#pragma unroll
    for (int off = 32; off >= 1; off /= 2) lsum += __shfl_xor(lsum, off, 64);
    if (lane == 0) s_inv[h] = 1.0f / lsum;
  }
  __syncthreads();
  // 3) weighted sum of the partial accumulators
  for (int idx = threadIdx.x; idx < G * D; idx += blockDim.x) {
    const int h = idx / D, d = idx % D;
    const float* pp = a.part + (first * G + h) * (D + 2) + d;
    const int64_t stride = int64_t(G) * (D + 2);
    float acc0 = 0.0f, acc1 = 0.0f, acc2 = 0.0f, acc3 = 0.0f;
    int c = 0;
    for (; c + 4 <= nchunk; c += 4) {
      acc0 += pp[(c + 0) * stride] * s_w[h][c + 0];
      acc1 += pp[(c + 1) * stride] * s_w[h][c + 1];
      acc2 += pp[(c + 2) * stride] * s_w[h][c + 2];
      acc3 += pp[(c + 3) * stride] * s_w[h][c + 3];
    }
    for (; c < nchunk; ++c) acc0 += pp[c * stride] * s_w[h][c];
    T* op = static_cast<T*>(a.o) + (int64_t(b) * a.hq + g * G + h) * D + d;
    *op = static_cast<T>(((acc0 + acc1) + (acc2 + acc3)) * s_inv[h]);
  }
}

template <typename T, int D, int G>
int launch_t(const DecodeArgs& a, void* stream) {
  const int64_t blocks = int64_t(a.batch) * a.items_per_seq;
  DecodeArgs copy = a;
  void* args[] = {&copy};
  hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(&decode_kernel<T, D, G>),
                                 dim3(static_cast<unsigned>(blocks)), dim3(256), args, 0,
                                 static_cast<hipStream_t>(stream));
  if (e != hipSuccess || (a.positions == nullptr && blocks == int64_t(a.batch) * a.hkv))
    return static_cast<int>(e);  // no cache spans several chunks
  e = hipLaunchKernel(reinterpret_cast<const void*>(&decode_combine_kernel<T, D, G>),
                      dim3(static_cast<unsigned>(a.batch * a.hkv)), dim3(256), args, 0,
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

int launch_decode(const DecodeArgs& a, int dtype, int head_dim, int group, void* stream) {
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
