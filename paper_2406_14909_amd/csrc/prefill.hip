// Prefill attention with a per-KV-head banded-plus-sink causal mask (paper
// Sec. 2.1, Eq. 1, with the Sec. 3.2 span: sink prefix + diagonal band of
// width w_g).  Query i sees key j iff j <= i and (j < s or i - j < w_g).
//
// One work-group = 4 waves = 128 query rows of one (sequence, query head);
// each wave owns 32 rows.  The work-group walks only the 64-key tiles that
// intersect the sink prefix or the band of its rows; every other tile is
// skipped without being read.  K and V tiles are staged in LDS (V stored
// transposed) and shared by the 4 waves.
//
// Matrix-core formulation (CDNA4 32x32 MFMA; bf16 32x32x16, fp32 32x32x2):
//   S^T = K Q^T  : A = K tile rows (keys), B = Q^T kept in registers.
//                  Output lane l holds the scores of query row l % 32 for
//                  16 keys, so the row softmax needs one cross-lane step.
//   O^T += V^T P^T : B = P^T taken straight from the score registers
//                  (converted to the input type), A = V^T read from LDS.
// The key order inside each 16-key MFMA step is permuted identically on both
// operands, which leaves the sum unchanged.
// Softmax is online (running max m and sum l per row) in base 2 with the
// scale folded into the exponent; the mask is evaluated only on tiles that
// are not entirely visible to the wave's rows.
#include "moa_device.h"

namespace moa {

namespace {

constexpr int BM = 128;   // query rows per work-group
constexpr int BN = 64;    // keys per tile
constexpr int NW = 4;     // waves per work-group

template <typename T> struct Mma;

template <> struct Mma<bf16> {
  static constexpr int K = 16;                 // reduction depth per instruction
  static constexpr int KPAD = 8;               // LDS row padding (elements)
  static constexpr int VPAD = 4;
  typedef bf16x8 frag;
  __device__ __forceinline__ static f32x16 mma(const frag& a, const frag& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

template <> struct Mma<float> {
  static constexpr int K = 2;
  static constexpr int KPAD = 4;
  static constexpr int VPAD = 4;
  typedef float frag;
  __device__ __forceinline__ static f32x16 mma(const frag& a, const frag& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

// Fragment of K / Q for reduction step kk: row `row` of a [*, ld] array,
// elements kk*K + (lane/32)*(K/2) ... (+K/2).
__device__ __forceinline__ bf16x8 load_frag(const bf16* base, int kk, int half) {
  return *reinterpret_cast<const bf16x8*>(base + kk * 16 + half * 8);
}
__device__ __forceinline__ float load_frag(const float* base, int kk, int half) {
  return base[kk * 2 + half];
}

template <typename T, int D>
__global__ void __launch_bounds__(256) prefill_kernel(PrefillArgs a) {
  using M = Mma<T>;
  constexpr int KS = D / M::K;            // MFMA steps over the head dimension
  constexpr int LDK = D + M::KPAD;        // LDS row stride of the K tile
  constexpr int LDV = BN + M::VPAD;       // LDS row stride of the V^T tile
  constexpr int EPL = Vec16<T>::N;        // elements per 16-byte load
  constexpr int CPR = D / EPL;            // 16-byte chunks per row

  __shared__ __attribute__((aligned(16))) T sK[BN * LDK];
  __shared__ __attribute__((aligned(16))) T sV[D * LDV];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int lrow = lane & 31;
  const int half = lane >> 5;

  // Work item: query tiles from last to first (heaviest first), then query
  // heads in decreasing window order, then sequences.
  const int per_tile = a.batch * a.hq;
  const int qt = a.n_qtiles - 1 - static_cast<int>(blockIdx.x / per_tile);
  const int rem = static_cast<int>(blockIdx.x % per_tile);
  const int h = a.head_order[rem / a.batch];
  const int b = rem % a.batch;
  const int g = h / a.group;
  const int64_t n = a.n;
  const int w = a.window[g];
  const int s = a.num_sink;

  const int i0 = qt * BM;
  const int i1 = static_cast<int>(min(n, int64_t(i0 + BM)));   // exclusive
  const int iw0 = i0 + wave * 32;                                // this wave's rows
  const int iw1 = min(i1, iw0 + 32);
  const bool wave_active = iw0 < i1;

  // Tiles to visit: sink tiles [0, ta) then band tiles [tb, tl].
  const int ta = (min(s, i1) + BN - 1) / BN;
  const int tl = (i1 - 1) / BN;
  const int tb = max(ta, max(0, i0 - w + 1) / BN);
  const int ntiles = ta + max(0, tl - tb + 1);

  const int64_t q_row_stride = int64_t(a.hq) * D;
  const int64_t kv_row_stride = int64_t(a.hkv) * D;
  const T* qg = static_cast<const T*>(a.q) + (int64_t(b) * n * a.hq + h) * D;
  const T* kg = static_cast<const T*>(a.k) + (int64_t(b) * n * a.hkv + g) * D;
  const T* vg = static_cast<const T*>(a.v) + (int64_t(b) * n * a.hkv + g) * D;

  // Q^T fragments of this lane's query row (zeros past the end).
  typename M::frag qf[KS];
  {
    const int i = iw0 + lrow;
    if (wave_active && i < i1) {
      const T* qrow = qg + int64_t(i) * q_row_stride;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) qf[kk] = load_frag(qrow, kk, half);
    } else {
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) qf[kk] = typename M::frag{};
    }
  }

  f32x16 oacc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt) oacc[dt] = f32x16{};
  float m_run = kNegBig, l_run = 0.0f;
  const int my_row = iw0 + lrow;

  for (int it = 0; it < ntiles; ++it) {
    const int t = it < ta ? it : tb + (it - ta);
    const int j0 = t * BN;

    // Stage K (row-major) and V (transposed) of keys j0 .. j0+BN-1.
    __syncthreads();
    for (int idx = threadIdx.x; idx < BN * CPR; idx += blockDim.x) {
      const int r = idx / CPR, cc = idx % CPR;
      const int j = j0 + r;
      Vec16<T> kx, vx;
      if (j < n) {
        kx = load16(kg + int64_t(j) * kv_row_stride + cc * EPL);
        vx = load16(vg + int64_t(j) * kv_row_stride + cc * EPL);
      } else {
        kx = zero16<T>();
        vx = zero16<T>();
      }
      store16(sK + r * LDK + cc * EPL, kx);
#pragma unroll
      for (int e = 0; e < EPL; ++e) sV[(cc * EPL + e) * LDV + r] = vx.v[e];
    }
    __syncthreads();

    if (!wave_active) continue;
    // Does any (row, key) pair of this wave fall inside the mask?
    const bool any_causal = j0 <= iw1 - 1;
    const bool any_vis = any_causal && (j0 < s || (iw0 - (j0 + BN - 1)) < w);
    if (!any_vis) continue;
    const bool all_vis = (j0 + BN - 1 <= iw0) && (iw1 - iw0 == 32) &&
                         ((j0 + BN <= s) || ((iw1 - 1) - j0 < w));

    // S^T = K Q^T for two 32-key sub-tiles.
    f32x16 sacc[2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      sacc[sub] = f32x16{};
      const T* krow = sK + (sub * 32 + lrow) * LDK;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) sacc[sub] = M::mma(load_frag(krow, kk, half), qf[kk], sacc[sub]);
    }

    // Scale into base 2, mask, tile row max.
    float tmax = -INFINITY;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float x = sacc[sub][r] * a.scale_log2;
        if (!all_vis) {
          const int j = j0 + sub * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
          const bool vis = (j <= my_row) && (j < s || my_row - j < w) && (my_row < i1);
          x = vis ? x : -INFINITY;
        }
        sacc[sub][r] = x;
        tmax = fmaxf(tmax, x);
      }
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float m_new = fmaxf(m_run, tmax);
    const float alpha = fast_exp2(m_run - m_new);
    m_run = m_new;

    float psum = 0.0f;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(sacc[sub][r] - m_new);
        sacc[sub][r] = p;
        psum += p;
      }
    }
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) oacc[dt] *= alpha;

    // O^T += V^T P^T.
    if constexpr (sizeof(T) == 2) {
      bf16x8 pf[2][2];
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int e = 0; e < 8; ++e) pf[sub][c][e] = static_cast<bf16>(sacc[sub][8 * c + e]);
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) {
        const T* vrow = sV + (dt * 32 + lrow) * LDV;
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const int kb = sub * 32 + 16 * c + half * 4;
            const bf16x4 lo4 = *reinterpret_cast<const bf16x4*>(vrow + kb);
            const bf16x4 hi4 = *reinterpret_cast<const bf16x4*>(vrow + kb + 8);
            const bf16x8 vf = __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7);
            oacc[dt] = M::mma(vf, pf[sub][c], oacc[dt]);
          }
        }
      }
    } else {
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) {
        const T* vrow = sV + (dt * 32 + lrow) * LDV;
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = sub * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
            oacc[dt] = M::mma(vrow[key], sacc[sub][r], oacc[dt]);
          }
        }
      }
    }
  }

  if (!wave_active || my_row >= i1) return;
  const float inv_l = 1.0f / l_run;
  T* orow = static_cast<T*>(a.o) + (int64_t(b) * n * a.hq + h) * D + int64_t(my_row) * q_row_stride;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
    for (int grp = 0; grp < 4; ++grp) {
      const int d0 = dt * 32 + grp * 8 + half * 4;
      if constexpr (sizeof(T) == 2) {
        bf16x4 outv;
#pragma unroll
        for (int e = 0; e < 4; ++e) outv[e] = static_cast<bf16>(oacc[dt][grp * 4 + e] * inv_l);
        *reinterpret_cast<bf16x4*>(orow + d0) = outv;
      } else {
        f32x4 outv;
#pragma unroll
        for (int e = 0; e < 4; ++e) outv[e] = oacc[dt][grp * 4 + e] * inv_l;
        *reinterpret_cast<f32x4*>(orow + d0) = outv;
      }
    }
  }
}

template <typename T, int D>
int launch_t(const PrefillArgs& a, void* stream) {
  const int64_t blocks = int64_t(a.n_qtiles) * a.batch * a.hq;
  PrefillArgs copy = a;
  void* args[] = {&copy};
  return static_cast<int>(hipLaunchKernel(reinterpret_cast<const void*>(&prefill_kernel<T, D>),
                                          dim3(static_cast<unsigned>(blocks)), dim3(NW * 64), args, 0,
                                          static_cast<hipStream_t>(stream)));
}

}  // namespace

int launch_prefill(const PrefillArgs& a, int dtype, int head_dim, void* stream) {
  if (dtype == MOA_BF16) {
    if (head_dim == 128) return launch_t<bf16, 128>(a, stream);
    if (head_dim == 64) return launch_t<bf16, 64>(a, stream);
  } else {
    if (head_dim == 128) return launch_t<float, 128>(a, stream);
    if (head_dim == 64) return launch_t<float, 64>(a, stream);
  }
  return static_cast<int>(hipErrorInvalidValue);
}

}  // namespace moa
