// Attention-influence profiling (paper Sec. 3.3 "Attention Influence
// Profiling", Eq. 3; Appendix "Derivation of Attention Influence"), fused.
//
// For dense causal attention A = softmax(scale * Q K^T) of every query head
// and a loss that reaches A through O = A V, dL/dA = dO V^T.  The influence
// of masking A_ij (first-order change of the loss, row renormalised) is
//     E_ij = -A_ij / (1 - A_ij) * (G_ij - D_i),   G = dO V^T,
//     D_i  = sum_n G_in A_in,
// and the profile keeps only its mean over 64 x 64 blocks and over the batch
// of calibration items.  Neither A nor G is ever stored: per 128-row tile of
// one query head the work-group makes two passes over the causal key tiles,
//   pass 1: S = Q K^T, dP = dO V^T; online row max m, row sum l of
//           e = exp(S - m) and u = sum e * dP, so D_i = u / l and
//           log-sum-exp = m + log l;
//   pass 2: S and dP again, A / (1 - A) = 1 / (exp(lse - S) - 1), E as
//           above, summed per (64-row block, 64-key block) into LDS,
// for every calibration item in turn, then writes the block means.
//
// Matrix-core formulation (CDNA4 32x32x16 bf16 MFMA): S^T = K Q^T and
// dP^T = V dO^T with the K / V tile rows as the A operand (double-buffered in
// LDS, filled by asynchronous buffer-to-LDS loads one tile ahead, 16-byte
// chunks XOR-swizzled per row) and Q^T / dO^T kept in registers, so lane l
// holds query row l % 32 for 16 keys and row reductions need one cross-lane
// step.
// Where 1 - A_ij of a row's largest weight is not resolved in fp32 (the
// row's other weights sum to less than about 2^-22 of it, e.g. row 0) the
// influence of the whole row is reported as 0.
#include "moa_device.h"

namespace moa {

namespace {

constexpr int IBM = 128;   // query rows per work-group
constexpr int IBN = 64;    // keys per tile (= profiling block)
constexpr int INW = 4;     // waves per work-group
constexpr int kMaxBlocks = kMaxInfluenceN / kInfluenceBlock;
static_assert(IBN == kInfluenceBlock, "one key tile per profiling block");

__device__ __forceinline__ f32x16 mma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
#else
  (void)a;
  (void)b;
  return c;
#endif
}

__device__ __forceinline__ float wave_sum(float x) {
  x = group_sum<16>(x);
  x += __shfl_xor(x, 16, 64);
  x += __shfl_xor(x, 32, 64);
  return x;
}

template <int D>
__global__ void __launch_bounds__(INW * 64, 2) influence_kernel(InfluenceArgs a) {
  constexpr int KS = D / 16;              // MFMA steps over the head dimension
  constexpr int RB = D * 2;               // bytes per K / V row
  constexpr int CPR = RB / 16;            // 16-byte chunks per row
  constexpr int TILE = IBN * RB;          // one K or V tile (rows unpadded)
  constexpr int DPW = TILE / 1024 / INW;  // 1 KB direct-to-LDS loads per wave per tile

  __shared__ __attribute__((aligned(1024))) char sK[2][TILE];
  __shared__ __attribute__((aligned(1024))) char sV[2][TILE];
  __shared__ float s_part[INW][kMaxBlocks];     // per-wave block sums

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lrow = lane & 31;
  const int half = lane >> 5;

  // Heaviest row tiles (most key tiles) first.
  const int h = static_cast<int>(blockIdx.x) % a.hq;
  const int t = a.n_tiles - 1 - static_cast<int>(blockIdx.x) / a.hq;
  const int g = h / a.group;
  const int n = a.n;
  const int i0 = t * IBM;
  const int i1 = min(n, i0 + IBM);
  const int iw0 = i0 + wave * 32;
  const bool wave_active = iw0 < i1;
  const int iw_last = min(i1, iw0 + 32) - 1;
  const int my_row = iw0 + lrow;
  const bool row_ok = wave_active && my_row < n;
  const int ntiles = (i1 - 1) / IBN + 1;
  const float c2 = a.scale_log2;

  for (int x = threadIdx.x; x < INW * kMaxBlocks; x += INW * 64) (&s_part[0][0])[x] = 0.0f;

  const int64_t q_stride = int64_t(a.hq) * D;     // elements between consecutive tokens
  const uint32_t kv_row_bytes = uint32_t(a.hkv) * RB;

  // K / V rows in LDS: 16-byte chunk c of row r sits at chunk position
  // c ^ swz(r), so the 16 rows read together by an MFMA operand load hit 16
  // different bank groups.  Tiles arrive by asynchronous buffer-to-LDS loads:
  // load i of this wave writes tile bytes [(wave * DPW + i) * 1024, +1024),
  // lane L's 16 bytes landing at chunk m = (wave * DPW + i) * 64 + L (row
  // m / CPR, position m % CPR) and carrying global chunk position ^ swz(row).
  auto swz = [](int r) { return CPR >= 16 ? (r & 15) : ((r >> 1) & 7); };
  uint32_t src[DPW];
  int src_row[DPW];
#pragma unroll
  for (int i = 0; i < DPW; ++i) {
    const int m = (wave * DPW + i) * 64 + lane;
    const int r = m / CPR, pos = m % CPR;
    src_row[i] = r;
    src[i] = uint32_t(r) * kv_row_bytes + uint32_t(pos ^ swz(r)) * 16u;
  }
  // Tile `it` of item b into buffer `buf`.  The buffer resource spans exactly
  // the tile's real key rows; rows past n re-read row n - 1 (never visible).
  auto issue = [&](int b, int it, int buf) {
    const int j0 = it * IBN;
    const int rows = min(IBN, n - j0);
    const int64_t first = (int64_t(b) * n + j0) * a.hkv + g;      // row j0 of head g, in rows of D
    const i32x4 kd = make_desc(static_cast<const char*>(a.k) + first * RB, uint32_t(rows - 1) * kv_row_bytes + RB);
    const i32x4 vd = make_desc(static_cast<const char*>(a.v) + first * RB, uint32_t(rows - 1) * kv_row_bytes + RB);
#pragma unroll
    for (int i = 0; i < DPW; ++i) {
      const uint32_t off = src_row[i] < rows ? src[i] : src[i] - uint32_t(src_row[i] - (rows - 1)) * kv_row_bytes;
      dma16_async(kd, off, &sK[buf][(wave * DPW + i) * 1024]);
      dma16_async(vd, off, &sV[buf][(wave * DPW + i) * 1024]);
    }
  };

  // S^T and dP^T of one 64-key tile (two 32-key halves), from LDS buffer buf.
  auto products = [&](int buf, const bf16x8* qf, const bf16x8* df, f32x16* sacc, f32x16* dacc) {
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      sacc[sub] = f32x16{};
      dacc[sub] = f32x16{};
      const int r = sub * 32 + lrow;
      const char* kb = &sK[buf][r * RB];
      const char* vb = &sV[buf][r * RB];
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const int off = ((2 * kk + half) ^ swz(r)) * 16;
        sacc[sub] = mma32(*reinterpret_cast<const bf16x8*>(kb + off), qf[kk], sacc[sub]);
        dacc[sub] = mma32(*reinterpret_cast<const bf16x8*>(vb + off), df[kk], dacc[sub]);
      }
    }
  };
  // Register r of half-tile `sub` holds, for this lane's query row, the key
  // j0 + sub * 32 + (r / 4) * 8 + half * 4 + r % 4 (32x32 MFMA output layout).

  int cnt = 0;                                      // tiles consumed so far (buffer parity)
  for (int b = 0; b < a.batch; ++b) {
    bf16x8 qf[KS], df[KS];
    if (row_ok) {
      const bf16* qr = static_cast<const bf16*>(a.q) + (int64_t(b) * n + my_row) * q_stride + h * D + 8 * half;
      const bf16* dr = static_cast<const bf16*>(a.dout) + (int64_t(b) * n + my_row) * q_stride + h * D + 8 * half;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        qf[kk] = *reinterpret_cast<const bf16x8*>(qr + 16 * kk);
        df[kk] = *reinterpret_cast<const bf16x8*>(dr + 16 * kk);
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        qf[kk] = bf16x8{};
        df[kk] = bf16x8{};
      }
    }
    issue(b, 0, cnt & 1);
    // Q / dO are waited for here, once: the tile loads are invisible to the
    // compiler's wait tracking, which would otherwise wait inside the loop.
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)

    // Running state per query row (both wave halves hold the same row):
    // mr = largest raw score so far, l = sum of exp2(c2 * s - c2 * mr),
    // u = sum of those weights times dP.
    float mr = kNegBig, l = 0.0f, u = 0.0f, lse2 = 0.0f, drow = 0.0f;
    for (int pass = 0; pass < 2; ++pass) {
      for (int it = 0; it < ntiles; ++it, ++cnt) {
        __builtin_amdgcn_s_waitcnt(0x0F70);     // this wave's loads of tile `it` have landed
        __syncthreads();                        // ... everyone's; the other buffer is free
        if (it + 1 < ntiles) issue(b, it + 1, (cnt + 1) & 1);
        else if (pass == 0) issue(b, 0, (cnt + 1) & 1);
        const int buf = cnt & 1;
        const int j0 = it * IBN;
        if (!wave_active || j0 > iw_last) continue;
        f32x16 sacc[2], dacc[2];
        products(buf, qf, df, sacc, dacc);
        // Only a tile reaching past the wave's first row holds keys after
        // some of its rows; there a hidden score becomes -inf, which both
        // passes below turn into a zero weight and a zero influence.
        if (j0 + IBN - 1 > iw0) {
          const int lim = my_row - j0 - half * 4;
#pragma unroll
          for (int sub = 0; sub < 2; ++sub)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              if (sub * 32 + (r >> 2) * 8 + (r & 3) > lim) sacc[sub][r] = -INFINITY;
        }
        if (pass == 0) {
          float tmax = -INFINITY;
#pragma unroll
          for (int sub = 0; sub < 2; ++sub)
#pragma unroll
            for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, sacc[sub][r]);
          tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
          const float mr_new = fmaxf(mr, tmax);
          const float m_new = mr_new * c2;          // scale > 0: the scaled maximum
          const float alpha = fast_exp2(mr * c2 - m_new);
          l *= alpha;
          u *= alpha;
#pragma unroll
          for (int sub = 0; sub < 2; ++sub)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const float e = fast_exp2(__builtin_fmaf(sacc[sub][r], c2, -m_new));
              l += e;
              u = __builtin_fmaf(e, dacc[sub][r], u);
            }
          mr = mr_new;
        } else {
          // A / (1 - A) = 1 / (2^(lse2 - c2 s) - 1), so the tile's influence
          // sum is  sum -ratio * (dP - D) = D * sum ratio - sum ratio * dP.
          float acc_dp = 0.0f, acc_r = 0.0f;
#pragma unroll
          for (int sub = 0; sub < 2; ++sub)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const float inv_p = fast_exp2(__builtin_fmaf(sacc[sub][r], -c2, lse2));
              const float ratio = __builtin_amdgcn_rcpf(inv_p - 1.0f);
              acc_dp = __builtin_fmaf(ratio, dacc[sub][r], acc_dp);
              acc_r += ratio;
            }
          const float esum = wave_sum(__builtin_fmaf(drow, acc_r, -acc_dp));
          if (lane == 0) s_part[wave][it] += esum;
        }
      }
      if (pass == 0) {
        l += __shfl_xor(l, 32, 64);
        u += __shfl_xor(u, 32, 64);
        lse2 = mr * c2 + __log2f(l);
        drow = u / l;
        // 1 / A of the row's largest weight, computed exactly as the second
        // pass will.  Where it lies within two fp32 ulps of 1, 1 - A is not
        // resolved: the whole row is reported as 0 (lse2 = +inf makes every
        // ratio 0), as is a row past n.  Elsewhere every key's 1 / A exceeds
        // 1, so no ratio divides by zero.
        const float inv_p_max = fast_exp2(__builtin_fmaf(mr, -c2, lse2));
        if (!row_ok || !(inv_p_max - 1.0f >= 0x1p-22f)) lse2 = INFINITY;
      }
    }
  }
  __syncthreads();

  // Block means of the (up to) two 64-row blocks of this tile; blocks above
  // the diagonal are 0.
  const int nb = a.nb;
  for (int x = threadIdx.x; x < 2 * nb; x += INW * 64) {
    const int ib = x / nb, jb = x - ib * nb;
    const int I = 2 * t + ib;
    if (I * IBN >= n) continue;
    float val = 0.0f;
    if (jb <= I) {
      const int rows = min(IBN, n - I * IBN), cols = min(IBN, n - jb * IBN);
      val = (s_part[2 * ib][jb] + s_part[2 * ib + 1][jb]) / (float(a.batch) * float(rows) * float(cols));
    }
    a.ebar[(int64_t(h) * nb + I) * nb + jb] = val;
  }
}

}  // namespace

int launch_influence(const InfluenceArgs& a, int head_dim, void* stream) {
  InfluenceArgs copy = a;
  void* args[] = {&copy};
  const void* kernel;
  if (head_dim == 128) kernel = reinterpret_cast<const void*>(&influence_kernel<128>);
  else if (head_dim == 64) kernel = reinterpret_cast<const void*>(&influence_kernel<64>);
  else return static_cast<int>(hipErrorInvalidValue);
  const unsigned blocks = static_cast<unsigned>(a.hq) * static_cast<unsigned>(a.n_tiles);
  return static_cast<int>(hipLaunchKernel(kernel, dim3(blocks), dim3(INW * 64), args, 0,
                                          static_cast<hipStream_t>(stream)));
}

}  // namespace moa
