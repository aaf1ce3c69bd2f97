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
// step.  Each pass is software-pipelined over 32-key halves: the products of
// the next half are written interleaved with the vector work on the current
// one, so the matrix cores and the vector unit of a wave overlap.
// Where 1 - A_ij of a row's largest weight is not resolved in fp32 (the
// row's other weights sum to less than about 2^-22 of it, e.g. row 0) the
// influence of the whole row is reported as 0.
#include <type_traits>

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
  uint32_t chunk_off[DPW];
  int src_row[DPW];
#pragma unroll
  for (int i = 0; i < DPW; ++i) {
    const int m = (wave * DPW + i) * 64 + lane;
    const int r = m / CPR, pos = m % CPR;
    src_row[i] = r;
    chunk_off[i] = uint32_t(pos ^ swz(r)) * 16u;
  }
  // Tile `it` of item b into buffer `buf`.  The buffer resource spans the
  // item's n key rows of head g; rows past n re-read row n - 1 (never
  // visible).
  const uint32_t span = uint32_t(n - 1) * kv_row_bytes + RB;
  auto issue = [&](int b, int it, int buf) {
    const int64_t first = int64_t(b) * n * a.hkv + g;             // row 0 of head g, in rows of D
    const i32x4 kd = make_desc(static_cast<const char*>(a.k) + first * RB, span);
    const i32x4 vd = make_desc(static_cast<const char*>(a.v) + first * RB, span);
#pragma unroll
    for (int i = 0; i < DPW; ++i) {
      const uint32_t off = uint32_t(min(it * IBN + src_row[i], n - 1)) * kv_row_bytes + chunk_off[i];
      dma16_async(kd, off, &sK[buf][(wave * DPW + i) * 1024]);
      dma16_async(vd, off, &sV[buf][(wave * DPW + i) * 1024]);
    }
  };

  struct Acc {                                    // S^T and dP^T of 32 keys
    f32x16 s, d;
  };
  // Register r of a 32-key half holds, for this lane's query row, key
  // (r / 4) * 8 + half * 4 + r % 4 of the half (32x32 MFMA output layout).
  // On the diagonal half (keys iw0 .. iw0 + 31) a key after the row gets
  // score -inf, which both passes turn into zero weight and zero influence.
  auto mask_diagonal = [&](Acc& acc) {
    const int lim = lrow - half * 4;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if ((r >> 2) * 8 + (r & 3) > lim) acc.s[r] = -INFINITY;
  };

  // Running state per query row (both wave halves hold the same row):
  // mr = largest raw score so far, l = sum of exp2(c2 * s - c2 * mr),
  // u = sum of those weights times dP; in pass 2, sums of ratio * dP and of
  // ratio over the current 64-key tile.
  float mr, l, u, lse2, drow, acc_dp, acc_r;
  // Pass 1, one 32-key half: new running maximum (returns the scaled one),
  // then each element's weight.
  auto rescale = [&](const Acc& acc) {
    float tmax = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, acc.s[r]);
    tmax = max_xor<32>(tmax);
    const float mr_new = fmaxf(mr, tmax);
    const float m_new = mr_new * c2;              // scale > 0: the scaled maximum
    const float alpha = fast_exp2(mr * c2 - m_new);
    l *= alpha;
    u *= alpha;
    mr = mr_new;
    return m_new;
  };
  auto weigh = [&](float sv, float dv, float m_new) {
    const float e = fast_exp2(__builtin_fmaf(sv, c2, -m_new));
    l += e;
    u = __builtin_fmaf(e, dv, u);
  };
  // Pass 2, one element: A / (1 - A) = 1 / (2^(lse2 - c2 s) - 1), and the
  // tile's influence sum is  sum -ratio * (dP - D) = D * sum ratio - sum ratio * dP.
  auto influence = [&](float sv, float dv) {
    const float inv_p = fast_exp2(__builtin_fmaf(sv, -c2, lse2));
    const float ratio = __builtin_amdgcn_rcpf(inv_p - 1.0f);
    acc_dp = __builtin_fmaf(ratio, dv, acc_dp);
    acc_r += ratio;
  };
  auto flush_tile = [&](int t) {
    const float esum = wave_sum_lane63(__builtin_fmaf(drow, acc_r, -acc_dp));
    if (lane == 63) s_part[wave][t] += esum;
    acc_dp = 0.0f;
    acc_r = 0.0f;
  };

  // Keys 0 .. iw0 - 1 precede every row of the wave: iw0 / 32 halves need no
  // mask.  The half after them is the diagonal one; later keys are hidden.
  const int n_plain = wave_active ? iw0 / 32 : 0;
  const int n_pairs = n_plain / 2;

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
    if (b == 0) issue(b, 0, cnt & 1);       // later items' first tiles come with the previous pass
    // Q / dO are waited for here, once: the tile loads are invisible to the
    // compiler's wait tracking, which would otherwise wait inside the loop.
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)

    mr = kNegBig;
    l = u = lse2 = drow = acc_dp = acc_r = 0.0f;

    // One pipelined step: the products of half `sub` of LDS buffer `buf`
    // into `out` (kProd), written interleaved with the vector work of the
    // previous half `in` (kWork) in KS groups: each group reads the operands
    // of two groups later from LDS, issues its two MFMAs and then 16 / KS elements of
    // vector work, which run while the matrix core is busy.  The scheduling
    // barrier after each group keeps that order.
    auto step = [&](auto second_c, auto prod_c, auto work_c, int buf, int sub, Acc& out, const Acc& in) {
      constexpr bool kSecond = decltype(second_c)::value;
      constexpr bool kProd = decltype(prod_c)::value;
      constexpr bool kWork = decltype(work_c)::value;
      constexpr int EPG = 16 / KS;                  // elements of work per group
      const int r = sub * 32 + lrow;
      const char* kb = &sK[buf][r * RB];
      const char* vb = &sV[buf][r * RB];
      auto frag = [&](const char* base, int kk) {
        return *reinterpret_cast<const bf16x8*>(base + ((2 * kk + half) ^ swz(r)) * 16);
      };
      bf16x8 kf[3], vf[3];                          // operands read two groups ahead
      float m_new = 0.0f;
      if constexpr (kProd) {
        out.s = f32x16{};
        out.d = f32x16{};
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          kf[kk] = frag(kb, kk);
          vf[kk] = frag(vb, kk);
        }
      }
      if constexpr (kWork && !kSecond) m_new = rescale(in);
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        if constexpr (kProd) {
          if (kk + 2 < KS) {
            kf[(kk + 2) % 3] = frag(kb, kk + 2);
            vf[(kk + 2) % 3] = frag(vb, kk + 2);
          }
          out.s = mma32(kf[kk % 3], qf[kk], out.s);
          out.d = mma32(vf[kk % 3], df[kk], out.d);
        }
        if constexpr (kWork) {
#pragma unroll
          for (int e = 0; e < EPG; ++e) {
            const int rr = kk * EPG + e;
            if constexpr (kSecond) influence(in.s[rr], in.d[rr]);
            else weigh(in.s[rr], in.d[rr], m_new);
          }
        }
        sched_fence();
      }
    };

    // One pass over the wave's key halves, software-pipelined: the products
    // of half k + 1 are computed in the same step as the vector work of half
    // k.  Every wave meets the work-group barrier once per tile of the
    // work-group (all ntiles of them), which is when the tile's loads are
    // complete and the next tile starts loading into the other buffer.
    auto run_pass = [&](auto second_c) {
      constexpr bool kSecond = decltype(second_c)::value;
      const std::true_type yes;
      const std::false_type no;
      auto buf = [&](int t) { return (cnt + t) & 1; };
      // The load issued after a pass's last tile is tile 0 of the next pass
      // or item (past the last item: this item's tile 0 again, unused), so
      // the loop body holds no branch.
      auto tile_ready = [&](int t) {
        __builtin_amdgcn_s_waitcnt(0x0F70);   // this wave's loads of tile t have landed
        __syncthreads();                      // ... everyone's; tile t - 1's buffer is free
        const bool last = t + 1 >= ntiles;
        const int next_b = (last && kSecond) ? min(b + 1, a.batch - 1) : b;
        issue(next_b, last ? 0 : t + 1, buf(t + 1));
      };
      Acc acc0, acc1;
      tile_ready(0);
      if (wave_active) {
        step(second_c, yes, no, buf(0), 0, acc0, acc1);
        for (int t = 0; t < n_pairs; ++t) {
          step(second_c, yes, yes, buf(t), 1, acc1, acc0);
          tile_ready(t + 1);
          step(second_c, yes, yes, buf(t + 1), 0, acc0, acc1);
          if constexpr (kSecond) flush_tile(t);
        }
        // Tile n_pairs: one more plain half when n_plain is odd, then the
        // diagonal half.
        if (n_plain & 1) {
          step(second_c, yes, yes, buf(n_pairs), 1, acc1, acc0);
          mask_diagonal(acc1);
          step(second_c, no, yes, 0, 0, acc0, acc1);
        } else {
          mask_diagonal(acc0);
          step(second_c, no, yes, 0, 0, acc1, acc0);
        }
        if constexpr (kSecond) flush_tile(n_pairs);
      }
      for (int t = (wave_active ? n_pairs : 0) + 1; t < ntiles; ++t) tile_ready(t);
      cnt += ntiles;
    };

    run_pass(std::false_type{});
    l = sum_xor<32>(l);
    u = sum_xor<32>(u);
    lse2 = mr * c2 + __log2f(l);
    drow = u / l;
    // 1 / A of the row's largest weight, computed exactly as the second pass
    // will.  Where it lies within two fp32 ulps of 1, 1 - A is not resolved:
    // the whole row is reported as 0 (lse2 = +inf makes every ratio 0), as is
    // a row past n.  Elsewhere every key's 1 / A exceeds 1, so no ratio
    // divides by zero.
    const float inv_p_max = fast_exp2(__builtin_fmaf(mr, -c2, lse2));
    if (!row_ok || !(inv_p_max - 1.0f >= 0x1p-22f)) lse2 = INFINITY;
    run_pass(std::true_type{});
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);       // the unused last load lands before LDS is released
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
