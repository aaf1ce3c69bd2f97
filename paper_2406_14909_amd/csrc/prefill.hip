// Prefill attention with a per-KV-head banded-plus-sink causal mask (paper
// Sec. 2.1, Eq. 1, with the Sec. 3.2 span: sink prefix + diagonal band of
// width w_g).  Query i sees key j iff j <= i and (j < s or i - j < w_g).
// With the block band (paper Appendix "Main Setup": 64-token blocks) the band
// of row i instead starts at the first token of block i/64 - ceil(w_g/64) + 1;
// both are "j >= band_start(i)" with band_start(i) = ((i >> sh) - W + 1) << sh.
//
// One work-group = 4 waves = 128 query rows of one (sequence, query head);
// each wave owns 32 rows.  The work-group walks only the 64-key tiles that
// intersect the sink prefix or the band of its rows; every other tile is
// skipped without being read.  K and V tiles are staged in LDS (double
// buffered: the global loads of tile t+1 are in flight while tile t is
// computed, one barrier per tile) and shared by the 4 waves.
//
// Matrix-core formulation (CDNA4 32x32 MFMA; bf16 32x32x16, fp32 32x32x2):
//   S^T = K Q^T  : A = K tile rows (keys), B = Q^T kept in registers.
//                  Output lane l holds the scores of query row l % 32 for
//                  16 keys, so the row softmax needs one cross-lane step.
//   O^T += V^T P^T : B = P^T taken straight from the score registers
//                  (converted to the input type), A = V^T.  For bf16 the V
//                  tile stays row-major in LDS and the transposing LDS read
//                  (ds_read_b64_tr_b16) delivers V^T fragments; the fp32
//                  instantiation stores V transposed instead.
// The key order inside each 16-key MFMA step is permuted identically on both
// operands, which leaves the sum unchanged.
// Softmax is online in base 2 with the scale folded into one FMA per score
// (bf16 instantiation); the row sum is accumulated over the bf16-rounded
// probabilities that the PV product uses.
// The running maximum used as the exponent offset is raised only when some
// row of the wave would otherwise see exponents above 2^8 (a wave-uniform
// test), so most tiles skip rescaling the output accumulator; the final
// normalisation by the running sum makes the result independent of that
// offset.  The mask is evaluated only on tiles that are not entirely visible
// to the wave's rows.
#include "moa_device.h"

namespace moa {

namespace {

constexpr int BM = 128;   // query rows per work-group
constexpr int BN = 64;    // keys per tile
constexpr int NW = 4;     // waves per work-group
constexpr float kRescaleSlack = 8.0f;   // log2 headroom before the offset is raised

typedef short i16x4 __attribute__((ext_vector_type(4)));

template <typename T> struct Mma;

template <> struct Mma<bf16> {
  static constexpr int K = 16;                 // reduction depth per instruction
  typedef bf16x8 frag;
  __device__ __forceinline__ static f32x16 mma(const frag& a, const frag& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

template <> struct Mma<float> {
  static constexpr int K = 2;
  typedef float frag;
  __device__ __forceinline__ static f32x16 mma(const frag& a, const frag& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

// Fragment of K / Q for reduction step kk: elements kk*K + half*(K/2) ... (+K/2).
__device__ __forceinline__ bf16x8 load_frag(const bf16* base, int kk, int half) {
  return *reinterpret_cast<const bf16x8*>(base + kk * 16 + half * 8);
}
__device__ __forceinline__ float load_frag(const float* base, int kk, int half) {
  return base[kk * 2 + half];
}

// Transposing LDS read of four bf16: within each 16-lane group, lane 4a+b
// receives element b of the 8-byte reads issued by lanes 4e+a (e = 0..3).
// (The builtin exists only in the device pass; the host pass, which merely
// emits kernel stubs, sees an empty body.)
__device__ __forceinline__ bf16x4 read_tr(const bf16* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  const i16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(const_cast<bf16*>(p)));
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

// x * y - z with the product rounded on its own (never fused).
__device__ __forceinline__ float mul_then_sub(float x, float y, float z) {
#pragma clang fp contract(off)
  return x * y - z;
}

template <typename T, int D>
struct Tiles {
  static constexpr bool kTr = sizeof(T) == 2;        // bf16: V via the transposing read
  static constexpr int RB = D * int(sizeof(T));      // bytes per K/V row
  static constexpr int CPR = RB / 16;                // 16-byte chunks per row
  static constexpr int TILE_BYTES = BN * RB;         // one K (or bf16 V) tile, rows unpadded
  static constexpr int DMA_PER_WAVE = TILE_BYTES / 1024 / NW;   // 1 KB direct-to-LDS loads
  // K stages in LDS: bf16 keeps K two tiles ahead (3 buffers, 80 KB per
  // work-group with V); the fp32 instantiation keeps one tile ahead.
  static constexpr int KSTAGES = kTr ? 3 : 2;
  static constexpr int EPL = Vec16<T>::N;            // elements per 16-byte chunk
  static constexpr int VT_LD = BN + 4;               // fp32 only: V^T row stride (elements)
  static constexpr int VT_BYTES = D * VT_LD * int(sizeof(T));
  static constexpr int V_BYTES = kTr ? TILE_BYTES : VT_BYTES;
  static constexpr int VREG = kTr ? 1 : BN * CPR / (NW * 64);   // fp32 V chunks staged per thread
  // K rows: chunk c of row r sits at chunk position c ^ swz_k(r), so the 16
  // rows read together by an MFMA operand load hit 16 different bank groups.
  __device__ __forceinline__ static int swz_k(int r) { return CPR >= 16 ? (r & 15) : ((r >> 1) & 7); }
  // V rows (bf16): depends on r mod 8 only; the 4 rows x 4 chunks read by half
  // a wave in one transposing load hit 16 different bank groups.
  __device__ __forceinline__ static int swz_v(int r) { return CPR >= 16 ? 4 * (r & 3) : 4 * ((r >> 1) & 1); }
};

template <typename T, int D>
__global__ void __launch_bounds__(NW * 64, 2) prefill_kernel(PrefillArgs a) {
  using M = Mma<T>;
  using TL = Tiles<T, D>;
  constexpr int KS = D / M::K;            // MFMA steps over the head dimension
  constexpr int RB = TL::RB, CPR = TL::CPR, EPL = TL::EPL, KST = TL::KSTAGES;

  __shared__ __attribute__((aligned(1024))) char sK[KST][TL::TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char sV[2][TL::V_BYTES];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform (scalar)
  const int lrow = lane & 31;
  const int half = lane >> 5;

  // Work item.  A dispatch unit is (KV head, sequence, qchunk consecutive
  // query tiles) with all `group` query heads of that KV head, so its work-
  // groups share K/V bands.  Units are ordered heaviest first (latest query
  // chunks first, then widest window) and dealt to the accelerator dies in
  // rounds of kNumXcd, alternating direction each round: work-group i runs on
  // die i % kNumXcd, which walks its units in order, so the work-groups
  // resident on one die at a time share that die's L2, and every die gets a
  // similar mix of heavy and light units.
  const int xcd = static_cast<int>(blockIdx.x % kNumXcd);
  const int local = static_cast<int>(blockIdx.x / kNumXcd);
  const int per_unit = a.group * a.qchunk;
  const int round = local / per_unit;
  const int unit = round * kNumXcd + ((round & 1) ? kNumXcd - 1 - xcd : xcd);
  if (unit >= a.n_units) return;                   // padding unit
  const int within = local % per_unit;
  const int hb = a.hkv * a.batch;
  const int cd = unit / hb;                        // chunk rank, heaviest first
  const int g = a.kv_order[(unit % hb) / a.batch];
  const int b = unit % a.batch;
  const int qt = (a.n_chunks - 1 - cd) * a.qchunk + (a.qchunk - 1 - within / a.group);
  if (qt >= a.n_qtiles) return;                     // past the last query tile
  const int h = g * a.group + within % a.group;
  const int64_t n = a.n;
  // Band of row i: keys from band_start(i) to i; token band (shift 0) or
  // block band (shift 6: whole 64-token blocks, window counted in blocks).
  const int wband = a.window[g];
  const int bsh = a.band_shift;
  auto band_start = [&](int i) { return ((i >> bsh) - wband + 1) * (1 << bsh); };
  const int s = a.num_sink;
  const float c2 = a.scale_log2;

  const int i0 = qt * BM;
  const int i1 = static_cast<int>(min(n, int64_t(i0 + BM)));   // exclusive
  const int iw0 = i0 + wave * 32;                                // this wave's rows
  const int iw1 = min(i1, iw0 + 32);
  const bool wave_active = iw0 < i1;

  // Tiles to visit: sink tiles [0, ta) then band tiles [tb, tl].
  const int ta = (min(s, i1) + BN - 1) / BN;
  const int tl = (i1 - 1) / BN;
  const int tb = max(ta, max(0, band_start(i0)) / BN);
  const int ntiles = ta + max(0, tl - tb + 1);

  const int64_t q_row_stride = int64_t(a.hq) * D;
  const int64_t kv_row_bytes = int64_t(a.hkv) * RB;
  const T* qg = static_cast<const T*>(a.q) + (int64_t(b) * n * a.hq + h) * D;
  const char* kg = static_cast<const char*>(a.k) + (int64_t(b) * n * a.hkv + g) * RB;
  const char* vg = static_cast<const char*>(a.v) + (int64_t(b) * n * a.hkv + g) * RB;

  // Q^T fragments of this lane's query row (loaded after the first tiles' DMA
  // is issued, see the pipeline prologue).
  typename M::frag qf[KS];

  // Direct-to-LDS tile loads: DMA instruction I writes buffer bytes
  // [I*1024, I*1024 + 1024) and lane L's 16 bytes land at chunk I*64 + L.
  // K: chunk m is row m / (CPR+1), column chunk m % (CPR+1); the last column
  // chunk of each row (and anything past the tile) is padding and re-reads the
  // row's first chunk.  V (bf16): chunk I*64 + L is row r, position p, and
  // carries global chunk p ^ swz_v(r).  Keys past the end re-read the last key
  // (always masked by causality).
  // Per-lane byte offsets of the DMA sources relative to the tile's first key
  // row (tile independent).  DMA instruction I writes tile bytes
  // [I*1024, I*1024 + 1024): lane L's 16 bytes land at chunk m = I*64 + L, i.e.
  // row m / CPR, chunk position m % CPR, and carry global chunk
  // position ^ swz(row).  Wave w issues instructions w*DMA_PER_WAVE + i.
  constexpr int DPW = TL::DMA_PER_WAVE;
  uint32_t k_src[DPW], v_src[TL::kTr ? DPW : 1];
  auto dma_row = [&](int i) { return ((wave * DPW + i) * 64 + lane) / CPR; };
#pragma unroll
  for (int i = 0; i < DPW; ++i) {
    const int m = (wave * DPW + i) * 64 + lane;
    const int r = m / CPR, p = m % CPR;
    k_src[i] = uint32_t(r) * uint32_t(kv_row_bytes) + uint32_t(p ^ TL::swz_k(r)) * 16u;
    if constexpr (TL::kTr) v_src[i] = uint32_t(r) * uint32_t(kv_row_bytes) + uint32_t(p ^ TL::swz_v(r)) * 16u;
  }
  // With a.rotate the band tiles are visited in a rotated order: from the
  // unit's common start tile tr (the first band tile of its last query tile,
  // clipped to this work-group's band) up to tl, then from tb up to tr - 1.
  // The work-groups of a unit run side by side on one die, so at every step
  // they read the same key tile (before the wrap: tile tr + step; after it:
  // tile tb + step - (tl - tr + 1), the same for every work-group since tb
  // and tl move with the query tile in step), and each tile comes from memory
  // about once per unit.  Softmax over a set does not depend on the order of
  // its members.  Without a.rotate (keys and values that fit the last-level
  // cache) the band is visited from tb up, which spreads the concurrent reads
  // of a unit over many tiles.
  const int qt_top = min(a.n_qtiles - 1, (a.n_chunks - 1 - cd) * a.qchunk + a.qchunk - 1);
  const int tr = a.rotate ? min(max(tb, max(ta, max(0, band_start(qt_top * BM)) / BN)), tl + 1) : tb;
  const int n_upper = tl - tr + 1;                    // band tiles tr .. tl
  auto tile_j0 = [&](int it) {
    if (it < ta) return it * BN;
    const int k = it - ta;
    return (k < n_upper ? tr + k : tb + (k - n_upper)) * BN;
  };
  // Tile loads go through a buffer resource that spans exactly the tile's real
  // key rows (at most BN), so no address outside the inputs is ever touched;
  // rows past the last key re-read key n-1 (always masked by causality).
  auto tile_dma = [&](const char* base, const auto& src, int it, char* lds) {
    const int j0 = tile_j0(it);
    const int64_t rows = min(int64_t(BN), n - j0);
    const i32x4 rs = make_desc(base + int64_t(j0) * kv_row_bytes, uint32_t((rows - 1) * kv_row_bytes + RB));
    if (rows == BN) {
#pragma unroll
      for (int i = 0; i < DPW; ++i) dma16_async(rs, src[i], lds + (wave * DPW + i) * 1024);
    } else {
#pragma unroll
      for (int i = 0; i < DPW; ++i) {
        const int r = dma_row(i);
        const uint32_t off = src[i] - uint32_t(r - min(r, int(rows) - 1)) * uint32_t(kv_row_bytes);
        dma16_async(rs, off, lds + (wave * DPW + i) * 1024);
      }
    }
  };
  auto issue_k = [&](int it) { tile_dma(kg, k_src, it, &sK[it % KST][0]); };
  Vec16<T> vreg[TL::VREG];
  auto issue_v = [&](int it) {
    if constexpr (TL::kTr) {
      tile_dma(vg, v_src, it, &sV[it & 1][0]);
    } else {
      const int j0 = tile_j0(it);
#pragma unroll
      for (int i = 0; i < TL::VREG; ++i) {
        const int idx = threadIdx.x + i * NW * 64;
        const int r = idx / CPR, cc = idx % CPR;
        const int64_t j = min(int64_t(j0 + r), n - 1);
        vreg[i] = load16(reinterpret_cast<const T*>(vg + j * kv_row_bytes) + cc * EPL);
      }
    }
  };
  // fp32: V^T[d][key] is written from the staged registers.
  auto store_vt = [&](int buf) {
    if constexpr (!TL::kTr) {
      T* vt = reinterpret_cast<T*>(&sV[buf][0]);
#pragma unroll
      for (int i = 0; i < TL::VREG; ++i) {
        const int idx = threadIdx.x + i * NW * 64;
        const int r = idx / CPR, cc = idx % CPR;
#pragma unroll
        for (int e = 0; e < EPL; ++e) vt[(cc * EPL + e) * TL::VT_LD + r] = vreg[i].v[e];
      }
    }
  };

  // Per-lane byte offsets of the MFMA operand reads (tile independent).
  // K operand: row lrow (+ 32 * sub; the swizzle depends on the row's low bits
  // only), head-dim elements [kk*K + half*K/2, +K/2).
  auto k_offset = [&](int kk) {
    if constexpr (TL::kTr) {
      return lrow * RB + (((2 * kk + half) ^ TL::swz_k(lrow)) * 16);
    } else {
      const int d = 2 * kk + half;
      return lrow * RB + (((d / 4) ^ TL::swz_k(lrow)) * 16) + (d % 4) * 4;
    }
  };
  int k_off[TL::kTr ? KS : 1];
  if constexpr (TL::kTr) {
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) k_off[kk] = k_offset(kk);
  }
  // Transposing V read: lane 16G + 4e + a points at row (G/2)*4 + e (+ kb0),
  // bf16 column 32*dt + 16*(G%2) + 4a.
  int v_off[D / 32];
  if constexpr (TL::kTr) {
    const int vr = (lane >> 5) * 4 + ((lane & 15) >> 2);    // row mod 8
    const int a4 = lane & 3;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
      const int q = dt * 4 + ((lane >> 4) & 1) * 2 + (a4 >> 1);
      v_off[dt] = vr * RB + ((q ^ TL::swz_v(vr)) * 16) + (a4 & 1) * 8;
    }
  } else {
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) v_off[dt] = (dt * 32 + lrow) * TL::VT_LD * int(sizeof(T));
  }

  f32x16 oacc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt) oacc[dt] = f32x16{};
  float m_run = kNegBig, l_run = 0.0f;
  const int my_row = iw0 + lrow;

  // Pipeline: during tile t, V(t+1) and then K(t+2) stream in; at the top of
  // tile t only the newest K loads may still be in flight.
  if (ntiles > 0) {
    issue_v(0);
    issue_k(0);
  }
  if (ntiles > 1) issue_k(1);
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
  // Wait for Q (and the first tiles) here, once.  The tile DMA is opaque to
  // the compiler's wait-count tracking, which would otherwise place waits for
  // the Q loads inside the tile loop, where they would also drain the
  // prefetches in flight.
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
  for (int it = 0; it < ntiles; ++it) {
    const int j0 = tile_j0(it);
    if constexpr (KST == 3) {
      if (it + 1 < ntiles) {
        // all but the last DPW loads (K(it+1)) have landed: K(it), V(it)
        __builtin_amdgcn_s_waitcnt(0x0F70 | DPW);
      } else {
        __builtin_amdgcn_s_waitcnt(0x0F70);
      }
    } else {
      __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    }
    store_vt(it & 1);
    __syncthreads();                      // ... for every thread; K(it-1), V(it-1) buffers are free
    if (it + 1 < ntiles) issue_v(it + 1);
    if constexpr (KST == 3) {
      if (it + 2 < ntiles) issue_k(it + 2);
    } else {
      if (it + 1 < ntiles) issue_k(it + 1);
    }
    const int buf = it & 1;
    const int kbuf = it % KST;

    if (!wave_active) continue;
    // Does any (row, key) pair of this wave fall inside the mask?
    const bool any_causal = j0 <= iw1 - 1;
    const bool any_vis = any_causal && (j0 < s || band_start(iw0) <= j0 + BN - 1);
    if (!any_vis) continue;
    const bool all_vis = (j0 + BN - 1 <= iw0) && (iw1 - iw0 == 32) &&
                         ((j0 + BN <= s) || band_start(iw1 - 1) <= j0);

    // S^T = K Q^T for two 32-key sub-tiles.
    // Fragments of step kk+1 are read while the MFMAs of step kk run; the two
    // 32-key chains alternate so consecutive MFMAs are independent.
    const char* kb = &sK[kbuf][0];
    auto kfrag = [&](int kk, int sub) {
      const int off = TL::kTr ? k_off[TL::kTr ? kk : 0] : k_offset(kk);
      return *reinterpret_cast<const typename M::frag*>(kb + sub * 32 * RB + off);
    };
    f32x16 sacc[2] = {f32x16{}, f32x16{}};
    typename M::frag kf[2][2];
    kf[0][0] = kfrag(0, 0);
    kf[0][1] = kfrag(0, 1);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      if (kk + 1 < KS) {
        kf[(kk + 1) & 1][0] = kfrag(kk + 1, 0);
        kf[(kk + 1) & 1][1] = kfrag(kk + 1, 1);
      }
      sacc[0] = M::mma(kf[kk & 1][0], qf[kk], sacc[0]);
      sacc[1] = M::mma(kf[kk & 1][1], qf[kk], sacc[1]);
    }

    // Mask (edge tiles only; branch-free selects) and the tile's raw row maximum.
    if (!all_vis) {
      const int jl = j0 + half * 4;                 // key of register 0 of this lane
      const int hi = my_row < i1 ? my_row - jl : -1;  // causal: key offset <= hi
      const int band = band_start(my_row) - jl;       // band: key offset >= band
      const int sink = s - jl;                        // sink: key offset < sink
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int dj = sub * 32 + (r >> 2) * 8 + (r & 3);
          const bool vis = (dj <= hi) & ((dj < sink) | (dj >= band));
          sacc[sub][r] = vis ? sacc[sub][r] : -INFINITY;
        }
      }
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, sacc[sub][r]);
    tmax = max_xor<32>(tmax) * c2;
    // Raise the exponent offset only when some row of the wave needs it.
    if (__any(tmax > m_run + kRescaleSlack)) {
      const float m_new = fmaxf(m_run, tmax);
      const float alpha = fast_exp2(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) oacc[dt] *= alpha;
    }

    const char* vb = &sV[buf][0];
    if constexpr (TL::kTr) {
      // P in bf16; the row sum is taken over the same rounded weights that
      // enter the PV product (dot2 with (1, 1)).
      bf16x8 pf[2][2];
      float psum = 0.0f;
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            pf[sub][c][e] = static_cast<bf16>(fast_exp2(__builtin_fmaf(sacc[sub][8 * c + e], c2, -m_run)));
#pragma unroll
          for (int e = 0; e < 8; e += 2) psum = dot2_ones(pf[sub][c][e], pf[sub][c][e + 1], psum);
        }
      }
      psum = sum_xor<32>(psum);
      l_run += psum;

      // O^T += V^T P^T: for each 16-key step the four d-tile accumulators are
      // independent; the V^T fragments of the next step are read meanwhile.
      auto vfrag = [&](int step, int dt) {
        const int kb0 = (step >> 1) * 32 + 16 * (step & 1);
        const bf16x4 lo4 = read_tr(reinterpret_cast<const bf16*>(vb + kb0 * RB + v_off[dt]));
        const bf16x4 hi4 = read_tr(reinterpret_cast<const bf16*>(vb + (kb0 + 8) * RB + v_off[dt]));
        return __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7);
      };
      bf16x8 vf[2][D / 32];
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) vf[0][dt] = vfrag(0, dt);
#pragma unroll
      for (int step = 0; step < 4; ++step) {
        if (step + 1 < 4) {
#pragma unroll
          for (int dt = 0; dt < D / 32; ++dt) vf[(step + 1) & 1][dt] = vfrag(step + 1, dt);
        }
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
          oacc[dt] = M::mma(vf[step & 1][dt], pf[step >> 1][step & 1], oacc[dt]);
      }
    } else {
      float psum = 0.0f;
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          // separately rounded product: a row's maximal score gives exactly
          // 2^0, so w = 1 returns v bit-exactly in fp32
          const float p = fast_exp2(mul_then_sub(sacc[sub][r], c2, m_run));
          sacc[sub][r] = p;
          psum += p;
        }
      }
      psum = sum_xor<32>(psum);
      l_run += psum;
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) {
        const T* vt = reinterpret_cast<const T*>(vb + v_off[dt]);
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = sub * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
            oacc[dt] = M::mma(vt[key], sacc[sub][r], oacc[dt]);
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
  const int64_t blocks = int64_t((a.n_units + kNumXcd - 1) / kNumXcd) * kNumXcd * a.group * a.qchunk;
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
