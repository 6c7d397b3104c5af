// fp32 GEMM on CDNA4 matrix cores (v_mfma_f32_16x16x4_f32) with fused
// epilogues for the surrogate's dense layers.
//
//   C[m, n] = sum_k A(m, k) * B(n, k)
//
// A(m, k) is stored k-contiguous (A[m * lda + k], "KMajor") or m-contiguous
// (A[k * lda + m], "MNMajor"); B(n, k) likewise.  The three products of a
// dense layer map onto it as
//   forward  Z  = A_in W^T : A = activations (KMajor), B = W (KMajor)
//   input grad dA = dZ W   : A = dZ (KMajor),         B = W viewed [k][n] (MNMajor)
//   weight grad dW = dZ^T A_in : A = dZ viewed [k][m] (MNMajor), B = A_in (MNMajor)
//
// Tiling: 64 * WGM * WGN threads (WGM x WGN wavefronts), block tile
// BM x BN = (16 FM WGM) x (16 FN WGN), k tile 16, double-buffered LDS tiles
// stored m/n-contiguous (As[k][m], Bs[k][n]).  Within a wavefront, fragment f
// of MFMA row i covers tile row 16*FM*wm + FM*i + f, so each lane fetches its
// FM A values (and FN B values) for one k with a single LDS vector read.
// MFMA lane layout (16x16x4 f32): lane l supplies A[i = l%16][k = l/16] and
// B[k = l/16][j = l%16]; accumulator element r of lane l is D[4*(l/16)+r][l%16].
// A lane therefore owns a (4 FM) x FN block of C: rows 4*FM*(l/16) + q,
// q = FM*r + f, and columns FN*(l%16) + g.
//
// Blocks are numbered so that the WGM-by-... m tiles that share one n tile
// are consecutive and land on the same XCD (L2) of the 8 on the chip.
#pragma once

#include "adam.h"
#include "common.h"

namespace ot {

enum class Lay : int { KMajor = 0, MNMajor = 1 };
enum class Epi : int {
  Store = 0,     // C = acc
  Bias = 1,      // C = acc + bias[n]
  BiasRelu = 2,  // C = max(acc + bias[n], 0)
  Mse = 3,       // Y = acc + bias[n]; R = Y - T; C = scale * R; partial sum of R^2 per block
  SplitK = 4,    // C[split] = acc (partial sums, reduced by a separate pass)
  Mask = 5,      // C = acc * (mask[m, n] > 0)
  Adam = 6       // acc is the gradient of the weights C: Adam updates C, adam_m, adam_v (same layout as C)
};

struct GemmArgs {
  const float* A;
  int64_t lda;
  const float* B;
  int64_t ldb;
  float* C;
  int64_t ldc;
  int64_t M, N, K;
  int64_t k_chunk;          // k range per split (multiple of 16); >= K without split
  int64_t split_stride;     // SplitK: elements between consecutive split slices of C
  const float* bias;        // Bias, BiasRelu, Mse
  const float* target;      // Mse
  int64_t ldt;
  const int32_t* target_rows;  // Mse (nullable): output row m compares with target row target_rows[m],
  int64_t target_rows_max;     //   clamped to [0, target_rows_max]
  float scale;              // Mse
  double* loss_partials;    // Mse: one per block
  const float* mask;        // Mask
  int64_t ldmask;
  float* rowsum;            // optional: sum_k A(m, k) for m of the block's rows (n tile 0 only)
  int64_t rowsum_stride;    // SplitK: elements between consecutive split slices of rowsum
  float* adam_m;            // Adam: moments at C's offsets
  float* adam_v;
  AdamArgs adam;
};

constexpr int kNumXcd = 8;

// Map the hardware block id to a logical tile id such that each XCD (blocks
// are dispatched round-robin over the 8 XCDs) receives a contiguous range of
// logical ids.
__device__ __forceinline__ int64_t xcd_remap(int64_t p, int64_t g) {
  const int64_t xcd = p % kNumXcd, q = p / kNumXcd;
  const int64_t per = g / kNumXcd, rem = g % kNumXcd;
  return xcd * per + (xcd < rem ? xcd : rem) + q;
}

template <int FM>
struct FragVec;
template <>
struct FragVec<4> { typedef f32x4 T; };
template <>
struct FragVec<2> { typedef f32x2 T; };
template <>
struct FragVec<1> { typedef float T; };

// ROLE only separates instantiations (0: hidden layers, 1: output layer) so
// that profiles attribute the output-layer products to their own kernels.
template <int WGM, int WGN, int FM, int FN, Lay LA, Lay LB, Epi EPI, int BK = 16, int ROLE = 0>
__global__ __launch_bounds__(64 * WGM * WGN)
__attribute__((amdgpu_waves_per_eu((EPI == Epi::Mse && FM * FN == 8) ? 5 : 1))) void gemm_f32_kernel(GemmArgs g) {
  constexpr int NT = 64 * WGM * WGN;
  static_assert(BK % 16 == 0, "k tile must be a multiple of 16");
  constexpr int BM = 16 * FM * WGM;
  constexpr int BN = 16 * FN * WGN;
  constexpr int PAD = 4;
  constexpr int LDA_S = BM + PAD;
  constexpr int LDB_S = BN + PAD;
  constexpr int VA = BM * BK / 4 / NT;  // float4 loads per thread per k tile
  constexpr int VB = BN * BK / 4 / NT;
  static_assert(VA >= 1 && VA * NT * 4 == BM * BK, "A tile does not split evenly");
  static_assert(VB >= 1 && VB * NT * 4 == BN * BK, "B tile does not split evenly");

  __shared__ __attribute__((aligned(16))) float As[2][BK * LDA_S];
  __shared__ __attribute__((aligned(16))) float Bs[2][BK * LDB_S];
  __shared__ double s_red[NT / 64];
  __shared__ int32_t s_trow[EPI == Epi::Mse ? BM : 1];   // target rows of the tile (Mse with target_rows)

  const int tid = threadIdx.x;
  const int lane = tid & 63, wid = tid >> 6;
  const int wm = wid % WGM, wn = wid / WGM;

  // Tile order: XCD remap over the whole grid (the blocks of one k split stay
  // on one XCD), and consecutive tiles walk the dimension with fewer tiles
  // first, so the blocks sharing the larger operand's tile run together.
  const int64_t tiles_m = (g.M + BM - 1) / BM;
  const int64_t tiles_n = (g.N + BN - 1) / BN;
  const int64_t lin = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
  // Wave priority by blockIdx.x / 256 (blocks of one CU come from different
  // rounds of 256), so that the blocks sharing a CU drift out of step and the
  // epilogues of some overlap the MFMAs of others.  Measured at the 100x100
  // net: the weight gradient (628 tiles x 2 k splits) 63.7 -> 58.7 us; the
  // linear block index in place of blockIdx.x gave no gain, and the forward
  // did not change either way.  Results do not depend on it.
  switch ((blockIdx.x >> 8) & 3) {
    case 0: __builtin_amdgcn_s_setprio(0); break;
    case 1: __builtin_amdgcn_s_setprio(1); break;
    case 2: __builtin_amdgcn_s_setprio(2); break;
    default: __builtin_amdgcn_s_setprio(3); break;
  }
  const int64_t l2 = xcd_remap(lin, (int64_t)gridDim.x * gridDim.y);
  const int64_t logical = l2 % gridDim.x, split = l2 / gridDim.x;
  int64_t tm, tn;
  if (tiles_m <= tiles_n) { tm = logical % tiles_m; tn = logical / tiles_m; }
  else { tn = logical % tiles_n; tm = logical / tiles_n; }
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int64_t kbeg = split * g.k_chunk;
  const int64_t kend = (kbeg + g.k_chunk < g.K) ? kbeg + g.k_chunk : g.K;
  const int64_t nk = (kend > kbeg) ? (kend - kbeg + BK - 1) / BK : 0;

  // Global -> register staging of one k tile.
  f32x4 ra[VA], rb[VB];
  // Blocks whose tile lies inside M x N load full k tiles without predication.
  const bool interior = (m0 + BM <= g.M) && (n0 + BN <= g.N);

  auto load_tile_fast = [&](int64_t k0) {
#pragma unroll
    for (int i = 0; i < VA; ++i) {
      const int v = tid + i * NT;
      if constexpr (LA == Lay::MNMajor) {
        const int kr = v / (BM / 4), mc = (v % (BM / 4)) * 4;
        ra[i] = *reinterpret_cast<const f32x4*>(g.A + (k0 + kr) * g.lda + m0 + mc);
      } else {
        const int mr = v / (BK / 4), kc = (v % (BK / 4)) * 4;
        ra[i] = *reinterpret_cast<const f32x4*>(g.A + (m0 + mr) * g.lda + k0 + kc);
      }
    }
#pragma unroll
    for (int i = 0; i < VB; ++i) {
      const int v = tid + i * NT;
      if constexpr (LB == Lay::MNMajor) {
        const int kr = v / (BN / 4), nc = (v % (BN / 4)) * 4;
        rb[i] = *reinterpret_cast<const f32x4*>(g.B + (k0 + kr) * g.ldb + n0 + nc);
      } else {
        const int nr = v / (BK / 4), kc = (v % (BK / 4)) * 4;
        rb[i] = *reinterpret_cast<const f32x4*>(g.B + (n0 + nr) * g.ldb + k0 + kc);
      }
    }
  };

  auto load_tile = [&](int64_t k0) {
    if (interior && k0 + BK <= kend) {
      load_tile_fast(k0);
      return;
    }
#pragma unroll
    for (int i = 0; i < VA; ++i) {
      const int v = tid + i * NT;
      if constexpr (LA == Lay::MNMajor) {
        const int kr = v / (BM / 4), mc = (v % (BM / 4)) * 4;
        const int64_t k = k0 + kr, m = m0 + mc;
        f32x4 t = {0.f, 0.f, 0.f, 0.f};
        if (k < kend) {
          const float* p = g.A + k * g.lda + m;
          if (m + 3 < g.M) t = *reinterpret_cast<const f32x4*>(p);
          else
            for (int c = 0; c < 4; ++c) t[c] = (m + c < g.M) ? p[c] : 0.f;
        }
        ra[i] = t;
      } else {
        const int mr = v / (BK / 4), kc = (v % (BK / 4)) * 4;
        const int64_t m = m0 + mr, k = k0 + kc;
        f32x4 t = {0.f, 0.f, 0.f, 0.f};
        if (m < g.M) {
          const float* p = g.A + m * g.lda + k;
          if (k + 3 < kend) t = *reinterpret_cast<const f32x4*>(p);
          else
            for (int c = 0; c < 4; ++c) t[c] = (k + c < kend) ? p[c] : 0.f;
        }
        ra[i] = t;
      }
    }
#pragma unroll
    for (int i = 0; i < VB; ++i) {
      const int v = tid + i * NT;
      if constexpr (LB == Lay::MNMajor) {
        const int kr = v / (BN / 4), nc = (v % (BN / 4)) * 4;
        const int64_t k = k0 + kr, n = n0 + nc;
        f32x4 t = {0.f, 0.f, 0.f, 0.f};
        if (k < kend) {
          const float* p = g.B + k * g.ldb + n;
          if (n + 3 < g.N) t = *reinterpret_cast<const f32x4*>(p);
          else
            for (int c = 0; c < 4; ++c) t[c] = (n + c < g.N) ? p[c] : 0.f;
        }
        rb[i] = t;
      } else {
        const int nr = v / (BK / 4), kc = (v % (BK / 4)) * 4;
        const int64_t n = n0 + nr, k = k0 + kc;
        f32x4 t = {0.f, 0.f, 0.f, 0.f};
        if (n < g.N) {
          const float* p = g.B + n * g.ldb + k;
          if (k + 3 < kend) t = *reinterpret_cast<const f32x4*>(p);
          else
            for (int c = 0; c < 4; ++c) t[c] = (k + c < kend) ? p[c] : 0.f;
        }
        rb[i] = t;
      }
    }
  };

  auto store_tile = [&](int buf) {
    float* as = As[buf];
    float* bs = Bs[buf];
#pragma unroll
    for (int i = 0; i < VA; ++i) {
      const int v = tid + i * NT;
      if constexpr (LA == Lay::MNMajor) {
        const int kr = v / (BM / 4), mc = (v % (BM / 4)) * 4;
        *reinterpret_cast<f32x4*>(as + kr * LDA_S + mc) = ra[i];
      } else {
        const int mr = v / (BK / 4), kc = (v % (BK / 4)) * 4;
#pragma unroll
        for (int c = 0; c < 4; ++c) as[(kc + c) * LDA_S + mr] = ra[i][c];
      }
    }
#pragma unroll
    for (int i = 0; i < VB; ++i) {
      const int v = tid + i * NT;
      if constexpr (LB == Lay::MNMajor) {
        const int kr = v / (BN / 4), nc = (v % (BN / 4)) * 4;
        *reinterpret_cast<f32x4*>(bs + kr * LDB_S + nc) = rb[i];
      } else {
        const int nr = v / (BK / 4), kc = (v % (BK / 4)) * 4;
#pragma unroll
        for (int c = 0; c < 4; ++c) bs[(kc + c) * LDB_S + nr] = rb[i][c];
      }
    }
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int f = 0; f < FM; ++f)
#pragma unroll
    for (int h = 0; h < FN; ++h) acc[f][h] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Optional row sums of A over k (bias gradient of the weight-gradient GEMM).
  const bool do_rowsum = (g.rowsum != nullptr) && (tn == 0);
  float rsum = 0.f;

  const int a_off = 16 * FM * wm + FM * (lane % 16);
  const int b_off = 16 * FN * wn + FN * (lane % 16);
  const int kl = lane / 16;

  // Indexed targets: the tile's row indices are read now, so that their
  // latency is hidden behind the main loop (its barriers publish them).
  if constexpr (EPI == Epi::Mse) {
    if (g.target_rows && tid < BM) {
      const int64_t m = min(m0 + tid, g.M - 1);
      s_trow[tid] = (int32_t)min(max((int64_t)g.target_rows[m], (int64_t)0), g.target_rows_max);
    }
  }
  if (nk > 0) {
    load_tile(kbeg);
    store_tile(0);
    __syncthreads();
  }
  for (int64_t kt = 0; kt < nk; ++kt) {
    const int buf = (int)(kt & 1);
    if (kt + 1 < nk) load_tile(kbeg + (kt + 1) * BK);
    const float* as = As[buf];
    const float* bs = Bs[buf];
    typedef typename FragVec<FM>::T FA;
    typedef typename FragVec<FN>::T FB;
    // fragments of step kk + 1 are read while step kk's MFMAs run
    FA an = *reinterpret_cast<const FA*>(as + kl * LDA_S + a_off);
    FB bn = *reinterpret_cast<const FB*>(bs + kl * LDB_S + b_off);
#pragma unroll
    for (int kk = 0; kk < BK / 4; ++kk) {
      const FA av = an;
      const FB bv = bn;
      if (kk + 1 < BK / 4) {
        const int kr = 4 * (kk + 1) + kl;
        an = *reinterpret_cast<const FA*>(as + kr * LDA_S + a_off);
        bn = *reinterpret_cast<const FB*>(bs + kr * LDB_S + b_off);
      }
#pragma unroll
      for (int f = 0; f < FM; ++f) {
        float a_f;
        if constexpr (FM == 1) a_f = av; else a_f = av[f];
#pragma unroll
        for (int h = 0; h < FN; ++h) {
          float b_h;
          if constexpr (FN == 1) b_h = bv; else b_h = bv[h];
          acc[f][h] = __builtin_amdgcn_mfma_f32_16x16x4f32(a_f, b_h, acc[f][h], 0, 0, 0);
        }
      }
    }
    if (do_rowsum && tid < BM) {
#pragma unroll
      for (int k = 0; k < BK; ++k) rsum += as[k * LDA_S + tid];
    }
    if (kt + 1 < nk) store_tile(buf ^ 1);
    __syncthreads();
  }
  if constexpr (EPI == Epi::Mse) {
    if (nk == 0) __syncthreads();       // publishes s_trow (the main loop's barriers do otherwise)
  }
  if (do_rowsum && tid < BM && m0 + tid < g.M) g.rowsum[split * g.rowsum_stride + m0 + tid] = rsum;

  // ---------------------------------------------------------------- epilogue
  float lsum = 0.f;
  [[maybe_unused]] const AdamArgs ad = (EPI == Epi::Adam) ? g.adam.resolved() : g.adam;
  const int64_t row_base = m0 + 16 * FM * wm + 4 * FM * (lane / 16);
  const int64_t col_base = n0 + 16 * FN * wn + FN * (lane % 16);
  float* Cb = g.C + (EPI == Epi::SplitK ? split * g.split_stride : 0);
  const bool full = (col_base + FN - 1 < g.N);
  // FN consecutive values starting at column col_base (zeros past N); the
  // pointers are 4 * FN-byte aligned because col_base is a multiple of FN
  // and every leading dimension is a multiple of 4.
  auto load_cols = [&](const float* p, float* out) {
    if (full) {
      if constexpr (FN == 4) {
        const f32x4 t = *reinterpret_cast<const f32x4*>(p);
        out[0] = t[0]; out[1] = t[1]; out[2] = t[2]; out[3] = t[3];
      } else if constexpr (FN == 2) {
        const f32x2 t = *reinterpret_cast<const f32x2*>(p);
        out[0] = t[0]; out[1] = t[1];
      } else {
#pragma unroll
        for (int h = 0; h < FN; ++h) out[h] = p[h];
      }
    } else {
#pragma unroll
      for (int h = 0; h < FN; ++h) out[h] = (col_base + h < g.N) ? p[h] : 0.f;
    }
  };
  float bv[FN];
  if constexpr (EPI == Epi::Bias || EPI == Epi::BiasRelu || EPI == Epi::Mse) load_cols(g.bias + col_base, bv);
  // Mse: the block's targets pass through LDS (the B staging buffer, free
  // after the main loop) in TP passes, each filled by direct global -> LDS
  // loads and waited for once: read row by row from global memory, every
  // row's wait would also wait for the previous row's dY stores (stores
  // count in vmcnt).  A lane's rows r of pass p are p RP .. p RP + RP - 1;
  // local row lr = ((wm 4 + lane / 16) RP + r - p RP) FM + f.  Tiles that
  // cross N, or unaligned targets, read row by row.
  constexpr int TB = 2 * BK * LDB_S;                              // floats of Bs
  constexpr int TP = (BM * BN <= TB) ? 1 : (BM * BN / 2 <= TB) ? 2 : 4;
  constexpr int RP = 4 / TP;
  static_assert(EPI != Epi::Mse || (BM * BN / TP <= TB && 256 % BN == 0), "target staging");
  const bool stage_t = (EPI == Epi::Mse) && (n0 + BN <= g.N) && (g.ldt % 4 == 0) &&
                       ((reinterpret_cast<uintptr_t>(g.target) & 15) == 0);
  float* Tl = &Bs[0][0];
  auto fill_targets = [&](int p) {
    typedef __attribute__((address_space(3))) void lds_void;
    constexpr int ROWS_KB = 256 / BN;                             // target rows per 1 KB chunk
    constexpr int CHUNKS = BM / TP * BN / 256;
    __syncthreads();                                              // Bs no longer read
    for (int c = wid; c < CHUNKS; c += NT / 64) {
      const int lr = c * ROWS_KB + lane / (BN / 4);
      const int ff = lr % FM, t = lr / FM, rr = t % RP, u = t / RP;
      const int R = 16 * FM * (u / 4) + 4 * FM * (u % 4) + FM * (p * RP + rr) + ff;
      const int64_t m = min(m0 + R, g.M - 1);
      const int64_t tr = g.target_rows ? (int64_t)s_trow[m - m0] : m;
      const float* src = g.target + tr * g.ldt + n0 + 4 * (lane % (BN / 4));
      __builtin_amdgcn_global_load_lds(src, (lds_void*)(Tl + c * 256), 16, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));        // vmcnt(0)
    __syncthreads();
  };
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if constexpr (EPI == Epi::Mse) {
      if (r % RP == 0 && stage_t) fill_targets(r / RP);
    }
#pragma unroll
    for (int f = 0; f < FM; ++f) {
      const int64_t m = row_base + FM * r + f;
      if (m >= g.M) continue;
      float v[FN];
#pragma unroll
      for (int h = 0; h < FN; ++h) v[h] = acc[f][h][r];
      if constexpr (EPI == Epi::Bias || EPI == Epi::BiasRelu || EPI == Epi::Mse) {
#pragma unroll
        for (int h = 0; h < FN; ++h) v[h] += bv[h];
      }
      if constexpr (EPI == Epi::BiasRelu) {
#pragma unroll
        for (int h = 0; h < FN; ++h) v[h] = v[h] > 0.f ? v[h] : 0.f;
      }
      if constexpr (EPI == Epi::Mse) {
        float tv[FN];
        if (stage_t) {
          const int lr = ((wm * 4 + lane / 16) * RP + r % RP) * FM + f;
          const float* tp = Tl + lr * BN + 16 * FN * wn + FN * (lane % 16);
#pragma unroll
          for (int h = 0; h < FN; ++h) tv[h] = tp[h];
        } else {
          const int64_t tr = g.target_rows ? (int64_t)s_trow[m - m0] : m;
          load_cols(g.target + tr * g.ldt + col_base, tv);
        }
#pragma unroll
        for (int h = 0; h < FN; ++h) {
          const float rr = (col_base + h < g.N) ? v[h] - tv[h] : 0.f;
          lsum += rr * rr;
          v[h] = g.scale * rr;
        }
      }
      if constexpr (EPI == Epi::Mask) {
        float mv[FN];
        load_cols(g.mask + m * g.ldmask + col_base, mv);
#pragma unroll
        for (int h = 0; h < FN; ++h) v[h] = mv[h] > 0.f ? v[h] : 0.f;
      }
      float* cp = Cb + m * g.ldc + col_base;
      if constexpr (EPI == Epi::Adam) {
        float* mp = g.adam_m + m * g.ldc + col_base;
        float* vp = g.adam_v + m * g.ldc + col_base;
        if (FN == 4 && full) {
          f32x4 P = *reinterpret_cast<const f32x4*>(cp), Mo = *reinterpret_cast<const f32x4*>(mp),
                V = *reinterpret_cast<const f32x4*>(vp);
          adam4(P, f32x4{v[0], v[FN > 1 ? 1 : 0], v[FN > 2 ? 2 : 0], v[FN > 3 ? 3 : 0]}, Mo, V, ad);
          *reinterpret_cast<f32x4*>(cp) = P;
          *reinterpret_cast<f32x4*>(mp) = Mo;
          *reinterpret_cast<f32x4*>(vp) = V;
        } else {
#pragma unroll
          for (int h = 0; h < FN; ++h) {
            if (col_base + h >= g.N) continue;
            float P = cp[h], Mo = mp[h], V = vp[h];
            adam1(P, v[h], Mo, V, ad);
            cp[h] = P;
            mp[h] = Mo;
            vp[h] = V;
          }
        }
        continue;
      }
      if (FN == 4 && full) {
        *reinterpret_cast<f32x4*>(cp) = f32x4{v[0], v[FN > 1 ? 1 : 0], v[FN > 2 ? 2 : 0], v[FN > 3 ? 3 : 0]};
      } else if (FN == 2 && full) {
        *reinterpret_cast<f32x2*>(cp) = f32x2{v[0], v[FN > 1 ? 1 : 0]};
      } else {
#pragma unroll
        for (int h = 0; h < FN; ++h)
          if (col_base + h < g.N) cp[h] = v[h];
      }
    }
  }
  if constexpr (EPI == Epi::Mse) {
    double ls = warp_sum((double)lsum);
    if (lane == 0) s_red[wid] = ls;
    __syncthreads();
    if (tid == 0) {
      double t = 0.0;
      for (int w = 0; w < NT / 64; ++w) t += s_red[w];
      g.loss_partials[blockIdx.y * gridDim.x + blockIdx.x] = t;
    }
  }
}

// Host launcher.  Returns the hipError_t of the launch.  t0 / t1 (nullable):
// events that take the kernel's own start and end times.
template <int WGM, int WGN, int FM, int FN, Lay LA, Lay LB, Epi EPI, int BK = 16, int ROLE = 0>
hipError_t launch_gemm_f32(const GemmArgs& g, int64_t splits, hipStream_t stream, hipEvent_t t0 = nullptr,
                           hipEvent_t t1 = nullptr) {
  constexpr int BM = 16 * FM * WGM, BN = 16 * FN * WGN;
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  dim3 grid((unsigned)tiles, (unsigned)splits);
  hipExtLaunchKernelGGL((gemm_f32_kernel<WGM, WGN, FM, FN, LA, LB, EPI, BK, ROLE>), grid, dim3(64 * WGM * WGN), 0,
                        stream, t0, t1, 0, g);
  return hipGetLastError();
}

template <int WGM, int WGN, int FM, int FN>
constexpr int64_t gemm_tiles(int64_t M, int64_t N) {
  return ((M + 16 * FM * WGM - 1) / (16 * FM * WGM)) * ((N + 16 * FN * WGN - 1) / (16 * FN * WGN));
}

}  // namespace ot
