// bf16 GEMM on CDNA4 matrix cores (v_mfma_f32_16x16x32_bf16), fp32
// accumulation, with fused epilogues for the mixed-precision surrogate.
//
//   C[m, n] = sum_k A(m, k) * B(n, k)      (A, B bf16; C fp32 or bf16)
//
// Operand storage as in the fp32 kernel: "KMajor" = k contiguous
// (A[m * lda + k]), "MNMajor" = m (or n) contiguous (A[k * lda + m]).
// Leading dimensions are multiples of 8 elements and bases 16-byte aligned.
//
// MFMA lane layout (16x16x32 bf16): lane l supplies A[i = l%16][k = 8(l/16)+e]
// and B[k = 8(l/16)+e][j = l%16], e = 0..7; accumulator element r of lane l is
// D[4(l/16)+r][l%16].
//
// LDS staging keeps each operand in its global layout, so every global load
// and LDS write is a 16-byte vector:
//   KMajor  -> tile [mn][BK + 8]: a lane's 8 k-values are one ds_read_b128;
//   MNMajor -> tile [BK][mn + 16]: a lane's 8 k-values are two
//              ds_read_b64_tr_b16 transpose reads (within each 16-lane group,
//              lane c addresses row k0 + c/4, columns 4 (c%4)..+3, and lane i
//              receives column i of those 4 rows).
// Block: 4 wavefronts (2 x 2), wave tile (16 FM) x (16 FN), fragment f
// covering rows 16 f .. 16 f + 15 of the wave tile.  The epilogue stages the
// fp32 accumulators through LDS so that each lane then handles 4 consecutive
// columns of a row: targets, bias and masks are read, and C written, with
// 16-byte (fp32) or 8-byte (bf16) vector accesses.
#pragma once

#include "adam.h"
#include "common.h"

namespace ot {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// fp32 -> bf16, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f2bf(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// Workgroup barrier that orders LDS accesses only.  __syncthreads() also
// waits for every outstanding global memory access (vmcnt(0)), which would
// drain loads that are meant to stay in flight across the barrier (k tiles of
// the pipelined loop, prefetched epilogue operands); code that needs a global
// load's data waits for it with its own vmcnt before this barrier.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

enum class LayB : int { KMajor = 0, MNMajor = 1 };
enum class EpiB : int {
  StoreF32 = 0,   // C (fp32) = acc
  SplitK = 1,     // C (fp32)[split] = acc
  BiasF32 = 2,    // C (fp32) = acc + bias[n]
  BiasReluBf = 3, // C (bf16) = bf16(max(acc + bias[n], 0))
  MaskBf = 4,     // C (bf16) = bf16(acc * (mask[m, n] > 0)), mask bf16
  MseBf = 5,      // R = acc + bias[n] - T[m, n] (T fp32); C (bf16) = bf16(scale R); per-block sum of R^2
  AdamF32 = 6     // acc is the gradient of the fp32 master weights C: Adam updates C, adam_m, adam_v
                  // (same layout as C) and writes bf16(C) to adam_pb; no gradient is stored
};

struct GemmBArgs {
  const uint16_t* A;
  int64_t lda;
  const uint16_t* B;
  int64_t ldb;
  void* C;
  int64_t ldc;
  int64_t M, N, K;
  int64_t k_chunk;          // per split, multiple of BK
  int64_t split_stride;     // SplitK: elements between split slices
  const float* bias;
  const float* target;      // MseBf (fp32)
  int64_t ldt;
  const int32_t* target_rows;  // MseBf (nullable): output row m compares with target row target_rows[m],
  int64_t target_rows_max;     //   clamped to [0, target_rows_max]
  float scale;
  double* loss_partials;
  const uint16_t* mask;     // MaskBf (bf16 activations)
  int64_t ldmask;
  float* rowsum;            // StoreF32 / SplitK with MNMajor A: sum_k A(m, k) (n tile 0)
  int64_t rowsum_stride;
  float* colsum;            // MseBf: per m-tile column sums of the bf16 dY, colsum[tm * colsum_ld + n]
  int64_t colsum_ld;
  float* adam_m;            // AdamF32: first and second moments, bf16 weight copy, all at C's offsets
  float* adam_v;
  uint16_t* adam_pb;
  AdamArgs adam;
};

__device__ __forceinline__ int64_t xcd_remap_b(int64_t p, int64_t g) {
  const int64_t xcd = p % 8, q = p / 8;
  const int64_t per = g / 8, rem = g % 8;
  return xcd * per + (xcd < rem ? xcd : rem) + q;
}

// Epilogue shared by the bf16 kernels.  A wavefront stages its fp32
// accumulators in LDS (`ep`, pitch WN + 4) for output rows mw.., columns nw..,
// in chunks of ROWS rows; each lane then handles 4 consecutive columns of a
// row, so targets, bias and masks are read, and C written, with vector
// accesses.  The reads of a chunk's targets / masks are issued before the chunk
// is staged, so their latency overlaps the staging.  MseBf also accumulates the
// loss partial of the block and, per m-tile, the column sums of the rounded dY
// (the output bias gradient) when g.colsum is set (finish()).
// Indexed targets (MseBf with target_rows): a block reads the row indices of
// its tile into LDS at its start, so that their latency is hidden behind the
// main loop, whose barriers publish them.
template <int BM>
__device__ __forceinline__ void load_target_rows(const GemmBArgs& g, int64_t m0, int32_t* s_trow) {
  if (g.target_rows)
    for (int i = threadIdx.x; i < BM; i += blockDim.x) {
      const int64_t m = min(m0 + i, g.M - 1);
      s_trow[i] = (int32_t)min(max((int64_t)g.target_rows[m], (int64_t)0), g.target_rows_max);
    }
}

template <int WN, EpiB EPI, int NW = 4>
struct BEpi {
  static constexpr int EP = WN + 4;
  static constexpr int CG = WN / 4;               // column groups of 4
  static constexpr int RPP = 64 / CG;             // rows per pass of a wavefront
  int cg, rl;
  int64_t col;
  bool cfull;
  const int32_t* s_trow = nullptr;   // MseBf with target_rows: row indices of the tile (LDS), row tile_m0 first
  int64_t tile_m0 = 0;
  __device__ __forceinline__ int64_t trow(const GemmBArgs& g, int64_t m) const {
    return g.target_rows ? (int64_t)s_trow[m - tile_m0] : m;
  }
  float lsum = 0.f;
  float csum[4] = {0.f, 0.f, 0.f, 0.f};
  float bias4[4] = {0.f, 0.f, 0.f, 0.f};

  __device__ __forceinline__ BEpi(const GemmBArgs& g, int64_t nw) {
    const int lane = threadIdx.x & 63;
    cg = lane % CG;
    rl = lane / CG;
    col = nw + 4 * cg;
    cfull = col + 3 < g.N;
    if constexpr (EPI == EpiB::BiasF32 || EPI == EpiB::BiasReluBf || EPI == EpiB::MseBf) {
      if (cfull) {
        const f32x4 t = *reinterpret_cast<const f32x4*>(g.bias + col);
        bias4[0] = t[0]; bias4[1] = t[1]; bias4[2] = t[2]; bias4[3] = t[3];
      } else {
        for (int c = 0; c < 4; ++c) bias4[c] = (col + c < g.N) ? g.bias[col + c] : 0.f;
      }
    }
  }

  // Rows m0 .. m0 + ROWS - 1 (ep row 0 = row m0).  stage() writes the chunk's
  // accumulators into ep and makes them visible to the wavefront.
  template <int ROWS, class Stage>
  __device__ __forceinline__ void rows(const GemmBArgs& g, const float* ep, int64_t m0, int64_t split, Stage stage) {
    static_assert(ROWS % RPP == 0, "chunk rows");
    constexpr int NP = ROWS / RPP;
    if constexpr (EPI == EpiB::AdamF32) {
      adam_rows<NP>(g, ep, m0, stage);
      return;
    }
    // targets (MseBf) or mask (MaskBf) of each pass; one branch around all
    // the loads of the chunk, so that they are all in flight together
    f32x4 pre[NP];
    if constexpr (EPI == EpiB::MseBf || EPI == EpiB::MaskBf) {
      if (cfull) {
#pragma unroll
        for (int i = 0; i < NP; ++i) {
          const int64_t m = min(m0 + rl + RPP * i, g.M - 1);
          if constexpr (EPI == EpiB::MseBf) {
            pre[i] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(g.target + trow(g, m) * g.ldt + col));
          } else {
            const u16x4 h = *reinterpret_cast<const u16x4*>(g.mask + m * g.ldmask + col);
            pre[i] = f32x4{bf2f(h[0]), bf2f(h[1]), bf2f(h[2]), bf2f(h[3])};
          }
        }
      } else {
#pragma unroll
        for (int i = 0; i < NP; ++i) {
          const int64_t m = min(m0 + rl + RPP * i, g.M - 1);
          for (int c = 0; c < 4; ++c) {
            if constexpr (EPI == EpiB::MseBf) pre[i][c] = (col + c < g.N) ? g.target[trow(g, m) * g.ldt + col + c] : 0.f;
            else pre[i][c] = (col + c < g.N) ? bf2f(g.mask[m * g.ldmask + col + c]) : 0.f;
          }
        }
      }
    }
    stage();
    // every prefetched operand of the chunk has landed (one wait here rather
    // than per row, where the row stores would be waited for too)
    if constexpr (EPI == EpiB::MseBf || EPI == EpiB::MaskBf)
      __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));            // vmcnt(0)
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const int rr = rl + RPP * i;
      const int64_t m = m0 + rr;
      if (m >= g.M || col >= g.N) continue;
      const f32x4 a4 = *reinterpret_cast<const f32x4*>(ep + rr * EP + 4 * cg);
      float v[4] = {a4[0], a4[1], a4[2], a4[3]};
      if constexpr (EPI == EpiB::StoreF32 || EPI == EpiB::SplitK || EPI == EpiB::BiasF32) {
        if constexpr (EPI == EpiB::BiasF32)
          for (int c = 0; c < 4; ++c) v[c] += bias4[c];
        float* C = reinterpret_cast<float*>(g.C) + (EPI == EpiB::SplitK ? split * g.split_stride : 0) + m * g.ldc + col;
        if (cfull) *reinterpret_cast<f32x4*>(C) = f32x4{v[0], v[1], v[2], v[3]};
        else
          for (int c = 0; c < 4; ++c)
            if (col + c < g.N) C[c] = v[c];
      } else {
        if constexpr (EPI == EpiB::BiasReluBf) {
          for (int c = 0; c < 4; ++c) { v[c] += bias4[c]; v[c] = v[c] > 0.f ? v[c] : 0.f; }
        }
        if constexpr (EPI == EpiB::MaskBf) {
          for (int c = 0; c < 4; ++c) v[c] = pre[i][c] > 0.f ? v[c] : 0.f;
        }
        if constexpr (EPI == EpiB::MseBf) {
          for (int c = 0; c < 4; ++c) {
            const float r = (col + c < g.N) ? (v[c] + bias4[c]) - pre[i][c] : 0.f;
            lsum += r * r;
            v[c] = g.scale * r;
          }
        }
        const uint16_t h4[4] = {f2bf(v[0]), f2bf(v[1]), f2bf(v[2]), f2bf(v[3])};
        if constexpr (EPI == EpiB::MseBf)
          for (int c = 0; c < 4; ++c) csum[c] += (col + c < g.N) ? bf2f(h4[c]) : 0.f;
        uint16_t* C = reinterpret_cast<uint16_t*>(g.C) + m * g.ldc + col;
        if (cfull) {
          *reinterpret_cast<u16x4*>(C) = u16x4{h4[0], h4[1], h4[2], h4[3]};
        } else {
          for (int c = 0; c < 4; ++c)
            if (col + c < g.N) C[c] = h4[c];
        }
      }
    }
  }

  // AdamF32: each lane updates 4 consecutive parameters of a row per pass,
  // passes taken in groups of G.  The master weights and both moments of a
  // group are loaded together (non-temporal: every parameter is touched once
  // per step), and the loads of group i + 1 are issued before group i is
  // updated and stored, so two groups are in flight; group 0's loads are
  // issued before the gradients are staged in LDS.
  template <int NP, class Stage>
  __device__ __forceinline__ void adam_rows(const GemmBArgs& g, const float* ep, int64_t m0, Stage stage) {
    constexpr int G = NP < 4 ? NP : 4;
    constexpr int NG = NP / G;
    static_assert(NP % G == 0, "pass groups");
    float* const P = reinterpret_cast<float*>(g.C);
    if (!cfull || col >= g.N) {
      stage();
      if (col >= g.N) return;
      for (int i = 0; i < NP; ++i) {
        const int rr = rl + RPP * i;
        const int64_t m = m0 + rr;
        if (m >= g.M) continue;
        for (int c = 0; c < 4; ++c) {
          if (col + c >= g.N) break;
          const int64_t o = m * g.ldc + col + c;
          float p = P[o], mo = g.adam_m[o], vo = g.adam_v[o];
          adam1(p, ep[rr * EP + 4 * cg + c], mo, vo, g.adam.resolved());
          P[o] = p;
          g.adam_m[o] = mo;
          g.adam_v[o] = vo;
          g.adam_pb[o] = f2bf(p);
        }
      }
      return;
    }
    const AdamArgs ad = g.adam.resolved();
    f32x4 pp[2][G], mm[2][G], vv[2][G];
    auto load = [&](int grp, int buf) {
#pragma unroll
      for (int u = 0; u < G; ++u) {
        const int64_t m = min(m0 + rl + RPP * (grp * G + u), g.M - 1);   // clamped rows are not stored
        const int64_t o = m * g.ldc + col;
        pp[buf][u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(P + o));
        mm[buf][u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(g.adam_m + o));
        vv[buf][u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(g.adam_v + o));
      }
    };
    load(0, 0);
    stage();
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
      const int buf = gi & 1;
      if (gi + 1 < NG) load(gi + 1, buf ^ 1);
#pragma unroll
      for (int u = 0; u < G; ++u) {
        const int rr = rl + RPP * (gi * G + u);
        const int64_t m = m0 + rr;
        if (m >= g.M) continue;
        const f32x4 gr = *reinterpret_cast<const f32x4*>(ep + rr * EP + 4 * cg);
        adam4(pp[buf][u], gr, mm[buf][u], vv[buf][u], ad);
        const int64_t o = m * g.ldc + col;
        __builtin_nontemporal_store(pp[buf][u], reinterpret_cast<f32x4*>(P + o));
        __builtin_nontemporal_store(mm[buf][u], reinterpret_cast<f32x4*>(g.adam_m + o));
        __builtin_nontemporal_store(vv[buf][u], reinterpret_cast<f32x4*>(g.adam_v + o));
        __builtin_nontemporal_store(
            u16x4{f2bf(pp[buf][u][0]), f2bf(pp[buf][u][1]), f2bf(pp[buf][u][2]), f2bf(pp[buf][u][3])},
            reinterpret_cast<u16x4*>(g.adam_pb + o));
      }
    }
  }

  // Block-level reductions of MseBf (loss partial, per-m-tile column sums)
  // over the block's NW wavefronts.  Waves 2 j and 2 j + 1 share column group
  // j.  s_red: >= 8 doubles + NW * WN floats of LDS.
  __device__ __forceinline__ void finish(const GemmBArgs& g, int64_t tm, double* s_red) {
    if constexpr (EPI == EpiB::MseBf) {
      const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
      const double ls = warp_sum((double)lsum);
      if (lane == 0) s_red[wid] = ls;
      // lanes with the same lane % CG hold the same 4 columns: fold the RPP
      // lanes, then the two wavefronts of each column half
      for (int c = 0; c < 4; ++c)
        for (int off = CG; off < 64; off <<= 1) csum[c] += __shfl_xor(csum[c], off, 64);
      float* xs = reinterpret_cast<float*>(s_red + 8);   // NW waves x WN floats
      if (rl == 0)
        for (int c = 0; c < 4; ++c) xs[wid * WN + 4 * cg + c] = csum[c];
      lds_barrier();
      if (tid == 0) {
        double t = s_red[0];
        for (int w = 1; w < NW; ++w) t += s_red[w];
        g.loss_partials[blockIdx.y * gridDim.x + blockIdx.x] = t;
      }
      if (g.colsum && (wid & 1) == 0 && rl == 0) {
        for (int c = 0; c < 4; ++c) {
          const int64_t n = col + c;
          if (n < g.N) g.colsum[tm * g.colsum_ld + n] = xs[wid * WN + 4 * cg + c] + xs[(wid + 1) * WN + 4 * cg + c];
        }
      }
    }
  }
};

template <int FM, int FN, LayB LA, LayB LB, EpiB EPI, int BK>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmBArgs g) {
  constexpr int NT = 256, WGM = 2, WGN = 2;
  constexpr int WM = 16 * FM, WN = 16 * FN;
  constexpr int BM = WGM * WM, BN = WGN * WN;
  static_assert(BK % 32 == 0, "k tile must be a multiple of 32");
  // LDS tile geometry (elements of 16 bits)
  constexpr int A_ROWS = (LA == LayB::KMajor) ? BM : BK;
  constexpr int A_PITCH = (LA == LayB::KMajor) ? BK + 8 : BM + 16;
  constexpr int B_ROWS = (LB == LayB::KMajor) ? BN : BK;
  constexpr int B_PITCH = (LB == LayB::KMajor) ? BK + 8 : BN + 16;
  constexpr int A_ELEMS = A_ROWS * A_PITCH, B_ELEMS = B_ROWS * B_PITCH;
  constexpr int VA = BM * BK / 8 / NT, VB = BN * BK / 8 / NT;   // 16-byte loads per thread
  static_assert(VA >= 1 && VA * NT * 8 == BM * BK && VB >= 1 && VB * NT * 8 == BN * BK, "tile split");
  constexpr int TILE_BYTES = 2 * 2 * (A_ELEMS + B_ELEMS);
  constexpr int EPI_BYTES = 4 * (WM * (WN + 4)) * 4;            // per-wave fp32 staging
  constexpr int LDS_BYTES = TILE_BYTES > EPI_BYTES ? TILE_BYTES : EPI_BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char smem[LDS_BYTES];
  __shared__ double s_red[8 + 2 * WN];   // loss partials + column-sum exchange (4 waves x WN floats)
  __shared__ int32_t s_trow[EPI == EpiB::MseBf ? BM : 1];
  uint16_t* const tiles16 = reinterpret_cast<uint16_t*>(smem);
  auto As = [&](int buf) { return tiles16 + buf * A_ELEMS; };
  auto Bs = [&](int buf) { return tiles16 + 2 * A_ELEMS + buf * B_ELEMS; };

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid % WGM, wn = wid / WGM;
  const int64_t tiles_m = (g.M + BM - 1) / BM;
  const int64_t logical = xcd_remap_b(blockIdx.x, (int64_t)gridDim.x);
  const int64_t tm = logical % tiles_m, tn = logical / tiles_m;
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int64_t split = blockIdx.y;
  const int64_t kbeg = split * g.k_chunk;
  const int64_t kend = (kbeg + g.k_chunk < g.K) ? kbeg + g.k_chunk : g.K;
  const int64_t nk = (kend > kbeg) ? (kend - kbeg + BK - 1) / BK : 0;
  const bool interior = (m0 + BM <= g.M) && (n0 + BN <= g.N);
  if constexpr (EPI == EpiB::MseBf) load_target_rows<BM>(g, m0, s_trow);

  u32x4 ra[VA], rb[VB];

  // 8 consecutive elements at p, zero where the predicate fails
  auto load8 = [&](const uint16_t* p, bool all, int valid) -> u32x4 {
    if (all) return *reinterpret_cast<const u32x4*>(p);
    uint16_t t[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) t[e] = e < valid ? p[e] : (uint16_t)0;
    u32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = (uint32_t)t[2 * e] | ((uint32_t)t[2 * e + 1] << 16);
    return r;
  };

  auto load_tile = [&](int64_t k0) {
    const bool fast = interior && (k0 + BK <= kend);
#pragma unroll
    for (int i = 0; i < VA; ++i) {
      const int v = tid + i * NT;
      if constexpr (LA == LayB::KMajor) {
        const int r = v / (BK / 8), c = (v % (BK / 8)) * 8;
        const int64_t m = m0 + r, k = k0 + c;
        if (fast) ra[i] = *reinterpret_cast<const u32x4*>(g.A + m * g.lda + k);
        else if (m < g.M && k < kend) ra[i] = load8(g.A + m * g.lda + k, k + 8 <= kend, (int)(kend - k));
        else ra[i] = u32x4{0, 0, 0, 0};
      } else {
        const int r = v / (BM / 8), c = (v % (BM / 8)) * 8;
        const int64_t k = k0 + r, m = m0 + c;
        if (fast) ra[i] = *reinterpret_cast<const u32x4*>(g.A + k * g.lda + m);
        else if (k < kend && m < g.M) ra[i] = load8(g.A + k * g.lda + m, m + 8 <= g.M, (int)(g.M - m));
        else ra[i] = u32x4{0, 0, 0, 0};
      }
    }
#pragma unroll
    for (int i = 0; i < VB; ++i) {
      const int v = tid + i * NT;
      if constexpr (LB == LayB::KMajor) {
        const int r = v / (BK / 8), c = (v % (BK / 8)) * 8;
        const int64_t n = n0 + r, k = k0 + c;
        if (fast) rb[i] = *reinterpret_cast<const u32x4*>(g.B + n * g.ldb + k);
        else if (n < g.N && k < kend) rb[i] = load8(g.B + n * g.ldb + k, k + 8 <= kend, (int)(kend - k));
        else rb[i] = u32x4{0, 0, 0, 0};
      } else {
        const int r = v / (BN / 8), c = (v % (BN / 8)) * 8;
        const int64_t k = k0 + r, n = n0 + c;
        if (fast) rb[i] = *reinterpret_cast<const u32x4*>(g.B + k * g.ldb + n);
        else if (k < kend && n < g.N) rb[i] = load8(g.B + k * g.ldb + n, n + 8 <= g.N, (int)(g.N - n));
        else rb[i] = u32x4{0, 0, 0, 0};
      }
    }
  };

  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < VA; ++i) {
      const int v = tid + i * NT;
      int r, c;
      if constexpr (LA == LayB::KMajor) { r = v / (BK / 8); c = (v % (BK / 8)) * 8; }
      else { r = v / (BM / 8); c = (v % (BM / 8)) * 8; }
      *reinterpret_cast<u32x4*>(As(buf) + r * A_PITCH + c) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < VB; ++i) {
      const int v = tid + i * NT;
      int r, c;
      if constexpr (LB == LayB::KMajor) { r = v / (BK / 8); c = (v % (BK / 8)) * 8; }
      else { r = v / (BN / 8); c = (v % (BN / 8)) * 8; }
      *reinterpret_cast<u32x4*>(Bs(buf) + r * B_PITCH + c) = rb[i];
    }
  };

  // Operand fragment (8 k-values for this lane) from an LDS tile.
  // KMajor: row `row`, k offset kofs.  MNMajor: k rows kofs.., column block col0.
  auto frag_k = [&](const uint16_t* t, int pitch, int row, int kofs) -> bf16x8 {
    return *reinterpret_cast<const bf16x8*>(t + row * pitch + kofs);
  };
  auto frag_mn = [&](const uint16_t* t, int pitch, int col0, int kofs) -> bf16x8 {
    const int c = lane % 16;
    typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
    const uint16_t* p0 = t + (kofs + c / 4) * pitch + col0 + 4 * (c % 4);
    const uint16_t* p1 = p0 + 4 * pitch;
    bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p0);
    bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p1);
    return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int f = 0; f < FM; ++f)
#pragma unroll
    for (int h = 0; h < FN; ++h) acc[f][h] = f32x4{0.f, 0.f, 0.f, 0.f};

  const bool do_rowsum = (g.rowsum != nullptr) && (tn == 0);
  float rsum = 0.f;
  const int kgrp = 8 * (lane / 16);

  if (nk > 0) {
    load_tile(kbeg);
    store_tile(0);
    __syncthreads();
  }
  for (int64_t kt = 0; kt < nk; ++kt) {
    const int buf = (int)(kt & 1);
    if (kt + 1 < nk) load_tile(kbeg + (kt + 1) * BK);
    const uint16_t* as = As(buf);
    const uint16_t* bs = Bs(buf);
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8 af[FM], bfr[FN];
#pragma unroll
      for (int f = 0; f < FM; ++f) {
        if constexpr (LA == LayB::KMajor) af[f] = frag_k(as, A_PITCH, WM * wm + 16 * f + lane % 16, 32 * ks + kgrp);
        else af[f] = frag_mn(as, A_PITCH, WM * wm + 16 * f, 32 * ks + kgrp);
      }
#pragma unroll
      for (int h = 0; h < FN; ++h) {
        if constexpr (LB == LayB::KMajor) bfr[h] = frag_k(bs, B_PITCH, WN * wn + 16 * h + lane % 16, 32 * ks + kgrp);
        else bfr[h] = frag_mn(bs, B_PITCH, WN * wn + 16 * h, 32 * ks + kgrp);
      }
#pragma unroll
      for (int f = 0; f < FM; ++f)
#pragma unroll
        for (int h = 0; h < FN; ++h)
          acc[f][h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[f], bfr[h], acc[f][h], 0, 0, 0);
    }
    if (do_rowsum && tid < BM) {
      static_assert(LA == LayB::MNMajor || EPI == EpiB::MaskBf || true, "");
      if constexpr (LA == LayB::MNMajor) {
#pragma unroll 8
        for (int k = 0; k < BK; ++k) rsum += bf2f(as[k * A_PITCH + tid]);
      }
    }
    if (kt + 1 < nk) store_tile(buf ^ 1);
    __syncthreads();
  }
  if (do_rowsum && tid < BM && m0 + tid < g.M) g.rowsum[split * g.rowsum_stride + m0 + tid] = rsum;

  // ---------------------------------------------------------------- epilogue
  // Stage this wave's WM x WN accumulators (fp32) in LDS, pitch WN + 4.
  constexpr int EP = WN + 4;
  float* ep = reinterpret_cast<float*>(smem) + wid * (WM * EP);
  // the main loop ended with a barrier, so the tile buffers are free
  BEpi<WN, EPI> e(g, n0 + WN * wn);
  if constexpr (EPI == EpiB::MseBf) {
    if (nk == 0) lds_barrier();        // publishes s_trow (the main loop's barriers do otherwise)
    e.s_trow = s_trow;
    e.tile_m0 = m0;
  }
  e.template rows<WM>(g, ep, m0 + WM * wm, split, [&] {
#pragma unroll
    for (int f = 0; f < FM; ++f)
#pragma unroll
      for (int h = 0; h < FN; ++h)
#pragma unroll
        for (int r = 0; r < 4; ++r) ep[(16 * f + 4 * (lane / 16) + r) * EP + 16 * h + lane % 16] = acc[f][h][r];
    lds_barrier();
  });
  e.finish(g, tm, s_red);
}

// t0 / t1 (nullable): events that take the kernel's own start and end times.
template <int FM, int FN, LayB LA, LayB LB, EpiB EPI, int BK>
hipError_t launch_gemm_bf16(const GemmBArgs& g, int64_t splits, hipStream_t stream, hipEvent_t t0 = nullptr,
                            hipEvent_t t1 = nullptr) {
  constexpr int BM = 32 * FM, BN = 32 * FN;
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  hipExtLaunchKernelGGL((gemm_bf16_kernel<FM, FN, LA, LB, EPI, BK>), dim3((unsigned)tiles, (unsigned)splits),
                        dim3(256), 0, stream, t0, t1, 0, g);
  return hipGetLastError();
}

template <int FM, int FN>
constexpr int64_t gemm_bf16_tiles(int64_t M, int64_t N) {
  return ((M + 32 * FM - 1) / (32 * FM)) * ((N + 32 * FN - 1) / (32 * FN));
}


// ---------------------------------------------------------------------------
// Pipelined bf16 GEMM for the large output-layer products.
//
// Block tile BM x BN (256 x 128 or 128 x 256), 4 wavefronts of (BM/2) x (BN/2)
// built from v_mfma_f32_32x32x16_bf16 (lane l supplies A[i = l%32][k =
// 8 (l/32) + e], B[k = 8 (l/32) + e][j = l%32]; accumulator element r of
// lane l is D[8 (r/4) + 4 (l/32) + r%4][l%32]), k tile BK (32 or 64), and a
// ring of S LDS stages filled by direct global -> LDS loads
// (global_load_lds_dwordx4: each lane's 16 bytes land at the wave's LDS base +
// 16 * lane), so S - 1 k tiles are in flight while the MFMAs consume one.
// OCC blocks share a CU (BK 32, 3 stages: 72 KB of LDS per block), so one
// block's prologue and epilogue overlap another's main loop.
//
// LDS rows are unpadded; the 16-byte chunks of a row are permuted by XOR with a
// function of the row (kswz / mswz), so that the operand reads of a quarter
// wavefront (16 lanes) touch 16 different 16-byte bank groups:
//   KMajor operand: stage tile [mn][BK] (BK / 8 chunks per row); lanes read 16
//     consecutive rows at one chunk;
//   MNMajor operand: stage tile [BK][mn] (mn / 8 chunks per row), read with
//     ds_read_b64_tr_b16 (within each 16-lane group, lane c addresses row
//     k0 + c/4, columns 4 (c%4)..+3 of a 16-column block, and lane i receives
//     column i of those 4 rows): 4 rows x 4 chunks per half wavefront.
//
// Tile order: consecutive blocks walk the dimension with fewer tiles first, so
// the blocks that share the large operand's tile run together (and, through
// the XCD remap, on one XCD's L2).  With M <= N that is the m tiles sharing a
// B tile; otherwise the n tiles sharing an A tile.  Split-K grids keep all
// tiles of one split together.
//
// The loss partial of an MseBf block is stored at its hardware index
// (blockIdx.y * gridDim.x + blockIdx.x); any fixed slot per block gives the
// same fixed-order sum.
//
// Requirements: K (and the split size) a multiple of BK.  Rows / columns past
// M or N are read from clamped addresses and their results are not stored.
template <int BK>
__device__ __forceinline__ int kswz(int row) {
  return BK == 64 ? ((row >> 1) & 7) : ((row >> 2) & 3);
}
__device__ __forceinline__ int mswz(int row) { return 4 * (row & 3); }

// Global offsets (elements, relative to the k tile's start) of a thread's
// 16-byte chunks of one operand: chunk ci = (i * NW + wid) * 64 + lane of a
// stage sits in LDS slot ci.  x0: the block tile's first row (KMajor) or
// column (MNMajor) of the operand, lim: its rows / columns (clamped: rows
// past the end are read from the last one), ld: its leading dimension.
template <LayB L, int TILE, int BK, int NW, int N>
__device__ __forceinline__ void stage_offsets(int64_t (&off)[N], int wid, int lane, int64_t x0, int64_t lim,
                                              int64_t ld) {
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const int ci = (i * NW + wid) * 64 + lane;
    if constexpr (L == LayB::KMajor) {
      constexpr int KC = BK / 8;
      const int row = ci / KC, pc = ci % KC, lc = pc ^ kswz<BK>(row);
      off[i] = min(x0 + row, lim - 1) * ld + 8 * lc;
    } else {
      constexpr int CPR = TILE / 8;
      const int row = ci / CPR, pc = ci % CPR, lc = pc ^ mswz(row);
      off[i] = (int64_t)row * ld + min(x0 + 8 * lc, (lim - 1) / 8 * 8);
    }
  }
}

// Direct global -> LDS loads of one operand's k tile starting at k0 into the
// stage area dst (global_load_lds_dwordx4: each lane's 16 bytes land at the
// wave's LDS base + 16 * lane).
template <LayB L, int NW, int N>
__device__ __forceinline__ void stage_load(const uint16_t* base, const int64_t (&off)[N], int64_t k0, int64_t ld,
                                           unsigned char* dst, int wid) {
  typedef __attribute__((address_space(3))) void lds_void;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const uint16_t* src = (L == LayB::KMajor) ? base + off[i] + k0 : base + off[i] + k0 * ld;
    __builtin_amdgcn_global_load_lds(src, (lds_void*)(dst + (i * NW + wid) * 1024), 16, 0, 0);
  }
}

// Operand of one 16-deep k step (kk) for the 32-wide fragment at `base` of a
// stage area (cpr: 16-byte chunks per MNMajor row).
// KMajor: lane l reads row base + l%32, 8 k-values at 16 kk + 8 (l/32).
// MNMajor: 16-lane group q covers columns base + 16 (q%2) .. +15 and k rows
// 16 kk + 8 (q/2) .. +7, read as two transposed 4-row blocks.
// The reads are inline assembly: the compiler cannot tell a read of one stage
// from the direct global -> LDS loads still in flight into the others, and
// before the first read of every k tile it would wait for all of them
// (vmcnt(0)), which removes the prefetch.  Stage completion is tracked by the
// kernels' own vmcnt waits and barriers; frag_fence() waits for the reads.
template <int BK>
__device__ __forceinline__ bf16x8 stage_frag(const unsigned char* st, int cpr, bool kmajor, int base, int kk,
                                             int lane) {
  typedef int i32x4 __attribute__((ext_vector_type(4)));
  typedef int i32x2 __attribute__((ext_vector_type(2)));
  typedef __attribute__((address_space(3))) const unsigned char lds_u8;
  constexpr int KC = BK / 8;
  auto lds_addr = [](const unsigned char* p) -> uint32_t { return (uint32_t)(size_t)(lds_u8*)p; };
  if (kmajor) {
    const int row = base + lane % 32;
    const int lc = 2 * kk + lane / 32;
    i32x4 v;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(lds_addr(st + (row * KC + (lc ^ kswz<BK>(row))) * 16)));
    return __builtin_bit_cast(bf16x8, v);
  }
  const int c = lane % 16, q = lane / 16;
  const int col = base + 16 * (q & 1) + 4 * (c % 4);
  const int r0 = 16 * kk + 8 * (q >> 1) + c / 4, r1 = r0 + 4;
  const int ch = col / 8, half = (col / 4) & 1;
  i32x2 lo, hi;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(lo) : "v"(lds_addr(st + (r0 * cpr + (ch ^ mswz(r0))) * 16 + half * 8)));
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(hi) : "v"(lds_addr(st + (r1 * cpr + (ch ^ mswz(r1))) * 16 + half * 8)));
  const bf16x4 l = __builtin_bit_cast(bf16x4, lo), h = __builtin_bit_cast(bf16x4, hi);
  return bf16x8{l[0], l[1], l[2], l[3], h[0], h[1], h[2], h[3]};
}

// Wait for the outstanding fragment reads; each fragment then passes through
// an empty statement, so that no use of it can move above the wait.
template <int N>
__device__ __forceinline__ void frag_fence_regs(bf16x8 (&x)[N]) {
  typedef int i32x4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int f = 0; f < N; ++f) {
    i32x4 v = __builtin_bit_cast(i32x4, x[f]);
    asm volatile("" : "+v"(v));
    x[f] = __builtin_bit_cast(bf16x8, v);
  }
}

template <int BM, int BN, int BK, int S, int OCC, LayB LA, LayB LB, EpiB EPI, int NWN = 2>
__global__ __launch_bounds__(128 * NWN, OCC) void gemm_bf16_pipe_kernel(GemmBArgs g) {
  constexpr int NW = 2 * NWN, NT = 64 * NW;                       // 2 x NWN wavefronts
  constexpr int WM = BM / 2, WN = BN / NWN, FM = WM / 32, FN = WN / 32;
  static_assert(NW <= 8, "loss partial slots");
  constexpr int A_CH = BM * BK / 8, B_CH = BN * BK / 8;          // 16-byte chunks per stage
  constexpr int LA_N = A_CH / NT, LB_N = B_CH / NT;               // loads per thread per k tile
  static_assert(A_CH % NT == 0 && B_CH % NT == 0, "tile split");
  static_assert(BK == 32 || BK == 64, "k tile");
  static_assert((LA == LayB::KMajor || BM >= 128) && (LB == LayB::KMajor || BN >= 128), "MNMajor swizzle needs >= 16 chunks per row");
  constexpr int STAGE_BYTES = (A_CH + B_CH) * 16;
  // epilogue chunk: CH_F fragments (32 CH_F rows) of each wave staged at once
  constexpr int EP = WN + 4;
  constexpr int CH_F = (NW * FM * 32 * EP * 4 <= S * STAGE_BYTES)         ? FM
                       : (NW * (FM / 2) * 32 * EP * 4 <= S * STAGE_BYTES) ? FM / 2
                                                                         : FM / 4;
  static_assert(CH_F >= 1 && NW * CH_F * 32 * EP * 4 <= S * STAGE_BYTES, "epilogue staging");
  __shared__ __attribute__((aligned(16))) unsigned char smem[S * STAGE_BYTES];
  __shared__ double s_red[8 + NW * WN / 2];
  __shared__ int32_t s_trow[EPI == EpiB::MseBf ? BM : 1];

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid % 2, wn = wid / 2;
  const int64_t tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  // XCD remap over the whole grid, tiles fastest: the blocks of one k split
  // run on one XCD and share its L2.
  const int64_t lin = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
  const int64_t l2 = xcd_remap_b(lin, (int64_t)gridDim.x * gridDim.y);
  const int64_t logical = l2 % gridDim.x, split = l2 / gridDim.x;
  int64_t tm, tn;
  if (tiles_m <= tiles_n) { tm = logical % tiles_m; tn = logical / tiles_m; }
  else { tn = logical % tiles_n; tm = logical / tiles_n; }
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int64_t kbeg = split * g.k_chunk;
  const int64_t kend = (kbeg + g.k_chunk < g.K) ? kbeg + g.k_chunk : g.K;
  const int nk = (int)((kend - kbeg) / BK);
  if constexpr (EPI == EpiB::MseBf) load_target_rows<BM>(g, m0, s_trow);

  int64_t a_off[LA_N], b_off[LB_N];
  stage_offsets<LA, BM, BK, NW>(a_off, wid, lane, m0, g.M, g.lda);
  stage_offsets<LB, BN, BK, NW>(b_off, wid, lane, n0, g.N, g.ldb);
  // k tile kt into stage st
  auto issue = [&](int kt, int st) {
    const int64_t k0 = kbeg + (int64_t)kt * BK;
    unsigned char* sa = smem + st * STAGE_BYTES;
    stage_load<LA, NW>(g.A, a_off, k0, g.lda, sa, wid);
    stage_load<LB, NW>(g.B, b_off, k0, g.ldb, sa + A_CH * 16, wid);
  };
  typedef float f32x16 __attribute__((ext_vector_type(16)));
  auto frag_wait = [](bf16x8 (&af)[FM], bf16x8 (&bf)[FN]) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    frag_fence_regs(af);
    frag_fence_regs(bf);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int f = 0; f < FM; ++f)
#pragma unroll
    for (int h = 0; h < FN; ++h) acc[f][h] = f32x16{};

  // vmcnt wait with lgkm / exp counters left unconstrained (gfx9 encoding)
#define OT_WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 0xF) | (0x7 << 4) | (0xF << 8) | (((n) >> 4) << 14))
  constexpr int PER_TILE = LA_N + LB_N;
  constexpr int KK = BK / 16;
  static_assert((S - 2) * PER_TILE <= 63, "vmcnt range");
  // Wait until tile t's loads (the oldest of tiles t .. min(t + S - 2, nk - 1)
  // still outstanding) have landed, then make every wave's loads visible.
  auto tile_ready = [&](int t) {
    const int ahead = min(S - 2, nk - 1 - t);
    if (ahead >= 2) OT_WAIT_VM(2 * PER_TILE);
    else if (ahead == 1) OT_WAIT_VM(PER_TILE);
    else OT_WAIT_VM(0);
    lds_barrier();
  };
  auto load_frags = [&](int t, int kk, bf16x8 (&af)[FM], bf16x8 (&bf)[FN]) {
    const unsigned char* sa = smem + (t % S) * STAGE_BYTES;
    const unsigned char* sb = sa + A_CH * 16;
#pragma unroll
    for (int f = 0; f < FM; ++f) af[f] = stage_frag<BK>(sa, BM / 8, LA == LayB::KMajor, WM * wm + 32 * f, kk, lane);
#pragma unroll
    for (int h = 0; h < FN; ++h) bf[h] = stage_frag<BK>(sb, BN / 8, LB == LayB::KMajor, WN * wn + 32 * h, kk, lane);
  };

  // Software pipeline: the fragments of the next 16-deep step are read while
  // the MFMAs of the current one run, across k tiles too.  The barrier that
  // publishes tile t + 1 comes before the MFMAs of tile t's last step, whose
  // fragments are already in registers, so stage t % S is free after it and
  // receives tile t + S.
  bf16x8 af[FM], bfr[FN];
  for (int s = 0; s < S - 1; ++s)
    if (s < nk) issue(s, s);
  if (nk > 0) {
    tile_ready(0);
    if (S - 1 < nk) issue(S - 1, S - 1);
    load_frags(0, 0, af, bfr);
    frag_wait(af, bfr);
  }
  for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      bf16x8 an[FM], bn[FN];
      const bool more = (kk + 1 < KK) || (kt + 1 < nk);
      if (kk + 1 < KK) {
        load_frags(kt, kk + 1, an, bn);
      } else if (kt + 1 < nk) {
        tile_ready(kt + 1);
        if (kt + S < nk) issue(kt + S, kt % S);
        load_frags(kt + 1, 0, an, bn);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int f = 0; f < FM; ++f)
#pragma unroll
        for (int h = 0; h < FN; ++h)
          acc[f][h] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[f], bfr[h], acc[f][h], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      if (more) {
        frag_wait(an, bn);
#pragma unroll
        for (int f = 0; f < FM; ++f) af[f] = an[f];
#pragma unroll
        for (int h = 0; h < FN; ++h) bfr[h] = bn[h];
      }
    }
  }
#undef OT_WAIT_VM
  static_assert(S <= 4, "wait depth");

  // Epilogue in FM / CH_F chunks of 32 CH_F rows per wave, staged through the
  // (now free) stage buffers.
  float* ep = reinterpret_cast<float*>(smem) + wid * (CH_F * 32 * EP);
  BEpi<WN, EPI, NW> e(g, n0 + WN * wn);
  if constexpr (EPI == EpiB::MseBf) {
    if (nk == 0) lds_barrier();        // publishes s_trow (the main loop's barriers do otherwise)
    e.s_trow = s_trow;
    e.tile_m0 = m0;
  }
#pragma unroll
  for (int c0 = 0; c0 < FM; c0 += CH_F) {
    e.template rows<CH_F * 32>(g, ep, m0 + WM * wm + 32 * c0, split, [&] {
      lds_barrier();                  // other waves are done with the stage buffers / previous chunk
#pragma unroll
      for (int f = 0; f < CH_F; ++f)
#pragma unroll
        for (int h = 0; h < FN; ++h)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            ep[(32 * f + 8 * (r / 4) + 4 * (lane / 32) + r % 4) * EP + 32 * h + lane % 32] = acc[c0 + f][h][r];
      lds_barrier();
    });
  }
  e.finish(g, tm, s_red);
}

template <int BM, int BN, int BK, int S, int OCC, LayB LA, LayB LB, EpiB EPI, int NWN = 2>
hipError_t launch_gemm_bf16_pipe(const GemmBArgs& g, int64_t splits, hipStream_t stream, hipEvent_t t0 = nullptr,
                                 hipEvent_t t1 = nullptr) {
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  hipExtLaunchKernelGGL((gemm_bf16_pipe_kernel<BM, BN, BK, S, OCC, LA, LB, EPI, NWN>),
                        dim3((unsigned)tiles, (unsigned)splits), dim3(128 * NWN), 0, stream, t0, t1, 0, g);
  return hipGetLastError();
}

template <int BM, int BN>
constexpr int64_t gemm_bf16_pipe_tiles(int64_t M, int64_t N) {
  return ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
}

// Ping-pong variant: 256 x 256 block tile, k tile 32, eight wavefronts in two
// groups of four (waves 0-3 and 4-7: waves w and w + 4 of a workgroup share a
// SIMD, so each SIMD holds one wave of each group), wave tile 128 x 64 as in
// the pipelined kernel.  The groups alternate between a fragment phase (read
// the wave's fragments of tile t from LDS, both 16-deep steps) and a compute
// phase (issue this thread's direct global -> LDS loads of tile t + S - 1,
// then the 16 MFMAs of tile t at raised wave priority), one phase apart, with
// a block barrier between phases:
//   phase 2t:     group 0 reads tile t,      group 1 computes tile t - 1
//   phase 2t + 1: group 0 computes tile t,   group 1 reads tile t
// so that on every SIMD one wave issues MFMAs while the other reads LDS.
// (Issuing the global loads in the fragment phase, ahead of the reads, slowed
// the reads: 4.49 -> 3.85 ms for the 1000x1000 deep net's input gradient when
// moved.)  Stage (t - 1) % S receives tile t + S - 1 from phase 2t + 1 on
// (group 0; group 1 at 2t + 2): both groups have read tile t - 1 by the end
// of phase 2t - 1.  Before phase 2t every thread waits for its own loads of
// tile t (vmcnt; loads complete in order) and the barrier publishes them.
template <int S, LayB LA, LayB LB, EpiB EPI>
__global__ __launch_bounds__(512, 1) void gemm_bf16_pp_kernel(GemmBArgs g) {
  constexpr int BM = 256, BN = 256, BK = 32, NW = 8, NT = 512;
  constexpr int WM = 128, WN = 64, FM = WM / 32, FN = WN / 32;
  constexpr int A_CH = BM * BK / 8, B_CH = BN * BK / 8;
  constexpr int LA_N = A_CH / NT, LB_N = B_CH / NT;
  constexpr int STAGE_BYTES = (A_CH + B_CH) * 16;
  constexpr int EP = WN + 4;
  constexpr int CH_F = (NW * FM * 32 * EP * 4 <= S * STAGE_BYTES)         ? FM
                       : (NW * (FM / 2) * 32 * EP * 4 <= S * STAGE_BYTES) ? FM / 2
                                                                         : FM / 4;
  static_assert(CH_F >= 1 && NW * CH_F * 32 * EP * 4 <= S * STAGE_BYTES, "epilogue staging");
  static_assert(S >= 3 && S <= 4, "stages");
  __shared__ __attribute__((aligned(16))) unsigned char smem[S * STAGE_BYTES];
  __shared__ double s_red[8 + NW * WN / 2];
  __shared__ int32_t s_trow[EPI == EpiB::MseBf ? BM : 1];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wid >> 2;
  const int wm = wid % 2, wn = wid / 2;
  const int64_t tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  const int64_t lin = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
  const int64_t l2 = xcd_remap_b(lin, (int64_t)gridDim.x * gridDim.y);
  const int64_t logical = l2 % gridDim.x, split = l2 / gridDim.x;
  int64_t tm, tn;
  if (tiles_m <= tiles_n) { tm = logical % tiles_m; tn = logical / tiles_m; }
  else { tn = logical % tiles_n; tm = logical / tiles_n; }
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int64_t kbeg = split * g.k_chunk;
  const int64_t kend = (kbeg + g.k_chunk < g.K) ? kbeg + g.k_chunk : g.K;
  const int nk = (int)((kend - kbeg) / BK);
  if constexpr (EPI == EpiB::MseBf) load_target_rows<BM>(g, m0, s_trow);

  int64_t a_off[LA_N], b_off[LB_N];
  stage_offsets<LA, BM, BK, NW>(a_off, wid, lane, m0, g.M, g.lda);
  stage_offsets<LB, BN, BK, NW>(b_off, wid, lane, n0, g.N, g.ldb);
  auto issue = [&](int kt) {
    const int64_t k0 = kbeg + (int64_t)kt * BK;
    unsigned char* sa = smem + (kt % S) * STAGE_BYTES;
    stage_load<LA, NW>(g.A, a_off, k0, g.lda, sa, wid);
    stage_load<LB, NW>(g.B, b_off, k0, g.ldb, sa + A_CH * 16, wid);
  };
  typedef float f32x16 __attribute__((ext_vector_type(16)));
  constexpr int KK = BK / 16;
  bf16x8 af[KK][FM], bfr[KK][FN];
  f32x16 acc[FM][FN];
#pragma unroll
  for (int f = 0; f < FM; ++f)
#pragma unroll
    for (int h = 0; h < FN; ++h) acc[f][h] = f32x16{};

#define OT_WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 0xF) | (0x7 << 4) | (0xF << 8) | (((n) >> 4) << 14))
  constexpr int PER_TILE = LA_N + LB_N;
  static_assert((S - 2) * PER_TILE <= 63, "vmcnt range");
  // this thread's loads of tile t have landed (its loads of up to S - 2 later tiles may be in flight)
  // this thread's loads of tile t have landed; `later`: how many of its later
  // tiles may still be in flight (group 0 has issued up to tile t + S - 2 when
  // it waits, group 1 up to t + S - 3)
  auto own_tile_landed = [&](int t, int later) {
    const int ahead = min(later, nk - 1 - t);
    if (ahead >= 2) OT_WAIT_VM(2 * PER_TILE);
    else if (ahead == 1) OT_WAIT_VM(PER_TILE);
    else OT_WAIT_VM(0);
  };
  auto frag_phase = [&](int t) {
    const unsigned char* sa = smem + (t % S) * STAGE_BYTES;
    const unsigned char* sb = sa + A_CH * 16;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
      for (int f = 0; f < FM; ++f) af[kk][f] = stage_frag<BK>(sa, BM / 8, LA == LayB::KMajor, WM * wm + 32 * f, kk, lane);
#pragma unroll
      for (int h = 0; h < FN; ++h) bfr[kk][h] = stage_frag<BK>(sb, BN / 8, LB == LayB::KMajor, WN * wn + 32 * h, kk, lane);
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      frag_fence_regs(af[kk]);
      frag_fence_regs(bfr[kk]);
    }
  };
  auto compute_phase = [&](int t) {
    if (t + S - 1 < nk) issue(t + S - 1);
    __builtin_amdgcn_s_setprio(1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
      for (int f = 0; f < FM; ++f)
#pragma unroll
        for (int h = 0; h < FN; ++h)
          acc[f][h] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[kk][f], bfr[kk][h], acc[f][h], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(0);
  };

  // prologue: tiles 0 .. S - 2 from every thread; tile 0 published
  for (int t = 0; t < S - 1; ++t)
    if (t < nk) issue(t);
  if (nk > 0) own_tile_landed(0, S - 2);
  lds_barrier();
  if (grp == 0) {
    for (int t = 0; t < nk; ++t) {
      frag_phase(t);
      lds_barrier();                                   // end of phase 2t
      compute_phase(t);
      if (t + 1 < nk) own_tile_landed(t + 1, S - 2);
      lds_barrier();                                   // end of phase 2t + 1
    }
    lds_barrier();                                     // end of phase 2 nk
  } else {
    lds_barrier();                                     // end of phase 0
    for (int t = 0; t < nk; ++t) {
      frag_phase(t);
      if (t + 1 < nk) own_tile_landed(t + 1, S - 3);
      lds_barrier();                                   // end of phase 2t + 1
      compute_phase(t);
      lds_barrier();                                   // end of phase 2t + 2
    }
  }
#undef OT_WAIT_VM

  float* ep = reinterpret_cast<float*>(smem) + wid * (CH_F * 32 * EP);
  BEpi<WN, EPI, NW> e(g, n0 + WN * wn);
  if constexpr (EPI == EpiB::MseBf) {
    e.s_trow = s_trow;
    e.tile_m0 = m0;
  }
#pragma unroll
  for (int c0 = 0; c0 < FM; c0 += CH_F) {
    e.template rows<CH_F * 32>(g, ep, m0 + WM * wm + 32 * c0, split, [&] {
      lds_barrier();
#pragma unroll
      for (int f = 0; f < CH_F; ++f)
#pragma unroll
        for (int h = 0; h < FN; ++h)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            ep[(32 * f + 8 * (r / 4) + 4 * (lane / 32) + r % 4) * EP + 32 * h + lane % 32] = acc[c0 + f][h][r];
      lds_barrier();
    });
  }
  e.finish(g, tm, s_red);
}

template <int S, LayB LA, LayB LB, EpiB EPI>
hipError_t launch_gemm_bf16_pp(const GemmBArgs& g, int64_t splits, hipStream_t stream, hipEvent_t t0 = nullptr,
                               hipEvent_t t1 = nullptr) {
  const int64_t tiles = ((g.M + 255) / 256) * ((g.N + 255) / 256);
  hipExtLaunchKernelGGL((gemm_bf16_pp_kernel<S, LA, LB, EPI>), dim3((unsigned)tiles, (unsigned)splits), dim3(512), 0,
                        stream, t0, t1, 0, g);
  return hipGetLastError();
}

}  // namespace ot
