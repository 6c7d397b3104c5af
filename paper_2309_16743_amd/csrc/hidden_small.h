// Narrow hidden layers (fp32): the two hidden layers of a 3-layer surrogate
// whose first layer has a small input width (<= 16) and whose hidden widths
// are <= 256, forward and backward, in three launches instead of nine.  At
// these widths the layers are a few hundred MFLOP per step and the cost is
// launch and latency, not arithmetic: each kernel stages its narrow operands
// in LDS with 16-byte loads issued together, then runs
// v_mfma_f32_16x16x4_f32 (lane l supplies A[l%16][l/16] and B[l/16][l%16];
// accumulator element r of lane l is D[4(l/16)+r][l%16]).
//
//   hidden_fwd_small_kernel   A1 = ReLU(X W1^T + b1), A2 = ReLU(A1 W2^T + b2)
//   hidden_bwd_small_kernel   role A: dZ1 = (dZ2 W2) * [A1 > 0] and, per row
//                             tile, partial sums of dW1 = dZ1^T X and db1;
//                             role B: k-split partials of dW2 = dZ2^T A1 and
//                             db2 = column sums of dZ2
//   hidden_bwd_reduce_kernel  dW2, db2, dW1, db1 from the partials, fixed order
//
// Every sum is taken in a fixed order, so results are deterministic.
//
// LDS row strides: operands read as A (16 rows at 4 consecutive k per MFMA)
// use a stride of 4 mod 64 floats, operands read as B (4 k rows at 16
// consecutive columns) a stride of 16 mod 64, so the 64 lanes of one operand
// read hit 64 different banks.
#pragma once

#include "common.h"

namespace ot {

constexpr int kSmallH = 256;     // widest hidden layer handled here
constexpr int kSmallIn = 16;     // widest input of layer 1
constexpr int kHfRows = 16;      // forward / role A: rows per block
constexpr int kHfCols = 64;      // forward / role A: output units per block
constexpr int kHbRows = 128;     // role B: batch rows per k split
constexpr int kHbTile = 64;      // role B: dW2 tile (64 x 64)
constexpr int kStrideA = kSmallH + 4;     // A-read rows of up to 256 values
constexpr int kStrideB = kHfCols + 16;    // B-read rows of 64 values

typedef float f32x4v __attribute__((ext_vector_type(4)));

// dst[r][c] (LDS, row stride ls) = src[r0 + r][c0 + c] for r < NR, c < NC
// (zero outside rows x cols); NR x NC / 4 vector loads spread over 256
// threads, all issued before the first LDS store.  The source rows must be
// 16-byte aligned with a leading dimension that is a multiple of 4.
template <int NR, int NC>
__device__ __forceinline__ void stage_tile(float* dst, int ls, const float* __restrict__ src, int64_t ld, int64_t r0,
                                           int64_t rows, int c0, int cols) {
  constexpr int NV = NR * NC / 4 / 256;
  static_assert(NV >= 1 && NV * 256 * 4 == NR * NC, "tile split");
  const int tid = threadIdx.x;
  f32x4v t[NV];
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    const int e = tid + 256 * q, r = e / (NC / 4), c = (e % (NC / 4)) * 4;
    const int64_t gr = r0 + r;
    const int gc = c0 + c;
    if (gr < rows && gc + 3 < cols) {
      t[q] = *reinterpret_cast<const f32x4v*>(src + gr * ld + gc);
    } else {
      f32x4v v = {0.f, 0.f, 0.f, 0.f};
      if (gr < rows)
        for (int u = 0; u < 4; ++u)
          if (gc + u < cols) v[u] = src[gr * ld + gc + u];
      t[q] = v;
    }
  }
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    const int e = tid + 256 * q, r = e / (NC / 4), c = (e % (NC / 4)) * 4;
    *reinterpret_cast<f32x4v*>(dst + r * ls + c) = t[q];
  }
}

// One 16 x 16 MFMA output block over kp (a multiple of 4) k values: lane l
// reads its A operand at pa[k * sa] and its B operand at pb[k * sb] for
// k = k0 (k0 = 0, 4, 8, ...; the lane's own k offset is folded into pa, pb).
// Four accumulator chains take the k steps in turn (four MFMAs in flight
// instead of one dependent chain), each step's operands are read while the
// previous steps run, and the chains are added in a fixed order at the end.
__device__ __forceinline__ void mfma_row_dot_chains(const float* pa, int sa, const float* pb, int sb, int kp,
                                                    f32x4v (&acc)[4]) {
  int k0 = 0;
  for (; k0 + 16 <= kp; k0 += 16) {
    float a[4], b[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      a[c] = pa[(k0 + 4 * c) * sa];
      b[c] = pb[(k0 + 4 * c) * sb];
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[c], b[c], acc[c], 0, 0, 0);
  }
  for (int c = 0; k0 < kp; k0 += 4, ++c) acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(pa[k0 * sa], pb[k0 * sb], acc[c], 0, 0, 0);
}
// The k range may be taken in pieces whose lengths before the last are
// multiples of 16: every k step then lands on the same chain as in one call.
__device__ __forceinline__ f32x4v mfma_row_dot(const float* pa, int sa, const float* pb, int sb, int kp) {
  f32x4v acc[4] = {};
  mfma_row_dot_chains(pa, sa, pb, sb, kp, acc);
  return (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

// Forward of layers 1 and 2 for rows r0 .. r0 + 15 and layer-2 units
// c0 .. c0 + 63.  Wave w computes the 16 x 16 output block of units
// c0 + 16 w .. c0 + 16 w + 15.  Blocks of column tile 0 also store A1.
__global__ __launch_bounds__(256) void hidden_fwd_small_kernel(
    const float* __restrict__ X, int64_t ldx, int in0, const float* __restrict__ W1, int64_t ldw1,
    const float* __restrict__ b1, int h1, const float* __restrict__ W2, int64_t ldw2, const float* __restrict__ b2,
    int h2, float* __restrict__ A1, int64_t lda1, float* __restrict__ A2, int64_t lda2, int64_t rows) {
  __shared__ __attribute__((aligned(16))) float sA1[kHfRows * kStrideA];
  __shared__ __attribute__((aligned(16))) float sW2[kHfCols * kStrideA];
  __shared__ float sX[kHfRows][kSmallIn];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t r0 = (int64_t)blockIdx.x * kHfRows;
  const int c0 = blockIdx.y * kHfCols;
  // W2 rows c0 .. c0 + 63 (all h1 columns) and X rows into LDS; thread j
  // keeps W1 row j and b1[j] in registers (layer 1 is one unit per thread)
  const int j = tid;
  float wj[kSmallIn], bj = 0.f;
#pragma unroll
  for (int k = 0; k < kSmallIn; ++k) wj[k] = (j < h1 && k < in0) ? W1[(int64_t)j * ldw1 + k] : 0.f;
  if (j < h1) bj = b1[j];
  stage_tile<kHfCols, kSmallH>(sW2, kStrideA, W2, ldw2, c0, h2, 0, h1);
  {
    const int r = tid / kSmallIn, k = tid % kSmallIn;
    sX[r][k] = (r0 + r < rows && k < in0) ? X[(r0 + r) * ldx + k] : 0.f;
  }
  __syncthreads();
  // layer 1 (K = in0 on the vector units; X and W1 are zero beyond in0, so the
  // padded terms add exact zeros); sX reads are broadcasts
  const int h1p = (h1 + 3) & ~3;
#pragma unroll 4
  for (int r = 0; r < kHfRows; ++r) {
    float z = bj;
#pragma unroll
    for (int k = 0; k < kSmallIn; ++k) z += sX[r][k] * wj[k];
    const float a = (j < h1 && z > 0.f) ? z : 0.f;
    if (j < h1 && blockIdx.y == 0 && r0 + r < rows) A1[(r0 + r) * lda1 + j] = a;
    sA1[r * kStrideA + j] = a;
  }
  __syncthreads();
  // layer 2: D[16 x 16] = A1 tile (16 x h1) * W2 block^T, k steps of 4
  const int ci = 16 * w + (lane & 15);
  f32x4v acc = mfma_row_dot(sA1 + (lane & 15) * kStrideA + (lane >> 4), 1, sW2 + ci * kStrideA + (lane >> 4), 1, h1p);
  const int c = c0 + ci;
  if (c < h2) {
    const float bias = b2[c];
    for (int q = 0; q < 4; ++q) {
      const int64_t row = r0 + 4 * (lane >> 4) + q;
      if (row < rows) {
        const float z = acc[q] + bias;
        A2[row * lda2 + c] = z > 0.f ? z : 0.f;
      }
    }
  }
}

constexpr int kMaskStride = kHfCols + 4;
// W2 is staged in two halves of its k range and role B's rows in two halves
// of the split, so that a block needs 67 KB of LDS and two fit on a CU.
constexpr int kWHalf = kSmallH / 2;
constexpr int kHbHalf = kHbRows / 2;
constexpr int kBwdSmem = kHfRows * kStrideA + kWHalf * kStrideB + kHfRows * (kHfCols + 1) + kHfRows * kSmallIn +
                         kHfRows * kMaskStride;
static_assert(2 * kHbHalf * kStrideB <= kBwdSmem, "role B staging");

// Backward, part 1.  Blocks [0, nA) (role A): rows r0 .. r0 + 15, layer-1
// units c0 .. c0 + 63: dA1 = dZ2 W2 (K = h2), dZ1 = dA1 * [A1 > 0] stored, and
// part1[rt][i][0 .. in0] = (sum_r dZ1[r][i] X[r][k] for k < in0, sum_r dZ1[r][i])
// over the tile's rows in order.  Blocks [nA, nA + nB) (role B): dW2 tile
// (j0 .. j0 + 63) x (i0 .. i0 + 63) over the batch rows of k split kc:
// part2[kc][j][i], and for i tile 0 the column sums part2b[kc][j].
__global__ __launch_bounds__(256) void hidden_bwd_small_kernel(
    const float* __restrict__ dZ2, int64_t ldd2, const float* __restrict__ A1, int64_t lda1,
    const float* __restrict__ X, int64_t ldx, int in0, const float* __restrict__ W2, int64_t ldw2, int h1, int h2,
    int64_t rows, float* __restrict__ dZ1, int64_t ldd1, float* __restrict__ part1, float* __restrict__ part2,
    float* __restrict__ part2b, int64_t nA) {
  __shared__ __attribute__((aligned(16))) float smem[kBwdSmem];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if ((int64_t)blockIdx.x < nA) {
    // ---------------- role A
    float* sD2 = smem;                                   // [16][kStrideA]
    float* sW = sD2 + kHfRows * kStrideA;                // [128][kStrideB]: one half of W2's k range
    float* sZ = sW + kWHalf * kStrideB;                  // [16][65]
    float* sX = sZ + kHfRows * (kHfCols + 1);            // [16][kSmallIn]
    float* sM = sX + kHfRows * kSmallIn;                 // [16][kMaskStride]: A1 tile (ReLU mask)
    const int tiles_c = (h1 + kHfCols - 1) / kHfCols;
    const int64_t rt = blockIdx.x / tiles_c;
    const int c0 = (int)(blockIdx.x % tiles_c) * kHfCols;
    const int64_t r0 = rt * kHfRows;
    stage_tile<kHfRows, kSmallH>(sD2, kStrideA, dZ2, ldd2, r0, rows, 0, h2);
    stage_tile<kWHalf, kHfCols>(sW, kStrideB, W2, ldw2, 0, h2, c0, h1);
    stage_tile<kHfRows, kHfCols>(sM, kMaskStride, A1, lda1, r0, rows, c0, h1);
    {
      const int r = tid / kSmallIn, k = tid % kSmallIn;
      sX[r * kSmallIn + k] = (r0 + r < rows && k < in0) ? X[(r0 + r) * ldx + k] : 0.f;
    }
    __syncthreads();
    const int h2p = (h2 + 3) & ~3;
    const int kh = h2p < kWHalf ? h2p : kWHalf;
    const int ci = 16 * w + (lane & 15);
    f32x4v ch[4] = {};
    mfma_row_dot_chains(sD2 + (lane & 15) * kStrideA + (lane >> 4), 1, sW + (lane >> 4) * kStrideB + ci, kStrideB, kh,
                        ch);
    if (h2p > kWHalf) {                                   // second half of W2's k range
      __syncthreads();
      stage_tile<kWHalf, kHfCols>(sW, kStrideB, W2, ldw2, kWHalf, h2, c0, h1);
      __syncthreads();
      mfma_row_dot_chains(sD2 + (lane & 15) * kStrideA + kWHalf + (lane >> 4), 1, sW + (lane >> 4) * kStrideB + ci,
                          kStrideB, h2p - kWHalf, ch);
    }
    const f32x4v acc = (ch[0] + ch[1]) + (ch[2] + ch[3]);
    const int i = c0 + ci;
    for (int q = 0; q < 4; ++q) {
      const int r = 4 * (lane >> 4) + q;
      const int64_t row = r0 + r;
      float d = 0.f;
      if (row < rows && i < h1) {
        d = sM[r * kMaskStride + ci] > 0.f ? acc[q] : 0.f;
        dZ1[row * ldd1 + i] = d;
      }
      sZ[r * (kHfCols + 1) + ci] = d;
    }
    __syncthreads();
    // partial dW1 / db1 of the tile: one (unit, k) pair per thread, rows in order
    for (int e = tid; e < kHfCols * (in0 + 1); e += 256) {
      const int c = e / (in0 + 1), k = e % (in0 + 1);
      if (c0 + c >= h1) continue;
      float s = 0.f;
      for (int r = 0; r < kHfRows; ++r) s += sZ[r * (kHfCols + 1) + c] * (k < in0 ? sX[r * kSmallIn + k] : 1.f);
      part1[(rt * h1 + c0 + c) * (in0 + 1) + k] = s;
    }
    return;
  }
  // ---------------- role B: dW2[j][i] = sum_b dZ2[b][j] A1[b][i] over the split's rows
  float* sD = smem;                          // [64][kStrideB]: one half of the split's rows
  float* sA = smem + kHbHalf * kStrideB;     // [64][kStrideB]
  const int64_t bid = blockIdx.x - nA;
  const int tj = (h2 + kHbTile - 1) / kHbTile, ti = (h1 + kHbTile - 1) / kHbTile;
  const int64_t kc = bid / (tj * ti);
  const int j0 = (int)((bid / ti) % tj) * kHbTile, i0 = (int)(bid % ti) * kHbTile;
  // wave w: rows j0 + 16 w .. +15 of the tile, all 64 columns (4 accumulators);
  // the split's rows are taken in two halves, in order
  f32x4v acc[4] = {};
  float csum = 0.f;
  for (int half = 0; half < 2; ++half) {
    const int64_t b0 = kc * kHbRows + half * kHbHalf;
    if (half) __syncthreads();
    stage_tile<kHbHalf, kHbTile>(sD, kStrideB, dZ2, ldd2, b0, rows, j0, h2);
    stage_tile<kHbHalf, kHbTile>(sA, kStrideB, A1, lda1, b0, rows, i0, h1);
    __syncthreads();
    const float* pa = sD + (lane >> 4) * kStrideB + 16 * w + (lane & 15);
    const float* pb = sA + (lane >> 4) * kStrideB + (lane & 15);
    float a = pa[0], b[4];
#pragma unroll
    for (int h = 0; h < 4; ++h) b[h] = pb[16 * h];
#pragma unroll 4
    for (int k0 = 0; k0 < kHbHalf; k0 += 4) {
      const int kn = (k0 + 4 < kHbHalf ? k0 + 4 : k0) * kStrideB;
      const float an = pa[kn];
      float bn[4];
#pragma unroll
      for (int h = 0; h < 4; ++h) bn[h] = pb[kn + 16 * h];
#pragma unroll
      for (int h = 0; h < 4; ++h) acc[h] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b[h], acc[h], 0, 0, 0);
      a = an;
#pragma unroll
      for (int h = 0; h < 4; ++h) b[h] = bn[h];
    }
    if (i0 == 0 && tid < kHbTile)
      for (int r = 0; r < kHbHalf; ++r) csum += sD[r * kStrideB + tid];
  }
  for (int h = 0; h < 4; ++h)
    for (int q = 0; q < 4; ++q) {
      const int j = j0 + 16 * w + 4 * (lane >> 4) + q, i = i0 + 16 * h + (lane & 15);
      if (j < h2 && i < h1) part2[(kc * h2 + j) * h1 + i] = acc[h][q];
    }
  if (i0 == 0 && tid < kHbTile && j0 + tid < h2) part2b[kc * h2 + j0 + tid] = csum;
}

// Backward, part 2: dW2[j][i] = sum_kc part2[kc][j][i], db2[j] = sum_kc
// part2b[kc][j], dW1[i][k] = sum_rt part1[rt][i][k], db1[i] = sum_rt
// part1[rt][i][in0], each in index order.  One thread per output element.
__global__ __launch_bounds__(256) void hidden_bwd_reduce_kernel(
    const float* __restrict__ part1, int64_t n_rt, const float* __restrict__ part2, const float* __restrict__ part2b,
    int64_t n_kc, int in0, int h1, int h2, float* __restrict__ dW1, int64_t ldw1, float* __restrict__ db1,
    float* __restrict__ dW2, int64_t ldw2, float* __restrict__ db2) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t n2 = (int64_t)h2 * h1, nb2 = h2, n1 = (int64_t)h1 * (in0 + 1);
  // the loads of 8 terms are issued together, the terms added in index order
  auto sum_strided = [](const float* p, int64_t n, int64_t stride) {
    float s = 0.f;
    int64_t q = 0;
    for (; q + 8 <= n; q += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = p[(q + u) * stride];
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; q < n; ++q) s += p[q * stride];
    return s;
  };
  if (t < n2) {
    dW2[(t / h1) * ldw2 + t % h1] = sum_strided(part2 + t, n_kc, n2);
  } else if (t < n2 + nb2) {
    const int64_t j = t - n2;
    db2[j] = sum_strided(part2b + j, n_kc, h2);
  } else if (t < n2 + nb2 + n1) {
    const int64_t e = t - n2 - nb2, i = e / (in0 + 1), k = e % (in0 + 1);
    const float s = sum_strided(part1 + i * (in0 + 1) + k, n_rt, (int64_t)h1 * (in0 + 1));
    if (k < in0) dW1[i * ldw1 + k] = s;
    else db1[i] = s;
  }
}

}  // namespace ot
