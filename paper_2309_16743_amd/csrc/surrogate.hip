// Surrogate MLP train step and prediction (the paper's deep surrogate of the
// heat equation, Sec. 4.1): forward through ReLU hidden layers and an
// identity output layer whose GEMM epilogue forms the mean-squared-error
// residual, back-propagation, and Adam.  By default the output layer's weights
// are updated inside the epilogue of their weight-gradient GEMM (or of its
// split-K reduction), so that gradient is never stored; one elementwise pass
// updates every other parameter.
//
// Parameter layout (device, fp32): one flat buffer; layer l holds W_l as
// out x ldw (ldw = round_up(in, 8), pad columns stay 0) followed by b_l, each
// segment starting on a 64-float boundary.  Gradients and the Adam moments
// use the same layout, so Adam is a single elementwise pass.
#include <algorithm>
#include <cmath>
#include <mutex>
#include <vector>

#include "common.h"
#include "gemm_bf16.h"
#include "gemm_f32.h"
#include "hidden_small.h"
#include "philox.h"
#include "surrogate.h"

namespace ot {

constexpr int kMaxSmallK = 16;   // layer 1 with in <= 16 uses the small-K kernels

// ------------------------------------------------------------------ small kernels
// Parameter initialisation: element e of layer `layer` (flat over W then b)
// is (2 m / 2^24 - 1) * bound rounded to fp32, m = top 24 bits of Philox word 0
// at counter (e, layer, INIT, 0), key (seed, 0).
__global__ void init_layer_kernel(float* __restrict__ W, float* __restrict__ b, int64_t in,
                                  int64_t out, int64_t ldw, uint64_t seed, uint64_t layer,
                                  double bound) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t nw = in * out;
  if (e >= nw + out) return;
  const uint64_t w = draw_word(seed, (uint64_t)e, layer, kKindInit);
  const double u = 2.0 * ((double)(w >> 40) / 16777216.0) - 1.0;
  const float val = (float)(u * bound);
  if (e < nw) W[(e / in) * ldw + (e % in)] = val;
  else b[e - nw] = val;
}

__global__ void fill_kernel(float* __restrict__ p, int64_t n, float v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// First layer with a small input width K (the 6 inputs (X, t)):
// A1[m][n] = max(sum_k X[m][k] W[n][k] + b[n], 0) (or without ReLU when the
// net has a single layer).  One thread per 4 consecutive outputs.
__global__ void small_k_forward_kernel(const float* __restrict__ X, int64_t ldx,
                                       const float* __restrict__ W, int64_t ldw,
                                       const float* __restrict__ bias, float* __restrict__ out,
                                       int64_t ldo, int64_t M, int64_t N, int64_t K, int relu,
                                       uint16_t* __restrict__ out16) {
  const int64_t groups = (N + 3) / 4;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= M * groups) return;
  const int64_t m = t / groups, n0 = (t % groups) * 4;
  float x[kMaxSmallK];
#pragma unroll
  for (int k = 0; k < kMaxSmallK; ++k) x[k] = k < K ? X[m * ldx + k] : 0.f;
  for (int c = 0; c < 4; ++c) {
    const int64_t n = n0 + c;
    if (n >= N) break;
    float acc = 0.f;
#pragma unroll
    for (int k = 0; k < kMaxSmallK; ++k)
      if (k < K) acc = fmaf(x[k], W[n * ldw + k], acc);
    acc += bias[n];
    const float y = relu ? (acc > 0.f ? acc : 0.f) : acc;
    if (out16) out16[m * ldo + n] = f2bf(y);   // bf16 activations feed the bf16 GEMMs
    else out[m * ldo + n] = y;
  }
}

// First-layer weight gradient, partial sums over a slice of rows:
// part[p][n][k] = sum_{m in slice p} dZ[m][n] X[m][k] (k < K), part[p][n][K] = sum dZ[m][n].
// grid = (ceil(N / 64), P); 256 threads = 64 columns x 4 row groups.
__global__ __launch_bounds__(256) void small_k_wgrad_partial_kernel(
    const float* __restrict__ dZ, int64_t ldz, const float* __restrict__ X, int64_t ldx,
    float* __restrict__ part, int64_t M, int64_t N, int64_t K, int64_t rows_per_part,
    const uint16_t* __restrict__ dZ16) {
  __shared__ float red[4][64][kMaxSmallK + 1];
  const int cn = threadIdx.x % 64, grp = threadIdx.x / 64;
  const int64_t n = (int64_t)blockIdx.x * 64 + cn;
  const int64_t mb = (int64_t)blockIdx.y * rows_per_part;
  const int64_t me = min(M, mb + rows_per_part);
  float acc[kMaxSmallK + 1];
#pragma unroll
  for (int k = 0; k <= kMaxSmallK; ++k) acc[k] = 0.f;
  if (n < N) {
    for (int64_t m = mb + grp; m < me; m += 4) {
      const float d = dZ16 ? bf2f(dZ16[m * ldz + n]) : dZ[m * ldz + n];
#pragma unroll
      for (int k = 0; k < kMaxSmallK; ++k)
        if (k < K) acc[k] = fmaf(d, X[m * ldx + k], acc[k]);
      acc[kMaxSmallK] += d;
    }
  }
#pragma unroll
  for (int k = 0; k <= kMaxSmallK; ++k) red[grp][cn][k] = acc[k];
  __syncthreads();
  if (grp == 0 && n < N) {
    float* dst = part + ((int64_t)blockIdx.y * N + n) * (K + 1);
    for (int k = 0; k < K; ++k) dst[k] = ((red[0][cn][k] + red[1][cn][k]) + red[2][cn][k]) + red[3][cn][k];
    dst[K] = ((red[0][cn][kMaxSmallK] + red[1][cn][kMaxSmallK]) + red[2][cn][kMaxSmallK]) +
             red[3][cn][kMaxSmallK];
  }
}

// Sum the P partial slices in order into dW (ld ldw) and db.
__global__ void small_k_wgrad_reduce_kernel(const float* __restrict__ part, int64_t P, int64_t N,
                                            int64_t K, float* __restrict__ dW, int64_t ldw,
                                            float* __restrict__ db) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= N * (K + 1)) return;
  const int64_t n = t / (K + 1), k = t % (K + 1);
  float s = 0.f;
  for (int64_t p = 0; p < P; ++p) s += part[(p * N + n) * (K + 1) + k];
  if (k < K) dW[n * ldw + k] = s;
  else db[n] = s;
}

// Split-K epilogue: out[m][n] = epi(sum_s ws[s][m][n]) with the splits summed
// in order; epi adds bias[n] (if given), applies ReLU (if relu) and the mask
// (mask[m][n] > 0, if given).  Threads of column group 0 also reduce the
// split row sums rs[s][m] into rowsum_out[m] (if given).
__global__ void splitk_epilogue_kernel(const float* __restrict__ ws, int64_t splits, int64_t split_stride,
                                       int64_t M, int64_t N, int64_t ldws, const float* __restrict__ bias, int relu,
                                       const float* __restrict__ mask, int64_t ldm, float* __restrict__ out,
                                       int64_t ldo, const float* __restrict__ rs, int64_t rs_stride,
                                       float* __restrict__ rowsum_out) {
  const int64_t groups = (N + 3) / 4;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= M * groups) return;
  const int64_t m = t / groups, n = (t % groups) * 4;
  if (rowsum_out && n == 0) {
    float r = rs[m];
    for (int64_t p = 1; p < splits; ++p) r += rs[p * rs_stride + m];
    rowsum_out[m] = r;
  }
  float v[4];
  const int cnt = (int)min((int64_t)4, N - n);
  if (cnt == 4) {
    const f32x4* src = reinterpret_cast<const f32x4*>(ws + m * ldws + n);
    const int64_t st4 = split_stride / 4;
    f32x4 acc = src[0];
    int64_t p = 1;
    // eight loads in flight, added in split order
    for (; p + 8 <= splits; p += 8) {
      f32x4 t[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) t[u] = src[(p + u) * st4];
#pragma unroll
      for (int u = 0; u < 8; ++u) acc += t[u];
    }
    for (; p < splits; ++p) acc += src[p * st4];
    for (int c = 0; c < 4; ++c) v[c] = acc[c];
  } else {
    for (int c = 0; c < cnt; ++c) {
      float a = ws[m * ldws + n + c];
      for (int64_t p = 1; p < splits; ++p) a += ws[p * split_stride + m * ldws + n + c];
      v[c] = a;
    }
  }
  for (int c = 0; c < cnt; ++c) {
    float x = v[c];
    if (bias) x += bias[n + c];
    if (relu) x = x > 0.f ? x : 0.f;
    if (mask) x = mask[m * ldm + n + c] > 0.f ? x : 0.f;
    v[c] = x;
  }
  if (cnt == 4 && ((ldo & 3) == 0) && ((reinterpret_cast<uintptr_t>(out) & 15) == 0)) {
    *reinterpret_cast<f32x4*>(out + m * ldo + n) = f32x4{v[0], v[1], v[2], v[3]};
  } else {
    for (int c = 0; c < cnt; ++c) out[m * ldo + n + c] = v[c];
  }
}

// Evaluation loss over row chunks: acc = (first ? 0 : acc) + sum(partials),
// partials added in a fixed order; the last chunk writes acc * inv_count.
__global__ __launch_bounds__(256) void loss_accumulate_kernel(const double* __restrict__ partials, int64_t n,
                                                              double* __restrict__ acc, int first, int last,
                                                              double inv_count, float* __restrict__ loss) {
  __shared__ double red[256];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 256) s += partials[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double t = (first ? 0.0 : *acc) + red[0];
    *acc = t;
    if (last && loss) *loss = (float)(t * inv_count);
  }
}

// The last pass of a train step: Adam over every parameter except the
// output-layer weights when their update is fused (the 16-byte groups
// [hole, hole + hole_len)), and the batch loss from the forward's partial sums.
struct AdamRest {
  float* p;
  const float* g;
  float* m;
  float* v;
  uint16_t* pb;            // bf16 copy of the weights (nullable)
  int64_t n4, hole, hole_len;
  const double* partials;  // loss partials of the output forward (nullable: no loss)
  int64_t n_partials;
  double inv_count;        // 1 / (B D)
  float* loss_a;           // receive the loss (each nullable)
  float* loss_b;
};

// loss = sum(partials) / count with the partials added in a fixed order
// (strided per thread, then a tree over the 256 threads).  One block of 256.
__device__ void reduce_loss_256(const AdamRest& r) {
  __shared__ double red[256];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < r.n_partials; i += 256) s += r.partials[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const float l = (float)(red[0] * r.inv_count);
    if (r.loss_a) *r.loss_a = l;
    if (r.loss_b) *r.loss_b = l;
  }
}

// Adam (adam1 in adam.h) over groups i = start, start + stride, ... of the
// non-hole 16-byte groups.  Two groups per thread and pass (eight loads in
// flight), non-temporal accesses (the state is touched once per step).
__device__ __forceinline__ void adam_groups(const AdamRest& r, const AdamArgs& a, int64_t i, int64_t stride) {
  f32x4* P = reinterpret_cast<f32x4*>(r.p);
  const f32x4* G = reinterpret_cast<const f32x4*>(r.g);
  f32x4* Mv = reinterpret_cast<f32x4*>(r.m);
  f32x4* V = reinterpret_cast<f32x4*>(r.v);
  u16x4* PB = reinterpret_cast<u16x4*>(r.pb);
  const int64_t n = r.n4 - r.hole_len;   // groups to update
  auto at = [&](int64_t k) { return k < r.hole ? k : k + r.hole_len; };
  for (; i + stride < n; i += 2 * stride) {
    f32x4 pp[2], gg[2], mm[2], vv[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t j = at(i + u * stride);
      pp[u] = __builtin_nontemporal_load(P + j);
      gg[u] = __builtin_nontemporal_load(G + j);
      mm[u] = __builtin_nontemporal_load(Mv + j);
      vv[u] = __builtin_nontemporal_load(V + j);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t j = at(i + u * stride);
      adam4(pp[u], gg[u], mm[u], vv[u], a);
      __builtin_nontemporal_store(pp[u], P + j);
      __builtin_nontemporal_store(mm[u], Mv + j);
      __builtin_nontemporal_store(vv[u], V + j);
      if (PB)   // bf16 copy of the updated master weights
        __builtin_nontemporal_store(u16x4{f2bf(pp[u][0]), f2bf(pp[u][1]), f2bf(pp[u][2]), f2bf(pp[u][3])}, PB + j);
    }
  }
  if (i < n) {
    const int64_t j = at(i);
    f32x4 pp = P[j], mm = Mv[j], vv = V[j];
    adam4(pp, G[j], mm, vv, a);
    P[j] = pp;
    Mv[j] = mm;
    V[j] = vv;
    if (PB) PB[j] = u16x4{f2bf(pp[0]), f2bf(pp[1]), f2bf(pp[2]), f2bf(pp[3])};
  }
}

// Standalone last pass: block 0 also forms the loss.
__global__ __launch_bounds__(256) void adam_kernel(AdamRest r, AdamArgs args) {
  const AdamArgs a = args.resolved();
  if (blockIdx.x == 0 && r.partials) reduce_loss_256(r);
  adam_groups(r, a, (int64_t)blockIdx.x * 256 + threadIdx.x, (int64_t)gridDim.x * 256);
}

// Device step counter of a captured step: one more step completed.
__global__ void step_done_kernel(long long* t_done) {
  if (threadIdx.x == 0 && blockIdx.x == 0) *t_done += 1;
}

// Split-K reduction fused with Adam (fp32 output layer), blocks of 256: the
// first main_blocks blocks take one 4-column group each: the weight gradient
// of element (m, n) is sum_s ws[s][m][n] in split order, exactly as the
// split-K epilogue would store it; Adam then updates p, mo, vo at m * ldp + n;
// threads of column group 0 also reduce the split row sums rs[s][m] into
// rowsum_out[m] (the bias gradient) and, when bias_p is given, apply Adam to
// the bias element m (bias_p, bias_m, bias_v).  The remaining blocks run the
// rest of the step's last pass (AdamRest: the parameters outside the output
// layer, then the loss in the first of them), so the step needs no separate
// Adam launch.
__global__ __launch_bounds__(256) void splitk_adam_kernel(const float* __restrict__ ws, int64_t splits,
                                                          int64_t split_stride, int64_t M, int64_t N, int64_t ldws,
                                                          float* __restrict__ p, float* __restrict__ mo,
                                                          float* __restrict__ vo, int64_t ldp, AdamArgs args,
                                                          const float* __restrict__ rs, int64_t rs_stride,
                                                          float* __restrict__ rowsum_out, float* __restrict__ bias_p,
                                                          float* __restrict__ bias_m, float* __restrict__ bias_v,
                                                          int64_t main_blocks, AdamRest rest) {
  const AdamArgs a = args.resolved();
  if ((int64_t)blockIdx.x >= main_blocks) {
    const int64_t rb = blockIdx.x - main_blocks;
    if (rb == 0 && rest.partials) reduce_loss_256(rest);
    adam_groups(rest, a, rb * 256 + threadIdx.x, ((int64_t)gridDim.x - main_blocks) * 256);
    return;
  }
  const int64_t groups = (N + 3) / 4;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= M * groups) return;
  const int64_t m = t / groups, n = (t % groups) * 4;
  if (rowsum_out && n == 0) {
    float r = rs[m];
    for (int64_t q = 1; q < splits; ++q) r += rs[q * rs_stride + m];
    rowsum_out[m] = r;
    if (bias_p) adam1(bias_p[m], r, bias_m[m], bias_v[m], a);
  }
  const int cnt = (int)min((int64_t)4, N - n);
  const int64_t o = m * ldp + n;
  if (cnt == 4) {
    const f32x4* src = reinterpret_cast<const f32x4*>(ws + m * ldws + n);
    const int64_t st4 = split_stride / 4;
    f32x4 pp = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + o));
    f32x4 mm = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(mo + o));
    f32x4 vv = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(vo + o));
    f32x4 acc = src[0];
    for (int64_t q = 1; q < splits; ++q) acc += src[q * st4];
    adam4(pp, acc, mm, vv, a);
    __builtin_nontemporal_store(pp, reinterpret_cast<f32x4*>(p + o));
    __builtin_nontemporal_store(mm, reinterpret_cast<f32x4*>(mo + o));
    __builtin_nontemporal_store(vv, reinterpret_cast<f32x4*>(vo + o));
  } else {
    for (int c = 0; c < cnt; ++c) {
      float gsum = ws[m * ldws + n + c];
      for (int64_t q = 1; q < splits; ++q) gsum += ws[q * split_stride + m * ldws + n + c];
      float pc = p[o + c], mc = mo[o + c], vc = vo[o + c];
      adam1(pc, gsum, mc, vc, a);
      p[o + c] = pc;
      mo[o + c] = mc;
      vo[o + c] = vc;
    }
  }
}

}  // namespace ot

namespace ot {

// db[n] = sum over m-tiles t (in order) of colsum[t * ld + n].
__global__ void colsum_reduce_kernel(const float* __restrict__ colsum, int64_t tiles, int64_t N, int64_t ld,
                                     float* __restrict__ db) {
  const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  float acc = 0.f;
  for (int64_t t = 0; t < tiles; ++t) acc += colsum[t * ld + n];
  db[n] = acc;
}

// bf16 copy of fp32 values (round to nearest even).
__global__ void to_bf16_kernel(const float* __restrict__ p, uint16_t* __restrict__ pb, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) pb[i] = f2bf(p[i]);
}

// Split-K epilogue with a bf16 result: out[m][n] = bf16(epi(sum_s ws[s][m][n])),
// epi = + bias[n] then ReLU (if relu), or * (mask[m][n] > 0) with a bf16 mask.
__global__ void splitk_epilogue_bf16_kernel(const float* __restrict__ ws, int64_t splits, int64_t split_stride,
                                            int64_t M, int64_t N, int64_t ldws, const float* __restrict__ bias,
                                            int relu, const uint16_t* __restrict__ mask, int64_t ldm,
                                            uint16_t* __restrict__ out, int64_t ldo) {
  const int64_t groups = (N + 3) / 4;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= M * groups) return;
  const int64_t m = t / groups, n = (t % groups) * 4;
  const int cnt = (int)min((int64_t)4, N - n);
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  if (cnt == 4) {
    const f32x4* src = reinterpret_cast<const f32x4*>(ws + m * ldws + n);
    const int64_t st4 = split_stride / 4;
    f32x4 acc = src[0];
    int64_t p = 1;
    for (; p + 8 <= splits; p += 8) {
      f32x4 tt[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) tt[u] = src[(p + u) * st4];
#pragma unroll
      for (int u = 0; u < 8; ++u) acc += tt[u];
    }
    for (; p < splits; ++p) acc += src[p * st4];
    for (int c = 0; c < 4; ++c) v[c] = acc[c];
  } else {
    for (int c = 0; c < cnt; ++c) {
      float a = ws[m * ldws + n + c];
      for (int64_t p = 1; p < splits; ++p) a += ws[p * split_stride + m * ldws + n + c];
      v[c] = a;
    }
  }
  for (int c = 0; c < cnt; ++c) {
    float x = v[c];
    if (bias) x += bias[n + c];
    if (relu) x = x > 0.f ? x : 0.f;
    if (mask) x = bf2f(mask[m * ldm + n + c]) > 0.f ? x : 0.f;
    out[m * ldo + n + c] = f2bf(x);
  }
}

}  // namespace ot

// ===================================================================== host side
namespace {

struct Layer {
  int64_t in = 0, out = 0, ldw = 0;
  int64_t w_off = 0, b_off = 0;
};

}  // namespace

struct ot_surrogate {
  int device = 0;
  int precision = OT_FP32;
  std::vector<int64_t> widths;
  std::vector<Layer> layers;
  int L = 0;
  int64_t n_flat = 0;
  float* params = nullptr;
  float* grads = nullptr;
  float* m = nullptr;
  float* v = nullptr;
  float lr = 1e-3f, beta1 = 0.9f, beta2 = 0.999f, eps = 1e-8f;
  int64_t t = 0;
  bool no_alloc = false;      // inside surrogate_predict_noalloc: workspaces must not grow
  bool fuse_out = false;      // output-layer Adam fused into its weight-gradient epilogue
  bool fused_step = false;    // ... and the current step took that path
  ot::AdamArgs step_adam{};   // Adam scalars of the current step
  // Device step counter (surrogate_set_device_step): steps completed, read by
  // the Adam kernels of every step and advanced by the step's last launch, so
  // that a step's launches can be captured once and replayed.
  long long* t_done_dev = nullptr;
  bool device_step = false;
  // Workspaces, sized for ws_rows batch rows.
  int64_t ws_rows = 0;
  std::vector<float*> act;   // act[l] = A_l, l = 1..L-1 (index 0 unused)
  std::vector<float*> dz;    // dz[l] = dZ_l, l = 1..L (dz[L] = dY)
  std::vector<int64_t> ld;   // ld[l] = round_up(widths[l], 4)
  float* splitws = nullptr;     // split-K partial products
  int64_t splitws_elems = 0;
  float* rsws = nullptr;        // split-K partial row sums (bias gradients)
  int64_t rsws_elems = 0;
  double* loss_partials = nullptr;
  int64_t n_partials_cap = 0;
  float* l1_part = nullptr;
  int64_t l1_part_elems = 0;
  bool small_hidden = false;    // fp32 6 -> H1 -> H2 -> D net with H1, H2 <= 256: fused narrow-layer kernels
  float* hs_part1 = nullptr;    // their partial sums (layer-1 gradient per row tile, layer-2 per k split)
  float* hs_part2 = nullptr;
  float* hs_part2b = nullptr;
  float* loss_last = nullptr;
  double* eval_acc = nullptr;   // running sum of squared residuals of surrogate_eval_loss
  ot::PhaseTimer timer;
  // OT_BF16 only
  uint16_t* pb = nullptr;                  // bf16 copy of the flat parameters
  std::vector<uint16_t*> act16;            // act16[l] = bf16(A_l), l = 1..L-1
  std::vector<uint16_t*> dz16;             // dz16[l] = bf16(dZ_l), l = 1..L (dz16[L] = dY)
  float* colsum = nullptr;                 // per m-tile column sums of dY (output bias gradient)
  int64_t colsum_elems = 0;
};

namespace {

using ot::Epi;
using ot::GemmArgs;
using ot::Lay;

int salloc(void** p, size_t bytes) {
  hipError_t e = hipMalloc(p, bytes ? bytes : 16);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    *p = nullptr;
    return ot::set_error(OT_E_NOMEM, "hipMalloc of %zu bytes failed: %s", bytes, hipGetErrorString(e));
  }
  return OT_OK;
}

void free_workspace(ot_surrogate* s) {
  for (float* p : s->act) (void)hipFree(p);
  for (float* p : s->dz) (void)hipFree(p);
  for (uint16_t* p : s->act16) (void)hipFree(p);
  for (uint16_t* p : s->dz16) (void)hipFree(p);
  s->act.assign(s->L + 1, nullptr);
  s->dz.assign(s->L + 1, nullptr);
  s->act16.assign(s->L + 1, nullptr);
  s->dz16.assign(s->L + 1, nullptr);
  (void)hipFree(s->splitws);
  (void)hipFree(s->rsws);
  (void)hipFree(s->loss_partials);
  (void)hipFree(s->l1_part);
  (void)hipFree(s->hs_part1);
  (void)hipFree(s->hs_part2);
  (void)hipFree(s->hs_part2b);
  s->hs_part1 = s->hs_part2 = s->hs_part2b = nullptr;
  s->splitws = nullptr;
  s->splitws_elems = 0;
  s->rsws = nullptr;
  s->rsws_elems = 0;
  s->loss_partials = nullptr;
  s->l1_part = nullptr;
  s->ws_rows = 0;
}

void free_surrogate(ot_surrogate* s) {
  if (!s) return;
  (void)hipDeviceSynchronize();
  free_workspace(s);
  s->timer.release();
  (void)hipFree(s->params);
  (void)hipFree(s->grads);
  (void)hipFree(s->m);
  (void)hipFree(s->v);
  (void)hipFree(s->loss_last);
  (void)hipFree(s->eval_acc);
  (void)hipFree(s->t_done_dev);
  (void)hipFree(s->pb);
  (void)hipFree(s->colsum);
  delete s;
}

constexpr int64_t kL1Parts = 32;

int refuse_alloc(const char* what) {
  return ot::set_error(OT_E_STATE, "%s would allocate inside surrogate_predict_noalloc", what);
}

int ensure_workspace(ot_surrogate* s, int64_t rows) {
  if (rows <= s->ws_rows) return OT_OK;
  if (s->no_alloc) return refuse_alloc("the batch workspace");
  OT_HIP(hipDeviceSynchronize());
  free_workspace(s);
  const int L = s->L;
  int rc;
  if (s->precision == OT_BF16) {
    for (int l = 1; l < L; ++l)
      if ((rc = salloc((void**)&s->act16[l], (size_t)rows * s->ld[l] * sizeof(uint16_t)))) return rc;
    for (int l = 1; l <= L; ++l)
      if ((rc = salloc((void**)&s->dz16[l], (size_t)rows * s->ld[l] * sizeof(uint16_t)))) return rc;
  } else {
    for (int l = 1; l < L; ++l)
      if ((rc = salloc((void**)&s->act[l], (size_t)rows * s->ld[l] * sizeof(float)))) return rc;
    for (int l = 1; l <= L; ++l)
      if ((rc = salloc((void**)&s->dz[l], (size_t)rows * s->ld[l] * sizeof(float)))) return rc;
  }
  // one loss partial per block of the output GEMM (64 x 64 tiles bound the count)
  s->n_partials_cap = ot::ceil_div(rows, 64) * ot::ceil_div(s->widths[L], 64) + 64;
  if ((rc = salloc((void**)&s->loss_partials, (size_t)s->n_partials_cap * sizeof(double)))) return rc;
  s->l1_part_elems = kL1Parts * s->widths[1] * (s->widths[0] + 1);
  if ((rc = salloc((void**)&s->l1_part, (size_t)s->l1_part_elems * sizeof(float)))) return rc;
  if (s->small_hidden) {
    const int64_t h1 = s->widths[1], h2 = s->widths[2], in0 = s->widths[0];
    const int64_t n_rt = ot::ceil_div(rows, ot::kHfRows), n_kc = ot::ceil_div(rows, ot::kHbRows);
    if ((rc = salloc((void**)&s->hs_part1, (size_t)(n_rt * h1 * (in0 + 1)) * sizeof(float)))) return rc;
    if ((rc = salloc((void**)&s->hs_part2, (size_t)(n_kc * h2 * h1) * sizeof(float)))) return rc;
    if ((rc = salloc((void**)&s->hs_part2b, (size_t)(n_kc * h2) * sizeof(float)))) return rc;
  }
  s->ws_rows = rows;
  return OT_OK;
}

// Tile shapes (4 wavefronts each): 128 x 128, 64 x 128, 64 x 64.
enum Cfg : int { kC128x128 = 0, kC64x128 = 1, kC64x64 = 2 };

int64_t tiles_of(int cfg, int64_t M, int64_t N) {
  switch (cfg) {
    case kC128x128: return ot::gemm_tiles<2, 2, 4, 4>(M, N);
    case kC64x128: return ot::gemm_tiles<2, 2, 2, 4>(M, N);
    default: return ot::gemm_tiles<2, 2, 2, 2>(M, N);
  }
}

struct Plan {
  int cfg = kC64x64;
  int64_t splits = 1;     // k ranges actually launched
  int64_t k_chunk = 0;
  int64_t blocks = 0;
};

// Tile and k-split choice (measured on MI355X at the surrogate's shapes).
// Whole tiles per CU matter more than tile size: a launch whose block count
// leaves some CUs a block more than others loses that fraction, so the plan
// aims for about 4 blocks per CU (960+) with 64 x 128 tiles, splits long k
// ranges (>= 4096) over 128 x 128 tiles, splits medium ones over 64 x 64
// tiles (>= 256 deep per split), and splits short problems down to 32-deep
// ranges until every CU has a block.  The MSE epilogue needs whole sums and
// is never split.
Plan make_plan(int64_t M, int64_t N, int64_t K, bool allow_split) {
  constexpr int64_t kCUs = 256;
  Plan p;
  if (tiles_of(kC64x128, M, N) >= 960 || !allow_split) {
    p.cfg = kC64x128;
    if (tiles_of(kC64x128, M, N) < kCUs) p.cfg = kC64x64;
    if (!allow_split && tiles_of(kC64x64, M, N) < kCUs) p.cfg = kC64x64;
  } else if (K >= 4096) {
    p.cfg = kC128x128;
    const int64_t t = tiles_of(kC128x128, M, N);
    while (t * p.splits < 2 * kCUs - 32 && K / (2 * p.splits) >= 256) p.splits *= 2;
  } else {
    p.cfg = kC64x64;
    const int64_t t = tiles_of(kC64x64, M, N);
    while (t * p.splits < 960 && K / (2 * p.splits) >= 256) p.splits *= 2;
    if (t * p.splits < kCUs)
      while (t * p.splits < kCUs && K / (2 * p.splits) >= 32) p.splits *= 2;
  }
  p.k_chunk = ot::round_up(ot::ceil_div(K, p.splits), 16);
  p.splits = std::max<int64_t>(1, ot::ceil_div(K, p.k_chunk));
  p.blocks = tiles_of(p.cfg, M, N) * p.splits;
  return p;
}

template <Lay LA, Lay LB, Epi EPI, int ROLE>
hipError_t launch_cfg(int cfg, const GemmArgs& g, int64_t splits, hipStream_t st, hipEvent_t t0, hipEvent_t t1) {
  switch (cfg) {
    case kC128x128: return ot::launch_gemm_f32<2, 2, 4, 4, LA, LB, EPI, 16, ROLE>(g, splits, st, t0, t1);
    case kC64x128: return ot::launch_gemm_f32<2, 2, 2, 4, LA, LB, EPI, 16, ROLE>(g, splits, st, t0, t1);
    default: return ot::launch_gemm_f32<2, 2, 2, 2, LA, LB, EPI, 16, ROLE>(g, splits, st, t0, t1);
  }
}

template <Lay LA, Lay LB, int ROLE>
hipError_t launch_epi(Epi epi, int cfg, const GemmArgs& g, int64_t splits, hipStream_t st, hipEvent_t t0 = nullptr,
                      hipEvent_t t1 = nullptr) {
  switch (epi) {
    case Epi::Store: return launch_cfg<LA, LB, Epi::Store, ROLE>(cfg, g, splits, st, t0, t1);
    case Epi::Bias: return launch_cfg<LA, LB, Epi::Bias, ROLE>(cfg, g, splits, st, t0, t1);
    case Epi::BiasRelu: return launch_cfg<LA, LB, Epi::BiasRelu, ROLE>(cfg, g, splits, st, t0, t1);
    case Epi::Mse: return launch_cfg<LA, LB, Epi::Mse, ROLE>(cfg, g, splits, st, t0, t1);
    case Epi::SplitK: return launch_cfg<LA, LB, Epi::SplitK, ROLE>(cfg, g, splits, st, t0, t1);
    case Epi::Adam: return launch_cfg<LA, LB, Epi::Adam, ROLE>(cfg, g, splits, st, t0, t1);
    default: return launch_cfg<LA, LB, Epi::Mask, ROLE>(cfg, g, splits, st, t0, t1);
  }
}

int ensure_colsum(ot_surrogate* s, int64_t elems) {
  if (elems <= s->colsum_elems) return OT_OK;
  if (s->no_alloc) return refuse_alloc("the column-sum buffer");
  OT_HIP(hipDeviceSynchronize());
  (void)hipFree(s->colsum);
  s->colsum = nullptr;
  s->colsum_elems = 0;
  int rc = salloc((void**)&s->colsum, (size_t)elems * sizeof(float));
  if (rc) return rc;
  s->colsum_elems = elems;
  return OT_OK;
}

int ensure_split_ws(ot_surrogate* s, int64_t elems, int64_t rs_elems) {
  if (s->no_alloc && (elems > s->splitws_elems || rs_elems > s->rsws_elems))
    return refuse_alloc("the split-K partials");
  if (elems > s->splitws_elems) {
    OT_HIP(hipDeviceSynchronize());
    (void)hipFree(s->splitws);
    s->splitws = nullptr;
    s->splitws_elems = 0;
    int rc = salloc((void**)&s->splitws, (size_t)elems * sizeof(float));
    if (rc) return rc;
    s->splitws_elems = elems;
  }
  if (rs_elems > s->rsws_elems) {
    OT_HIP(hipDeviceSynchronize());
    (void)hipFree(s->rsws);
    s->rsws = nullptr;
    s->rsws_elems = 0;
    int rc = salloc((void**)&s->rsws, (size_t)rs_elems * sizeof(float));
    if (rc) return rc;
    s->rsws_elems = rs_elems;
  }
  return OT_OK;
}

// C = epi(A B) with the plan's tile shape; split-K runs write partial sums to
// the workspace and a second kernel applies the epilogue (fixed split order).
// ph_gemm / ph_reduce: timing phases of the two halves (-1: not timed).
// rest (Adam epilogue only, nullable): the step's last pass (other parameters
// and loss); when the product is split it runs in extra blocks of the split-K
// Adam reduction and *rest_done is set.
template <Lay LA, Lay LB, int ROLE = 0>
int run_gemm(ot_surrogate* s, GemmArgs g, Epi epi, hipStream_t st, const char* what, bool allow_split,
             int ph_gemm = -1, int ph_reduce = -1, int64_t* blocks_out = nullptr,
             const ot::AdamRest* rest = nullptr, bool* rest_done = nullptr) {
  const Plan p = make_plan(g.M, g.N, g.K, allow_split && epi != Epi::Mse);
  if (blocks_out) *blocks_out = p.blocks;
  ot::PhaseTimer& tm = s->timer;
  if (p.splits == 1) {
    g.k_chunk = g.K;
    hipEvent_t t0 = nullptr, t1 = nullptr;
    if (ph_gemm >= 0) tm.kernel_events(ph_gemm, &t0, &t1);
    hipError_t e = launch_epi<LA, LB, ROLE>(epi, p.cfg, g, 1, st, t0, t1);
    if (e != hipSuccess) return ot::set_error(OT_E_HIP, "launch of %s GEMM failed: %s", what, hipGetErrorString(e));
    return OT_OK;
  }
  const int64_t ldws = ot::round_up(g.N, 4);
  int rc = ensure_split_ws(s, p.splits * g.M * ldws, g.rowsum ? p.splits * g.M : 0);
  if (rc) return rc;
  GemmArgs h = g;
  h.C = s->splitws;
  h.ldc = ldws;
  h.split_stride = g.M * ldws;
  h.k_chunk = p.k_chunk;
  h.rowsum = g.rowsum ? s->rsws : nullptr;
  h.rowsum_stride = g.M;
  hipEvent_t t0 = nullptr, t1 = nullptr;
  if (ph_gemm >= 0) tm.kernel_events(ph_gemm, &t0, &t1);
  hipError_t e = launch_epi<LA, LB, ROLE>(Epi::SplitK, p.cfg, h, p.splits, st, t0, t1);
  if (e != hipSuccess) return ot::set_error(OT_E_HIP, "launch of %s GEMM failed: %s", what, hipGetErrorString(e));
  if (ph_reduce >= 0) tm.mark(st, ph_reduce, 0);
  const int64_t work = g.M * ot::ceil_div(g.N, 4);
  if (epi == Epi::Adam) {
    const int64_t main_blocks = ot::ceil_div(work, 256);
    int64_t rest_blocks = 0;
    ot::AdamRest r{};
    float *bp = nullptr, *bm = nullptr, *bv = nullptr;
    if (rest && g.rowsum) {
      // the output layer is the last segment of the flat buffer: its bias gets
      // its update from the thread that reduces its gradient, the rest pass
      // covers the layers before it
      r = *rest;
      r.hole_len = r.n4 - r.hole;
      const int64_t boff = g.rowsum - s->grads;
      bp = s->params + boff;
      bm = s->m + boff;
      bv = s->v + boff;
      rest_blocks = std::max<int64_t>(1, std::min<int64_t>(ot::ceil_div(r.n4 - r.hole_len, 512), 4096));
      if (rest_done) *rest_done = true;
    }
    hipLaunchKernelGGL(ot::splitk_adam_kernel, dim3((unsigned)(main_blocks + rest_blocks)), dim3(256), 0, st,
                       s->splitws, p.splits, h.split_stride, g.M, g.N, ldws, g.C, g.adam_m, g.adam_v, g.ldc, g.adam,
                       h.rowsum, h.rowsum_stride, g.rowsum, bp, bm, bv, main_blocks, r);
    OT_LAUNCHED("splitk_adam_kernel");
    if (ph_reduce >= 0) tm.mark(st, ph_reduce, 1);
    return OT_OK;
  }
  const bool bias = (epi == Epi::Bias || epi == Epi::BiasRelu);
  hipLaunchKernelGGL(ot::splitk_epilogue_kernel, dim3((unsigned)ot::ceil_div(work, 128)), dim3(128), 0, st,
                     s->splitws, p.splits, h.split_stride, g.M, g.N, ldws, bias ? g.bias : nullptr,
                     epi == Epi::BiasRelu ? 1 : 0, epi == Epi::Mask ? g.mask : nullptr, g.ldmask, g.C, g.ldc,
                     h.rowsum, h.rowsum_stride, g.rowsum);
  OT_LAUNCHED("splitk_epilogue_kernel");
  if (ph_reduce >= 0) tm.mark(st, ph_reduce, 1);
  return OT_OK;
}

GemmArgs args0() {
  GemmArgs g{};
  return g;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Forward pass of layers 1..L-1 into act[]; rows x widths[0] input at X.
int forward_hidden(ot_surrogate* s, const float* X, int64_t ldx, int64_t rows, hipStream_t st) {
  const int L = s->L;
  if (s->small_hidden) {
    const Layer &l1 = s->layers[0], &l2 = s->layers[1];
    const dim3 grid((unsigned)ot::ceil_div(rows, ot::kHfRows), (unsigned)ot::ceil_div(l2.out, ot::kHfCols));
    hipLaunchKernelGGL(ot::hidden_fwd_small_kernel, grid, dim3(256), 0, st, X, ldx, (int)l1.in,
                       s->params + l1.w_off, l1.ldw, s->params + l1.b_off, (int)l1.out, s->params + l2.w_off, l2.ldw,
                       s->params + l2.b_off, (int)l2.out, s->act[1], s->ld[1], s->act[2], s->ld[2], rows);
    OT_LAUNCHED("hidden_fwd_small_kernel");
    return OT_OK;
  }
  for (int l = 1; l < L; ++l) {
    const Layer& ly = s->layers[l - 1];
    const float* W = s->params + ly.w_off;
    const float* b = s->params + ly.b_off;
    if (l == 1 && ly.in <= ot::kMaxSmallK) {
      const int64_t work = rows * ot::ceil_div(ly.out, 4);
      hipLaunchKernelGGL(ot::small_k_forward_kernel, dim3((unsigned)ot::ceil_div(work, 256)), dim3(256), 0, st, X,
                         ldx, W, ly.ldw, b, s->act[1], s->ld[1], rows, ly.out, ly.in, 1, (uint16_t*)nullptr);
      OT_LAUNCHED("small_k_forward_kernel");
      continue;
    }
    GemmArgs g = args0();
    g.A = (l == 1) ? X : s->act[l - 1];
    g.lda = (l == 1) ? ldx : s->ld[l - 1];
    g.B = W;
    g.ldb = ly.ldw;
    g.C = s->act[l];
    g.ldc = s->ld[l];
    g.M = rows;
    g.N = ly.out;
    g.K = ly.in;
    g.bias = b;
    int rc = run_gemm<Lay::KMajor, Lay::KMajor>(s, g, Epi::BiasRelu, st, "hidden forward", true);
    if (rc) return rc;
  }
  return OT_OK;
}

// ------------------------------------------------------------------ bf16 path
using ot::EpiB;
using ot::GemmBArgs;
using ot::LayB;

// bf16 tiles: for large products the pipelined 256 x 128 kernel (k tile 32,
// direct-to-LDS loads, two blocks per CU) or the ping-pong 256 x 256 kernel
// (eight wavefronts, one block per CU); 128 x 128 (4 x 4 fragments per wave)
// and 64 x 64 (2 x 2) with a k tile of 32 otherwise.
enum CfgB : int { kB128 = 0, kB64 = 1, kBPipe = 2, kBPipeW = 3 };
constexpr int kBK = 32;
constexpr int kPipeBK = 32;

int64_t tiles_b(int cfg, int64_t M, int64_t N) {
  if (cfg == kBPipe) return ot::gemm_bf16_pipe_tiles<256, 128>(M, N);
  if (cfg == kBPipeW) return ot::gemm_bf16_pipe_tiles<256, 256>(M, N);
  return cfg == kB128 ? ot::gemm_bf16_tiles<4, 4>(M, N) : ot::gemm_bf16_tiles<2, 2>(M, N);
}

// The 32-deep k tile kernels when k is a multiple of 32 and the tiles give
// about one block per CU or more: products split over long k ranges take the
// ping-pong kernel's 256 x 256 tiles (splits until about two blocks per CU,
// keeping at least 32 k tiles per split), and so do unsplit products with the
// fused MSE epilogue when wide_ok; the others 256 x 128 tiles of the
// pipelined kernel (two blocks per CU).  Else 128 x 128 tiles when they give
// about two blocks per CU; long k ranges are split over 128 x 128 tiles,
// shorter ones over 64 x 64.
// pipe_ok: the 32-deep k tile kernels may be used (they have no row-sum output).
Plan make_plan_b(int64_t M, int64_t N, int64_t K, bool allow_split, bool pipe_ok = true, bool wide_ok = false) {
  constexpr int64_t kCUs = 256;
  Plan p;
  if (wide_ok && pipe_ok && !allow_split && K % kPipeBK == 0 && M >= 256 && N >= 256 &&
      tiles_b(kBPipeW, M, N) >= kCUs - 16) {
    p.cfg = kBPipeW;
    p.k_chunk = K;
    p.splits = 1;
    p.blocks = tiles_b(kBPipeW, M, N);
    return p;
  }
  if (pipe_ok && allow_split && K % kPipeBK == 0 && M >= 256 && N >= 256) {
    const int64_t t = tiles_b(kBPipeW, M, N);
    int64_t sp = 1;
    while (t * sp < 2 * kCUs - 32 && K / (2 * sp) >= 32 * kPipeBK) sp *= 2;
    if (sp > 1 && t * sp >= kCUs - 16) {
      p.cfg = kBPipeW;
      p.k_chunk = ot::round_up(ot::ceil_div(K, sp), kPipeBK);
      p.splits = std::max<int64_t>(1, ot::ceil_div(K, p.k_chunk));
      p.blocks = t * p.splits;
      return p;
    }
  }
  if (pipe_ok && K % kPipeBK == 0 && M >= 256 && N >= 128) {
    const int64_t t = tiles_b(kBPipe, M, N);
    int64_t sp = 1;
    if (allow_split)
      while (t * sp < 4 * kCUs - 64 && K / (2 * sp) >= 32 * kPipeBK) sp *= 2;
    if (t * sp >= kCUs - 16) {
      p.cfg = kBPipe;
      p.k_chunk = ot::round_up(ot::ceil_div(K, sp), kPipeBK);
      p.splits = std::max<int64_t>(1, ot::ceil_div(K, p.k_chunk));
      p.blocks = t * p.splits;
      return p;
    }
  }
  const int64_t t128 = tiles_b(kB128, M, N);
  if (t128 >= 2 * kCUs - 32) {
    p.cfg = kB128;
  } else if (!allow_split) {
    p.cfg = t128 >= kCUs - 16 ? kB128 : kB64;
  } else {
    p.cfg = K >= 4096 ? kB128 : kB64;
    const int64_t t = tiles_b(p.cfg, M, N);
    while (t * p.splits < 2 * kCUs - 32 && K / (2 * p.splits) >= 256) p.splits *= 2;
    if (t * p.splits < kCUs)
      while (t * p.splits < kCUs && K / (2 * p.splits) >= 64) p.splits *= 2;
  }
  p.k_chunk = ot::round_up(ot::ceil_div(K, p.splits), kBK);
  p.splits = std::max<int64_t>(1, ot::ceil_div(K, p.k_chunk));
  p.blocks = tiles_b(p.cfg, M, N) * p.splits;
  return p;
}

template <LayB LA, LayB LB, EpiB E>
hipError_t launch_cfg_b(int cfg, const GemmBArgs& g, int64_t splits, hipStream_t st, hipEvent_t t0 = nullptr,
                        hipEvent_t t1 = nullptr) {
  // 256 x 128 tile, k tile 32, 3 stages, 2 blocks per CU
  if constexpr (E == EpiB::AdamF32) {
    // fused Adam: 128 x 256 tiles, so each tile row of the updated parameters is 1 KB contiguous
    if (cfg == kBPipe) return ot::launch_gemm_bf16_pipe<128, 256, kPipeBK, 3, 2, LA, LB, E>(g, splits, st, t0, t1);
  }
  if (cfg == kBPipe) return ot::launch_gemm_bf16_pipe<256, 128, kPipeBK, 3, 2, LA, LB, E>(g, splits, st, t0, t1);
  if constexpr (E != EpiB::AdamF32) {
    // 256 x 256 tile, eight wavefronts in ping-pong, 4 stages (128 KB of LDS), one block per CU
    if (cfg == kBPipeW) return ot::launch_gemm_bf16_pp<4, LA, LB, E>(g, splits, st, t0, t1);
  }
  if (cfg == kB128) return ot::launch_gemm_bf16<4, 4, LA, LB, E, kBK>(g, splits, st, t0, t1);
  return ot::launch_gemm_bf16<2, 2, LA, LB, E, kBK>(g, splits, st, t0, t1);
}

// C = epi(A B) on bf16 operands; split-K runs write fp32 partials and a
// fixed-order pass applies the epilogue.
template <LayB LA, LayB LB, EpiB E>
int run_gemm_b(ot_surrogate* s, GemmBArgs g, hipStream_t st, const char* what, bool allow_split,
               int ph_gemm = -1, int ph_reduce = -1, int64_t* blocks_out = nullptr) {
  const Plan p = make_plan_b(g.M, g.N, g.K, allow_split && E != EpiB::MseBf && E != EpiB::AdamF32, g.rowsum == nullptr,
                             E == EpiB::MseBf);
  if (blocks_out) *blocks_out = p.blocks;
  ot::PhaseTimer& tm = s->timer;
  if (p.splits == 1) {
    g.k_chunk = p.k_chunk;
    hipEvent_t t0 = nullptr, t1 = nullptr;
    if (ph_gemm >= 0) tm.kernel_events(ph_gemm, &t0, &t1);
    hipError_t e = launch_cfg_b<LA, LB, E>(p.cfg, g, 1, st, t0, t1);
    if (e != hipSuccess) return ot::set_error(OT_E_HIP, "launch of %s GEMM failed: %s", what, hipGetErrorString(e));
    return OT_OK;
  }
  if constexpr (E == EpiB::MseBf || E == EpiB::AdamF32) {
    return ot::set_error(OT_E_STATE, "%s: the MSE and Adam epilogues cannot be split", what);
  } else {
    const int64_t ldws = ot::round_up(g.N, 4);
    int rc = ensure_split_ws(s, p.splits * g.M * ldws, g.rowsum ? p.splits * g.M : 0);
    if (rc) return rc;
    GemmBArgs h = g;
    h.C = s->splitws;
    h.ldc = ldws;
    h.split_stride = g.M * ldws;
    h.k_chunk = p.k_chunk;
    h.rowsum = g.rowsum ? s->rsws : nullptr;
    h.rowsum_stride = g.M;
    hipEvent_t t0 = nullptr, t1 = nullptr;
    if (ph_gemm >= 0) tm.kernel_events(ph_gemm, &t0, &t1);
    hipError_t e = launch_cfg_b<LA, LB, EpiB::SplitK>(p.cfg, h, p.splits, st, t0, t1);
    if (e != hipSuccess) return ot::set_error(OT_E_HIP, "launch of %s GEMM failed: %s", what, hipGetErrorString(e));
    if (ph_reduce >= 0) tm.mark(st, ph_reduce, 0);
    const int64_t work = g.M * ot::ceil_div(g.N, 4);
    if constexpr (E == EpiB::StoreF32 || E == EpiB::BiasF32) {
      hipLaunchKernelGGL(ot::splitk_epilogue_kernel, dim3((unsigned)ot::ceil_div(work, 128)), dim3(128), 0, st,
                         s->splitws, p.splits, h.split_stride, g.M, g.N, ldws,
                         E == EpiB::BiasF32 ? g.bias : nullptr, 0, (const float*)nullptr, (int64_t)0,
                         reinterpret_cast<float*>(g.C), g.ldc, h.rowsum, h.rowsum_stride, g.rowsum);
      OT_LAUNCHED("splitk_epilogue_kernel");
    } else {
      hipLaunchKernelGGL(ot::splitk_epilogue_bf16_kernel, dim3((unsigned)ot::ceil_div(work, 128)), dim3(128), 0, st,
                         s->splitws, p.splits, h.split_stride, g.M, g.N, ldws,
                         E == EpiB::BiasReluBf ? g.bias : nullptr, E == EpiB::BiasReluBf ? 1 : 0,
                         E == EpiB::MaskBf ? g.mask : nullptr, g.ldmask, reinterpret_cast<uint16_t*>(g.C), g.ldc);
      OT_LAUNCHED("splitk_epilogue_bf16_kernel");
    }
    if (ph_reduce >= 0) tm.mark(st, ph_reduce, 1);
    return OT_OK;
  }
}

GemmBArgs bargs0() {
  GemmBArgs g{};
  return g;
}

// bf16 forward of layers 1..L-1 into act16[]: layer 1 in fp32 (K = input width).
int forward_hidden_bf16(ot_surrogate* s, const float* X, int64_t ldx, int64_t rows, hipStream_t st) {
  const int L = s->L;
  for (int l = 1; l < L; ++l) {
    const Layer& ly = s->layers[l - 1];
    if (l == 1) {
      const int64_t work = rows * ot::ceil_div(ly.out, 4);
      hipLaunchKernelGGL(ot::small_k_forward_kernel, dim3((unsigned)ot::ceil_div(work, 256)), dim3(256), 0, st, X,
                         ldx, s->params + ly.w_off, ly.ldw, s->params + ly.b_off, (float*)nullptr, s->ld[1], rows,
                         ly.out, ly.in, 1, s->act16[1]);
      OT_LAUNCHED("small_k_forward_kernel");
      continue;
    }
    GemmBArgs g = bargs0();
    g.A = s->act16[l - 1];
    g.lda = s->ld[l - 1];
    g.B = s->pb + ly.w_off;
    g.ldb = ly.ldw;
    g.C = s->act16[l];
    g.ldc = s->ld[l];
    g.M = rows;
    g.N = ly.out;
    g.K = ly.in;
    g.bias = s->params + ly.b_off;
    int rc = run_gemm_b<LayB::KMajor, LayB::KMajor, EpiB::BiasReluBf>(s, g, st, "bf16 hidden forward", true);
    if (rc) return rc;
  }
  return OT_OK;
}

// bf16 forward of b rows and the output layer's fused MSE epilogue: dY (bf16)
// into dz16[L], per-block loss partials; with bias_grad also the output bias
// gradient (column sums of the rounded dY) into grads.  *n_partials receives
// the number of loss partials.
int forward_mse_bf16(ot_surrogate* s, const float* x, int64_t ldx, const float* u, int64_t ldu, const int32_t* u_rows,
                     int64_t u_rows_max, int64_t b, hipStream_t st, bool bias_grad, int64_t* n_partials) {
  const int L = s->L;
  const int64_t D = s->widths[L];
  ot::PhaseTimer& tm = s->timer;
  int rc;
  tm.mark(st, OT_PH_FWD_HIDDEN, 0);
  if ((rc = forward_hidden_bf16(s, x, ldx, b, st))) return rc;
  tm.mark(st, OT_PH_FWD_HIDDEN, 1);
  const Layer& lo = s->layers[L - 1];
  GemmBArgs g = bargs0();
  g.A = s->act16[L - 1];
  g.lda = s->ld[L - 1];
  g.B = s->pb + lo.w_off;
  g.ldb = lo.ldw;
  g.C = s->dz16[L];
  g.ldc = s->ld[L];
  g.M = b;
  g.N = D;
  g.K = lo.in;
  g.bias = s->params + lo.b_off;
  g.target = u;
  g.ldt = ldu;
  g.target_rows = u_rows;
  g.target_rows_max = u_rows_max;
  g.scale = (float)(2.0 / ((double)b * (double)D));
  g.loss_partials = s->loss_partials;
  if (bias_grad) {
    // output bias gradient: per m-tile column sums of the rounded dY
    const int64_t mtiles = ot::ceil_div(b, 64);
    if ((rc = ensure_colsum(s, mtiles * s->ld[L]))) return rc;
    g.colsum = s->colsum;
    g.colsum_ld = s->ld[L];
  }
  const Plan pf = make_plan_b(g.M, g.N, g.K, false, true, true);
  *n_partials = pf.blocks;
  if (pf.blocks > s->n_partials_cap) return ot::set_error(OT_E_STATE, "loss partial buffer too small");
  if ((rc = run_gemm_b<LayB::KMajor, LayB::KMajor, EpiB::MseBf>(s, g, st, "bf16 output forward+MSE", false,
                                                                OT_PH_FWD_OUTPUT)))
    return rc;
  if (bias_grad) {
    const int64_t used_mtiles = ot::ceil_div(b, (pf.cfg == kBPipe || pf.cfg == kBPipeW) ? 256 : (pf.cfg == kB128 ? 128 : 64));
    hipLaunchKernelGGL(ot::colsum_reduce_kernel, dim3((unsigned)ot::ceil_div(D, 256)), dim3(256), 0, st, s->colsum,
                       used_mtiles, D, s->ld[L], s->grads + lo.b_off);
    OT_LAUNCHED("colsum_reduce_kernel");
  }
  return OT_OK;
}

// Forward, fused MSE and backward of the bf16 path (the loss is reduced and
// Adam applied by the step's last pass); *n_partials: loss partials written.
int train_step_bf16(ot_surrogate* s, const float* x, int64_t ldx, const float* u, int64_t ldu, const int32_t* u_rows,
                    int64_t u_rows_max, int64_t b, hipStream_t st, hipEvent_t targets_read, int64_t* n_partials) {
  const int L = s->L;
  ot::PhaseTimer& tm = s->timer;
  int rc;
  if ((rc = forward_mse_bf16(s, x, ldx, u, ldu, u_rows, u_rows_max, b, st, true, n_partials))) return rc;
  if (targets_read) OT_HIP(hipEventRecord(targets_read, st));

  for (int l = L; l >= 1; --l) {
    if (l == L - 1) tm.mark(st, OT_PH_BWD_HIDDEN, 0);
    const Layer& ly = s->layers[l - 1];
    float* dW = s->grads + ly.w_off;
    float* db = s->grads + ly.b_off;
    if (l == 1) {
      const int64_t rows_per = ot::ceil_div(b, kL1Parts);
      const int64_t P = ot::ceil_div(b, rows_per);
      hipLaunchKernelGGL(ot::small_k_wgrad_partial_kernel, dim3((unsigned)ot::ceil_div(ly.out, 64), (unsigned)P),
                         dim3(256), 0, st, (const float*)nullptr, s->ld[1], x, ldx, s->l1_part, b, ly.out, ly.in,
                         rows_per, s->dz16[1]);
      OT_LAUNCHED("small_k_wgrad_partial_kernel");
      const int64_t n = ly.out * (ly.in + 1);
      hipLaunchKernelGGL(ot::small_k_wgrad_reduce_kernel, dim3((unsigned)ot::ceil_div(n, 256)), dim3(256), 0, st,
                         s->l1_part, P, ly.out, ly.in, dW, ly.ldw, db);
      OT_LAUNCHED("small_k_wgrad_reduce_kernel");
      break;
    }
    const int ph_w = (l == L) ? OT_PH_WGRAD_OUTPUT : -1;
    const bool fused = (l == L) && s->fused_step;
    // weight gradient dW = dZ^T A (the output bias gradient came from the
    // forward epilogue); fused: Adam on W_L in the epilogue instead of a store
    auto wgrad = [&]() -> int {
      GemmBArgs g = bargs0();
      g.A = s->dz16[l];
      g.lda = s->ld[l];
      g.B = s->act16[l - 1];
      g.ldb = s->ld[l - 1];
      g.ldc = ly.ldw;
      g.M = ly.out;
      g.N = ly.in;
      g.K = b;
      if (fused) {
        g.C = s->params + ly.w_off;
        g.adam_m = s->m + ly.w_off;
        g.adam_v = s->v + ly.w_off;
        g.adam_pb = s->pb + ly.w_off;
        g.adam = s->step_adam;
        return run_gemm_b<LayB::MNMajor, LayB::MNMajor, EpiB::AdamF32>(s, g, st, "bf16 weight gradient + Adam",
                                                                       false, ph_w);
      }
      g.C = dW;
      g.rowsum = (l == L) ? nullptr : db;
      return run_gemm_b<LayB::MNMajor, LayB::MNMajor, EpiB::StoreF32>(s, g, st, "bf16 weight gradient", true, ph_w,
                                                                      ph_w >= 0 ? OT_PH_WGRAD_REDUCE : -1);
    };
    // input gradient dA_{l-1} = dZ_l W_l (bf16 copy of W), then the ReLU mask
    auto igrad = [&]() -> int {
      GemmBArgs g = bargs0();
      g.A = s->dz16[l];
      g.lda = s->ld[l];
      g.B = s->pb + ly.w_off;
      g.ldb = ly.ldw;
      g.C = s->dz16[l - 1];
      g.ldc = s->ld[l - 1];
      g.M = b;
      g.N = ly.in;
      g.K = ly.out;
      g.mask = s->act16[l - 1];
      g.ldmask = s->ld[l - 1];
      return run_gemm_b<LayB::KMajor, LayB::MNMajor, EpiB::MaskBf>(s, g, st, "bf16 input gradient", true,
                                                                   l == L ? OT_PH_IGRAD_OUTPUT : -1,
                                                                   l == L ? OT_PH_IGRAD_REDUCE : -1);
    };
    // the fused update rewrites W_L, which the input gradient reads first
    if (fused) {
      if ((rc = igrad()) || (rc = wgrad())) return rc;
    } else {
      if ((rc = wgrad()) || (rc = igrad())) return rc;
    }
  }
  tm.mark(st, OT_PH_BWD_HIDDEN, 1);
  return OT_OK;
}

int predict_bf16(ot_surrogate* s, const float* xr, int64_t ldx, int64_t rows, float* yr, int64_t ldy,
                 hipStream_t st) {
  int rc = forward_hidden_bf16(s, xr, ldx, rows, st);
  if (rc) return rc;
  const int L = s->L;
  const Layer& lo = s->layers[L - 1];
  GemmBArgs g = bargs0();
  g.A = s->act16[L - 1];
  g.lda = s->ld[L - 1];
  g.B = s->pb + lo.w_off;
  g.ldb = lo.ldw;
  g.C = yr;
  g.ldc = ldy;
  g.M = rows;
  g.N = s->widths[L];
  g.K = lo.in;
  g.bias = s->params + lo.b_off;
  return run_gemm_b<LayB::KMajor, LayB::KMajor, EpiB::BiasF32>(s, g, st, "bf16 output forward", true);
}

int check_input(ot_surrogate* s, const float* X, int64_t ldx) {
  OT_REQUIRE(X != nullptr, "input x is NULL");
  OT_REQUIRE(ldx >= s->widths[0], "ldx < input width");
  if (s->widths[0] > ot::kMaxSmallK)
    OT_REQUIRE(aligned16(X) && ldx % 4 == 0, "input width > %d needs 16-byte aligned x and ldx %% 4 == 0",
               ot::kMaxSmallK);
  return OT_OK;
}

}  // namespace

extern "C" int surrogate_create(ot_surrogate** out, const int64_t* widths, int32_t n_widths, int32_t precision,
                                float lr, float beta1, float beta2, float eps, uint64_t seed, int64_t max_batch,
                                uint32_t flags) {
  ot::clear_error();
  OT_REQUIRE(out != nullptr && widths != nullptr, "surrogate_create: NULL argument");
  *out = nullptr;
  OT_REQUIRE(n_widths >= 2 && n_widths <= 16, "surrogate_create: n_widths outside [2, 16]");
  for (int i = 0; i < n_widths; ++i)
    OT_REQUIRE(widths[i] >= 1 && widths[i] <= (1LL << 26), "surrogate_create: width %d outside [1, 2^26]", i);
  OT_REQUIRE(precision == OT_FP32 || precision == OT_BF16, "surrogate_create: unknown precision %d",
             (int)precision);
  if (precision == OT_BF16)
    OT_REQUIRE(n_widths >= 3 && widths[0] <= 16,
               "surrogate_create: bf16 nets need >= 2 layers and an input width <= 16 (first layer runs in fp32)");
  OT_REQUIRE((flags & ~(uint32_t)OT_SURROGATE_KEEP_GRADS) == 0, "surrogate_create: unknown flags 0x%x",
             (unsigned)flags);
  OT_REQUIRE(max_batch >= 1 && max_batch <= (1LL << 20), "surrogate_create: max_batch outside [1, 2^20]");
  OT_REQUIRE(lr >= 0.f && beta1 >= 0.f && beta1 < 1.f && beta2 >= 0.f && beta2 < 1.f && eps > 0.f,
             "surrogate_create: bad Adam hyper-parameters");
  ot_surrogate* s = new ot_surrogate();
  s->precision = precision;
  s->widths.assign(widths, widths + n_widths);
  s->L = n_widths - 1;
  s->lr = lr;
  s->beta1 = beta1;
  s->beta2 = beta2;
  s->eps = eps;
  s->fuse_out = (flags & OT_SURROGATE_KEEP_GRADS) == 0;
  s->small_hidden = precision == OT_FP32 && n_widths == 4 && widths[0] <= ot::kSmallIn &&
                    widths[1] <= ot::kSmallH && widths[2] <= ot::kSmallH;
  s->ld.resize(n_widths);
  for (int i = 0; i < n_widths; ++i) s->ld[i] = ot::round_up(widths[i], 8);
  int64_t off = 0;
  for (int l = 0; l < s->L; ++l) {
    Layer ly;
    ly.in = widths[l];
    ly.out = widths[l + 1];
    ly.ldw = ot::round_up(ly.in, 8);
    ly.w_off = off;
    off = ot::round_up(off + ly.out * ly.ldw, 64);
    ly.b_off = off;
    off = ot::round_up(off + ly.out, 64);
    s->layers.push_back(ly);
  }
  s->n_flat = off;
  s->act.assign(s->L + 1, nullptr);
  s->dz.assign(s->L + 1, nullptr);
  s->act16.assign(s->L + 1, nullptr);
  s->dz16.assign(s->L + 1, nullptr);
  auto fail = [&](int code) {
    free_surrogate(s);
    return code;
  };
  if (hipGetDevice(&s->device) != hipSuccess) return fail(ot::set_error(OT_E_HIP, "hipGetDevice failed"));
  int rc;
  const size_t bytes = (size_t)s->n_flat * sizeof(float);
  if ((rc = salloc((void**)&s->params, bytes))) return fail(rc);
  if ((rc = salloc((void**)&s->grads, bytes))) return fail(rc);
  if ((rc = salloc((void**)&s->m, bytes))) return fail(rc);
  if ((rc = salloc((void**)&s->v, bytes))) return fail(rc);
  if ((rc = salloc((void**)&s->loss_last, 16))) return fail(rc);
  if ((rc = salloc((void**)&s->eval_acc, 16))) return fail(rc);
  const unsigned fb = (unsigned)ot::ceil_div(s->n_flat, 256);
  for (float* p : {s->params, s->grads, s->m, s->v}) {
    hipLaunchKernelGGL(ot::fill_kernel, dim3(fb), dim3(256), 0, 0, p, s->n_flat, 0.f);
  }
  for (int l = 0; l < s->L; ++l) {
    const Layer& ly = s->layers[l];
    const int64_t n = ly.in * ly.out + ly.out;
    hipLaunchKernelGGL(ot::init_layer_kernel, dim3((unsigned)ot::ceil_div(n, 256)), dim3(256), 0, 0,
                       s->params + ly.w_off, s->params + ly.b_off, ly.in, ly.out, ly.ldw, seed, (uint64_t)l,
                       1.0 / std::sqrt((double)ly.in));
  }
  if (precision == OT_BF16) {
    if ((rc = salloc((void**)&s->pb, (size_t)s->n_flat * sizeof(uint16_t)))) return fail(rc);
    hipLaunchKernelGGL(ot::to_bf16_kernel, dim3(fb), dim3(256), 0, 0, s->params, s->pb, s->n_flat);
  }
  if (hipGetLastError() != hipSuccess) return fail(ot::set_error(OT_E_HIP, "initialisation launch failed"));
  if ((rc = ensure_workspace(s, max_batch))) return fail(rc);
  if (hipDeviceSynchronize() != hipSuccess) return fail(ot::set_error(OT_E_HIP, "initialisation failed"));
  *out = s;
  return OT_OK;
}

extern "C" int surrogate_destroy(ot_surrogate* s) {
  ot::clear_error();
  free_surrogate(s);
  return OT_OK;
}

namespace {

int copy_layer(ot_surrogate* s, int32_t layer, const float* buf, float* W_host, float* b_host) {
  OT_REQUIRE(s != nullptr && layer >= 0 && layer < s->L, "layer index out of range");
  const Layer& ly = s->layers[layer];
  OT_HIP(hipDeviceSynchronize());
  if (W_host)
    OT_HIP(hipMemcpy2D(W_host, ly.in * sizeof(float), buf + ly.w_off, ly.ldw * sizeof(float), ly.in * sizeof(float),
                       ly.out, hipMemcpyDeviceToHost));
  if (b_host) OT_HIP(hipMemcpy(b_host, buf + ly.b_off, ly.out * sizeof(float), hipMemcpyDeviceToHost));
  return OT_OK;
}

}  // namespace

extern "C" int surrogate_set_params(ot_surrogate* s, int32_t layer, const float* W_host, const float* b_host) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr && layer >= 0 && layer < s->L, "surrogate_set_params: layer index out of range");
  const Layer& ly = s->layers[layer];
  OT_HIP(hipDeviceSynchronize());
  if (W_host)
    OT_HIP(hipMemcpy2D(s->params + ly.w_off, ly.ldw * sizeof(float), W_host, ly.in * sizeof(float),
                       ly.in * sizeof(float), ly.out, hipMemcpyHostToDevice));
  if (b_host) OT_HIP(hipMemcpy(s->params + ly.b_off, b_host, ly.out * sizeof(float), hipMemcpyHostToDevice));
  if (s->pb) {
    hipLaunchKernelGGL(ot::to_bf16_kernel, dim3((unsigned)ot::ceil_div(s->n_flat, 256)), dim3(256), 0, 0, s->params,
                       s->pb, s->n_flat);
    OT_LAUNCHED("to_bf16_kernel");
    OT_HIP(hipDeviceSynchronize());
  }
  return OT_OK;
}

extern "C" int surrogate_get_params(ot_surrogate* s, int32_t layer, float* W_host, float* b_host) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr, "surrogate_get_params: NULL surrogate");
  return copy_layer(s, layer, s->params, W_host, b_host);
}

extern "C" int surrogate_get_grads(ot_surrogate* s, int32_t layer, float* dW_host, float* db_host) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr, "surrogate_get_grads: NULL surrogate");
  if (s->fused_step && layer == s->L - 1 && dW_host != nullptr)
    return ot::set_error(OT_E_STATE,
                         "surrogate_get_grads: the output-layer weight gradient is not stored when its Adam update "
                         "is fused (create the surrogate with OT_SURROGATE_KEEP_GRADS)");
  return copy_layer(s, layer, s->grads, dW_host, db_host);
}

// The host's step count after steps that ran with the device counter (a
// captured step replayed advances only the device's).
static int sync_step_count(ot_surrogate* s) {
  if (!s->device_step) return OT_OK;
  OT_HIP(hipDeviceSynchronize());
  long long t = 0;
  OT_HIP(hipMemcpy(&t, s->t_done_dev, sizeof t, hipMemcpyDeviceToHost));
  s->t = t;
  return OT_OK;
}

extern "C" int surrogate_get_adam_state(ot_surrogate* s, int32_t layer, float* mW_host, float* mb_host,
                                        float* vW_host, float* vb_host, int64_t* t_out) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr, "surrogate_get_adam_state: NULL surrogate");
  int rc = sync_step_count(s);
  if (rc) return rc;
  rc = copy_layer(s, layer, s->m, mW_host, mb_host);
  if (rc) return rc;
  rc = copy_layer(s, layer, s->v, vW_host, vb_host);
  if (rc) return rc;
  if (t_out) *t_out = s->t;
  return OT_OK;
}

extern "C" int surrogate_set_lr(ot_surrogate* s, float lr) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr && lr >= 0.f, "surrogate_set_lr: bad argument");
  s->lr = lr;
  return OT_OK;
}

// Adam scalars of the step about to run (t counts from 1).
static void begin_step(ot_surrogate* s) {
  s->t += 1;
  s->step_adam = ot::AdamArgs{s->lr, s->beta1, s->beta2, s->eps, ot::bias_correction(s->beta1, s->t),
                              ot::bias_correction(s->beta2, s->t), s->device_step ? s->t_done_dev : nullptr};
  const Layer& lo = s->layers[s->L - 1];
  // a single layer with a small input width takes the small-K gradient kernels, which store
  s->fused_step = s->fuse_out && !(s->L == 1 && lo.in <= ot::kMaxSmallK);
}

// The step's last pass: Adam over every parameter (and the bf16 weight copy
// in OT_BF16 mode) except the output-layer weights when the step updated them
// in the fused epilogue, with the loss from the forward's partial sums
// reduced in its first block.
static ot::AdamRest make_rest(ot_surrogate* s, int64_t n_partials, int64_t rows, float* loss_dev) {
  const Layer& lo = s->layers[s->L - 1];
  ot::AdamRest r{};
  r.p = s->params;
  r.g = s->grads;
  r.m = s->m;
  r.v = s->v;
  r.pb = s->pb;
  r.n4 = s->n_flat / 4;
  r.hole = s->fused_step ? lo.w_off / 4 : 0;
  r.hole_len = s->fused_step ? (lo.b_off - lo.w_off) / 4 : 0;
  r.partials = s->loss_partials;
  r.n_partials = n_partials;
  r.inv_count = 1.0 / ((double)rows * (double)s->widths[s->L]);
  r.loss_a = loss_dev;
  r.loss_b = s->loss_last;
  return r;
}

static int adam_step(ot_surrogate* s, hipStream_t st, const ot::AdamRest& r) {
  ot::PhaseTimer& tm = s->timer;
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>(ot::ceil_div(r.n4 - r.hole_len, 256), 32768));
  tm.mark(st, OT_PH_ADAM, 0);
  hipLaunchKernelGGL(ot::adam_kernel, dim3((unsigned)blocks), dim3(256), 0, st, r, s->step_adam);
  OT_LAUNCHED("adam_kernel");
  tm.mark(st, OT_PH_ADAM, 1);
  return OT_OK;
}

// fp32 forward of b rows and the output layer's fused bias + MSE epilogue:
// dY = 2 (Y - U) / (B D) into dz[L], per-block loss partials.
static int forward_mse_f32(ot_surrogate* s, const float* x, int64_t ldx, const float* u, int64_t ldu,
                           const int32_t* u_rows, int64_t u_rows_max, int64_t b, hipStream_t st,
                           int64_t* n_partials) {
  const int L = s->L;
  const int64_t D = s->widths[L];
  ot::PhaseTimer& tm = s->timer;
  int rc;
  tm.mark(st, OT_PH_FWD_HIDDEN, 0);
  if ((rc = forward_hidden(s, x, ldx, b, st))) return rc;
  tm.mark(st, OT_PH_FWD_HIDDEN, 1);
  const Layer& lo = s->layers[L - 1];
  GemmArgs g = args0();
  g.A = (L == 1) ? x : s->act[L - 1];
  g.lda = (L == 1) ? ldx : s->ld[L - 1];
  g.B = s->params + lo.w_off;
  g.ldb = lo.ldw;
  g.C = s->dz[L];
  g.ldc = s->ld[L];
  g.M = b;
  g.N = D;
  g.K = lo.in;
  g.bias = s->params + lo.b_off;
  g.target = u;
  g.ldt = ldu;
  g.target_rows = u_rows;
  g.target_rows_max = u_rows_max;
  g.scale = (float)(2.0 / ((double)b * (double)D));
  g.loss_partials = s->loss_partials;
  *n_partials = make_plan(g.M, g.N, g.K, false).blocks;
  if (*n_partials > s->n_partials_cap) return ot::set_error(OT_E_STATE, "loss partial buffer too small");
  return run_gemm<Lay::KMajor, Lay::KMajor, 1>(s, g, Epi::Mse, st, "output forward+MSE", false, OT_PH_FWD_OUTPUT);
}

// Input checks shared by train_step and eval_loss (before any state changes).
static int check_batch(ot_surrogate* s, const float* x, int64_t ldx, const float* u, int64_t ldu, const char* what) {
  int rc = check_input(s, x, ldx);
  if (rc) return rc;
  const int L = s->L;
  OT_REQUIRE(u != nullptr && ldu >= s->widths[L] && ldu % 4 == 0 && aligned16(u),
             "%s: targets need 16-byte alignment and ldu >= D, ldu %% 4 == 0", what);
  if (L == 1 && s->layers[0].in <= ot::kMaxSmallK)
    OT_REQUIRE(aligned16(x) && ldx % 4 == 0, "single-layer nets need 16-byte aligned x, ldx %% 4 == 0");
  return OT_OK;
}

// The train step.  u_rows (nullable): target row j is u + u_rows[j] * ldu
// (indices clamped to [0, u_rows_max]); targets_read (nullable): recorded on
// the stream once every target has been read.
static int train_step_launches(ot_surrogate* s, const float* x, int64_t ldx, const float* u, int64_t ldu,
                               const int32_t* u_rows, int64_t u_rows_max, int64_t b, void* stream, float* loss_dev,
                               hipEvent_t targets_read) {
  const int L = s->L;
  int rc;
  const int64_t D = s->widths[L];
  if ((rc = ensure_workspace(s, b))) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  begin_step(s);

  ot::PhaseTimer& tm = s->timer;
  int64_t n_partials = 0;
  if (s->precision == OT_BF16) {
    if ((rc = train_step_bf16(s, x, ldx, u, ldu, u_rows, u_rows_max, b, st, targets_read, &n_partials))) return rc;
    rc = adam_step(s, st, make_rest(s, n_partials, b, loss_dev));
    tm.next_call();
    return rc;
  }
  if ((rc = forward_mse_f32(s, x, ldx, u, ldu, u_rows, u_rows_max, b, st, &n_partials))) return rc;
  if (targets_read) OT_HIP(hipEventRecord(targets_read, st));
  const ot::AdamRest rest = make_rest(s, n_partials, b, loss_dev);
  bool rest_done = false;

  // weight and bias gradient of layer l: dW = dZ^T A_in, db = column sums of
  // dZ; for the output layer of a fused step, Adam on W_L in the epilogue (or
  // the split-K reduction, which then also runs the step's last pass)
  auto wgrad = [&](int l) -> int {
    const int ph_w = (l == L) ? OT_PH_WGRAD_OUTPUT : -1;
    const Layer& ly = s->layers[l - 1];
    const float* A_in = (l == 1) ? x : s->act[l - 1];
    const int64_t ld_in = (l == 1) ? ldx : s->ld[l - 1];
    float* dW = s->grads + ly.w_off;
    float* db = s->grads + ly.b_off;
    if (l == 1 && ly.in <= ot::kMaxSmallK) {
      if (ph_w >= 0) tm.mark(st, ph_w, 0);
      const int64_t rows_per = ot::ceil_div(b, kL1Parts);
      const int64_t P = ot::ceil_div(b, rows_per);
      hipLaunchKernelGGL(ot::small_k_wgrad_partial_kernel, dim3((unsigned)ot::ceil_div(ly.out, 64), (unsigned)P),
                         dim3(256), 0, st, s->dz[1], s->ld[1], x, ldx, s->l1_part, b, ly.out, ly.in, rows_per,
                         (const uint16_t*)nullptr);
      OT_LAUNCHED("small_k_wgrad_partial_kernel");
      const int64_t n = ly.out * (ly.in + 1);
      hipLaunchKernelGGL(ot::small_k_wgrad_reduce_kernel, dim3((unsigned)ot::ceil_div(n, 256)), dim3(256), 0, st,
                         s->l1_part, P, ly.out, ly.in, dW, ly.ldw, db);
      OT_LAUNCHED("small_k_wgrad_reduce_kernel");
      if (ph_w >= 0) tm.mark(st, ph_w, 1);
      return OT_OK;
    }
    GemmArgs g = args0();
    g.A = s->dz[l];
    g.lda = s->ld[l];
    g.B = A_in;
    g.ldb = ld_in;
    g.C = dW;
    g.ldc = ly.ldw;
    g.M = ly.out;
    g.N = ly.in;
    g.K = b;
    g.rowsum = db;
    if (l == L && s->fused_step) {
      g.C = s->params + ly.w_off;
      g.adam_m = s->m + ly.w_off;
      g.adam_v = s->v + ly.w_off;
      g.adam = s->step_adam;
      return run_gemm<Lay::MNMajor, Lay::MNMajor, 1>(s, g, Epi::Adam, st, "weight gradient + Adam", true, ph_w,
                                                     OT_PH_WGRAD_REDUCE, nullptr, &rest, &rest_done);
    }
    return (l == L) ? run_gemm<Lay::MNMajor, Lay::MNMajor, 1>(s, g, Epi::Store, st, "weight gradient", true, ph_w,
                                                              OT_PH_WGRAD_REDUCE)
                    : run_gemm<Lay::MNMajor, Lay::MNMajor, 0>(s, g, Epi::Store, st, "weight gradient", true);
  };
  // input gradient dA_{l-1} = dZ_l W_l, then the ReLU mask of layer l-1
  auto igrad = [&](int l) -> int {
    const Layer& ly = s->layers[l - 1];
    GemmArgs g = args0();
    g.A = s->dz[l];
    g.lda = s->ld[l];
    g.B = s->params + ly.w_off;
    g.ldb = ly.ldw;
    g.M = b;
    g.N = ly.in;
    g.K = ly.out;
    g.C = s->dz[l - 1];
    g.ldc = s->ld[l - 1];
    g.mask = s->act[l - 1];
    g.ldmask = s->ld[l - 1];
    return (l == L) ? run_gemm<Lay::KMajor, Lay::MNMajor, 1>(s, g, Epi::Mask, st, "input gradient", true,
                                                             OT_PH_IGRAD_OUTPUT, OT_PH_IGRAD_REDUCE)
                    : run_gemm<Lay::KMajor, Lay::MNMajor, 0>(s, g, Epi::Mask, st, "input gradient", true);
  };

  // ---- backward, layer by layer from the output.  A fused step computes the
  // output layer's input gradient first (it reads W_L), runs the hidden
  // layers, and updates W_L last, so that its split-K reduction can carry the
  // step's last pass.
  const bool defer_out = s->fused_step && L >= 2;
  for (int l = L; l >= 1; --l) {
    if (l == L - 1) {
      tm.mark(st, OT_PH_BWD_HIDDEN, 0);
      if (s->small_hidden) {   // layers 2 and 1 in two launches
        const Layer &l1 = s->layers[0], &l2 = s->layers[1];
        const int64_t n_rt = ot::ceil_div(b, ot::kHfRows), n_kc = ot::ceil_div(b, ot::kHbRows);
        const int64_t nA = n_rt * ot::ceil_div(l1.out, ot::kHfCols);
        const int64_t nB = n_kc * ot::ceil_div(l2.out, ot::kHbTile) * ot::ceil_div(l1.out, ot::kHbTile);
        hipLaunchKernelGGL(ot::hidden_bwd_small_kernel, dim3((unsigned)(nA + nB)), dim3(256), 0, st, s->dz[2],
                           s->ld[2], s->act[1], s->ld[1], x, ldx, (int)l1.in, s->params + l2.w_off, l2.ldw,
                           (int)l1.out, (int)l2.out, b, s->dz[1], s->ld[1], s->hs_part1, s->hs_part2, s->hs_part2b,
                           nA);
        OT_LAUNCHED("hidden_bwd_small_kernel");
        const int64_t n_out = l2.out * l1.out + l2.out + l1.out * (l1.in + 1);
        hipLaunchKernelGGL(ot::hidden_bwd_reduce_kernel, dim3((unsigned)ot::ceil_div(n_out, 256)), dim3(256), 0, st,
                           s->hs_part1, n_rt, s->hs_part2, s->hs_part2b, n_kc, (int)l1.in, (int)l1.out, (int)l2.out,
                           s->grads + l1.w_off, l1.ldw, s->grads + l1.b_off, s->grads + l2.w_off, l2.ldw,
                           s->grads + l2.b_off);
        OT_LAUNCHED("hidden_bwd_reduce_kernel");
        break;
      }
    }
    if (l == 1) {
      if ((rc = wgrad(1))) return rc;
      break;
    }
    if (l == L && defer_out) {
      if ((rc = igrad(l))) return rc;
      continue;
    }
    if ((rc = wgrad(l)) || (rc = igrad(l))) return rc;
  }
  if (L >= 2) tm.mark(st, OT_PH_BWD_HIDDEN, 1);
  if (defer_out && (rc = wgrad(L))) return rc;
  if (!rest_done) rc = adam_step(s, st, rest);
  tm.next_call();
  return rc;
}

// One train step; with the device step counter on, its last launch advances
// the counter that the step's Adam kernels read.
static int train_step(ot_surrogate* s, const float* x, int64_t ldx, const float* u, int64_t ldu,
                      const int32_t* u_rows, int64_t u_rows_max, int64_t b, void* stream, float* loss_dev,
                      hipEvent_t targets_read) {
  int rc = train_step_launches(s, x, ldx, u, ldu, u_rows, u_rows_max, b, stream, loss_dev, targets_read);
  if (rc == OT_OK && s->device_step) {
    hipLaunchKernelGGL(ot::step_done_kernel, dim3(1), dim3(64), 0, static_cast<hipStream_t>(stream), s->t_done_dev);
    OT_LAUNCHED("step_done_kernel");
  }
  return rc;
}

extern "C" int surrogate_set_device_step(ot_surrogate* s, int32_t enable) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr, "surrogate_set_device_step: NULL surrogate");
  OT_REQUIRE(enable == 0 || enable == 1, "surrogate_set_device_step: enable must be 0 or 1");
  if ((enable != 0) == s->device_step) return OT_OK;
  if (enable) {
    if (!s->t_done_dev) {
      int rc = salloc((void**)&s->t_done_dev, sizeof(long long));
      if (rc) return rc;
    }
    OT_HIP(hipDeviceSynchronize());
    const long long t = s->t;
    OT_HIP(hipMemcpy(s->t_done_dev, &t, sizeof t, hipMemcpyHostToDevice));
    s->device_step = true;
    return OT_OK;
  }
  int rc = sync_step_count(s);
  s->device_step = false;
  return rc;
}

extern "C" int surrogate_train_step(ot_surrogate* s, const float* x, int64_t ldx, const float* u, int64_t ldu,
                                    int64_t b, void* stream, float* loss_dev) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr, "surrogate_train_step: NULL surrogate");
  OT_REQUIRE(b >= 1 && b <= (1LL << 20), "surrogate_train_step: b outside [1, 2^20]");
  int rc = check_batch(s, x, ldx, u, ldu, "surrogate_train_step");
  if (rc) return rc;
  return train_step(s, x, ldx, u, ldu, nullptr, 0, b, stream, loss_dev, nullptr);
}

extern "C" int surrogate_train_step_rows(ot_surrogate* s, const float* x, int64_t ldx, const float* u, int64_t ldu,
                                         const int32_t* rows, int64_t n_rows, int64_t b, void* stream,
                                         float* loss_dev, void* targets_read) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr, "surrogate_train_step_rows: NULL surrogate");
  OT_REQUIRE(b >= 1 && b <= (1LL << 20), "surrogate_train_step_rows: b outside [1, 2^20]");
  OT_REQUIRE(rows != nullptr && (reinterpret_cast<uintptr_t>(rows) & 3u) == 0,
             "surrogate_train_step_rows: rows must be a 4-byte aligned device int32 array");
  OT_REQUIRE(n_rows >= 1 && n_rows <= (1LL << 31), "surrogate_train_step_rows: n_rows outside [1, 2^31]");
  int rc = check_batch(s, x, ldx, u, ldu, "surrogate_train_step_rows");
  if (rc) return rc;
  return train_step(s, x, ldx, u, ldu, rows, n_rows - 1, b, stream, loss_dev, static_cast<hipEvent_t>(targets_read));
}

extern "C" int surrogate_eval_loss(ot_surrogate* s, const float* x, int64_t ldx, const float* u, int64_t ldu,
                                   int64_t n, void* stream, float* loss_dev) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr, "surrogate_eval_loss: NULL surrogate");
  OT_REQUIRE(n >= 1, "surrogate_eval_loss: n < 1");
  OT_REQUIRE(loss_dev != nullptr, "surrogate_eval_loss: loss_dev is NULL");
  int rc = check_batch(s, x, ldx, u, ldu, "surrogate_eval_loss");
  if (rc) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t chunk = std::max<int64_t>(s->ws_rows, 1);
  const int64_t D = s->widths[s->L];
  for (int64_t r0 = 0; r0 < n; r0 += chunk) {
    const int64_t rows = std::min(chunk, n - r0);
    int64_t n_partials = 0;
    rc = (s->precision == OT_BF16)
             ? forward_mse_bf16(s, x + r0 * ldx, ldx, u + r0 * ldu, ldu, nullptr, 0, rows, st, false, &n_partials)
             : forward_mse_f32(s, x + r0 * ldx, ldx, u + r0 * ldu, ldu, nullptr, 0, rows, st, &n_partials);
    if (rc) return rc;
    hipLaunchKernelGGL(ot::loss_accumulate_kernel, dim3(1), dim3(256), 0, st, s->loss_partials, n_partials,
                       s->eval_acc, r0 == 0 ? 1 : 0, r0 + rows >= n ? 1 : 0, 1.0 / ((double)n * (double)D),
                       loss_dev);
    OT_LAUNCHED("loss_accumulate_kernel");
  }
  return OT_OK;
}

// ------------------------------------------------------------------ checkpoint
// Blob layout (host memory, native byte order): magic "OTSURV1", int64
// precision, n_widths, widths[n_widths], t, n_flat; float lr, beta1, beta2,
// eps; then the flat fp32 parameters, first and second Adam moments
// (n_flat each, the device layout).  Gradients are not state (every step
// recomputes them); the bf16 weight copy is rounded again from the restored
// master weights.
namespace {
constexpr char kSurMagic[8] = {'O', 'T', 'S', 'U', 'R', 'V', '1', 0};

int64_t sur_blob_bytes(const ot_surrogate* s) {
  return 8 + 8 * (2 + (int64_t)s->widths.size() + 2) + 4 * 4 + 3 * s->n_flat * 4;
}
}  // namespace

extern "C" int surrogate_checkpoint_size(ot_surrogate* s, int64_t* bytes) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr && bytes != nullptr, "surrogate_checkpoint_size: NULL argument");
  *bytes = sur_blob_bytes(s);
  return OT_OK;
}

extern "C" int surrogate_checkpoint(ot_surrogate* s, void* buf, int64_t bytes) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr && buf != nullptr, "surrogate_checkpoint: NULL argument");
  OT_REQUIRE(bytes >= sur_blob_bytes(s), "surrogate_checkpoint: buffer of %lld bytes, %lld needed",
             (long long)bytes, (long long)sur_blob_bytes(s));
  int rc = sync_step_count(s);
  if (rc) return rc;
  OT_HIP(hipDeviceSynchronize());
  ot::BlobWriter w(buf, bytes);
  __builtin_memcpy(w.take(8), kSurMagic, 8);
  w.put((int64_t)s->precision);
  w.put((int64_t)s->widths.size());
  for (int64_t v : s->widths) w.put(v);
  w.put(s->t);
  w.put(s->n_flat);
  for (float v : {s->lr, s->beta1, s->beta2, s->eps}) w.put(v);
  for (const float* src : {s->params, s->m, s->v})
    OT_HIP(hipMemcpy(w.take(s->n_flat * 4), src, s->n_flat * 4, hipMemcpyDeviceToHost));
  return w.good ? OT_OK : ot::set_error(OT_E_STATE, "surrogate_checkpoint: blob overrun");
}

extern "C" int surrogate_restore(ot_surrogate* s, const void* buf, int64_t bytes) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr && buf != nullptr, "surrogate_restore: NULL argument");
  ot::BlobReader rd(buf, bytes);
  const unsigned char* magic = rd.take(8);
  OT_REQUIRE(magic != nullptr && __builtin_memcmp(magic, kSurMagic, 8) == 0,
             "surrogate_restore: not a surrogate checkpoint");
  const int64_t precision = rd.get<int64_t>(), nw = rd.get<int64_t>();
  OT_REQUIRE(rd.good && precision == s->precision && nw == (int64_t)s->widths.size(),
             "surrogate_restore: checkpoint of a different surrogate (precision or depth)");
  for (int64_t i = 0; i < nw; ++i)
    OT_REQUIRE(rd.get<int64_t>() == s->widths[i], "surrogate_restore: width %lld differs", (long long)i);
  const int64_t t = rd.get<int64_t>(), n_flat = rd.get<int64_t>();
  float hp[4];
  for (float& v : hp) v = rd.get<float>();
  OT_REQUIRE(rd.good && n_flat == s->n_flat && t >= 0, "surrogate_restore: inconsistent checkpoint header");
  OT_REQUIRE(bytes >= sur_blob_bytes(s), "surrogate_restore: checkpoint truncated");
  OT_HIP(hipDeviceSynchronize());
  for (float* dst : {s->params, s->m, s->v}) OT_HIP(hipMemcpy(dst, rd.take(n_flat * 4), n_flat * 4, hipMemcpyHostToDevice));
  if (s->pb) {
    hipLaunchKernelGGL(ot::to_bf16_kernel, dim3((unsigned)ot::ceil_div(n_flat, 256)), dim3(256), 0, 0, s->params, s->pb,
                       n_flat);
    OT_LAUNCHED("to_bf16_kernel");
    OT_HIP(hipDeviceSynchronize());
  }
  s->t = t;
  s->lr = hp[0];
  s->beta1 = hp[1];
  s->beta2 = hp[2];
  s->eps = hp[3];
  if (s->device_step) {
    const long long td = t;
    OT_HIP(hipMemcpy(s->t_done_dev, &td, sizeof td, hipMemcpyHostToDevice));
  }
  return OT_OK;
}

extern "C" int surrogate_timing_begin(ot_surrogate* s, uint32_t phase_mask, int64_t max_steps) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr, "surrogate_timing_begin: NULL surrogate");
  OT_REQUIRE(phase_mask != 0 && phase_mask < (1u << OT_SURROGATE_PHASES), "surrogate_timing_begin: bad mask");
  return s->timer.begin(phase_mask, OT_SURROGATE_PHASES, max_steps);
}

extern "C" int surrogate_timing_end(ot_surrogate* s, double* ms_total, int64_t* count) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr, "surrogate_timing_end: NULL surrogate");
  return s->timer.end(ms_total, count);
}

namespace {

// Argument checks of the predict entry points (before anything is enqueued).
int check_predict(ot_surrogate* s, const float* x, int64_t ldx, float* y, int64_t ldy, const char* what) {
  int rc = check_input(s, x, ldx);
  if (rc) return rc;
  const int L = s->L;
  OT_REQUIRE(y != nullptr && ldy >= s->widths[L] && ldy % 4 == 0 && aligned16(y),
             "%s: y needs 16-byte alignment and ldy >= D, ldy %% 4 == 0", what);
  if (L == 1)
    OT_REQUIRE(aligned16(x) && ldx % 4 == 0, "single-layer nets need 16-byte aligned x, ldx %% 4 == 0");
  return OT_OK;
}

// Forward of `rows` rows (at most the workspace's) into y with the output bias epilogue.
int predict_rows(ot_surrogate* s, const float* xr, int64_t ldx, int64_t rows, float* yr, int64_t ldy,
                 hipStream_t st) {
  if (s->precision == OT_BF16) return predict_bf16(s, xr, ldx, rows, yr, ldy, st);
  int rc = forward_hidden(s, xr, ldx, rows, st);
  if (rc) return rc;
  const int L = s->L;
  const Layer& lo = s->layers[L - 1];
  GemmArgs g = args0();
  g.A = (L == 1) ? xr : s->act[L - 1];
  g.lda = (L == 1) ? ldx : s->ld[L - 1];
  g.B = s->params + lo.w_off;
  g.ldb = lo.ldw;
  g.C = yr;
  g.ldc = ldy;
  g.M = rows;
  g.N = s->widths[L];
  g.K = lo.in;
  g.bias = s->params + lo.b_off;
  return run_gemm<Lay::KMajor, Lay::KMajor, 1>(s, g, Epi::Bias, st, "output forward", true);
}

}  // namespace

extern "C" int surrogate_predict(ot_surrogate* s, const float* x, int64_t ldx, int64_t n, float* y, int64_t ldy,
                                 void* stream) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr, "surrogate_predict: NULL surrogate");
  OT_REQUIRE(n >= 0, "surrogate_predict: n < 0");
  if (n == 0) return OT_OK;
  int rc = check_predict(s, x, ldx, y, ldy, "surrogate_predict");
  if (rc) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t chunk = std::max<int64_t>(s->ws_rows, 1);
  for (int64_t r0 = 0; r0 < n; r0 += chunk) {
    const int64_t rows = std::min(chunk, n - r0);
    if ((rc = predict_rows(s, x + r0 * ldx, ldx, rows, y + r0 * ldy, ldy, st))) return rc;
  }
  return OT_OK;
}

// ------------------------------------------------------------------ prediction without allocation
// surrogate_predict_noalloc keeps the hidden activations and the split-K
// partial products of one call in this array instead of the surrogate's
// workspaces: one copy per device, held until the process ends.  On the host
// the name `scratch` denotes a host-side stand-in, not device memory: host
// code passes only the address hipGetSymbolAddress returns for a device.
static __device__ __align__(256) unsigned char scratch[OT_PREDICT_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
unsigned char* g_scratch_addr[kMaxScratchDevices] = {};

// Device address of `scratch` on `device` (which must be current), looked up
// once per device.
int scratch_address(int device, unsigned char** out) {
  OT_REQUIRE(device >= 0 && device < kMaxScratchDevices, "surrogate_predict_noalloc: device %d above %d", device,
             kMaxScratchDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_addr[device] == nullptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return ot::set_error(OT_E_HIP, "hipGetSymbolAddress of the prediction scratch failed: %s",
                           hipGetErrorString(e));
    g_scratch_addr[device] = static_cast<unsigned char*>(p);
  }
  *out = g_scratch_addr[device];
  return OT_OK;
}

// Where one no-allocation prediction over `rows` rows keeps its data in the
// scratch: each hidden activation (rows x ld[l], fp32 or bf16) on a 256-byte
// boundary, then the largest split-K partial buffer of its GEMMs (the plans
// predict_rows will take).
struct NoAllocLayout {
  int64_t act_off[16] = {};
  int64_t split_off = 0;
  int64_t split_elems = 0;
  int64_t total = 0;
};

NoAllocLayout noalloc_layout(const ot_surrogate* s, int64_t rows) {
  const int L = s->L;
  const bool bf = s->precision == OT_BF16;
  NoAllocLayout lay;
  int64_t off = 0;
  for (int l = 1; l < L; ++l) {
    lay.act_off[l] = off;
    off = ot::round_up(off + rows * s->ld[l] * (bf ? 2 : 4), 256);
  }
  int64_t split = 0;
  for (int l = 1; l <= L; ++l) {
    const Layer& ly = s->layers[l - 1];
    // hidden layers without a GEMM: bf16 layer 1, the fp32 small-K layer 1
    // and the fp32 narrow-hidden kernels
    if (l < L && (bf ? l == 1 : (s->small_hidden || (l == 1 && ly.in <= ot::kMaxSmallK)))) continue;
    const Plan p = bf ? make_plan_b(rows, ly.out, ly.in, true) : make_plan(rows, ly.out, ly.in, true);
    if (p.splits > 1) split = std::max(split, p.splits * rows * ot::round_up(ly.out, 4));
  }
  lay.split_off = off;
  lay.split_elems = split;
  lay.total = off + split * 4;
  return lay;
}

// Points the surrogate's activation and split-K workspaces at the scratch for
// one call and forbids growing them; restores both on destruction.
struct ScratchWorkspace {
  ot_surrogate* s;
  float* act[16];
  uint16_t* act16[16];
  float* splitws;
  int64_t splitws_elems;
  float* rsws;
  int64_t rsws_elems;
  ScratchWorkspace(ot_surrogate* sur, unsigned char* base, const NoAllocLayout& lay)
      : s(sur), splitws(sur->splitws), splitws_elems(sur->splitws_elems), rsws(sur->rsws),
        rsws_elems(sur->rsws_elems) {
    for (int l = 1; l < s->L; ++l) {
      act[l] = s->act[l];
      act16[l] = s->act16[l];
      if (s->precision == OT_BF16)
        s->act16[l] = reinterpret_cast<uint16_t*>(base + lay.act_off[l]);
      else
        s->act[l] = reinterpret_cast<float*>(base + lay.act_off[l]);
    }
    s->splitws = lay.split_elems ? reinterpret_cast<float*>(base + lay.split_off) : nullptr;
    s->splitws_elems = lay.split_elems;
    s->rsws = nullptr;
    s->rsws_elems = 0;
    s->no_alloc = true;
  }
  ~ScratchWorkspace() {
    for (int l = 1; l < s->L; ++l) {
      s->act[l] = act[l];
      s->act16[l] = act16[l];
    }
    s->splitws = splitws;
    s->splitws_elems = splitws_elems;
    s->rsws = rsws;
    s->rsws_elems = rsws_elems;
    s->no_alloc = false;
  }
};

}  // namespace

extern "C" int surrogate_predict_noalloc(ot_surrogate* s, const float* x, int64_t ldx, int64_t n, float* y,
                                         int64_t ldy, void* stream) {
  ot::clear_error();
  OT_REQUIRE(s != nullptr, "surrogate_predict_noalloc: NULL surrogate");
  OT_REQUIRE(n >= 0 && n <= (1LL << 20), "surrogate_predict_noalloc: n outside [0, 2^20]");
  if (n == 0) return OT_OK;
  int rc = check_predict(s, x, ldx, y, ldy, "surrogate_predict_noalloc");
  if (rc) return rc;
  int device = -1;
  OT_HIP(hipGetDevice(&device));
  if (device != s->device)
    return ot::set_error(OT_E_STATE, "surrogate_predict_noalloc: device %d is current, the surrogate lives on %d",
                         device, s->device);
  const NoAllocLayout lay = noalloc_layout(s, n);
  OT_REQUIRE(lay.total <= (int64_t)OT_PREDICT_NOALLOC_SCRATCH_BYTES,
             "surrogate_predict_noalloc: %lld rows need %lld bytes of scratch, above its %lld bytes (use fewer rows)",
             (long long)n, (long long)lay.total, (long long)OT_PREDICT_NOALLOC_SCRATCH_BYTES);
  unsigned char* base = nullptr;
  if ((rc = scratch_address(device, &base))) return rc;
  ScratchWorkspace ws(s, base, lay);
  return predict_rows(s, x, ldx, n, y, ldy, static_cast<hipStream_t>(stream));
}
