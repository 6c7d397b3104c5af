// Adam (Kingma and Ba, 2015, Algorithm 1) update of one parameter, fp32, in
// the fixed operation order every kernel of the library uses:
//   m = b1 m + (1 - b1) g;  v = b2 v + (1 - b2) g^2;
//   p = p - lr * (m / c1) / (sqrt(v / c2) + eps),  c1 = 1 - b1^t, c2 = 1 - b2^t.
// The standalone pass over the flat parameter buffer and the update fused into
// the output layer's weight-gradient epilogue both call adam1(), so a fused
// step and a step with materialised gradients agree bit for bit when the
// gradients do.
#pragma once

#include "common.h"

namespace ot {

// 1 - beta^t, the bias correction of step t (t >= 1), in double by binary
// exponentiation: the same operations on the host and on the device, so a
// step whose t is read from device memory uses the same corrections as one
// whose corrections the host computed.
__host__ __device__ inline float bias_correction(float beta, long long t) {
  double r = 1.0, b = (double)beta;
  for (long long e = t; e > 0; e >>= 1) {
    if (e & 1) r *= b;
    b *= b;
  }
  return (float)(1.0 - r);
}

struct AdamArgs {
  float lr, b1, b2, eps;
  float c1, c2;   // bias corrections 1 - b1^t, 1 - b2^t of the step being taken
  // When set, the step is t = *t_done + 1 (steps completed, in device memory)
  // and the kernel forms c1, c2 itself (resolved()), so that a captured step
  // replays with the same arguments.
  const long long* t_done;

#ifdef __HIPCC__
  __device__ __forceinline__ AdamArgs resolved() const {
    AdamArgs a = *this;
    if (t_done) {
      const long long t = *t_done + 1;
      a.c1 = bias_correction(b1, t);
      a.c2 = bias_correction(b2, t);
    }
    return a;
  }
#endif
};

#ifdef __HIPCC__
__device__ __forceinline__ void adam1(float& p, float g, float& m, float& v, const AdamArgs& a) {
  m = a.b1 * m + (1.0f - a.b1) * g;
  v = a.b2 * v + (1.0f - a.b2) * (g * g);
  const float mhat = m / a.c1;
  const float vhat = v / a.c2;
  p = p - a.lr * mhat / (sqrtf(vhat) + a.eps);
}

__device__ __forceinline__ void adam4(f32x4& p, const f32x4 g, f32x4& m, f32x4& v, const AdamArgs& a) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    float pc = p[c], mc = m[c], vc = v[c];
    adam1(pc, g[c], mc, vc, a);
    p[c] = pc;
    m[c] = mc;
    v[c] = vc;
  }
}
#endif

}  // namespace ot
