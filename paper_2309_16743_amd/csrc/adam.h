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

struct AdamArgs {
  float lr, b1, b2, eps;
  float c1, c2;   // bias corrections 1 - b1^t, 1 - b2^t of the step being taken
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
