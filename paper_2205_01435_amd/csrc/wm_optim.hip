// Optimiser step of the world-model training (section 4.7 fits the model on
// its log-likelihood loss with a learning rate decayed by a second-degree
// polynomial): Adam with bias correction on fp32 parameters, in place.
// Element-wise and bound by HBM: 16 bytes read and 12 written per parameter,
// moved in 16-byte pieces by a grid-stride loop.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "wm_kernels.h"
#include "wm_profile.h"

namespace wm {
namespace {

struct AdamArgs {
  long n;
  float* p;
  const float* g;
  float* m;
  float* v;
  float lr, b1, b2, eps, c1, c2;  // c1 = 1 - b1^t, c2 = 1 - b2^t
};

__device__ __forceinline__ void adam1(const AdamArgs& a, float& p, float g, float& m, float& v) {
  m = a.b1 * m + (1.0f - a.b1) * g;
  v = a.b2 * v + (1.0f - a.b2) * g * g;
  const float mh = m / a.c1, vh = v / a.c2;
  p = p - a.lr * mh / (sqrtf(vh) + a.eps);
}

__global__ void __launch_bounds__(256) k_adam(const AdamArgs a) {
  const long n4 = a.n >> 2;
  const long stride = (long)gridDim.x * blockDim.x;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    float4 p = reinterpret_cast<const float4*>(a.p)[i];
    const float4 g = reinterpret_cast<const float4*>(a.g)[i];
    float4 m = reinterpret_cast<const float4*>(a.m)[i];
    float4 v = reinterpret_cast<const float4*>(a.v)[i];
    adam1(a, p.x, g.x, m.x, v.x);
    adam1(a, p.y, g.y, m.y, v.y);
    adam1(a, p.z, g.z, m.z, v.z);
    adam1(a, p.w, g.w, m.w, v.w);
    reinterpret_cast<float4*>(a.p)[i] = p;
    reinterpret_cast<float4*>(a.m)[i] = m;
    reinterpret_cast<float4*>(a.v)[i] = v;
  }
  // the tail beyond a multiple of four
  for (long i = 4 * n4 + (long)blockIdx.x * blockDim.x + threadIdx.x; i < a.n; i += stride)
    adam1(a, a.p[i], a.g[i], a.m[i], a.v[i]);
}

}  // namespace

hipError_t launch_adam(long n, float* p, const float* g, float* m, float* v, int step, float lr,
                       float beta1, float beta2, float eps, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  AdamArgs a{n, p, g, m, v, lr, beta1, beta2, eps,
             (float)(1.0 - pow((double)beta1, step)), (float)(1.0 - pow((double)beta2, step))};
  long blocks = ((n >> 2) + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 2048) blocks = 2048;  // eight per CU, grid-stride beyond
  return launch("adam", k_adam, dim3((unsigned)blocks), dim3(256), 0, s, a);
}

}  // namespace wm
