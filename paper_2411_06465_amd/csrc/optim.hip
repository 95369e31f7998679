// One Adam step over a shard of the model states (Sec. 3.1): the optimizer
// keeps an FP32 master weight, momentum and variance per parameter, reads the
// FP32 accumulated gradient and writes the BF16 weight the layers read.
//
// Every element is touched once: 16 bytes read (gradient, master, momentum,
// variance) and 14 written (master, momentum, variance, weight), 4 more when
// the gradient is cleared for the next accumulation.  The kernel is a stream:
// each thread moves one 16-byte vector of four parameters of every array,
// consecutive threads consecutive vectors, with non-temporal loads and stores
// (nothing is read twice, so nothing is worth keeping in the caches).  One
// 256-thread workgroup per 1024 parameters, with no loop: on the 300M-parameter
// shard of a 70B rank this streams at about 6 TB/s, where a grid of eight
// workgroups per CU looping over the shard reached 4.2 TB/s and two or four
// vectors per thread were 4-6% slower.
#include "kernels.h"

namespace l4d {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

// Square root rounded to nearest.  The hardware square root is within one
// ulp; the nearest float is that estimate or a neighbour, and the neighbour
// wins exactly when the residual x - s_nb * s (one fma, so its sign is exact)
// says the midpoint between the two lies on the far side of sqrt(x).
// Inputs below 2^-96 are scaled by 2^32 first, to stay off the denormal range.
__device__ __forceinline__ float sqrt_rn(float x) {
  const bool tiny = x < 0x1p-96f;
  const float xs = tiny ? x * 0x1p32f : x;
  const float s = __builtin_amdgcn_sqrtf(xs);
  const float dn = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, s) - 1u);
  const float up = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, s) + 1u);
  float r = s;
  if (__builtin_fmaf(-dn, s, xs) <= 0.f) r = dn;
  if (__builtin_fmaf(-up, s, xs) > 0.f) r = up;
  return tiny ? r * 0x1p-16f : r;
}

// w <- w - lr (m_hat / (sqrt(v_hat) + eps)) - lr wd w, in the order
// m_hat / (sqrt(v_hat) + eps) = (m r1) / (sqrt(v) rs2 + eps).
__device__ __forceinline__ void adam1(const AdamConsts& k, float s, float g, float& w, float& m, float& v) {
  g *= s;
  m = k.beta1 * m + k.one_m_beta1 * g;
  v = k.beta2 * v + k.one_m_beta2 * (g * g);
  const float u = (m * k.r1) / (sqrt_rn(v) * k.rs2 + k.eps);
  w = w - (k.lr * u + k.decay * w);
}

template <bool ZERO>
__global__ void __launch_bounds__(256) adam_kernel(AdamConsts k, int64_t n, float* __restrict__ grad,
                                                   float* __restrict__ master, float* __restrict__ mom,
                                                   float* __restrict__ var, uint16_t* __restrict__ weight) {
  const float s = k.scale_dev ? k.scale * *k.scale_dev : k.scale;
  const int64_t n4 = n >> 2;
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (j < n4) {
    f32x4* g4 = reinterpret_cast<f32x4*>(grad) + j;
    f32x4* w4 = reinterpret_cast<f32x4*>(master) + j;
    f32x4* m4 = reinterpret_cast<f32x4*>(mom) + j;
    f32x4* v4 = reinterpret_cast<f32x4*>(var) + j;
    const f32x4 g = __builtin_nontemporal_load(g4);
    f32x4 w = __builtin_nontemporal_load(w4);
    f32x4 m = __builtin_nontemporal_load(m4);
    f32x4 v = __builtin_nontemporal_load(v4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float we = w[e], me = m[e], ve = v[e];
      adam1(k, s, g[e], we, me, ve);
      w[e] = we;
      m[e] = me;
      v[e] = ve;
    }
    __builtin_nontemporal_store(w, w4);
    __builtin_nontemporal_store(m, m4);
    __builtin_nontemporal_store(v, v4);
    const u16x4 b = {f2bf(w.x), f2bf(w.y), f2bf(w.z), f2bf(w.w)};
    __builtin_nontemporal_store(b, reinterpret_cast<u16x4*>(weight) + j);
    if (ZERO) __builtin_nontemporal_store(f32x4{0.f, 0.f, 0.f, 0.f}, g4);
  }
  // the last n % 4 parameters, one per thread of the last workgroup
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x < (n & 3)) {
    const int64_t i = (n4 << 2) + threadIdx.x;
    float w = master[i], m = mom[i], v = var[i];
    adam1(k, s, grad[i], w, m, v);
    master[i] = w;
    mom[i] = m;
    var[i] = v;
    weight[i] = f2bf(w);
    if (ZERO) grad[i] = 0.f;
  }
}

}  // namespace

hipError_t adam_step(const AdamConsts& c, int64_t n, float* grad, float* master, float* m, float* v,
                     uint16_t* weight, int32_t zero_grad, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t groups = ((n >> 2) + 255) / 256;
  const unsigned grid = static_cast<unsigned>(groups < 1 ? 1 : groups);
  if (zero_grad)
    hipLaunchKernelGGL(adam_kernel<true>, dim3(grid), dim3(256), 0, stream, c, n, grad, master, m, v, weight);
  else
    hipLaunchKernelGGL(adam_kernel<false>, dim3(grid), dim3(256), 0, stream, c, n, grad, master, m, v, weight);
  return hipGetLastError();
}

}  // namespace l4d
