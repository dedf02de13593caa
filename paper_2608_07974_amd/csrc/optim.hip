// Local update (Eq. (6)) / on-device AdamW: one streaming pass over the flat
// fp32 buffers.  AdamW reads master, grad, m, v and writes master, m, v and
// the bf16 shadow; SGD reads master and grad and writes master and shadow.
#include "common.h"

namespace zl {

__global__ void __launch_bounds__(256) optimizer_kernel(OptDesc o) {
  const size_t n4 = o.n / 4;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  float4* P = reinterpret_cast<float4*>(o.master);
  const float4* G = reinterpret_cast<const float4*>(o.grad);
  float4* M = reinterpret_cast<float4*>(o.m);
  float4* Vv = reinterpret_cast<float4*>(o.v);
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n4; i += stride) {
    float4 p = P[i];
    const float4 g = G[i];
    float pa[4] = {p.x, p.y, p.z, p.w};
    const float ga[4] = {g.x, g.y, g.z, g.w};
    if (o.optimizer == 0) {
      float4 m = M[i], v = Vv[i];
      float ma[4] = {m.x, m.y, m.z, m.w}, va[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        ma[k] = o.beta1 * ma[k] + (1.f - o.beta1) * ga[k];
        va[k] = o.beta2 * va[k] + (1.f - o.beta2) * ga[k] * ga[k];
        const float mh = ma[k] / o.bc1;
        const float vh = va[k] / o.bc2;
        pa[k] = pa[k] - o.lr * (mh / (sqrtf(vh) + o.eps) + o.wd * pa[k]);
      }
      M[i] = make_float4(ma[0], ma[1], ma[2], ma[3]);
      Vv[i] = make_float4(va[0], va[1], va[2], va[3]);
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) pa[k] = pa[k] - o.lr * ga[k];
    }
    P[i] = make_float4(pa[0], pa[1], pa[2], pa[3]);
    if (o.shadow) {
      ushort4 sh = make_ushort4(f32_to_bf16(pa[0]), f32_to_bf16(pa[1]), f32_to_bf16(pa[2]),
                                f32_to_bf16(pa[3]));
      reinterpret_cast<ushort4*>(o.shadow)[i] = sh;
    }
  }
}

hipError_t launch_optimizer(const OptDesc& o, hipStream_t s) {
  if (o.n == 0) return hipSuccess;
  size_t blocks = (o.n / 4 + 255) / 256;
  if (blocks > 65536) blocks = 65536;  // a few float4 per thread, many waves in flight
  if (blocks == 0) blocks = 1;
  hipLaunchKernelGGL(optimizer_kernel, dim3((unsigned)blocks), dim3(256), 0, s, o);
  return hipGetLastError();
}

__global__ void shadow_kernel(const float* __restrict__ master, bf16_t* __restrict__ shadow,
                              size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    shadow[i] = f32_to_bf16(master[i]);
}

hipError_t launch_shadow(const float* master, bf16_t* shadow, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(shadow_kernel, dim3((unsigned)blocks), dim3(256), 0, s, master, shadow, n);
  return hipGetLastError();
}

__global__ void zero_block_kernel(float* __restrict__ p, int64_t ld, int64_t r0, int64_t r1,
                                  int64_t c0, int64_t c1) {
  const int64_t w = c1 - c0, n = (r1 - r0) * w;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[(r0 + i / w) * ld + c0 + i % w] = 0.f;
}

hipError_t launch_zero_block(float* p, int64_t ld, int64_t r0, int64_t r1, int64_t c0, int64_t c1,
                             hipStream_t s) {
  if (r1 <= r0 || c1 <= c0) return hipSuccess;
  int64_t blocks = ((r1 - r0) * (c1 - c0) + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(zero_block_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, ld, r0, r1, c0,
                     c1);
  return hipGetLastError();
}

}  // namespace zl
