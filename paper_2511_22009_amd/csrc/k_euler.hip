// K6: the per-sample Euler update x' = x + dt_k v_k (Sec. 3.1.1 discretization; the
// final update of Alg. 1, with each slot's own signed step dt_k = t_next - t) fused
// with the pipeline shift of Alg. 2 (fresh noise enters slot 0, every latent moves one
// slot on, the oldest leaves finished), and the guidance combine v = v_u + w (v_c - v_u).
//
// In place without a race: each thread owns four elements of the latent and walks the
// slots from the oldest to the newest, reading slot k before it writes slot k + 1.
// Products and sums are rounded separately (contraction into FMA is switched off for
// these functions), so the result is bit-identical to a plain fp32 x + dt * v.
#include "sf_device.h"

namespace sf {

__device__ __forceinline__ float4 guided(float4 vc, float4 vu, float w) {
#pragma clang fp contract(off)
  return make_float4(vu.x + w * (vc.x - vu.x), vu.y + w * (vc.y - vu.y), vu.z + w * (vc.z - vu.z),
                     vu.w + w * (vc.w - vu.w));
}

__global__ __launch_bounds__(256) void euler_shift_kernel(EulerArgs a) {
#pragma clang fp contract(off)
  const int e4 = blockIdx.x * blockDim.x + threadIdx.x;
  const int n4 = a.E >> 2;
  if (e4 >= n4) return;
  float4* x = (float4*)a.x;
  const float4* v = (const float4*)a.v;
  for (int k = a.B - 1; k >= 0; --k) {
    float4 vk = v[(size_t)k * n4 + e4];
    if (a.guided) vk = guided(vk, v[(size_t)(a.B + k) * n4 + e4], a.w);
    const float4 xk = x[(size_t)k * n4 + e4];
    const float d = a.dt.v[k];
    const float4 xn = make_float4(xk.x + d * vk.x, xk.y + d * vk.y, xk.z + d * vk.z, xk.w + d * vk.w);
    if (k == a.B - 1 && a.x_done)
      ((float4*)a.x_done)[e4] = xn;
    else
      x[(size_t)(k + 1) * n4 + e4] = xn;
  }
  x[e4] = ((const float4*)a.z_new)[e4];
}

hipError_t launch_euler_shift(const EulerArgs& a, hipStream_t s) {
  const int n4 = a.E >> 2;
  launch(euler_shift_kernel, dim3((n4 + 255) / 256), dim3(256), 0, s, a);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void cfg_combine_kernel(const float* v, int B, int E, float w, float* out) {
  const int n4 = E >> 2;
  const size_t total = (size_t)B * n4;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const size_t k = i / n4, e4 = i - k * n4;
  const float4* v4 = (const float4*)v;
  ((float4*)out)[i] = guided(v4[k * n4 + e4], v4[(B + k) * n4 + e4], w);
}

hipError_t launch_cfg_combine(const float* v, int B, int E, float w, float* v_out, hipStream_t s) {
  const size_t total = (size_t)B * (E >> 2);
  launch(cfg_combine_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, v, B, E, w, v_out);
  return hipGetLastError();
}

}  // namespace sf
