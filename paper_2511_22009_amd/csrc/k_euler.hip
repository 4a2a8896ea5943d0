// K6: the per-sample Euler update x' = x + dt_k v_k (Sec. 3.1.1 discretization; the
// final update of Alg. 1, with each slot's own signed step dt_k = t_next - t) fused
// with the pipeline shift of Alg. 2 (fresh noise enters slot 0, every latent moves one
// slot on, the oldest leaves finished), and the guidance combine v = v_u + w (v_c - v_u).
// With time windows set, the network output is a noise prediction and the update is
// PeRFlow's window conversion (Sec. 2 time windows, Sec. 3.3, Alg. 1): per slot,
// x' = x + dt (lambda_t x + eta_t eps - x) / (t^e - t) = A_k x + B_k eps, with A_k and
// B_k computed once per slot in fp64 at the start of every workgroup.
//
// In place without a race: each thread owns one element of the latent, reads it from
// every slot, then writes the slots from the oldest to the newest.
// Products and sums are rounded separately (contraction into FMA is switched off for
// these functions), so the result is bit-identical to a plain fp32 x + dt * v.
#include "sf_device.h"

namespace sf {

__device__ __forceinline__ float4 guided(float4 vc, float4 vu, float w) {
#pragma clang fp contract(off)
  return make_float4(vu.x + w * (vc.x - vu.x), vu.y + w * (vc.y - vu.y), vu.z + w * (vc.z - vu.z),
                     vu.w + w * (vc.w - vu.w));
}

// Window coefficients of one slot at normalised time t with step dt: the window is
// k = #{j < W : t > j / W + eps} (at least 1), running from t^s = k / W down to
// t^e = (k - 1) / W; gamma = sqrt(abar(t^s) / abar(t^e)) with abar read at index
// round(u (n - 1)); lambda_s = 1 / gamma, eta_s = -sqrt(1 - gamma^2) / gamma;
// denom = lambda_s (t - t^s) + (t^e - t); lambda_t = lambda_s (t^e - t^s) / denom,
// eta_t = eta_s (t^e - t) / denom; with c = dt / (t^e - t): A = 1 + c (lambda_t - 1),
// B = c eta_t.
__device__ void window_coeffs(const EulerArgs& a, int k, float* A, float* B) {
  const double t = a.t.v[k], dt = a.dt.v[k];
  int kw = 0;
  for (int j = 0; j < a.windows; ++j) kw += t > (double)j / a.windows + a.eps ? 1 : 0;
  kw = kw < 1 ? 1 : kw;
  const double ts = (double)kw / a.windows, te = (double)(kw - 1) / a.windows;
  const double as = a.abar[(int)rint(ts * (a.n_abar - 1))], ae = a.abar[(int)rint(te * (a.n_abar - 1))];
  const double g = sqrt(as / ae);
  const double lam_s = 1.0 / g, eta_s = -sqrt(1.0 - g * g) / g;
  const double den = lam_s * (t - ts) + (te - t);
  const double lam_t = lam_s * (te - ts) / den, eta_t = eta_s * (te - t) / den;
  const double c = dt / (te - t);
  *A = (float)(1.0 + c * (lam_t - 1.0));
  *B = (float)(c * eta_t);
}

// One thread per element: it loads the element of every slot (and both guidance rows)
// first, then writes the updated values oldest first, so every read of slot k precedes
// the write of slot k + 1 and all of a thread's loads are in flight together. The
// latent's elements spread over E / 256 workgroups (64 at 512^2).
template <int BMAX>
__global__ __launch_bounds__(256) void euler_shift_kernel(EulerArgs a) {
#pragma clang fp contract(off)
  __shared__ float coef[2][kMaxRows];
  if (a.windows > 0) {
    if ((int)threadIdx.x < a.B) window_coeffs(a, threadIdx.x, &coef[0][threadIdx.x], &coef[1][threadIdx.x]);
    __syncthreads();
  }
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= a.E) return;
  const size_t E = a.E;
  float xs[BMAX], vs[BMAX];
#pragma unroll
  for (int k = 0; k < BMAX; ++k) {
    if (k < a.B) {
      xs[k] = a.x[k * E + e];
      vs[k] = a.v[k * E + e];
      if (a.guided) {
        const float vu = a.v[(a.B + k) * E + e];
        vs[k] = vu + a.w * (vs[k] - vu);
      }
    }
  }
  const float z = a.z_new[e];
#pragma unroll
  for (int k = BMAX - 1; k >= 0; --k) {
    if (k >= a.B) continue;
    const float xn = a.windows > 0 ? coef[0][k] * xs[k] + coef[1][k] * vs[k] : xs[k] + a.dt.v[k] * vs[k];
    if (k == a.B - 1 && a.x_done)
      a.x_done[e] = xn;
    else
      a.x[(k + 1) * E + e] = xn;
  }
  a.x[e] = z;
}

hipError_t launch_euler_shift(const EulerArgs& a, hipStream_t s) {
  const dim3 grid((a.E + 255) / 256);
  if (a.B <= 4)
    launch(euler_shift_kernel<4>, grid, dim3(256), 0, s, a);
  else if (a.B <= 16)
    launch(euler_shift_kernel<16>, grid, dim3(256), 0, s, a);
  else
    launch(euler_shift_kernel<kMaxRows>, grid, dim3(256), 0, s, a);
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

// The admitted latent of an image-to-image run: the straight-path point between the
// reference and the noise at the schedule's first time t0 (t = 1 is noise).
__global__ __launch_bounds__(256) void noise_latent_kernel(const float* x_ref, const float* z, float t0, int n4,
                                                            float* out) {
#pragma clang fp contract(off)
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  const float a = 1.0f - t0;
  const float4 r = ((const float4*)x_ref)[i], q = ((const float4*)z)[i];
  ((float4*)out)[i] = make_float4(a * r.x + t0 * q.x, a * r.y + t0 * q.y, a * r.z + t0 * q.z, a * r.w + t0 * q.w);
}

hipError_t launch_noise_latent(const float* x_ref, const float* z, float t0, int E, float* out, hipStream_t s) {
  const int n4 = E >> 2;
  launch(noise_latent_kernel, dim3((n4 + 255) / 256), dim3(256), 0, s, x_ref, z, t0, n4, out);
  return hipGetLastError();
}

}  // namespace sf
