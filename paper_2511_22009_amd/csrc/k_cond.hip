// Per-sample conditioning kernels:
//  * K1, the timestep path: each sample's own t enters as the sinusoidal embedding of
//    1000 t, goes through the two-layer timestep MLP, and every adaLN projection of
//    every block reads SiLU(c). All three stages are batched GEMVs (one weight row
//    read from HBM serves every sample), so the heterogeneous timesteps of Sec. 3.2
//    cost no more than one shared t would.
//  * K2, patchify + patch embedding + position table.
//  * context assembly for the cross-attention K/V projection.
#include "sf_device.h"

namespace sf {

constexpr int kGemvSamples = 8;  // samples staged in LDS per pass

template <typename WT>
__device__ __forceinline__ void load4(const WT* p, float* w);

template <>
__device__ __forceinline__ void load4<float>(const float* p, float* w) {
  float4 v = *(const float4*)p;
  w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
}

template <>
__device__ __forceinline__ void load4<bf16>(const bf16* p, float* w) {
  bf16x4 v = *(const bf16x4*)p;
  w[0] = (float)v[0]; w[1] = (float)v[1]; w[2] = (float)v[2]; w[3] = (float)v[3];
}

// One wavefront per output row j; lanes stride the row four elements at a time and
// the samples' input vectors sit in LDS.
template <typename WT>
__global__ __launch_bounds__(256) void gemv_kernel(GemvArgs a) {
  extern __shared__ float xs[];  // [kGemvSamples][K]
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const WT* W = (const WT*)a.W;
  for (int b0 = 0; b0 < a.B; b0 += kGemvSamples) {
    const int nb = min(kGemvSamples, a.B - b0);
    for (int i = threadIdx.x; i < nb * a.K; i += blockDim.x) {
      const int bb = i / a.K, k = i - bb * a.K;
      float val;
      if (a.x_mode == 1) {
        const int half = a.K >> 1;
        const int f = k < half ? k : k - half;
        const float tau = 1000.0f * a.t.v[b0 + bb];
        const float phi = tau * a.freqs[f];
        val = k < half ? cosf(phi) : sinf(phi);
      } else {
        val = a.X[(size_t)(b0 + bb) * a.ldx + k];
      }
      xs[bb * a.K + k] = val;
    }
    __syncthreads();
    for (int j = blockIdx.x * 4 + wave; j < a.R; j += gridDim.x * 4) {
      float acc[kGemvSamples];
#pragma unroll
      for (int bb = 0; bb < kGemvSamples; ++bb) acc[bb] = 0.0f;
      const WT* wr = W + (size_t)j * a.K;
      for (int k = lane * 4; k < a.K; k += 256) {
        float w[4];
        load4<WT>(wr + k, w);
#pragma unroll
        for (int bb = 0; bb < kGemvSamples; ++bb) {
          if (bb < nb) {
            const float* xp = xs + bb * a.K + k;
            acc[bb] += w[0] * xp[0] + w[1] * xp[1] + w[2] * xp[2] + w[3] * xp[3];
          }
        }
      }
#pragma unroll
      for (int bb = 0; bb < kGemvSamples; ++bb) {
        if (bb < nb) {
          float s = wave_sum(acc[bb]);
          if (lane == 0) {
            s += a.bias[j];
            if (a.act == 1) s = silu(s);
            a.Y[(size_t)(b0 + bb) * a.ldy + j] = s;
          }
        }
      }
    }
    __syncthreads();
  }
}

hipError_t launch_gemv(bool w_bf16, const GemvArgs& a, hipStream_t s) {
  const int rows_per_block = 4;
  int grid = (a.R + rows_per_block - 1) / rows_per_block;
  if (grid > 2048) grid = 2048;
  const size_t lds = sizeof(float) * kGemvSamples * a.K;
  if (w_bf16)
    hipLaunchKernelGGL(gemv_kernel<bf16>, dim3(grid), dim3(256), lds, s, a);
  else
    hipLaunchKernelGGL(gemv_kernel<float>, dim3(grid), dim3(256), lds, s, a);
  return hipGetLastError();
}

// One workgroup per token: gather the token's p*p*C patch values (feature
// (i*p + j)*C + c of token gh*(W/p) + gw reads x[c][gh*p + i][gw*p + j]), then each
// thread produces columns of h = tok . W_pe^T + b_pe + pos[n].
__global__ __launch_bounds__(256) void embed_kernel(EmbedArgs a) {
  __shared__ float tok[kMaxPatch];
  const int m = blockIdx.x;
  const int r = m / a.N;
  const int n = m - r * a.N;
  const int lat = r % a.n_lat;
  const int gwn = a.W / a.p;
  const int gh = n / gwn, gw = n - gh * gwn;
  const int P = a.p * a.p * a.C;
  if (threadIdx.x < P) {
    const int f = threadIdx.x;
    const int c = f % a.C, ij = f / a.C;
    const int i = ij / a.p, j = ij - i * a.p;
    tok[f] = a.x[(((size_t)lat * a.C + c) * a.H + gh * a.p + i) * a.W + gw * a.p + j];
  }
  __syncthreads();
  for (int d = threadIdx.x; d < a.D; d += blockDim.x) {
    const float* wr = a.W_pe + (size_t)d * P;
    float acc = 0.0f;
    for (int f = 0; f < P; ++f) acc += tok[f] * wr[f];
    a.h[(size_t)m * a.D + d] = (acc + a.b_pe[d]) + a.pos[(size_t)n * a.D + d];
  }
}

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(embed_kernel, dim3(a.rows * a.N), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void ctx_assemble_kernel(const float* ctx, const float* null_ctx,
                                                           int n_cond, int rows, int per_row, T* out) {
  const size_t total = (size_t)rows * per_row;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    const int r = (int)(i / per_row);
    const size_t e = i - (size_t)r * per_row;
    const float v = r < n_cond ? ctx[(size_t)r * per_row + e] : null_ctx[e];
    out[i] = from_f32<T>(v);
  }
}

hipError_t launch_ctx_assemble(bool use_bf16, const float* ctx, const float* null_ctx, int n_cond,
                               int rows, int ctx_len, int ctx_dim, void* out, hipStream_t s) {
  const int per_row = ctx_len * ctx_dim;
  int grid = (int)(((size_t)rows * per_row + 255) / 256);
  if (grid > 4096) grid = 4096;
  if (use_bf16)
    hipLaunchKernelGGL(ctx_assemble_kernel<bf16>, dim3(grid), dim3(256), 0, s, ctx, null_ctx,
                       n_cond, rows, per_row, (bf16*)out);
  else
    hipLaunchKernelGGL(ctx_assemble_kernel<float>, dim3(grid), dim3(256), 0, s, ctx, null_ctx,
                       n_cond, rows, per_row, (float*)out);
  return hipGetLastError();
}

}  // namespace sf
