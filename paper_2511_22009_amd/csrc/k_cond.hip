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

constexpr int kGemvSamples = 4;  // samples per pass (inputs held in registers)

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

// Lane `lane` owns elements 4*(lane + 64 c) .. +3 of the input width for c < NCH, so its
// slice of every sample's input vector stays in registers for all rows; a wavefront
// streams kGemvRows weight rows at a time (independent loads in flight) and reduces
// each row's partial sums across the 64 lanes at the end.
template <typename WT, int NCH, int kGemvRows>
__global__ __launch_bounds__(256) void gemv_kernel(GemvArgs a) {
  const int lane = threadIdx.x & 63;
  const int gw = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int nw = gridDim.x * 4;
  const WT* W = (const WT*)a.W;
  for (int b0 = 0; b0 < a.B; b0 += kGemvSamples) {
    const int nb = min(kGemvSamples, a.B - b0);
    float x[kGemvSamples][NCH][4];
#pragma unroll
    for (int bb = 0; bb < kGemvSamples; ++bb)
#pragma unroll
      for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int k = 4 * (lane + 64 * c) + e;
          float v = 0.0f;
          if (bb < nb && k < a.K) {
            if (a.x_mode == 1) {
              const int half = a.K >> 1;
              const int f = k < half ? k : k - half;
              const float tau = 1000.0f * a.t.v[b0 + bb];
              const float phi = tau * a.freqs[f];
              v = k < half ? cosf(phi) : sinf(phi);
            } else {
              v = a.X[(size_t)(b0 + bb) * a.ldx + k];
            }
          }
          x[bb][c][e] = v;
        }
    for (int j0 = gw * kGemvRows; j0 < a.R; j0 += nw * kGemvRows) {
      float acc[kGemvRows][kGemvSamples];
#pragma unroll
      for (int rr = 0; rr < kGemvRows; ++rr)
#pragma unroll
        for (int bb = 0; bb < kGemvSamples; ++bb) acc[rr][bb] = 0.0f;
#pragma unroll
      for (int rr = 0; rr < kGemvRows; ++rr) {
        const int j = min(j0 + rr, a.R - 1);
        const WT* wr = W + (size_t)j * a.K;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          const int k = 4 * (lane + 64 * c);
          if (k < a.K) {
            float w[4];
            load4<WT>(wr + k, w);
            // explicit fma chain: every sample slot runs the same operation sequence, so
            // a sample's result does not depend on which slot of the batch it sits in
#pragma unroll
            for (int bb = 0; bb < kGemvSamples; ++bb) {
              float t = acc[rr][bb];
              t = fmaf(w[0], x[bb][c][0], t);
              t = fmaf(w[1], x[bb][c][1], t);
              t = fmaf(w[2], x[bb][c][2], t);
              t = fmaf(w[3], x[bb][c][3], t);
              acc[rr][bb] = t;
            }
          }
        }
      }
      if constexpr (kGemvRows * kGemvSamples == 16) {
        float v16[16];
#pragma unroll
        for (int rr = 0; rr < kGemvRows; ++rr)
#pragma unroll
          for (int bb = 0; bb < kGemvSamples; ++bb) v16[rr * kGemvSamples + bb] = acc[rr][bb];
        float sum = wave_reduce16(v16);
        const int idx = (lane >> 2) & 15;
        const int rr = idx / kGemvSamples, bb = idx % kGemvSamples;
        const int j = j0 + rr;
        if ((lane & 3) == 0 && bb < nb && j < a.R) {
          sum += a.bias[j];
          if (a.act == 1) sum = silu(sum);
          a.Y[(size_t)(b0 + bb) * a.ldy + j] = sum;
        }
      } else {
#pragma unroll
        for (int rr = 0; rr < kGemvRows; ++rr)
#pragma unroll
          for (int bb = 0; bb < kGemvSamples; ++bb) {
            if (bb >= nb) continue;
            float sum = wave_sum(acc[rr][bb]);
            const int j = j0 + rr;
            if (lane == 0 && j < a.R) {
              sum += a.bias[j];
              if (a.act == 1) sum = silu(sum);
              a.Y[(size_t)(b0 + bb) * a.ldy + j] = sum;
            }
          }
      }
    }
  }
}

template <typename WT, int ROWS>
static hipError_t launch_gemv_rows(const GemvArgs& a, hipStream_t s) {
  const int nch = (a.K + 255) / 256;
  int grid = (a.R + 4 * ROWS - 1) / (4 * ROWS);
  if (grid > 2048) grid = 2048;
  switch (nch) {
#define SF_GEMV_CASE(n) \
  case n: launch((gemv_kernel<WT, n, ROWS>), dim3(grid), dim3(256), 0, s, a); break;
    SF_GEMV_CASE(1) SF_GEMV_CASE(2) SF_GEMV_CASE(3) SF_GEMV_CASE(4) SF_GEMV_CASE(5)
    SF_GEMV_CASE(6) SF_GEMV_CASE(7) SF_GEMV_CASE(8)
#undef SF_GEMV_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Few rows (the timestep MLP): one row per wavefront for parallelism. Many rows (the
// adaLN table): four rows per wavefront and one butterfly reduction per row group.
template <typename WT>
static hipError_t launch_gemv_t(const GemvArgs& a, hipStream_t s) {
  return a.R < 16384 ? launch_gemv_rows<WT, 1>(a, s) : launch_gemv_rows<WT, 4>(a, s);
}

hipError_t launch_gemv(bool w_bf16, const GemvArgs& a, hipStream_t s) {
  return w_bf16 ? launch_gemv_t<bf16>(a, s) : launch_gemv_t<float>(a, s);
}

// One thread per four consecutive outputs of one token: the token's p*p*C patch values
// (feature (i*p + j)*C + c of token gh*(W/p) + gw reads x[c][gh*p + i][gw*p + j]) times
// the transposed patch-embedding weight W_peT [P][D], plus bias and position row.
__global__ __launch_bounds__(256) void embed_kernel(EmbedArgs a) {
  const int d4n = a.D >> 2;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= a.rows * a.N * d4n) return;
  const int m = idx / d4n, d = (idx - m * d4n) * 4;
  const int r = m / a.N;
  const int n = m - r * a.N;
  const int lat = r % a.n_lat;
  const int gwn = a.W / a.p;
  const int gh = n / gwn, gw = n - gh * gwn;
  const int P = a.p * a.p * a.C;
  float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  for (int f = 0; f < P; ++f) {
    const int c = f % a.C, ij = f / a.C;
    const int i = ij / a.p, j = ij - i * a.p;
    const float t = a.x[(((size_t)lat * a.C + c) * a.H + gh * a.p + i) * a.W + gw * a.p + j];
    const float4 w = *(const float4*)(a.W_pe + (size_t)f * a.D + d);
    acc.x += t * w.x; acc.y += t * w.y; acc.z += t * w.z; acc.w += t * w.w;
  }
  const float4 b = *(const float4*)(a.b_pe + d);
  const float4 ps = *(const float4*)(a.pos + (size_t)n * a.D + d);
  *(float4*)(a.h + (size_t)m * a.D + d) =
      make_float4((acc.x + b.x) + ps.x, (acc.y + b.y) + ps.y, (acc.z + b.z) + ps.z, (acc.w + b.w) + ps.w);
}

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
  const int total = a.rows * a.N * (a.D >> 2);
  launch(embed_kernel, dim3((total + 255) / 256), dim3(256), 0, s, a);
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
    launch(ctx_assemble_kernel<bf16>, dim3(grid), dim3(256), 0, s, ctx, null_ctx,
                       n_cond, rows, per_row, (bf16*)out);
  else
    launch(ctx_assemble_kernel<float>, dim3(grid), dim3(256), 0, s, ctx, null_ctx,
                       n_cond, rows, per_row, (float*)out);
  return hipGetLastError();
}

}  // namespace sf
