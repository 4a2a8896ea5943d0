// Row kernels over the fp32 residual stream, one wavefront per token row:
//  * K5: LayerNorm (biased variance, eps 1e-6, no affine) followed by the per-sample
//    adaLN modulate LN(h) (1 + scale) + shift, where the row's sample selects its own
//    row of the modulation table, so each sample is conditioned on its own t;
//  * K7: the same LN + modulate with the final layer's table entries, the linear map
//    D -> p*p*C, and unpatchify into the velocity latent.
#include "sf_device.h"

namespace sf {

constexpr float kLnEps = 1e-6f;
constexpr int kLnVec = kMaxWidth / 4 / 64;  // float4 per lane for the widest row

// Loads one row (D floats, D % 4 == 0) into per-lane registers and returns mean/rstd.
__device__ __forceinline__ void row_stats(const float* row, int D, int lane, float4 (&v)[kLnVec],
                                          float& mean, float& rstd) {
  const int nv = D >> 2;
  const float4* r4 = (const float4*)row;
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < kLnVec; ++i) {
    const int c = lane + i * 64;
    if (c < nv) {
      v[i] = r4[c];
      s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
    }
  }
  mean = wave_sum(s) / (float)D;
  float ss = 0.0f;
#pragma unroll
  for (int i = 0; i < kLnVec; ++i) {
    const int c = lane + i * 64;
    if (c < nv) {
      const float a = v[i].x - mean, b = v[i].y - mean, cc = v[i].z - mean, d = v[i].w - mean;
      ss += (a * a + b * b) + (cc * cc + d * d);
    }
  }
  const float var = wave_sum(ss) / (float)D;
  rstd = 1.0f / sqrtf(var + kLnEps);
}

template <typename OT> struct Store4;
template <> struct Store4<float> {
  __device__ static void run(float* p, float a, float b, float c, float d) {
    *(float4*)p = make_float4(a, b, c, d);
  }
};
template <> struct Store4<bf16> {
  __device__ static void run(bf16* p, float a, float b, float c, float d) {
    bf16x4 o = {(bf16)a, (bf16)b, (bf16)c, (bf16)d};
    *(bf16x4*)p = o;
  }
};

template <typename OT>
__device__ __forceinline__ void ln_store_row(const LnArgs& a, int m, int lane, const float4 (&v)[kLnVec], float mean,
                                             float rstd) {
  const float* sh = nullptr;
  const float* sc = nullptr;
  if (a.table) {
    const int r = (int)fdiv((uint32_t)m, a.tok);
    const int slot = r < a.n_slots ? r : r - a.n_slots;
    sh = a.table + (size_t)slot * a.ldt + a.shift_off;
    sc = a.table + (size_t)slot * a.ldt + a.scale_off;
  }
  OT* out = (OT*)a.out + (size_t)m * a.D;
  const int nv = a.D >> 2;
#pragma unroll
  for (int i = 0; i < kLnVec; ++i) {
    const int c = lane + i * 64;
    if (c < nv) {
      float y0 = (v[i].x - mean) * rstd, y1 = (v[i].y - mean) * rstd;
      float y2 = (v[i].z - mean) * rstd, y3 = (v[i].w - mean) * rstd;
      if (sc) {
        const float4 s4 = *(const float4*)(sc + 4 * c);
        const float4 h4 = *(const float4*)(sh + 4 * c);
        y0 = y0 * (1.0f + s4.x) + h4.x;
        y1 = y1 * (1.0f + s4.y) + h4.y;
        y2 = y2 * (1.0f + s4.z) + h4.z;
        y3 = y3 * (1.0f + s4.w) + h4.w;
      }
      Store4<OT>::run(out + 4 * c, y0, y1, y2, y3);
    }
  }
}

// RPW rows per wavefront, NV float4 per lane per row (D <= 256 NV). Every load of
// the wavefront's rows and of their table entries (shift and scale) is issued before
// the first reduction, so the kernel pays one memory latency per row group.
template <typename OT, int NV, int RPW>
__global__ __launch_bounds__(256) void ln_mod_kernel(LnArgs a) {
  const int lane = threadIdx.x & 63;
  const int mb = (blockIdx.x * 4 + (threadIdx.x >> 6)) * RPW;
  if (mb >= a.M) return;
  const int nv = a.D >> 2;
  float4 v[RPW][NV], sc[RPW][NV], sh[RPW][NV];
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int m = min(mb + r, a.M - 1);
    const float4* row = (const float4*)(a.h + (size_t)m * a.D);
    const float* tsh = nullptr;
    const float* tsc = nullptr;
    if (a.table) {
      const int q = (int)fdiv((uint32_t)m, a.tok);
      const int slot = q < a.n_slots ? q : q - a.n_slots;
      tsh = a.table + (size_t)slot * a.ldt + a.shift_off;
      tsc = a.table + (size_t)slot * a.ldt + a.scale_off;
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = lane + i * 64;
      const bool in = c < nv;
      v[r][i] = in ? row[c] : make_float4(0.f, 0.f, 0.f, 0.f);
      if (a.table && in) {
        sc[r][i] = *(const float4*)(tsc + 4 * c);
        sh[r][i] = *(const float4*)(tsh + 4 * c);
      } else {
        sc[r][i] = make_float4(0.f, 0.f, 0.f, 0.f);
        sh[r][i] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
  }
  float mean[RPW], rstd[RPW];
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < NV; ++i) s += (v[r][i].x + v[r][i].y) + (v[r][i].z + v[r][i].w);
    mean[r] = wave_sum(s) / (float)a.D;
  }
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    float q = 0.0f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      if (lane + i * 64 < nv) {
        float d;
        d = v[r][i].x - mean[r]; q += d * d; d = v[r][i].y - mean[r]; q += d * d;
        d = v[r][i].z - mean[r]; q += d * d; d = v[r][i].w - mean[r]; q += d * d;
      }
    }
    rstd[r] = 1.0f / sqrtf(wave_sum(q) / (float)a.D + kLnEps);
  }
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int m = mb + r;
    if (m >= a.M) break;
    OT* out = (OT*)a.out + (size_t)m * a.D;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = lane + i * 64;
      if (c < nv) {
        float y0 = (v[r][i].x - mean[r]) * rstd[r], y1 = (v[r][i].y - mean[r]) * rstd[r];
        float y2 = (v[r][i].z - mean[r]) * rstd[r], y3 = (v[r][i].w - mean[r]) * rstd[r];
        if (a.table) {
          y0 = y0 * (1.0f + sc[r][i].x) + sh[r][i].x;
          y1 = y1 * (1.0f + sc[r][i].y) + sh[r][i].y;
          y2 = y2 * (1.0f + sc[r][i].z) + sh[r][i].z;
          y3 = y3 * (1.0f + sc[r][i].w) + sh[r][i].w;
        }
        Store4<OT>::run(out + 4 * c, y0, y1, y2, y3);
      }
    }
  }
}

template <typename OT, int NV>
static void launch_ln_nv(const LnArgs& a, hipStream_t s) {
  constexpr int RPW = NV <= 4 ? 2 : 1;
  const int grid = (a.M + 4 * RPW - 1) / (4 * RPW);
  launch((ln_mod_kernel<OT, NV, RPW>), dim3(grid), dim3(256), 0, s, a);
}

template <typename OT>
static hipError_t launch_ln_t(const LnArgs& a, hipStream_t s) {
  switch ((a.D + 255) / 256) {
    case 1: launch_ln_nv<OT, 1>(a, s); break;
    case 2: launch_ln_nv<OT, 2>(a, s); break;
    case 3: launch_ln_nv<OT, 3>(a, s); break;
    case 4: launch_ln_nv<OT, 4>(a, s); break;
    case 5: launch_ln_nv<OT, 5>(a, s); break;
    case 6: launch_ln_nv<OT, 6>(a, s); break;
    case 7: launch_ln_nv<OT, 7>(a, s); break;
    case 8: launch_ln_nv<OT, 8>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_ln(bool out_bf16, const LnArgs& a, hipStream_t s) {
  return out_bf16 ? launch_ln_t<bf16>(a, s) : launch_ln_t<float>(a, s);
}

// W_f lives in LDS for the whole workgroup (staged with independent 16-byte loads);
// each wavefront walks token rows.
__global__ __launch_bounds__(256) void head_kernel(HeadArgs a) {
  extern __shared__ float wf[];  // [P][D]
  {
    const int n4 = (a.P * a.D) >> 2;
    const float4* src = (const float4*)a.W_f;
    float4* dst = (float4*)wf;
    constexpr int kStage = kMaxPatch * kMaxWidth / 4 / 256;
#pragma unroll
    for (int k = 0; k < kStage; ++k) {
      const int i = threadIdx.x + k * 256;
      if (i < n4) dst[i] = src[i];
    }
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int M = a.rows * a.N;
  const int nv = a.D >> 2;
  const int gwn = a.W / a.p;
  for (int m = blockIdx.x * 4 + wave; m < M; m += gridDim.x * 4) {
    float4 v[kLnVec];
    float mean, rstd;
    row_stats(a.h + (size_t)m * a.D, a.D, lane, v, mean, rstd);
    const int r = (int)fdiv((uint32_t)m, a.tok);
    const int n = m - r * a.N;
    const int slot = r < a.n_slots ? r : r - a.n_slots;
    const float* sh = a.table + (size_t)slot * a.ldt + a.shift_off;
    const float* sc = a.table + (size_t)slot * a.ldt + a.scale_off;
#pragma unroll
    for (int i = 0; i < kLnVec; ++i) {
      const int c = lane + i * 64;
      if (c < nv) {
        const float4 s4 = *(const float4*)(sc + 4 * c);
        const float4 h4 = *(const float4*)(sh + 4 * c);
        v[i].x = (v[i].x - mean) * rstd * (1.0f + s4.x) + h4.x;
        v[i].y = (v[i].y - mean) * rstd * (1.0f + s4.y) + h4.y;
        v[i].z = (v[i].z - mean) * rstd * (1.0f + s4.z) + h4.z;
        v[i].w = (v[i].w - mean) * rstd * (1.0f + s4.w) + h4.w;
      }
    }
    const int gh = n / gwn, gw = n - gh * gwn;
    for (int o0 = 0; o0 < a.P; o0 += 16) {
      float acc[16];
#pragma unroll
      for (int o = 0; o < 16; ++o) {
        acc[o] = 0.0f;
        if (o0 + o < a.P) {
          const float* wr = wf + (o0 + o) * a.D;
#pragma unroll
          for (int i = 0; i < kLnVec; ++i) {
            const int c = lane + i * 64;
            if (c < nv) {
              const float4 w4 = *(const float4*)(wr + 4 * c);
              acc[o] += (v[i].x * w4.x + v[i].y * w4.y) + (v[i].z * w4.z + v[i].w * w4.w);
            }
          }
        }
      }
      const float mine = wave_reduce16(acc);
      const int f = o0 + ((lane >> 2) & 15);
      if ((lane & 3) == 0 && f < a.P) {
        const int c = f % a.C, ij = f / a.C;
        const int i = ij / a.p, j = ij - i * a.p;
        a.v[(((size_t)r * a.C + c) * a.H + gh * a.p + i) * a.W + gw * a.p + j] = mine + a.b_f[f];
      }
    }
  }
}

hipError_t launch_head(const HeadArgs& a, hipStream_t s) {
  const int M = a.rows * a.N;
  int grid = (M + 15) / 16;
  if (grid > 512) grid = 512;
  const size_t lds = sizeof(float) * a.P * a.D;
  launch(head_kernel, dim3(grid), dim3(256), lds, s, a);
  return hipGetLastError();
}

}  // namespace sf
