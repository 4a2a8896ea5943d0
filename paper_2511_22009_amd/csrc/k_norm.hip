// Row kernels over the fp32 residual stream, one wavefront per token row:
//  * K5: LayerNorm (biased variance, eps 1e-6, no affine) followed by the per-sample
//    adaLN modulate LN(h) (1 + scale) + shift, where the row's sample selects its own
//    row of the modulation table, so each sample is conditioned on its own t;
//  * K7: the same LN + modulate with the final layer's table entries, the linear map
//    D -> p*p*C, and unpatchify into the velocity latent.
#include "sf_device.h"

namespace sf {

constexpr float kLnEps = 1e-6f;
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

// RPW rows per wavefront, NV float4 per lane per row (D <= 256 NV). Every load of
// the wavefront's rows and of their table entries (shift and scale) is issued before
// the first reduction, so the kernel pays one memory latency per row group. The loads
// are unconditional, at in-bounds indices (chunk 0 stands in for chunks past the row's
// end; a plain LN reads its unused shift and scale from the row itself), and the zeros
// of the chunks past the end are selected once all loads are issued: a load under a
// lane condition makes the compiler wait for it before the other path writes the same
// registers, which would cost one memory latency per chunk.
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
    const float* tsh = (const float*)row;
    const float* tsc = (const float*)row;
    if (a.table) {
      const int q = (int)fdiv((uint32_t)m, a.tok);
      const int slot = q < a.n_slots ? q : q - a.n_slots;
      tsh = a.table + (size_t)slot * a.ldt + a.shift_off;
      tsc = a.table + (size_t)slot * a.ldt + a.scale_off;
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = lane + i * 64;
      const int cc = c < nv ? c : 0;
      v[r][i] = row[cc];
      sc[r][i] = *(const float4*)(tsc + 4 * cc);
      sh[r][i] = *(const float4*)(tsh + 4 * cc);
    }
  }
#pragma unroll
  for (int r = 0; r < RPW; ++r)
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (lane + i * 64 >= nv) v[r][i] = make_float4(0.f, 0.f, 0.f, 0.f);
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
  // one row per wavefront: more wavefronts in flight beat more rows per wavefront
  // (4096 x 768: 4.5 us against 5.1 us with two rows)
  constexpr int RPW = 1;
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

// Four token rows per wavefront. Every load of the rows and of their final
// shift/scale entries is issued before the first reduction; the linear map D -> P then
// runs in groups of four outputs: the lane's slice of four W_f rows (read from L2, the
// next group's while this one is used) is applied to all four rows, and the 16 row x
// output sums leave through one butterfly reduction. The result is written straight to
// its unpatchified position.
template <int NV>
__global__ __launch_bounds__(256) void head_kernel(HeadArgs a) {
  constexpr int RH = 4;
  const int lane = threadIdx.x & 63;
  const int M = a.rows * a.N;
  const int mb = (blockIdx.x * 4 + (threadIdx.x >> 6)) * RH;
  if (mb >= M) return;
  const int nv = a.D >> 2;
  float4 v[RH][NV];
  {
    float4 sc[RH][NV], sh[RH][NV];
#pragma unroll
    for (int r = 0; r < RH; ++r) {
      const int m = min(mb + r, M - 1);
      const float4* row = (const float4*)(a.h + (size_t)m * a.D);
      const int q = (int)fdiv((uint32_t)m, a.tok);
      const int slot = q < a.n_slots ? q : q - a.n_slots;
      const float* tsh = a.table + (size_t)slot * a.ldt + a.shift_off;
      const float* tsc = a.table + (size_t)slot * a.ldt + a.scale_off;
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        // unconditional loads at in-bounds indices, zeros selected after all are issued
        const int c = lane + i * 64;
        const int cc = c < nv ? c : 0;
        v[r][i] = row[cc];
        sc[r][i] = *(const float4*)(tsc + 4 * cc);
        sh[r][i] = *(const float4*)(tsh + 4 * cc);
      }
    }
#pragma unroll
    for (int r = 0; r < RH; ++r)
#pragma unroll
      for (int i = 0; i < NV; ++i)
        if (lane + i * 64 >= nv) v[r][i] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int r = 0; r < RH; ++r) {
      float s = 0.0f;
#pragma unroll
      for (int i = 0; i < NV; ++i) s += (v[r][i].x + v[r][i].y) + (v[r][i].z + v[r][i].w);
      const float mean = wave_sum(s) / (float)a.D;
      float q = 0.0f;
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        if (lane + i * 64 < nv) {
          const float d0 = v[r][i].x - mean, d1 = v[r][i].y - mean, d2 = v[r][i].z - mean, d3 = v[r][i].w - mean;
          q += (d0 * d0 + d1 * d1) + (d2 * d2 + d3 * d3);
        }
      }
      const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)a.D + kLnEps);
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const bool in = lane + i * 64 < nv;
        v[r][i].x = in ? (v[r][i].x - mean) * rstd * (1.0f + sc[r][i].x) + sh[r][i].x : 0.0f;
        v[r][i].y = in ? (v[r][i].y - mean) * rstd * (1.0f + sc[r][i].y) + sh[r][i].y : 0.0f;
        v[r][i].z = in ? (v[r][i].z - mean) * rstd * (1.0f + sc[r][i].z) + sh[r][i].z : 0.0f;
        v[r][i].w = in ? (v[r][i].w - mean) * rstd * (1.0f + sc[r][i].w) + sh[r][i].w : 0.0f;
      }
    }
  }
  const int gwn = a.W / a.p;
  // output groups of four, with the next group's weight rows loaded while this group's
  // dot products run (two register sets, the loop unrolled by two)
  auto load_w = [&](float4 (&w)[4][NV], int o0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float* wr = a.W_f + (size_t)min(o0 + q, a.P - 1) * a.D;
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int c = lane + i * 64;
        w[q][i] = *(const float4*)(wr + 4 * (c < nv ? c : 0));
      }
    }
  };
  auto group = [&](const float4 (&w)[4][NV], int o0) {
    float acc[16];
#pragma unroll
    for (int r = 0; r < RH; ++r)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float t = 0.0f;
#pragma unroll
        for (int i = 0; i < NV; ++i)
          t += (v[r][i].x * w[q][i].x + v[r][i].y * w[q][i].y) + (v[r][i].z * w[q][i].z + v[r][i].w * w[q][i].w);
        acc[r * 4 + q] = t;
      }
    const float tot = wave_reduce16(acc);
    const int idx = (lane >> 2) & 15;
    const int r = idx >> 2, f = o0 + (idx & 3);
    const int m = mb + r;
    if ((lane & 3) == 0 && f < a.P && m < M) {
      const int row = (int)fdiv((uint32_t)m, a.tok);
      const int n = m - row * a.N;
      const int gh = n / gwn, gw = n - gh * gwn;
      const int c = f % a.C, ij = f / a.C;
      const int i = ij / a.p, j = ij - i * a.p;
      a.v[(((size_t)row * a.C + c) * a.H + gh * a.p + i) * a.W + gw * a.p + j] = tot + a.b_f[f];
    }
  };
  float4 wa[4][NV], wb[4][NV];
  load_w(wa, 0);
  for (int o0 = 0; o0 < a.P; o0 += 8) {
    if (o0 + 4 < a.P) load_w(wb, o0 + 4);
    group(wa, o0);
    if (o0 + 4 < a.P) {
      if (o0 + 8 < a.P) load_w(wa, o0 + 8);
      group(wb, o0 + 4);
    }
  }
}

hipError_t launch_head(const HeadArgs& a, hipStream_t s) {
  const int M = a.rows * a.N;
  const dim3 grid((M + 15) / 16);
  switch ((a.D + 255) / 256) {
    case 1: launch(head_kernel<1>, grid, dim3(256), 0, s, a); break;
    case 2: launch(head_kernel<2>, grid, dim3(256), 0, s, a); break;
    case 3: launch(head_kernel<3>, grid, dim3(256), 0, s, a); break;
    case 4: launch(head_kernel<4>, grid, dim3(256), 0, s, a); break;
    case 5: launch(head_kernel<5>, grid, dim3(256), 0, s, a); break;
    case 6: launch(head_kernel<6>, grid, dim3(256), 0, s, a); break;
    case 7: launch(head_kernel<7>, grid, dim3(256), 0, s, a); break;
    case 8: launch(head_kernel<8>, grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sf
