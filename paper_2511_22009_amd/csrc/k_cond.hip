// Per-sample conditioning kernels:
//  * K1, the timestep path: each sample's own t enters as the sinusoidal embedding of
//    1000 t, goes through the two-layer timestep MLP, and every adaLN projection of
//    every block reads SiLU(c). All three stages are batched GEMVs (one weight row
//    read from HBM serves every sample), so the heterogeneous timesteps of Sec. 3.2
//    cost no more than one shared t would.
//  * K2, patchify + patch embedding + position table.
//  * the context entries of the cross-attention keys and values (assembly, and the
//    bitwise lookup that reuses an entry while its context stays in the queue).
#include <mutex>

#include "sf_device.h"

namespace sf {

constexpr int kGemvSamples = 4;  // samples per pass (inputs held in registers)

// Batched GEMV. Each wavefront takes RW consecutive weight rows and reads them with
// 16-byte buffer loads (lane l holds 16-byte chunks l + 64 c of every row; chunks past
// the row read as zeros), so all RW * NC loads of a lane are in flight at once and no
// load sits behind a branch. Four samples' input slices stay in registers (read from
// X, or built as the sinusoids of 1000 t). The RW x 4 row/sample partial sums leave
// through butterfly reductions of 16 values. One task (RW rows) per wavefront.
template <typename WT, int NC, int RW, int XMODE>
__device__ __forceinline__ void gemv_body(const GemvArgs& a, int bid) {
  constexpr int E = 16 / sizeof(WT);  // elements per 16-byte chunk
  static_assert(RW * kGemvSamples % 16 == 0, "rows x samples must fill butterfly groups");
  const int lane = threadIdx.x & 63;
  const int j0 = (bid * 4 + (threadIdx.x >> 6)) * RW;
  // the sinusoid mode builds each batch's embedding once per workgroup in LDS (with a
  // barrier), so there every wavefront stays to the end
  if (XMODE == 0 && j0 >= a.R) return;
  __shared__ float emb[XMODE == 1 ? kGemvSamples * kMaxWidth : 1];
  const int nchunk = a.K / E;
  const __amdgpu_buffer_rsrc_t w_src = buffer_rsrc(a.W, (uint32_t)((size_t)a.R * a.K * sizeof(WT)));
  const __amdgpu_buffer_rsrc_t x_src = buffer_rsrc(a.X, a.X ? (uint32_t)((size_t)a.B * a.ldx * 4) : 0u);
  for (int b0 = 0; b0 < a.B; b0 += kGemvSamples) {
    const int nb = min(kGemvSamples, a.B - b0);
    if constexpr (XMODE == 1) {
      // [cos | sin] of 1000 t times the frequency table, for this batch's samples
      const int half = a.K >> 1;
      __syncthreads();
      for (int i = threadIdx.x; i < nb * a.K; i += blockDim.x) {
        const int bb = i / a.K, k = i - bb * a.K;
        const int f = k < half ? k : k - half;
        const float phi = (1000.0f * a.t.v[b0 + bb]) * a.freqs[f];
        emb[i] = k < half ? cosf(phi) : sinf(phi);
      }
      __syncthreads();
    }
    u32x4 w[RW][NC];
#pragma unroll
    for (int rr = 0; rr < RW; ++rr) {
      const int j = min(j0 + rr, a.R - 1);
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int ch = lane + 64 * c;
        w[rr][c] = buffer_load16_stream(w_src, ch < nchunk ? (int)(((uint32_t)j * a.K + ch * E) * sizeof(WT)) : kOffOOB);
      }
    }
    float x[kGemvSamples][NC][E];
#pragma unroll
    for (int bb = 0; bb < kGemvSamples; ++bb)
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int ch = lane + 64 * c;
        const bool in = bb < nb && ch < nchunk;
        if constexpr (XMODE == 1) {
#pragma unroll
          for (int e = 0; e < E; ++e) x[bb][c][e] = in ? emb[bb * a.K + ch * E + e] : 0.0f;
        } else {
#pragma unroll
          for (int q = 0; q < E / 4; ++q) {
            const u32x4 v = buffer_load16(x_src, in ? ((b0 + bb) * a.ldx + ch * E + 4 * q) * 4 : kOffOOB);
            const float4 f = __builtin_bit_cast(float4, v);
            x[bb][c][4 * q + 0] = f.x; x[bb][c][4 * q + 1] = f.y;
            x[bb][c][4 * q + 2] = f.z; x[bb][c][4 * q + 3] = f.w;
          }
        }
      }
    float acc[RW][kGemvSamples];
#pragma unroll
    for (int rr = 0; rr < RW; ++rr) {
#pragma unroll
      for (int bb = 0; bb < kGemvSamples; ++bb) acc[rr][bb] = 0.0f;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        float wf[E];
        if constexpr (E == 8) {
          const bf16x8 v = __builtin_bit_cast(bf16x8, w[rr][c]);
#pragma unroll
          for (int e = 0; e < 8; ++e) wf[e] = (float)v[e];
        } else {
          const float4 v = __builtin_bit_cast(float4, w[rr][c]);
          wf[0] = v.x; wf[1] = v.y; wf[2] = v.z; wf[3] = v.w;
        }
        // the same fma sequence for every sample slot, so a sample's result does not
        // depend on its slot in the batch
#pragma unroll
        for (int bb = 0; bb < kGemvSamples; ++bb) {
          float t = acc[rr][bb];
#pragma unroll
          for (int e = 0; e < E; ++e) t = fmaf(wf[e], x[bb][c][e], t);
          acc[rr][bb] = t;
        }
      }
    }
#pragma unroll
    for (int grp = 0; grp < RW * kGemvSamples / 16; ++grp) {
      constexpr int RG = 16 / kGemvSamples;  // rows per butterfly group
      float v16[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) v16[q] = acc[grp * RG + q / kGemvSamples][q % kGemvSamples];
      float sum = wave_reduce16(v16);
      const int idx = (lane >> 2) & 15;
      const int rr = grp * RG + idx / kGemvSamples, bb = idx % kGemvSamples;
      const int j = j0 + rr;
      if ((lane & 3) == 0 && bb < nb && j < a.R) {
        sum += a.bias[j];
        if (a.act == 1) sum = silu(sum);
        a.Y[(size_t)(b0 + bb) * a.ldy + j] = sum;
      }
    }
  }
}

template <typename WT, int NC, int RW, int XMODE>
__global__ __launch_bounds__(256) void gemv_kernel(GemvArgs a) {
  gemv_body<WT, NC, RW, XMODE>(a, blockIdx.x);
}

// Rows per wavefront: keep the loads of a task within the register file. Eight rows up
// to three fp32 chunks per lane (a 768-wide fp32 layer: 143 VGPRs, 5.3 against 6.4 us
// with four rows), four beyond.
template <typename WT, int NC>
constexpr int gemv_rows_per_wave() {
  return NC <= 2 || (NC == 3 && sizeof(WT) == 4) ? 8 : 4;
}

template <typename WT, int NC>
static void launch_gemv_nc(const GemvArgs& a, hipStream_t s) {
  constexpr int RW = gemv_rows_per_wave<WT, NC>();
  const int tasks = (a.R + RW - 1) / RW;
  if (a.x_mode == 1)
    launch((gemv_kernel<WT, NC, RW, 1>), dim3((tasks + 3) / 4), dim3(256), 0, s, a);
  else
    launch((gemv_kernel<WT, NC, RW, 0>), dim3((tasks + 3) / 4), dim3(256), 0, s, a);
}

template <typename WT>
static hipError_t launch_gemv_t(const GemvArgs& a, hipStream_t s) {
  constexpr int E = 16 / sizeof(WT);
  if (a.K % E || (size_t)a.R * a.K * sizeof(WT) >= (1ull << 31)) return hipErrorInvalidValue;
  switch ((a.K / E + 63) / 64) {
    case 1: launch_gemv_nc<WT, 1>(a, s); break;
    case 2: launch_gemv_nc<WT, 2>(a, s); break;
    case 3: launch_gemv_nc<WT, 3>(a, s); break;
    case 4: launch_gemv_nc<WT, 4>(a, s); break;
    case 5: launch_gemv_nc<WT, 5>(a, s); break;
    case 6: launch_gemv_nc<WT, 6>(a, s); break;
    case 7: launch_gemv_nc<WT, 7>(a, s); break;
    case 8: launch_gemv_nc<WT, 8>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gemv(bool w_bf16, const GemvArgs& a, hipStream_t s) {
  return w_bf16 ? launch_gemv_t<bf16>(a, s) : launch_gemv_t<float>(a, s);
}

// Patch embedding, h = patches . W_peT + b_pe + pos. The token's p*p*C patch values
// (feature (i*p + j)*C + c of token gh*(W/p) + gw reads x[c][gh*p + i][gw*p + j]) times
// the transposed patch-embedding weight W_peT [P][D], plus bias and position row.
//
// 2x2 patches of 4 channels, one workgroup per kEmbedWgTok consecutive tokens: the
// tokens' 16 patch values each are staged in LDS once (one 8-byte load per value pair)
// and read back as broadcasts, and each thread keeps the sixteen W_peT rows of its four
// output columns in registers for all of the workgroup's tokens, so the weight is read
// once per kEmbedWgTok tokens (not once per four, as with a thread per four tokens:
// 8.8 -> 6.5 us at 4096 tokens x 768, 41.8 -> 24.0 us at 16384 x 1152, same bits).
// All of a thread's weight, bias and position-row loads for its first column group are
// issued before the patch values are staged, so the two memory latencies overlap
// instead of following each other across the barrier.
constexpr int kEmbedWgTok = 8;

__device__ __forceinline__ void embed_p2c4_body(const EmbedArgs& a, int bid) {
  __shared__ float4 px_s[kEmbedWgTok][4];  // token t: feature (2i + j) * 4 + c at [t][f / 4][f % 4]
  const int M = a.rows * a.N;
  const int m0 = bid * kEmbedWgTok;
  const int tid = threadIdx.x;
  const int gwn = a.W / 2;
  const int d4n = a.D >> 2;
  const int nt = min(kEmbedWgTok, M - m0);
  struct Cols {
    float4 w[16], b, pos[kEmbedWgTok];
  };
  // loads of column group c4 (clamped to an in-bounds group; its results are used only
  // if c4 < d4n)
  auto load_cols = [&](int c4, Cols& k) {
    const int d = 4 * min(c4, d4n - 1);
#pragma unroll
    for (int f = 0; f < 16; ++f) k.w[f] = *(const float4*)(a.W_pe + (size_t)f * a.D + d);
    k.b = *(const float4*)(a.b_pe + d);
#pragma unroll
    for (int t = 0; t < kEmbedWgTok; ++t) {
      const int m = min(m0 + t, M - 1);
      const int n = m - (m / a.N) * a.N;
      k.pos[t] = *(const float4*)(a.pos + (size_t)n * a.D + d);
    }
  };
  auto compute_cols = [&](int c4, const Cols& k) {
    const int d = 4 * c4;
#pragma unroll
    for (int t = 0; t < kEmbedWgTok; ++t) {
      if (t >= nt) break;
      float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 pv = px_s[t][q];
        const float p4[4] = {pv.x, pv.y, pv.z, pv.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float4 wf = k.w[4 * q + e];
          acc.x += p4[e] * wf.x; acc.y += p4[e] * wf.y; acc.z += p4[e] * wf.z; acc.w += p4[e] * wf.w;
        }
      }
      *(float4*)(a.h + (size_t)(m0 + t) * a.D + d) =
          make_float4((acc.x + k.b.x) + k.pos[t].x, (acc.y + k.b.y) + k.pos[t].y, (acc.z + k.b.z) + k.pos[t].z,
                      (acc.w + k.b.w) + k.pos[t].w);
    }
  };
  // the patch-value load first, so that staging it waits for it alone
  const bool stager = tid < kEmbedWgTok * 8;
  const int st = tid >> 3, sc = (tid >> 1) & 3, si = tid & 1;
  float2 pxv;
  {
    const int m = min(m0 + st, M - 1);
    const int r = m / a.N, n = m - r * a.N;
    const int lat = r % a.n_lat;
    const int gh = n / gwn, gw = n - gh * gwn;
    // threads past the stagers load the first stager's value (in bounds, unused)
    pxv = *(const float2*)(a.x + (((size_t)lat * 4 + (stager ? sc : 0)) * a.H + gh * 2 + (stager ? si : 0)) * a.W + gw * 2);
  }
  __builtin_amdgcn_sched_barrier(0);  // keep it ahead of the column loads
  Cols first;
  load_cols(tid, first);
  if (stager) {
    float* ps = (float*)&px_s[st][0];
    ps[(2 * si + 0) * 4 + sc] = pxv.x;
    ps[(2 * si + 1) * 4 + sc] = pxv.y;
  }
  __syncthreads();
  if (tid < d4n) compute_cols(tid, first);
  for (int c4 = tid + 256; c4 < d4n; c4 += 256) {
    Cols k;
    load_cols(c4, k);
    compute_cols(c4, k);
  }
}

__global__ __launch_bounds__(256) void embed_p2c4_kernel(EmbedArgs a) { embed_p2c4_body(a, blockIdx.x); }

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
  if (a.p == 2 && a.C == 4) {
    launch(embed_p2c4_kernel, dim3((a.rows * a.N + kEmbedWgTok - 1) / kEmbedWgTok), dim3(256), 0, s, a);
  } else {
    launch(embed_kernel, dim3((total + 255) / 256), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

// The adaLN GEMV and the patch embed in one grid. They are independent (the embed does
// not read the conditioning), and the GEMV's workgroups leave most of the chip idle in
// their last round (1776 of them at 512^2, three per CU: 2.3 rounds). So the embed's
// workgroups follow the GEMV's in the same launch, filling that round, instead of
// running as a launch of their own. Each part computes exactly what its own kernel does.
template <typename WT, int NC, int RW>
__global__ __launch_bounds__(256) void gemv_embed_kernel(GemvArgs g, EmbedArgs e, int n_gemv) {
  if ((int)blockIdx.x < n_gemv)
    gemv_body<WT, NC, RW, 0>(g, blockIdx.x);
  else
    embed_p2c4_body(e, blockIdx.x - n_gemv);
}

bool gemv_embed_supported(bool w_bf16, const GemvArgs& g, const EmbedArgs& e) {
  const int E = w_bf16 ? 8 : 4;
  const int nc = (g.K / E + 63) / 64;
  return g.x_mode == 0 && e.p == 2 && e.C == 4 && g.K % E == 0 && nc >= 1 && nc <= 3 &&
         (size_t)g.R * g.K * (w_bf16 ? 2 : 4) < (1ull << 31);
}

template <typename WT, int NC>
static void launch_gemv_embed_nc(const GemvArgs& g, const EmbedArgs& e, hipStream_t s) {
  constexpr int RW = gemv_rows_per_wave<WT, NC>();
  const int n_gemv = ((g.R + RW - 1) / RW + 3) / 4;
  const int n_embed = (e.rows * e.N + kEmbedWgTok - 1) / kEmbedWgTok;
  launch((gemv_embed_kernel<WT, NC, RW>), dim3(n_gemv + n_embed), dim3(256), 0, s, g, e, n_gemv);
}

hipError_t launch_gemv_embed(bool w_bf16, const GemvArgs& g, const EmbedArgs& e, hipStream_t s) {
  if (!gemv_embed_supported(w_bf16, g, e)) return hipErrorInvalidValue;
  const int nc = (g.K / (w_bf16 ? 8 : 4) + 63) / 64;
  if (w_bf16) {
    if (nc == 1) launch_gemv_embed_nc<bf16, 1>(g, e, s);
    else if (nc == 2) launch_gemv_embed_nc<bf16, 2>(g, e, s);
    else launch_gemv_embed_nc<bf16, 3>(g, e, s);
  } else {
    if (nc == 1) launch_gemv_embed_nc<float, 1>(g, e, s);
    else if (nc == 2) launch_gemv_embed_nc<float, 2>(g, e, s);
    else launch_gemv_embed_nc<float, 3>(g, e, s);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------- context entries
// Network row r of a call with B slots: r < B conditional (entry of slot r), r >= B
// unconditional (the null-context entry, context row B).
__device__ __forceinline__ void write_kv_map(CtxState* st, int B, int guided, const int* ent) {
  const int rows = guided ? 2 * B : B;
  for (int r = threadIdx.x; r < rows; r += blockDim.x) st->kv_map[r] = ent[r < B ? r : B];
}

// Without reuse: entry j is context row j (j < B: ctx[j], j == B: the null context).
template <typename T>
__global__ __launch_bounds__(256) void ctx_prepare_kernel(CtxArgs a) {
  if (blockIdx.x == 0) {
    __shared__ int ent[kMaxRows + 1];
    for (int j = threadIdx.x; j <= a.B; j += blockDim.x) ent[j] = j;
    __syncthreads();
    write_kv_map(a.st, a.B, a.guided, ent);
  }
  const size_t total = (size_t)(a.B + a.guided) * a.per_row;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int j = (int)(i / a.per_row);
    const size_t e = i - (size_t)j * a.per_row;
    const float v = j < a.B ? a.ctx[i] : a.null_ctx[e];
    ((T*)a.ctxA)[(size_t)j * a.pitch + e] = from_f32<T>(v);
  }
}

// The two entries context row j may reuse: c0 the entry its slot held in the previous
// call, c1 the entry of the slot before it (Alg. 2's shift moves a latent and its
// context one slot on per step); the null row has only the previous null entry.
__device__ __forceinline__ void ctx_candidates(const CtxState* st, int B, int j, int& c0, int& c1) {
  if (j == B) {
    c0 = st->prev_null - 1;
    c1 = -1;
  } else {
    c0 = j < st->prev_B ? st->prev_slot[j] : -1;
    c1 = (j >= 1 && j - 1 < st->prev_B) ? st->prev_slot[j - 1] : -1;
  }
}

constexpr int kCtxPer = 16;                // floats per thread and workgroup pass
constexpr int kCtxChunk = 256 * kCtxPer;    // floats compared / copied per workgroup

// grid (context rows, chunks): bitwise comparison of each context row with the stored
// context of its candidate entries (both in one pass over the row, every load of a
// thread issued before the first comparison); a difference anywhere sets the
// candidate's bit. The workgroup's finding leaves in one atomic, so rows that differ
// everywhere (the shifted slots against their own old entry) do not serialise hundreds
// of atomics on one word.
__global__ __launch_bounds__(256) void ctx_compare_kernel(CtxArgs a) {
  const int j = blockIdx.x;
  int c0, c1;
  ctx_candidates(a.st, a.B, j, c0, c1);
  const float* row = j < a.B ? a.ctx + (size_t)j * a.per_row : a.null_ctx;
  const float* k0 = a.keep + (size_t)(c0 < 0 ? 0 : c0) * a.per_row;
  const float* k1 = a.keep + (size_t)(c1 < 0 ? 0 : c1) * a.per_row;
  const int i0 = blockIdx.y * kCtxChunk + threadIdx.x;
  uint32_t x[kCtxPer], y0[kCtxPer], y1[kCtxPer];
#pragma unroll
  for (int u = 0; u < kCtxPer; ++u) {
    const int i = min(i0 + u * 256, a.per_row - 1);  // past the row: a repeat of its last element
    x[u] = __float_as_uint(row[i]);
    y0[u] = __float_as_uint(k0[i]);
    y1[u] = __float_as_uint(k1[i]);
  }
  bool d0 = false, d1 = false;
#pragma unroll
  for (int u = 0; u < kCtxPer; ++u) {
    d0 |= x[u] != y0[u];
    d1 |= x[u] != y1[u];
  }
  d0 &= c0 >= 0;
  d1 &= c1 >= 0;
  __shared__ int bits;
  if (threadIdx.x == 0) bits = 0;
  __syncthreads();
  const int mine = (__any(d0) ? 1 : 0) | (__any(d1) ? 2 : 0);
  if ((threadIdx.x & 63) == 0 && mine) atomicOr(&bits, mine);
  __syncthreads();
  if (threadIdx.x == 0 && bits) atomicOr(&a.st->flags[j], bits);
}

// Picks each context row's entry (a matching candidate, else an entry no row of this
// call uses), marks the new ones live, writes kv_map, and keeps this call's slot entries
// as the next call's candidates. The state moves between global memory and LDS with all
// 64 lanes; the choice itself is one lane's short loop over LDS only (dependent global
// or scratch accesses in that loop would cost a memory latency each).
__global__ __launch_bounds__(64) void ctx_assign_kernel(CtxArgs a) {
  CtxState* st = a.st;
  const int tid = threadIdx.x;
  const int rc = a.B + a.guided;
  __shared__ int prev[kMaxRows], flags[kMaxRows + 1], ent[kMaxRows + 1], live[kMaxRows + 1], src[kMaxRows + 1];
  __shared__ int s_prevB, s_prevNull, s_fresh;
  for (int j = tid; j <= kMaxRows; j += 64) {
    if (j < kMaxRows) prev[j] = st->prev_slot[j];
    flags[j] = st->flags[j];
    live[j] = 0;
    src[j] = -1;
  }
  if (tid == 0) {
    s_prevB = st->prev_B;
    s_prevNull = st->prev_null;
  }
  __syncthreads();
  __shared__ bool taken[kMaxRows + 1];
  for (int e = tid; e <= kMaxRows; e += 64) taken[e] = false;
  __syncthreads();
  if (tid == 0) {
    for (int j = 0; j < rc; ++j) {
      int c0, c1;
      if (j == a.B) {
        c0 = s_prevNull - 1;
        c1 = -1;
      } else {
        c0 = j < s_prevB ? prev[j] : -1;
        c1 = (j >= 1 && j - 1 < s_prevB) ? prev[j - 1] : -1;
      }
      const int fl = flags[j];
      int e = -1;
      if (c0 >= 0 && !(fl & 1)) e = c0;
      else if (c1 >= 0 && !(fl & 2)) e = c1;
      ent[j] = e;
      if (e >= 0) taken[e] = true;
    }
    int next = 0, fresh = 0;
    for (int j = 0; j < rc; ++j) {
      if (ent[j] >= 0) continue;
      while (taken[next]) ++next;  // rc <= n_entries, so a free entry exists
      ent[j] = next;
      taken[next] = true;
      live[next] = 1;
      src[next] = j;
      ++fresh;
    }
    s_fresh = fresh;
  }
  __syncthreads();
  const int rows = a.guided ? 2 * a.B : a.B;
  for (int r = tid; r < rows; r += 64) st->kv_map[r] = ent[r < a.B ? r : a.B];
  for (int e = tid; e <= kMaxRows; e += 64) {
    st->live[e] = live[e];
    st->src[e] = src[e];
    st->flags[e] = 0;
  }
  for (int j = tid; j < a.B; j += 64) st->prev_slot[j] = ent[j];
  if (tid == 0) {
    st->prev_B = a.B;
    st->prev_null = a.guided ? ent[a.B] + 1 : 0;
    st->calls += 1;
    st->computed += (unsigned long long)s_fresh;
  }
}

// grid (entries, chunks): a live entry takes its context row (kept in fp32 for later
// comparisons, and in the compute type as the K/V GEMM operand).
template <typename T>
__global__ __launch_bounds__(256) void ctx_fill_kernel(CtxArgs a) {
  const int e = blockIdx.x;
  if (!a.st->live[e]) return;
  const int j = a.st->src[e];
  const float* row = j < a.B ? a.ctx + (size_t)j * a.per_row : a.null_ctx;
  const int i0 = blockIdx.y * kCtxChunk + threadIdx.x;
  float v[kCtxPer];
#pragma unroll
  for (int u = 0; u < kCtxPer; ++u) v[u] = row[min(i0 + u * 256, a.per_row - 1)];
#pragma unroll
  for (int u = 0; u < kCtxPer; ++u) {
    const int i = i0 + u * 256;
    if (i < a.per_row) {
      a.keep[(size_t)e * a.per_row + i] = v[u];
      ((T*)a.ctxA)[(size_t)e * a.pitch + i] = from_f32<T>(v[u]);
    }
  }
}

__global__ __launch_bounds__(64) void ctx_reset_kernel(CtxState* st) {
  int* p = (int*)st;
  for (int i = threadIdx.x; i < (int)(sizeof(CtxState) / sizeof(int)); i += 64) p[i] = 0;
}

hipError_t launch_ctx_prepare(bool use_bf16, const CtxArgs& a, hipStream_t s) {
  int grid = (int)(((size_t)(a.B + a.guided) * a.per_row + 255) / 256);
  if (grid > 4096) grid = 4096;
  if (use_bf16)
    launch(ctx_prepare_kernel<bf16>, dim3(grid), dim3(256), 0, s, a);
  else
    launch(ctx_prepare_kernel<float>, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_ctx_lookup(bool use_bf16, const CtxArgs& a, hipStream_t s) {
  const int chunks = (a.per_row + kCtxChunk - 1) / kCtxChunk;
  launch(ctx_compare_kernel, dim3(a.B + a.guided, chunks), dim3(256), 0, s, a);
  launch(ctx_assign_kernel, dim3(1), dim3(64), 0, s, a);
  if (use_bf16)
    launch(ctx_fill_kernel<bf16>, dim3(a.n_entries, chunks), dim3(256), 0, s, a);
  else
    launch(ctx_fill_kernel<float>, dim3(a.n_entries, chunks), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_ctx_reset(CtxState* st, hipStream_t s) {
  launch(ctx_reset_kernel, dim3(1), dim3(64), 0, s, st);
  return hipGetLastError();
}

// Scratch of the allocation-free conditioning call: the timestep MLP's hidden layer and
// SiLU(c), each [kMaxRows][kMaxWidth] fp32 (1 MiB in all). One copy per GPU, allocated
// with the code object and held until the process ends. Host code never passes the
// symbol itself to a kernel: it looks up the device address once per device
// (modulation_scratch) and uses that.
static __device__ __align__(256) float scratch[2 * kMaxRows * kMaxWidth];

hipError_t modulation_scratch(float** out, size_t* floats) {
  constexpr int kDevices = 64;
  static std::mutex mu;
  static float* addr[kDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return e != hipSuccess ? e : hipErrorInvalidSymbol;
    addr[dev] = (float*)p;
  }
  *out = addr[dev];
  *floats = sizeof(scratch) / sizeof(float);
  return hipSuccess;
}

}  // namespace sf
