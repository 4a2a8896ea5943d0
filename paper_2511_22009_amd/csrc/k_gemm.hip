// K3: the velocity network's dense projections, C[M][N] = A[M][K] . B[N][K]^T (both
// operands K-contiguous, weights stored [out][in]) with the epilogue fused:
//   QKV      + bias, scattered to head-major q, k and transposed v (the layout the
//            attention kernel consumes without a transpose);
//   RES_GATE h += gate[sample][n] * (acc + bias), the gate row picked by the token's
//            sample, i.e. each sample's own timestep (adaLN gate);
//   GELU     out = GELU_tanh(acc + bias);
//   RES      h += acc + bias.
//
// bf16 path: v_mfma_f32_32x32x16_bf16 on 128x128x64 workgroup tiles, four wavefronts
// each owning a 64x64 sub-tile (2x2 MFMA blocks), both operand tiles double-buffered in
// LDS with a 16-byte row pad so the 16-byte fragment reads of a 32-lane column are free
// of bank conflicts, and the next K-slice fetched into registers while the current one
// feeds the matrix cores. fp32 path: LDS-tiled FMA GEMM (exact fp32 arithmetic for
// the parity mode).
#include "sf_device.h"

namespace sf {

template <EpiKind KIND, typename OT>
__device__ __forceinline__ void epilogue(const GemmArgs& a, int m, int n, float acc) {
  const float val = acc + a.bias[n];
  if constexpr (KIND == EPI_QKV) {
    const int part = (int)fdiv((uint32_t)n, a.div_D);
    const int rem = n - part * a.D;
    const int head = (int)fdiv((uint32_t)rem, a.div_dh);
    const int d = rem - head * a.dh;
    const int r = (int)fdiv((uint32_t)m, a.div_ntok);
    const int tok = m - r * a.ntok;
    const size_t bh = (size_t)r * a.heads + head;
    const int which = a.which_base + part;
    // Destination picked with selects, not a three-way branch: this compiler lowered
    // the divergent if / else-if / else form to code that stored the v part through
    // the k pointer.
    const size_t i_qk = (bh * a.ntok + tok) * a.dh + d;
    const size_t i_v = (bh * a.dh + d) * a.ldv + tok;
    OT* const p_qk = (OT*)(which == 0 ? a.q : a.k);
    OT* const dst = which >= 2 ? (OT*)a.vT + i_v : p_qk + i_qk;
    *dst = from_f32<OT>(val);
  } else if constexpr (KIND == EPI_RES_GATE) {
    const int r = (int)fdiv((uint32_t)m, a.div_ntok);
    const int slot = r < a.n_slots ? r : r - a.n_slots;
    const float g = a.table[(size_t)slot * a.ldt + a.gate_off + n];
    float* hp = a.h + (size_t)m * a.ldh + n;
    *hp = *hp + g * val;
  } else if constexpr (KIND == EPI_GELU) {
    ((OT*)a.out)[(size_t)m * a.ldo + n] = from_f32<OT>(gelu_tanh(val));
  } else {
    float* hp = a.h + (size_t)m * a.ldh + n;
    *hp = *hp + val;
  }
}

// ------------------------------------------------------------------ bf16 / MFMA
constexpr int kBK = 64;
constexpr int kLdk = kBK + 8;  // LDS row pitch in bf16 (144 bytes)

__device__ __forceinline__ void store4(bf16* p, float a, float b, float c, float d) {
  const bf16x4 v = {(bf16)a, (bf16)b, (bf16)c, (bf16)d};
  *(bf16x4*)p = v;
}

// Epilogue over the C tile staged in LDS (fp32, row pitch CP), four outputs per
// thread and step: row-contiguous for h, GELU output, q and k; token-contiguous for the
// transposed v.
template <EpiKind KIND, int BM, int BN, int NT>
__device__ __forceinline__ void staged_epilogue(const GemmArgs& a, const float* Cs, int CP, int m0, int n0,
                                                int tid) {
  constexpr int C4 = BN / 4;
  for (int c = tid; c < BM * C4; c += NT) {
    const int row = c / C4, c4 = c - row * C4;
    const int m = m0 + row, n = n0 + c4 * 4;
    if (m >= a.M || n >= a.N) continue;
    const float4 acc = *(const float4*)&Cs[row * CP + c4 * 4];
    const float4 b = *(const float4*)(a.bias + n);
    const float v0 = acc.x + b.x, v1 = acc.y + b.y, v2 = acc.z + b.z, v3 = acc.w + b.w;
    if constexpr (KIND == EPI_QKV) {
      const int part = (int)fdiv((uint32_t)n, a.div_D);
      const int which = a.which_base + part;
      if (which >= 2) continue;  // v columns: second pass
      const int rem = n - part * a.D;
      const int head = (int)fdiv((uint32_t)rem, a.div_dh);
      const int d = rem - head * a.dh;
      const int r = (int)fdiv((uint32_t)m, a.div_ntok);
      const int tok = m - r * a.ntok;
      bf16* base = (bf16*)(which == 0 ? a.q : a.k);
      store4(base + (((size_t)r * a.heads + head) * a.ntok + tok) * a.dh + d, v0, v1, v2, v3);
    } else if constexpr (KIND == EPI_RES_GATE) {
      const int r = (int)fdiv((uint32_t)m, a.div_ntok);
      const int slot = r < a.n_slots ? r : r - a.n_slots;
      const float4 g = *(const float4*)(a.table + (size_t)slot * a.ldt + a.gate_off + n);
      float4* hp = (float4*)(a.h + (size_t)m * a.ldh + n);
      float4 h = *hp;
      h.x += g.x * v0; h.y += g.y * v1; h.z += g.z * v2; h.w += g.w * v3;
      *hp = h;
    } else if constexpr (KIND == EPI_GELU) {
      store4((bf16*)a.out + (size_t)m * a.ldo + n, gelu_tanh(v0), gelu_tanh(v1), gelu_tanh(v2), gelu_tanh(v3));
    } else {
      float4* hp = (float4*)(a.h + (size_t)m * a.ldh + n);
      float4 h = *hp;
      h.x += v0; h.y += v1; h.z += v2; h.w += v3;
      *hp = h;
    }
  }
  if constexpr (KIND == EPI_QKV) {
    constexpr int R4 = BM / 4;
    for (int c = tid; c < R4 * BN; c += NT) {
      const int col = c / R4, r4 = c - col * R4;
      const int n = n0 + col, m = m0 + r4 * 4;
      if (n >= a.N || m >= a.M) continue;
      const int part = (int)fdiv((uint32_t)n, a.div_D);
      if (a.which_base + part < 2) continue;
      const int rem = n - part * a.D;
      const int head = (int)fdiv((uint32_t)rem, a.div_dh);
      const int d = rem - head * a.dh;
      const int r = (int)fdiv((uint32_t)m, a.div_ntok);
      const int tok = m - r * a.ntok;
      const float bn = a.bias[n];
      bf16* vt = (bf16*)a.vT + (((size_t)r * a.heads + head) * a.dh + d) * a.ldv;
      const float* cp = Cs + (r4 * 4) * CP + col;
      if (tok + 3 < a.ntok && m + 3 < a.M && (tok & 3) == 0) {
        store4(vt + tok, cp[0] + bn, cp[CP] + bn, cp[2 * CP] + bn, cp[3 * CP] + bn);
      } else {
        for (int q = 0; q < 4 && m + q < a.M; ++q) {
          const int mq = m + q;
          const int rq = (int)fdiv((uint32_t)mq, a.div_ntok);
          const int tq = mq - rq * a.ntok;
          ((bf16*)a.vT)[(((size_t)rq * a.heads + head) * a.dh + d) * a.ldv + tq] = (bf16)(cp[q * CP] + bn);
        }
      }
    }
  }
}

// Operand tiles come in through raw buffer loads: rows past M or N and columns past K
// get an out-of-range offset and read as zeros, so the loads carry no branches and stay
// in flight while the matrix cores work on the previous K slice.
template <int BM, int BN, int WM, int WN, EpiKind KIND>
__global__ __launch_bounds__(WM * WN * 64) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM / 32;
  constexpr int TN = BN / WN / 32;
  constexpr int CPR = kBK / 8;  // 16-byte chunks per tile row
  constexpr int ACH = BM * CPR / NT;
  constexpr int BCH = BN * CPR / NT;
  static_assert(ACH * NT == BM * CPR && BCH * NT == BN * CPR, "tile / thread mismatch");
  constexpr int AB_BYTES = 2 * (BM + BN) * kLdk * 2;
  constexpr int CP = BN + 4;
  constexpr int C_BYTES = BM * CP * 4;
  constexpr int SMEM = AB_BYTES > C_BYTES ? AB_BYTES : C_BYTES;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  bf16* As = (bf16*)smem;
  bf16* Bs = As + 2 * BM * kLdk;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int l32 = lane & 31, g = lane >> 5;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;

  const __amdgpu_buffer_rsrc_t ra_src = buffer_rsrc(a.A, (uint32_t)a.M * a.lda * 2);
  const __amdgpu_buffer_rsrc_t rb_src = buffer_rsrc(a.B, (uint32_t)a.N * a.ldb * 2);
  int a_off[ACH], b_off[BCH], a_kc[ACH], b_kc[BCH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    const int c = tid + i * NT, row = c / CPR;
    a_kc[i] = (c % CPR) * 8;
    a_off[i] = (m0 + row < a.M) ? ((m0 + row) * a.lda + a_kc[i]) * 2 : kOffOOB;
  }
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int c = tid + i * NT, row = c / CPR;
    b_kc[i] = (c % CPR) * 8;
    b_off[i] = (n0 + row < a.N) ? ((n0 + row) * a.ldb + b_kc[i]) * 2 : kOffOOB;
  }
  u32x4 ra[ACH], rb[BCH];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < ACH; ++i)
      ra[i] = buffer_load16(ra_src, (k0 + a_kc[i] < a.K && a_off[i] != kOffOOB) ? a_off[i] + 2 * k0 : kOffOOB);
#pragma unroll
    for (int i = 0; i < BCH; ++i)
      rb[i] = buffer_load16(rb_src, (k0 + b_kc[i] < a.K && b_off[i] != kOffOOB) ? b_off[i] + 2 * k0 : kOffOOB);
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + i * NT, row = c / CPR;
      *(u32x4*)&As[buf * BM * kLdk + row * kLdk + a_kc[i]] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + i * NT, row = c / CPR;
      *(u32x4*)&Bs[buf * BN * kLdk + row * kLdk + b_kc[i]] = rb[i];
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = (a.K + kBK - 1) / kBK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * kBK);
    const bf16* Ab = As + cur * BM * kLdk + (wm * TM * 32 + l32) * kLdk + g * 8;
    const bf16* Bb = Bs + cur * BN * kLdk + (wn * TN * 32 + l32) * kLdk + g * 8;
    bf16x8 af[2][TM], bfr[2][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) af[0][i] = *(const bf16x8*)(Ab + i * 32 * kLdk);
#pragma unroll
    for (int j = 0; j < TN; ++j) bfr[0][j] = *(const bf16x8*)(Bb + j * 32 * kLdk);
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      const int cb = kk & 1;
      if (kk + 1 < kBK / 16) {
#pragma unroll
        for (int i = 0; i < TM; ++i) af[cb ^ 1][i] = *(const bf16x8*)(Ab + i * 32 * kLdk + (kk + 1) * 16);
#pragma unroll
        for (int j = 0; j < TN; ++j) bfr[cb ^ 1][j] = *(const bf16x8*)(Bb + j * 32 * kLdk + (kk + 1) * 16);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cb][i], bfr[cb][j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // stage C (lane holds column l32, rows (r/4)*8 + g*4 + r%4 of each 32x32 block)
  float* Cs = (float*)smem;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = (wm * TM + i) * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
        const int col = (wn * TN + j) * 32 + l32;
        Cs[row * CP + col] = acc[i][j][r];
      }
  __syncthreads();
  staged_epilogue<KIND, BM, BN, NT>(a, Cs, CP, m0, n0, tid);
}

// ------------------------------------------------------------------ fp32 / FMA
constexpr int kFT = 64;   // tile edge
constexpr int kFK = 16;   // K slice

template <EpiKind KIND>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  __shared__ float As[kFK][kFT + 4];
  __shared__ float Bs[kFK][kFT + 4];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * kFT, n0 = blockIdx.x * kFT;
  const float* A = (const float*)a.A;
  const float* B = (const float*)a.B;
  float acc[4][4] = {};
  const int lr = tid >> 2, lk = (tid & 3) * 4;  // loader: row lr, k offset lk
  for (int k0 = 0; k0 < a.K; k0 += kFK) {
    {
      const int gm = m0 + lr, gk = k0 + lk;
      float4 v = (gm < a.M && gk < a.K) ? *(const float4*)(A + (size_t)gm * a.lda + gk) : make_float4(0, 0, 0, 0);
      As[lk + 0][lr] = v.x; As[lk + 1][lr] = v.y; As[lk + 2][lr] = v.z; As[lk + 3][lr] = v.w;
      const int gn = n0 + lr;
      float4 w = (gn < a.N && gk < a.K) ? *(const float4*)(B + (size_t)gn * a.ldb + gk) : make_float4(0, 0, 0, 0);
      Bs[lk + 0][lr] = w.x; Bs[lk + 1][lr] = w.y; Bs[lk + 2][lr] = w.z; Bs[lk + 3][lr] = w.w;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kFK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += av[i] * bv[j];
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty + 16 * i;
    if (m >= a.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx + 16 * j;
      if (n < a.N) epilogue<KIND, float>(a, m, n, acc[i][j]);
    }
  }
}

template <EpiKind KIND>
static hipError_t launch_kind(bool use_bf16, const GemmArgs& a, hipStream_t s) {
  if (use_bf16) {
    constexpr int BM = 128, BN = 128;
    dim3 grid((a.N + BN - 1) / BN, (a.M + BM - 1) / BM);
    hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, 2, 2, KIND>), grid, dim3(256), 0, s, a);
  } else {
    dim3 grid((a.N + kFT - 1) / kFT, (a.M + kFT - 1) / kFT);
    hipLaunchKernelGGL(gemm_f32_kernel<KIND>, grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_gemm(bool use_bf16, EpiKind kind, const GemmArgs& a, hipStream_t s) {
  switch (kind) {
    case EPI_QKV: return launch_kind<EPI_QKV>(use_bf16, a, s);
    case EPI_RES_GATE: return launch_kind<EPI_RES_GATE>(use_bf16, a, s);
    case EPI_GELU: return launch_kind<EPI_GELU>(use_bf16, a, s);
    case EPI_RES: return launch_kind<EPI_RES>(use_bf16, a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace sf
