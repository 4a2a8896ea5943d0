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

template <int BM, int BN, int WGM, int WGN, EpiKind KIND>
__global__ __launch_bounds__(WGM * WGN * 64) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int NT = WGM * WGN * 64;
  constexpr int TM = BM / WGM / 32;
  constexpr int TN = BN / WGN / 32;
  constexpr int CPR = kBK / 8;                 // 16-byte chunks per tile row
  constexpr int ACH = BM * CPR / NT;
  constexpr int BCH = BN * CPR / NT;
  static_assert(ACH * NT == BM * CPR && BCH * NT == BN * CPR, "tile / thread mismatch");
  __shared__ bf16 As[2][BM * kLdk];
  __shared__ bf16 Bs[2][BN * kLdk];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int l32 = lane & 31, g = lane >> 5;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const bf16* A = (const bf16*)a.A;
  const bf16* B = (const bf16*)a.B;

  uint4 ra[ACH], rb[BCH];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + i * NT, row = c / CPR, kc = c % CPR;
      const int gm = m0 + row, gk = k0 + kc * 8;
      ra[i] = (gm < a.M && gk < a.K) ? *(const uint4*)(A + (size_t)gm * a.lda + gk) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + i * NT, row = c / CPR, kc = c % CPR;
      const int gn = n0 + row, gk = k0 + kc * 8;
      rb[i] = (gn < a.N && gk < a.K) ? *(const uint4*)(B + (size_t)gn * a.ldb + gk) : make_uint4(0, 0, 0, 0);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + i * NT, row = c / CPR, kc = c % CPR;
      *(uint4*)&As[buf][row * kLdk + kc * 8] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + i * NT, row = c / CPR, kc = c % CPR;
      *(uint4*)&Bs[buf][row * kLdk + kc * 8] = rb[i];
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
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *(const bf16x8*)&As[cur][((wm * TM + i) * 32 + l32) * kLdk + kk * 16 + g * 8];
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *(const bf16x8*)&Bs[cur][((wn * TN + j) * 32 + l32) * kLdk + kk * 16 + g * 8];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // C block layout: lane holds column l32 and rows (r/4)*8 + g*4 + r%4.
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + (wn * TN + j) * 32 + l32;
      if (n >= a.N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + (wm * TM + i) * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
        if (m < a.M) epilogue<KIND, bf16>(a, m, n, acc[i][j][r]);
      }
    }
  }
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
