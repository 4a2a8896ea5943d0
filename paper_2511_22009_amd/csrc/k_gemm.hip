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
#include <cmath>

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

// Block -> tile map. The hardware hands workgroup b to XCD b % 8 and each XCD has its
// own L2, so each XCD gets a contiguous range of logical tiles; inside it tiles go in
// groups of kGroupM tile rows, M fastest, so the A rows and B columns a group touches
// are reused from one L2. Bijective for any tile count.
constexpr int kXcds = 8;
constexpr int kGroupM = 8;
__device__ __forceinline__ void tile_coords(int nbm, int nbn, int& mt, int& nt) {
  const int T = nbm * nbn;
  const int b = blockIdx.x;
  const int xcd = b % kXcds, local = b / kXcds;
  const int base = T / kXcds, rem = T % kXcds;
  const int logical = xcd * base + min(xcd, rem) + local;
  const int per_group = kGroupM * nbn;
  const int group = logical / per_group;
  const int first_m = group * kGroupM;
  const int gsize = min(kGroupM, nbm - first_m);
  const int in = logical - group * per_group;
  mt = first_m + in % gsize;
  nt = in / gsize;
}

// Operand tiles come in through raw buffer loads: rows past M or N and columns past K
// get an out-of-range offset and read as zeros, so the loads carry no branches. Two
// register stages keep the tile two K slices ahead in flight while the matrix cores
// work on the current one from LDS (double-buffered, 16-byte row pad). PF = 1 keeps
// one register stage (tiles with many wavefronts, where other wavefronts hide the
// latency and registers are scarce), PF = 2 keeps two.
template <int BM, int BN, int WM, int WN, int PF, EpiKind KIND>
__global__ __launch_bounds__(WM * WN * 64) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM / 32;
  constexpr int TN = BN / WN / 32;
  static_assert(TM * WM * 32 == BM && TN * WN * 32 == BN, "wave grid must tile the block");
  constexpr int CPR = kBK / 8;  // 16-byte chunks per tile row
  constexpr int ATOT = BM * CPR, BTOT = BN * CPR;
  constexpr int ACH = (ATOT + NT - 1) / NT;
  constexpr int BCH = (BTOT + NT - 1) / NT;
  constexpr int AB_BYTES = 2 * (BM + BN) * kLdk * 2;
  constexpr int CP = BN + 4;
  constexpr int LDS_CAP = 160 * 1024;
  constexpr int NP = (BM * CP * 4 <= LDS_CAP) ? 1 : ((BM / 2) * CP * 4 <= LDS_CAP ? 2 : 4);
  constexpr int RP = BM / NP;  // C rows staged per pass
  static_assert(RP % 32 == 0, "staging pass must hold whole MFMA blocks");
  constexpr int C_BYTES = RP * CP * 4;
  constexpr int SMEM = AB_BYTES > C_BYTES ? AB_BYTES : C_BYTES;
  static_assert(SMEM <= LDS_CAP, "tile does not fit in LDS");
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  bf16* As = (bf16*)smem;
  bf16* Bs = As + 2 * BM * kLdk;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int l32 = lane & 31, g = lane >> 5;
  int mt, nt;
  tile_coords((a.M + BM - 1) / BM, (a.N + BN - 1) / BN, mt, nt);
  const int m0 = mt * BM, n0 = nt * BN;

  const __amdgpu_buffer_rsrc_t ra_src = buffer_rsrc(a.A, (uint32_t)a.M * a.lda * 2);
  const __amdgpu_buffer_rsrc_t rb_src = buffer_rsrc(a.B, (uint32_t)a.N * a.ldb * 2);
  int a_off[ACH], b_off[BCH], a_lds[ACH], b_lds[BCH], a_kc[ACH], b_kc[BCH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    const int c = tid + i * NT, row = c / CPR;
    a_kc[i] = (c % CPR) * 8;
    a_lds[i] = row * kLdk + a_kc[i];
    a_off[i] = (c < ATOT && m0 + row < a.M) ? ((m0 + row) * a.lda + a_kc[i]) * 2 : kOffOOB;
  }
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int c = tid + i * NT, row = c / CPR;
    b_kc[i] = (c % CPR) * 8;
    b_lds[i] = row * kLdk + b_kc[i];
    b_off[i] = (c < BTOT && n0 + row < a.N) ? ((n0 + row) * a.ldb + b_kc[i]) * 2 : kOffOOB;
  }
  u32x4 ra[PF][ACH], rb[PF][BCH];
  auto gload = [&](u32x4 (&va)[ACH], u32x4 (&vb)[BCH], int kt) {
    const int k0 = kt * kBK;
#pragma unroll
    for (int i = 0; i < ACH; ++i)
      va[i] = buffer_load16(ra_src, (k0 + a_kc[i] < a.K && a_off[i] != kOffOOB) ? a_off[i] + 2 * k0 : kOffOOB);
#pragma unroll
    for (int i = 0; i < BCH; ++i)
      vb[i] = buffer_load16(rb_src, (k0 + b_kc[i] < a.K && b_off[i] != kOffOOB) ? b_off[i] + 2 * k0 : kOffOOB);
  };
  auto lstore = [&](const u32x4 (&va)[ACH], const u32x4 (&vb)[BCH], int buf) {
#pragma unroll
    for (int i = 0; i < ACH; ++i)
      if (ATOT % NT == 0 || tid + i * NT < ATOT) *(u32x4*)&As[buf * BM * kLdk + a_lds[i]] = va[i];
#pragma unroll
    for (int i = 0; i < BCH; ++i)
      if (BTOT % NT == 0 || tid + i * NT < BTOT) *(u32x4*)&Bs[buf * BN * kLdk + b_lds[i]] = vb[i];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  auto compute = [&](int buf) {
    const bf16* Ab = As + buf * BM * kLdk + (wm * TM * 32 + l32) * kLdk + g * 8;
    const bf16* Bb = Bs + buf * BN * kLdk + (wn * TN * 32 + l32) * kLdk + g * 8;
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
  };

  const int nk = (a.K + kBK - 1) / kBK;
  if constexpr (PF == 2) {
    gload(ra[0], rb[0], 0);
    if (nk > 1) gload(ra[PF - 1], rb[PF - 1], 1);
    lstore(ra[0], rb[0], 0);
    if (nk > 2) gload(ra[0], rb[0], 2);
    __syncthreads();
    for (int kt = 0; kt < nk; kt += 2) {
      compute(0);  // tile kt
      if (kt + 1 < nk) {
        lstore(ra[PF - 1], rb[PF - 1], 1);  // tile kt+1
        if (kt + 3 < nk) gload(ra[PF - 1], rb[PF - 1], kt + 3);
      }
      __syncthreads();
      if (kt + 1 >= nk) break;
      compute(1);  // tile kt+1
      if (kt + 2 < nk) {
        lstore(ra[0], rb[0], 0);  // tile kt+2
        if (kt + 4 < nk) gload(ra[0], rb[0], kt + 4);
      }
      __syncthreads();
    }
  } else {
    gload(ra[0], rb[0], 0);
    lstore(ra[0], rb[0], 0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + 1 < nk) gload(ra[0], rb[0], kt + 1);
      compute(kt & 1);
      if (kt + 1 < nk) lstore(ra[0], rb[0], (kt + 1) & 1);
      __syncthreads();
    }
  }

  // stage C in passes of RP rows (lane holds column l32 and rows (r/4)*8 + g*4 + r%4
  // of each 32x32 block), then run the fused epilogue on each pass
  float* Cs = (float*)smem;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int rb0 = (wm * TM + i) * 32;
      if (rb0 < p * RP || rb0 >= (p + 1) * RP) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = rb0 - p * RP + (r >> 2) * 8 + g * 4 + (r & 3);
          Cs[row * CP + (wn * TN + j) * 32 + l32] = acc[i][j][r];
        }
    }
    __syncthreads();
    staged_epilogue<KIND, RP, BN, NT>(a, Cs, CP, m0 + p * RP, n0, tid);
    if (p + 1 < NP) __syncthreads();
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

// The same GEMM with an explicitly interleaved main loop. Each K step is one straight
// block: the matrix-core instructions of tile k are interleaved (sched_group_barrier)
// with the LDS fragment reads of tile k, the LDS writes of tile k+1 (already in
// registers) and the buffer loads of tile k+2, so memory work issues under the MFMAs
// instead of in stalls between them.
template <int BM, int BN, int WM, int WN, EpiKind KIND>
__global__ __launch_bounds__(WM * WN * 64) void gemm_bf16_sched_kernel(GemmArgs a) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM / 32;
  constexpr int TN = BN / WN / 32;
  static_assert(TM * WM * 32 == BM && TN * WN * 32 == BN, "wave grid must tile the block");
  constexpr int CPR = kBK / 8;
  constexpr int ATOT = BM * CPR, BTOT = BN * CPR;
  constexpr int ACH = (ATOT + NT - 1) / NT;
  constexpr int BCH = (BTOT + NT - 1) / NT;
  static_assert(ATOT % NT == 0 && BTOT % NT == 0, "scheduled variant needs whole chunks per thread");
  constexpr int AB_BYTES = 2 * (BM + BN) * kLdk * 2;
  constexpr int CP = BN + 4;
  constexpr int LDS_CAP = 160 * 1024;
  constexpr int NP = (BM * CP * 4 <= LDS_CAP) ? 1 : ((BM / 2) * CP * 4 <= LDS_CAP ? 2 : 4);
  constexpr int RP = BM / NP;
  constexpr int C_BYTES = RP * CP * 4;
  constexpr int SMEM = AB_BYTES > C_BYTES ? AB_BYTES : C_BYTES;
  static_assert(SMEM <= LDS_CAP, "tile does not fit in LDS");
  constexpr int NMFMA = TM * TN * (kBK / 16);
  constexpr int NDSR = (TM + TN) * (kBK / 16);
  constexpr int NDSW = ACH + BCH;
  constexpr int NVMEM = ACH + BCH;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  bf16* As = (bf16*)smem;
  bf16* Bs = As + 2 * BM * kLdk;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int l32 = lane & 31, g = lane >> 5;
  int mt, nt;
  tile_coords((a.M + BM - 1) / BM, (a.N + BN - 1) / BN, mt, nt);
  const int m0 = mt * BM, n0 = nt * BN;

  const __amdgpu_buffer_rsrc_t ra_src = buffer_rsrc(a.A, (uint32_t)a.M * a.lda * 2);
  const __amdgpu_buffer_rsrc_t rb_src = buffer_rsrc(a.B, (uint32_t)a.N * a.ldb * 2);
  int a_off[ACH], b_off[BCH], a_lds[ACH], b_lds[BCH], a_kc[ACH], b_kc[BCH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    const int c = tid + i * NT, row = c / CPR;
    a_kc[i] = (c % CPR) * 8;
    a_lds[i] = row * kLdk + a_kc[i];
    a_off[i] = (m0 + row < a.M) ? ((m0 + row) * a.lda + a_kc[i]) * 2 : kOffOOB;
  }
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int c = tid + i * NT, row = c / CPR;
    b_kc[i] = (c % CPR) * 8;
    b_lds[i] = row * kLdk + b_kc[i];
    b_off[i] = (n0 + row < a.N) ? ((n0 + row) * a.ldb + b_kc[i]) * 2 : kOffOOB;
  }
  u32x4 ra[ACH], rb[BCH];
  auto gload = [&](int kt) {
    const int k0 = kt * kBK;
#pragma unroll
    for (int i = 0; i < ACH; ++i)
      ra[i] = buffer_load16(ra_src, (k0 + a_kc[i] < a.K && a_off[i] != kOffOOB) ? a_off[i] + 2 * k0 : kOffOOB);
#pragma unroll
    for (int i = 0; i < BCH; ++i)
      rb[i] = buffer_load16(rb_src, (k0 + b_kc[i] < a.K && b_off[i] != kOffOOB) ? b_off[i] + 2 * k0 : kOffOOB);
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) *(u32x4*)&As[buf * BM * kLdk + a_lds[i]] = ra[i];
#pragma unroll
    for (int i = 0; i < BCH; ++i) *(u32x4*)&Bs[buf * BN * kLdk + b_lds[i]] = rb[i];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // one K step on LDS buffer `cur`; optionally writes the next tile (registers -> LDS
  // buffer cur^1) and fetches the one after into registers
  auto step = [&](int cur, int kt, bool write_next, bool load_next) {
    const bf16* Ab = As + cur * BM * kLdk + (wm * TM * 32 + l32) * kLdk + g * 8;
    const bf16* Bb = Bs + cur * BN * kLdk + (wn * TN * 32 + l32) * kLdk + g * 8;
    bf16x8 af[kBK / 16][TM], bfr[kBK / 16][TN];
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
#pragma unroll
      for (int i = 0; i < TM; ++i) af[kk][i] = *(const bf16x8*)(Ab + i * 32 * kLdk + kk * 16);
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[kk][j] = *(const bf16x8*)(Bb + j * 32 * kLdk + kk * 16);
    }
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[kk][i], bfr[kk][j], acc[i][j], 0, 0, 0);
    if (write_next) lstore(cur ^ 1);
    if (load_next) gload(kt + 2);
    // interleave: fragment reads ahead of their MFMAs, then LDS writes and global loads
    // spread across the remaining MFMAs
    constexpr int R_PER = (NDSR + NMFMA - 1) / NMFMA;
#pragma unroll
    for (int i = 0; i < NMFMA / 2; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2 * R_PER, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
#pragma unroll
    for (int i = 0; i < NMFMA - NMFMA / 2; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x200, (NDSW + NMFMA / 2 - 1) / (NMFMA / 2), 0);
      __builtin_amdgcn_sched_group_barrier(0x020, (NVMEM + NMFMA / 2 - 1) / (NMFMA / 2), 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
  };

  const int nk = (a.K + kBK - 1) / kBK;
  gload(0);
  lstore(0);
  if (nk > 1) gload(1);
  __syncthreads();
  int kt = 0;
  for (; kt + 2 < nk; ++kt) {
    step(kt & 1, kt, true, true);
    __syncthreads();
  }
  if (kt + 1 < nk) {
    step(kt & 1, kt, true, false);
    __syncthreads();
    ++kt;
  }
  step(kt & 1, kt, false, false);
  __syncthreads();

  float* Cs = (float*)smem;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int rb0 = (wm * TM + i) * 32;
      if (rb0 < p * RP || rb0 >= (p + 1) * RP) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = rb0 - p * RP + (r >> 2) * 8 + g * 4 + (r & 3);
          Cs[row * CP + (wn * TN + j) * 32 + l32] = acc[i][j][r];
        }
    }
    __syncthreads();
    staged_epilogue<KIND, RP, BN, NT>(a, Cs, CP, m0 + p * RP, n0, tid);
    if (p + 1 < NP) __syncthreads();
  }
}

// Tile shapes (BM x BN, wave grid WM x WN, register prefetch stages). Per-wave tiles
// are 64x64, 64x96 or 32x96.
#define SF_GEMM_TILES(X)    \
  X(0, 128, 128, 2, 2, 2)   \
  X(1, 128, 96, 4, 1, 2)    \
  X(2, 128, 96, 2, 1, 2)    \
  X(3, 128, 288, 2, 3, 1)   \
  X(4, 128, 384, 2, 4, 1)   \
  X(5, 256, 128, 4, 2, 1)   \
  X(6, 64, 192, 1, 2, 2)    \
  X(7, 128, 192, 2, 2, 2)   \
  X(8, 256, 96, 4, 1, 2)    \
  X(9, 128, 128, 2, 2, 1)   \
  X(10, 256, 256, 2, 4, 1)  \
  X(11, 256, 128, 2, 2, 1)  \
  X(12, 256, 128, 2, 2, 2)  \
  X(13, 128, 256, 2, 2, 1)  \
  X(14, 256, 256, 4, 2, 1)  \
  X(15, 128, 128, 2, 2, 0)  \
  X(16, 256, 256, 2, 4, 0)  \
  X(17, 128, 256, 2, 2, 0)  \
  X(18, 256, 128, 4, 2, 0)

struct TileInfo {
  int bm, bn, waves;
};
static const TileInfo kTiles[] = {
#define SF_TILE_INFO(id, bm, bn, wm, wn, pf) {bm, bn, wm * wn},
    SF_GEMM_TILES(SF_TILE_INFO)
#undef SF_TILE_INFO
};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);

template <EpiKind KIND>
static hipError_t launch_bf16_tile(int tile, const GemmArgs& a, hipStream_t s) {
  switch (tile) {
#define SF_TILE_CASE(id, bm, bn, wm, wn, pf)                                                      \
  case id:                                                                                         \
    if constexpr (pf == 0)                                                                         \
      hipLaunchKernelGGL((gemm_bf16_sched_kernel<bm, bn, wm, wn, KIND>),                            \
                         dim3(((a.N + bn - 1) / bn) * ((a.M + bm - 1) / bm)), dim3(wm * wn * 64), 0, s, a); \
    else                                                                                           \
      hipLaunchKernelGGL((gemm_bf16_kernel<bm, bn, wm, wn, (pf == 0 ? 1 : pf), KIND>),               \
                         dim3(((a.N + bn - 1) / bn) * ((a.M + bm - 1) / bm)), dim3(wm * wn * 64), 0, s, a); \
    break;
    SF_GEMM_TILES(SF_TILE_CASE)
#undef SF_TILE_CASE
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// The interleaved 128x128 tile (id 15) measured fastest on every projection shape of
// the 512^2 and 1024^2 networks (M = 4096 / 16384, N in {768, 1152, 2304, 3072, 3456,
// 4608}); the other shapes stay available to launch_gemm_tile.
int choose_gemm_tile(int M, int N, int K) {
  (void)M;
  (void)N;
  (void)K;
  return 15;
}

template <EpiKind KIND>
static hipError_t launch_kind(bool use_bf16, int tile, const GemmArgs& a, hipStream_t s) {
  if (use_bf16) return launch_bf16_tile<KIND>(tile < 0 ? choose_gemm_tile(a.M, a.N, a.K) : tile, a, s);
  dim3 grid((a.N + kFT - 1) / kFT, (a.M + kFT - 1) / kFT);
  hipLaunchKernelGGL(gemm_f32_kernel<KIND>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gemm_tile(bool use_bf16, int tile, EpiKind kind, const GemmArgs& a, hipStream_t s) {
  switch (kind) {
    case EPI_QKV: return launch_kind<EPI_QKV>(use_bf16, tile, a, s);
    case EPI_RES_GATE: return launch_kind<EPI_RES_GATE>(use_bf16, tile, a, s);
    case EPI_GELU: return launch_kind<EPI_GELU>(use_bf16, tile, a, s);
    case EPI_RES: return launch_kind<EPI_RES>(use_bf16, tile, a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm(bool use_bf16, EpiKind kind, const GemmArgs& a, hipStream_t s) {
  return launch_gemm_tile(use_bf16, -1, kind, a, s);
}

}  // namespace sf
