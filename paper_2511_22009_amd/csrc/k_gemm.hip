// K3: the velocity network's dense projections, C[M][N] = A[M][K] . B[N][K]^T (both
// operands K-contiguous, weights stored [out][in]) with the epilogue fused:
//   QKV      + bias, scattered to head-major q, k and transposed v (the layout the
//            attention kernel consumes without a transpose);
//   RES_GATE h += gate[sample][n] * (acc + bias), the gate row picked by the token's
//            sample, i.e. each sample's own timestep (adaLN gate);
//   GELU     out = GELU_tanh(acc + bias);
//   RES      h += acc + bias;
//   KVX      + bias, the cross-attention keys and transposed values of every block at
//            once (one context entry per network row).
//
// bf16 path: v_mfma_f32_32x32x16_bf16 on BM x BN x BK workgroup tiles (BK 64 or 128;
// table at the end), each wavefront owning a 64x64, 64x96 or 32x96 sub-tile, optionally with
// the K slice split over two sets of wavefronts; both operand tiles are
// double-buffered in LDS with a 16-byte row pad so the 16-byte fragment reads of a
// 32-lane column are free of bank conflicts, and the next K-slice is fetched into
// registers while the current one feeds the matrix cores. The MFMAs take the weight
// fragment as the first operand, so each lane ends up holding four adjacent output
// columns of one row, which the epilogues move in 8- and 16-byte pieces. fp32 path:
// LDS-tiled FMA GEMM (exact fp32 arithmetic for the parity mode).
#include <cmath>

#include "sf_device.h"

namespace sf {

// Destination of a projection column in part `part` (= n / D) of network row r: QKV
// part which_base + part (0 q, 1 k, 2 v) of row r; KVX the key (even part) or value of
// block part / 2, stored as row r * L + block of the [rows][heads][...] layouts.
template <EpiKind KIND>
__device__ __forceinline__ void qkv_dest(const GemmArgs& a, int part, int r, int& which, int& rr) {
  if constexpr (KIND == EPI_KVX) {
    which = 1 + (part & 1);
    rr = r * a.kv_blocks + (part >> 1);
  } else {
    which = a.which_base + part;
    rr = r;
  }
}

// True when the tile of rows m0 .. m0 + BM - 1 holds a row whose entry is live (or no
// liveness is given): the caller skips the whole tile otherwise.
template <EpiKind KIND, int BM>
__device__ __forceinline__ bool tile_live(const GemmArgs& a, int m0) {
  if constexpr (KIND != EPI_KVX) return true;
  if (!a.row_live) return true;
  const int r0 = (int)fdiv((uint32_t)m0, a.div_ntok);
  const int r1 = (int)fdiv((uint32_t)(min(m0 + BM, a.M) - 1), a.div_ntok);
  for (int r = r0; r <= r1; ++r)
    if (a.row_live[r]) return true;
  return false;
}

template <EpiKind KIND, typename OT>
__device__ __forceinline__ void epilogue(const GemmArgs& a, int m, int n, float acc) {
  const float val = acc + a.bias[n];
  if constexpr (KIND == EPI_QKV || KIND == EPI_KVX) {
    const int part = (int)fdiv((uint32_t)n, a.div_D);
    const int rem = n - part * a.D;
    const int head = (int)fdiv((uint32_t)rem, a.div_dh);
    const int d = rem - head * a.dh;
    const int r0 = (int)fdiv((uint32_t)m, a.div_ntok);
    const int tok = m - r0 * a.ntok;
    int which, r;
    qkv_dest<KIND>(a, part, r0, which, r);
    const size_t bh = (size_t)r * a.heads + head;
    // Destination picked with selects, not a three-way branch: this compiler lowered
    // the divergent if / else-if / else form to code that stored the v part through
    // the k pointer.
    const size_t i_qk = (bh * a.ntok + tok) * a.dh + d;
    const size_t i_v = (bh * a.dh + d) * a.ldv + (a.vperm ? vt_pos(tok) : tok);
    OT* const p_qk = (OT*)(which == 0 ? a.q : a.k);
    OT* const dst = which >= 2 ? (OT*)a.vT + i_v : p_qk + i_qk;
    *dst = from_f32<OT>(val);
  } else if constexpr (KIND == EPI_RES_GATE || KIND == EPI_RES_GATE_MLP) {
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

// Largest divisor of n that is at most cap: the number of epilogue items a thread
// handles per batch.
constexpr int batch_of(int n, int cap) {
  for (int u = cap; u > 1; --u)
    if (n % u == 0) return u;
  return 1;
}

// Epilogue of the fp32 residual projections (h += gate[sample] * (acc + bias) and
// h += acc + bias) over the C tile staged in LDS (fp32, row pitch CP), four adjacent
// outputs of a row per item. Items are processed in batches: every load of a batch (C
// from LDS, bias, gate, residual) is issued before any of its results is used, with
// out-of-tile items reading a clamped in-range address, so a batch pays one memory
// latency instead of one per item. Only the stores are predicated.
template <EpiKind KIND, int BM, int BN, int NT>
__device__ __forceinline__ void staged_epilogue(const GemmArgs& a, const float* Cs, int CP, int m0, int n0,
                                                int tid) {
  static_assert(KIND == EPI_RES || KIND == EPI_RES_GATE || KIND == EPI_RES_GATE_MLP, "residual epilogues only");
  constexpr bool kGate = KIND == EPI_RES_GATE || KIND == EPI_RES_GATE_MLP;
  constexpr int C4 = BN / 4;
  constexpr int TOTAL = BM * C4;
  constexpr int IT = (TOTAL + NT - 1) / NT;
  constexpr int U = batch_of(IT, kGate && NT > 256 ? 4 : 8);  // four live float4 loads per gated item
  for (int i0 = 0; i0 < IT; i0 += U) {
    float4 cv[U], bv[U], hv[U], gv[U];
    int mm[U], nn[U];
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = tid + (i0 + u) * NT;
      const int row = c / C4, c4 = c - row * C4;
      const int m = m0 + row, n = n0 + c4 * 4;
      ok[u] = (TOTAL % NT == 0 || c < TOTAL) && m < a.M && n < a.N;
      mm[u] = ok[u] ? m : m0;
      nn[u] = ok[u] ? n : 0;
      cv[u] = *(const float4*)&Cs[(ok[u] ? row : 0) * CP + (ok[u] ? c4 * 4 : 0)];
      bv[u] = *(const float4*)(a.bias + nn[u]);
      hv[u] = *(const float4*)(a.h + (size_t)mm[u] * a.ldh + nn[u]);
      if constexpr (kGate) {
        const int r = (int)fdiv((uint32_t)mm[u], a.div_ntok);
        const int slot = r < a.n_slots ? r : r - a.n_slots;
        gv[u] = *(const float4*)(a.table + (size_t)slot * a.ldt + a.gate_off + nn[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int m = mm[u], n = nn[u];
      const float v0 = cv[u].x + bv[u].x, v1 = cv[u].y + bv[u].y, v2 = cv[u].z + bv[u].z, v3 = cv[u].w + bv[u].w;
      float4 h = hv[u];
      if constexpr (kGate) {
        h.x += gv[u].x * v0; h.y += gv[u].y * v1; h.z += gv[u].z * v2; h.w += gv[u].w * v3;
      } else {
        h.x += v0; h.y += v1; h.z += v2; h.w += v3;
      }
      if (ok[u]) *(float4*)(a.h + (size_t)m * a.ldh + n) = h;
    }
  }
}

// The same residual epilogue with its global operands loaded ahead of time: load()
// issues, for one pass of RP tile rows, the bias, gate-row and residual loads of a
// thread's items (clamped in-range addresses for items outside the tile), so their
// latency can pass under other work; apply() combines them with the C tile staged in
// LDS, with the arithmetic of staged_epilogue, and stores.
template <EpiKind KIND, int RP, int BN, int NT>
struct ResItems {
  static_assert(KIND == EPI_RES || KIND == EPI_RES_GATE || KIND == EPI_RES_GATE_MLP || KIND == EPI_GELU ||
                    KIND == EPI_QKV || KIND == EPI_KVX,
                "epilogue kind");
  static constexpr bool kGate = KIND == EPI_RES_GATE || KIND == EPI_RES_GATE_MLP;
  static constexpr int C4 = BN / 4;
  static constexpr int TOTAL = RP * C4;
  static constexpr int IT = (TOTAL + NT - 1) / NT;
  float4 b[IT], h[IT], g[IT];

  __device__ __forceinline__ static bool item(const GemmArgs& a, int m0, int n0, int tid, int u, int& row, int& c4,
                                              int& m, int& n) {
    const int c = tid + u * NT;
    row = c / C4;
    c4 = c - row * C4;
    m = m0 + row;
    n = n0 + c4 * 4;
    return (TOTAL % NT == 0 || c < TOTAL) && m < a.M && n < a.N;
  }
  __device__ __forceinline__ void load(const GemmArgs& a, int m0, int n0, int tid) {
#pragma unroll
    for (int u = 0; u < IT; ++u) {
      int row, c4, m, n;
      const bool ok = item(a, m0, n0, tid, u, row, c4, m, n);
      const int mm = ok ? m : m0, nn = ok ? n : 0;
      b[u] = *(const float4*)(a.bias + nn);
      h[u] = *(const float4*)(a.h + (size_t)mm * a.ldh + nn);
      if constexpr (kGate) {
        const int r = (int)fdiv((uint32_t)mm, a.div_ntok);
        const int slot = r < a.n_slots ? r : r - a.n_slots;
        g[u] = *(const float4*)(a.table + (size_t)slot * a.ldt + a.gate_off + nn);
      }
    }
  }
  __device__ __forceinline__ void apply(const GemmArgs& a, const float* Cs, int CP, int m0, int n0, int tid) const {
#pragma unroll
    for (int u = 0; u < IT; ++u) {
      int row, c4, m, n;
      const bool ok = item(a, m0, n0, tid, u, row, c4, m, n);
      const float4 cv = *(const float4*)&Cs[(ok ? row : 0) * CP + (ok ? c4 * 4 : 0)];
      const float v0 = cv.x + b[u].x, v1 = cv.y + b[u].y, v2 = cv.z + b[u].z, v3 = cv.w + b[u].w;
      float4 hh = h[u];
      if constexpr (kGate) {
        hh.x += g[u].x * v0; hh.y += g[u].y * v1; hh.z += g[u].z * v2; hh.w += g[u].w * v3;
      } else {
        hh.x += v0; hh.y += v1; hh.z += v2; hh.w += v3;
      }
      if (ok) *(float4*)(a.h + (size_t)m * a.ldh + n) = hh;
    }
  }
};

// Epilogue of the bf16-output projections (GELU for the MLP up-projection, the head
// split for QKV). Bias and activation are applied in registers, where every lane holds
// four adjacent columns of one row; the bf16 results are staged in LDS (8-byte writes)
// and leave in 16-byte chunks: 8 adjacent columns of a row for the GELU output and for
// q / k (a chunk never straddles a head since the head width is a multiple of 8), and 8
// adjacent tokens of one column for the transposed v.
constexpr int kEpiPad = 8;  // bf16 row pad of the staged tile (16 bytes)

template <EpiKind KIND, int BM, int BN, int TM, int TN, int NT>
__device__ __forceinline__ void bf16_epilogue(const GemmArgs& a, const f32x16 (&acc)[TM][TN], bf16* Cs,
                                              const float* bias_s, int m0, int n0, int wm, int wn, int l32, int g,
                                              bool owner, int tid) {
  constexpr int CPB = BN + kEpiPad;
  f32x4 bias[TN][4];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) bias[j][q] = *(const f32x4*)&bias_s[(wn * TN + j) * 32 + q * 8 + g * 4];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    if (!owner) break;
    const int row = (wm * TM + i) * 32 + l32;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[e] = acc[i][j][4 * q + e] + bias[j][q][e];
          if constexpr (KIND == EPI_GELU) v[e] = gelu_tanh(v[e]);
        }
        const bf16x4 o = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
        *(bf16x4*)&Cs[row * CPB + (wn * TN + j) * 32 + q * 8 + g * 4] = o;
      }
  }
  __syncthreads();
  // row-major 16-byte chunks: the whole GELU tile; the q and k columns of QKV
  constexpr int C8 = BN / 8;
  constexpr int TOTAL = BM * C8;
  constexpr int IT = (TOTAL + NT - 1) / NT;
  constexpr int U = batch_of(IT, 8);
  for (int i0 = 0; i0 < IT; i0 += U) {
    u32x4 val[U];
    int mm[U], nn[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = tid + (i0 + u) * NT;
      const int row = c / C8, c8 = c - row * C8;
      const bool in = TOTAL % NT == 0 || c < TOTAL;
      mm[u] = in ? m0 + row : a.M;
      nn[u] = n0 + c8 * 8;
      val[u] = *(const u32x4*)&Cs[(in ? row : 0) * CPB + c8 * 8];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int m = mm[u], n = nn[u];
      if (m >= a.M || n >= a.N) continue;
      if constexpr (KIND == EPI_GELU) {
        *(u32x4*)((bf16*)a.out + (size_t)m * a.ldo + n) = val[u];
      } else {
        const int part = (int)fdiv((uint32_t)n, a.div_D);
        const int rem = n - part * a.D;
        const int head = (int)fdiv((uint32_t)rem, a.div_dh);
        const int d = rem - head * a.dh;
        const int r0 = (int)fdiv((uint32_t)m, a.div_ntok);
        const int tok = m - r0 * a.ntok;
        int which, r;
        qkv_dest<KIND>(a, part, r0, which, r);
        bf16* base = (bf16*)(which == 0 ? a.q : a.k);
        if (which < 2) *(u32x4*)(base + (((size_t)r * a.heads + head) * a.ntok + tok) * a.dh + d) = val[u];
      }
    }
  }
  if constexpr (KIND == EPI_QKV || KIND == EPI_KVX) {
    // transposed v, skipped unless the tile reaches the v columns. Plain layout: item =
    // (column, 8 consecutive rows), one 16-byte store. Items that end a network row early
    // or start unaligned go element-wise.
    if (KIND == EPI_QKV && a.which_base + (int)fdiv((uint32_t)min(n0 + BN, a.N) - 1, a.div_D) < 2) return;
    auto v_items = [&]() {
      constexpr int RG = 8;
      constexpr int VT = BM / RG * BN;
      constexpr int VIT = (VT + NT - 1) / NT;
      for (int it = 0; it < VIT; ++it) {
        const int c = tid + it * NT;
        const int rb = c / BN, col = c - rb * BN;  // adjacent lanes: adjacent columns
        const int n = n0 + col, m = m0 + rb * RG;
        if ((VT % NT != 0 && c >= VT) || n >= a.N || m >= a.M) continue;
        const int part = (int)fdiv((uint32_t)n, a.div_D);
        const int rem = n - part * a.D;
        const int head = (int)fdiv((uint32_t)rem, a.div_dh);
        const int d = rem - head * a.dh;
        const int r0 = (int)fdiv((uint32_t)m, a.div_ntok);
        const int tok = m - r0 * a.ntok;
        int which, r;
        qkv_dest<KIND>(a, part, r0, which, r);
        if (which < 2) continue;
        const bf16* cp = Cs + (rb * RG) * CPB + col;
        bf16* vt = (bf16*)a.vT + (((size_t)r * a.heads + head) * a.dh + d) * a.ldv;
        if (tok + RG <= a.ntok && m + RG <= a.M && (tok & (RG - 1)) == 0) {
          bf16x8 o;
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = cp[e * CPB];
          *(bf16x8*)(vt + tok) = o;
        } else {
          for (int e = 0; e < RG && m + e < a.M; ++e) {
            const int me = m + e;
            const int re0 = (int)fdiv((uint32_t)me, a.div_ntok);
            const int te = me - re0 * a.ntok;
            int we, re;
            qkv_dest<KIND>(a, part, re0, we, re);
            ((bf16*)a.vT)[(((size_t)re * a.heads + head) * a.dh + d) * a.ldv + te] =
                cp[e * CPB];
          }
        }
      }
    };
    // permuted layout: item = (8 adjacent columns, 16 consecutive rows). The 16 rows come
    // from LDS as one 16-byte read each and are transposed in registers (two bf16 per
    // v_perm); each column leaves as two 16-byte stores in the permuted key order.
    auto v_items_perm = [&]() {
      constexpr int CG = BN / 8;
      constexpr int VT = BM / 16 * CG;
      constexpr int VIT = (VT + NT - 1) / NT;
      for (int it = 0; it < VIT; ++it) {
        const int c = tid + it * NT;
        const int rb = c / CG, cg = c - rb * CG;  // adjacent lanes: adjacent column groups
        const int n = n0 + cg * 8, m = m0 + rb * 16;
        if ((VT % NT != 0 && c >= VT) || n >= a.N || m >= a.M) continue;
        const int part = (int)fdiv((uint32_t)n, a.div_D);
        const int rem = n - part * a.D;
        const int head = (int)fdiv((uint32_t)rem, a.div_dh);
        const int d0 = rem - head * a.dh;  // the 8 columns are dims d0.. of one head (dh % 8 == 0)
        const int r0 = (int)fdiv((uint32_t)m, a.div_ntok);
        const int tok = m - r0 * a.ntok;
        int which, r;
        qkv_dest<KIND>(a, part, r0, which, r);
        if (which < 2) continue;
        if (tok + 16 <= a.ntok && m + 16 <= a.M && (tok & 15) == 0 && n + 8 <= a.N) {
          u32x4 rows[16];
#pragma unroll
          for (int e = 0; e < 16; ++e) rows[e] = *(const u32x4*)&Cs[(rb * 16 + e) * CPB + cg * 8];
          bf16* vt = (bf16*)a.vT + (((size_t)r * a.heads + head) * a.dh + d0) * a.ldv + tok;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            // column j: bf16 j of every row; a word packs tokens (t0, t1) low to high
            const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
            auto pk = [&](int t0, int t1) { return __builtin_amdgcn_perm(rows[t1][j >> 1], rows[t0][j >> 1], sel); };
            // key columns tok..tok+7 hold keys 0-3, 8-11; tok+8..tok+15 keys 4-7, 12-15
            *(u32x4*)(vt + (size_t)j * a.ldv) = u32x4{pk(0, 1), pk(2, 3), pk(8, 9), pk(10, 11)};
            *(u32x4*)(vt + (size_t)j * a.ldv + 8) = u32x4{pk(4, 5), pk(6, 7), pk(12, 13), pk(14, 15)};
          }
        } else {
          for (int e = 0; e < 16 && m + e < a.M; ++e) {
            const int me = m + e;
            const int re0 = (int)fdiv((uint32_t)me, a.div_ntok);
            const int te = me - re0 * a.ntok;
            int we, re;
            qkv_dest<KIND>(a, part, re0, we, re);
            for (int j = 0; j < 8 && n + j < a.N; ++j)
              ((bf16*)a.vT)[(((size_t)re * a.heads + head) * a.dh + d0 + j) * a.ldv + vt_pos(te)] =
                  Cs[(rb * 16 + e) * CPB + cg * 8 + j];
          }
        }
      }
    };
    if (a.vperm)
      v_items_perm();
    else
      v_items();
  }
}

// Block -> tile map. The hardware hands workgroup b to XCD b % 8 and each XCD has its
// own L2, so each XCD gets a contiguous range of logical tiles; inside it tiles go in
// groups of GM tile rows, M fastest, so the A rows and B columns a group touches are
// reused from one L2. Bijective for any tile count and group size. The QKV projection
// takes groups of four where that measured faster (at 4096 x 2304 each XCD then owns
// four whole A row panels and every column tile; also at 16384 rows), but not for 4096
// rows of 128 x 128 tiles over 27 column tiles (width 1152), where eight are faster. The
// MLP up-projection, and the directly staged narrow GEMMs other than the MLP
// down-projection, take four on grids of at least 64 tile rows; everything else eight.
constexpr int kXcds = 8;
constexpr int kGroupM = 8;
__device__ __forceinline__ void tile_coords(int nbm, int nbn, int& mt, int& nt, int GM = kGroupM) {
  const int T = nbm * nbn;
  const int b = blockIdx.x;
  const int xcd = b % kXcds, local = b / kXcds;
  const int base = T / kXcds, rem = T % kXcds;
  const int logical = xcd * base + min(xcd, rem) + local;
  const int per_group = GM * nbn;
  const int group = logical / per_group;
  const int first_m = group * GM;
  const int gsize = min(GM, nbm - first_m);
  const int in = logical - group * per_group;
  mt = first_m + in % gsize;
  nt = in / gsize;
}

// The bf16 GEMM with an explicitly interleaved main loop. Operand tiles come in through
// raw buffer loads (rows past M or N and columns past K get an out-of-range offset and
// read as zeros, so the loads carry no branches). Each K step is one straight
// block: the matrix-core instructions of tile k are interleaved (sched_group_barrier)
// with the LDS fragment reads of tile k, the LDS writes of tile k+1 (already in
// registers) and the buffer loads of tile k+2, so memory work issues under the MFMAs
// instead of in stalls between them. Loader chunks past the tile (when the chunk count
// is not a multiple of the thread count) read zeros and land in a spare LDS slot, so
// the block stays branch-free.
template <int BM, int BN, int BK, int WM, int WN, int KSPLIT, EpiKind KIND>
__global__ __launch_bounds__(WM * WN * KSPLIT * 64) void gemm_bf16_sched_kernel(GemmArgs a) {
  constexpr int NT = WM * WN * KSPLIT * 64;
  constexpr int LDK = BK + 8;  // LDS row pitch in bf16 (a 16-byte pad)
  constexpr int TM = BM / WM / 32;
  constexpr int TN = BN / WN / 32;
  static_assert(TM * WM * 32 == BM && TN * WN * 32 == BN, "wave grid must tile the block");
  constexpr int CPR = BK / 8;
  constexpr int ATOT = BM * CPR, BTOT = BN * CPR;
  constexpr int ACH = (ATOT + NT - 1) / NT;
  constexpr int BCH = (BTOT + NT - 1) / NT;
  constexpr int AB_BYTES = 2 * (BM + BN) * LDK * 2 + 16;  // + spare slot
  constexpr int CP = BN + 4;
  constexpr int LDS_CAP = 160 * 1024;
  constexpr int NP = (BM * CP * 4 <= LDS_CAP) ? 1 : ((BM / 2) * CP * 4 <= LDS_CAP ? 2 : 4);
  constexpr int RP = BM / NP;
  constexpr int C_BYTES = RP * CP * 4;
  constexpr int SMEM = AB_BYTES > C_BYTES ? AB_BYTES : C_BYTES;
  static_assert(SMEM <= LDS_CAP, "tile does not fit in LDS");
  static_assert(BM * (BN + kEpiPad) * 2 <= SMEM, "staged bf16 tile does not fit in LDS");
  constexpr int KS = BK / 16 / KSPLIT;        // MFMA K steps per tile and wavefront
  static_assert(KS * 16 * KSPLIT == BK, "K split must divide the K slice");
  static_assert(KSPLIT == 1 || BM * CP * 4 <= AB_BYTES, "K-split partials must fit in LDS");
  constexpr int NMFMA = TM * TN * KS;
  constexpr int NDSR = (TM + TN) * KS;
  constexpr int NDSW = ACH + BCH;
  constexpr int NVMEM = ACH + BCH;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  bf16* As = (bf16*)smem;
  bf16* Bs = As + 2 * BM * LDK;
  constexpr int SPARE = 2 * (BM + BN) * LDK;  // bf16 index of the spare slot

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // wavefront (kg, wm, wn): sub-tile (wm, wn) over K quarter-slices kg*KS .. kg*KS+KS-1
  // of every 64-wide K slice
  const int kg = wave / (WM * WN), wmn = wave - kg * (WM * WN);
  const int wm = wmn / WN, wn = wmn % WN;
  const int l32 = lane & 31, g = lane >> 5;
  int mt, nt;
  {
    const int nbm = (a.M + BM - 1) / BM, nbn = (a.N + BN - 1) / BN;
    tile_coords(nbm, nbn, mt, nt,
                (KIND == EPI_QKV && (nbm >= 64 || nbn <= 8)) || (KIND == EPI_GELU && nbm >= 64) ? 4 : kGroupM);
  }
  const int m0 = mt * BM, n0 = nt * BN;
  if (!tile_live<KIND, BM>(a, m0)) return;  // uniform across the workgroup
  // the tile's bias columns go to LDS now, so the epilogue does not wait on them
  constexpr bool kBf16Out = KIND == EPI_GELU || KIND == EPI_QKV || KIND == EPI_KVX;
  __shared__ __attribute__((aligned(16))) float bias_s[kBf16Out ? BN : 4];
  if constexpr (kBf16Out) {
    for (int c = tid; c < BN / 4; c += NT) {
      const int n = n0 + 4 * c;
      *(f32x4*)&bias_s[4 * c] = n < a.N ? *(const f32x4*)(a.bias + n) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }

  const __amdgpu_buffer_rsrc_t ra_src = buffer_rsrc(a.A, (uint32_t)a.M * a.lda * 2);
  const __amdgpu_buffer_rsrc_t rb_src = buffer_rsrc(a.B, (uint32_t)a.N * a.ldb * 2);
  // per chunk: global byte offset at k = 0 (or out of range), K column, and LDS index
  // relative to the buffer base (the spare slot minus the buffer base for chunks past
  // the tile, so `buffer base + index` always lands in the spare slot)
  int a_off[ACH], b_off[BCH], a_kc[ACH], b_kc[BCH], a_lds[ACH], b_lds[BCH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    const int c = tid + i * NT, row = c / CPR;
    const bool in = c < ATOT;
    a_kc[i] = (c % CPR) * 8;
    a_lds[i] = in ? row * LDK + a_kc[i] : -1;
    a_off[i] = (in && m0 + row < a.M) ? ((m0 + row) * a.lda + a_kc[i]) * 2 : kOffOOB;
  }
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int c = tid + i * NT, row = c / CPR;
    const bool in = c < BTOT;
    b_kc[i] = (c % CPR) * 8;
    b_lds[i] = in ? row * LDK + b_kc[i] : -1;
    b_off[i] = (in && n0 + row < a.N) ? ((n0 + row) * a.ldb + b_kc[i]) * 2 : kOffOOB;
  }
  u32x4 ra[ACH], rb[BCH];
  // FAST (K a multiple of BK): every slice lies wholly inside K or wholly past it, so
  // the loads go through resources based at the slice's first column and each thread's
  // offsets are the fixed ones of k = 0 (rows past M keep the out-of-range offset); a
  // slice past K gets empty resources and reads zeros. The main loop is compiled once
  // per form and chosen by K, so neither carries a per-slice branch.
  auto gload = [&](auto fastc, int kt) {
    const int k0 = kt * BK;
    if constexpr (decltype(fastc)::value) {
      const bool live = k0 < a.K;
      const __amdgpu_buffer_rsrc_t ra1 =
          buffer_rsrc((const char*)a.A + 2 * (size_t)k0, live ? (uint32_t)a.M * a.lda * 2 - 2 * k0 : 0u);
      const __amdgpu_buffer_rsrc_t rb1 =
          buffer_rsrc((const char*)a.B + 2 * (size_t)k0, live ? (uint32_t)a.N * a.ldb * 2 - 2 * k0 : 0u);
#pragma unroll
      for (int i = 0; i < ACH; ++i) ra[i] = buffer_load16(ra1, a_off[i]);
#pragma unroll
      for (int i = 0; i < BCH; ++i) rb[i] = buffer_load16(rb1, b_off[i]);
      return;
    }
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
      const int idx = (ATOT % NT == 0 || a_lds[i] >= 0) ? buf * BM * LDK + a_lds[i] : SPARE;
      *(u32x4*)&As[idx] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int idx = (BTOT % NT == 0 || b_lds[i] >= 0) ? buf * BN * LDK + b_lds[i] : SPARE - 2 * BM * LDK;
      *(u32x4*)&Bs[idx] = rb[i];
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  auto step = [&](auto fastc, int cur, int kt, bool write_next, bool load_next) {
    const bf16* Ab = As + cur * BM * LDK + (wm * TM * 32 + l32) * LDK + g * 8 + kg * KS * 16;
    const bf16* Bb = Bs + cur * BN * LDK + (wn * TN * 32 + l32) * LDK + g * 8 + kg * KS * 16;
    bf16x8 af[2][TM], bfr[2][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) af[0][i] = *(const bf16x8*)(Ab + i * 32 * LDK);
#pragma unroll
    for (int j = 0; j < TN; ++j) bfr[0][j] = *(const bf16x8*)(Bb + j * 32 * LDK);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int cb = kk & 1;
      if (kk + 1 < KS) {
#pragma unroll
        for (int i = 0; i < TM; ++i) af[cb ^ 1][i] = *(const bf16x8*)(Ab + i * 32 * LDK + (kk + 1) * 16);
#pragma unroll
        for (int j = 0; j < TN; ++j) bfr[cb ^ 1][j] = *(const bf16x8*)(Bb + j * 32 * LDK + (kk + 1) * 16);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[cb][j], af[cb][i], acc[i][j], 0, 0, 0);
    }
    if (write_next) lstore(cur ^ 1);
    if (load_next) gload(fastc, kt + 2);
    // interleave: the fragment reads ahead of their MFMAs over the first half of the
    // MFMAs, the LDS writes and global loads over the second half
    constexpr int H1 = NMFMA / 2, H2 = NMFMA - NMFMA / 2;
#pragma unroll
    for (int i = 0; i < H1; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x100, (NDSR + H1 - 1) / H1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
#pragma unroll
    for (int i = 0; i < H2; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x200, (NDSW + H2 - 1) / H2, 0);
      __builtin_amdgcn_sched_group_barrier(0x020, (NVMEM + H2 - 1) / H2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
  };

  const int nk = (a.K + BK - 1) / BK;
  auto main_loop = [&](auto fastc) {
    gload(fastc, 0);
    lstore(0);
    if (nk > 1) gload(fastc, 1);
    __syncthreads();
    int kt = 0;
    for (; kt + 2 < nk; ++kt) {
      step(fastc, kt & 1, kt, true, true);
      __syncthreads();
    }
    if (kt + 1 < nk) {
      step(fastc, kt & 1, kt, true, false);
      __syncthreads();
      ++kt;
    }
    step(fastc, kt & 1, kt, false, false);
    __syncthreads();
  };
  if (a.K % BK == 0)
    main_loop(std::true_type{});
  else
    main_loop(std::false_type{});

  // The MFMAs compute C^T blocks (weights as the first operand), so in acc[i][j]
  // lane (l32, g) holds row (wm*TM + i)*32 + l32 of the tile and, in registers
  // 4q..4q+3, the four adjacent columns (wn*TN + j)*32 + 8q + 4g + 0..3.
  if constexpr (KSPLIT == 2) {
    // the second K half's partial sums go through LDS to the first half's wavefronts:
    // one fixed order (first half + second half) for every element
    float* P = (float*)smem;
    if (kg == 1) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
            *(f32x4*)&P[((wm * TM + i) * 32 + l32) * CP + (wn * TN + j) * 32 + q * 8 + g * 4] = v;
          }
    }
    __syncthreads();
    if (kg == 0) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 v = *(const f32x4*)&P[((wm * TM + i) * 32 + l32) * CP + (wn * TN + j) * 32 + q * 8 + g * 4];
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[i][j][4 * q + e] += v[e];
          }
    }
    __syncthreads();
  }
  if constexpr (kBf16Out) {
    bf16_epilogue<KIND, BM, BN, TM, TN, NT>(a, acc, (bf16*)smem, bias_s, m0, n0, wm, wn, l32, g, kg == 0, tid);
  } else {
    float* Cs = (float*)smem;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int rb0 = (wm * TM + i) * 32;
        if (kg != 0 || rb0 < p * RP || rb0 >= (p + 1) * RP) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
            *(f32x4*)&Cs[(rb0 - p * RP + l32) * CP + (wn * TN + j) * 32 + q * 8 + g * 4] = v;
          }
      }
      __syncthreads();
      staged_epilogue<KIND, RP, BN, NT>(a, Cs, CP, m0 + p * RP, n0, tid);
      if (p + 1 < NP) __syncthreads();
    }
  }
}

// ------------------------------------------------- bf16 / MFMA, direct LDS staging
//
// The same tile computation with operand slices moved by buffer_load ... lds straight
// from global memory into a ring of STAGES LDS buffers (no VGPR round trip, no LDS
// write instructions), fetched STAGES - 1 slices ahead.
//
// Each stage is its own __shared__ variable and the main loop is unrolled by STAGES, so
// every LDS access names one variable: the compiler then tells the in-flight loads into
// other stages apart from the stage being read and waits only for the right ones.
// The loop's barrier is a bare s_barrier (ordered by compiler-only fences) after an
// explicit wait for this slice's loads: the workgroup-scope release fence of
// __syncthreads would wait for every outstanding LDS-bound load, i.e. for all stages.
//
// Stage layout: rows of BK bf16 without padding, 16-byte chunks swizzled by dma_swz.

template <int BM, int BN, int BK, int WM, int WN, int KSPLIT, int STAGES, EpiKind KIND>
__global__ __launch_bounds__(WM * WN * KSPLIT * 64) void gemm_bf16_dma_kernel(GemmArgs a) {
  constexpr int NT = WM * WN * KSPLIT * 64;
  constexpr int TM = BM / WM / 32;
  constexpr int TN = BN / WN / 32;
  static_assert(TM * WM * 32 == BM && TN * WN * 32 == BN, "wave grid must tile the block");
  constexpr int CPR = BK / 8;
  constexpr int ATOT = BM * CPR, BTOT = BN * CPR;
  static_assert(ATOT % 64 == 0 && BTOT % 64 == 0, "whole wavefronts of 16-byte chunks per slice");
  constexpr int ACH = (ATOT + NT - 1) / NT, BCH = (BTOT + NT - 1) / NT, LPT = ACH + BCH;
  constexpr int KS = BK / 16 / KSPLIT;  // MFMA K steps per slice and wavefront
  static_assert(KS * 16 * KSPLIT == BK, "K split must divide the K slice");
  static_assert(STAGES == 3 || STAGES == 4, "three or four stages");
  constexpr bool kBf16Out = KIND == EPI_GELU || KIND == EPI_QKV || KIND == EPI_KVX;
  // each stage buffer also holds, after the main loop, one row block of the K-split
  // partial sums, one half of the fp32 output tile, or the whole bf16 output tile
  constexpr int CP = BN + 4;
  constexpr int RP = BM / 2;
  constexpr int SLICE = (BM + BN) * BK * 2;
  // K-split partials: MFMA block b = i * TN + j of every first-set wavefront (4 KB each)
  // goes to stage b % STAGES at block slot b / STAGES
  constexpr int PBLK = WM * WN * 16 * 64 * 4;
  constexpr int PART = KSPLIT == 2 ? (TM * TN + STAGES - 1) / STAGES * PBLK : 0;
  constexpr int EPI = kBf16Out ? BM * (BN + kEpiPad) * 2 : RP * CP * 4;
  constexpr int SBA = SLICE > PART ? (SLICE > EPI ? SLICE : EPI) : (PART > EPI ? PART : EPI);
  static_assert(KSPLIT == 1 || KSPLIT == 2, "K split of one or two");
  static_assert(STAGES * SBA + (kBf16Out ? BN * 4 : 16) <= 160 * 1024, "stages do not fit in LDS");
  constexpr int NMFMA = TM * TN * KS;
  constexpr int NDSR = (TM + TN) * KS;
  __shared__ __attribute__((aligned(16))) char st0[SBA];
  __shared__ __attribute__((aligned(16))) char st1[SBA];
  __shared__ __attribute__((aligned(16))) char st2[SBA];
  __shared__ __attribute__((aligned(16))) char st3[STAGES > 3 ? SBA : 16];
  // destination of the loads of wavefronts whose chunk round lies past the tile (they
  // read zeros; nothing reads this back)
  constexpr bool kSpare = ATOT % NT != 0 || BTOT % NT != 0;
  __shared__ __attribute__((aligned(16))) char spare[kSpare ? 1024 : 16];
  auto stage = [&](auto s) -> char* {
    constexpr int S = decltype(s)::value % STAGES;
    if constexpr (S == 0) return st0;
    else if constexpr (S == 1) return st1;
    else if constexpr (S == 2) return st2;
    else return st3;
  };

  const int tid = threadIdx.x;
  // the wavefront index is uniform: kept scalar, so the LDS destinations of the direct
  // loads (M0) need no readfirstlane
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = wave / (WM * WN), wmn = wave - kg * (WM * WN);
  const int wm = wmn / WN, wn = wmn % WN;
  const int l32 = lane & 31, g = lane >> 5;
  int mt, nt;
  {
    const int nbm = (a.M + BM - 1) / BM, nbn = (a.N + BN - 1) / BN;
    tile_coords(nbm, nbn, mt, nt, nbm >= 64 && KIND != EPI_RES_GATE_MLP ? 4 : kGroupM);
  }
  const int m0 = mt * BM, n0 = nt * BN;
  if (!tile_live<KIND, BM>(a, m0)) return;  // uniform across the workgroup
  __shared__ __attribute__((aligned(16))) float bias_s[kBf16Out ? BN : 4];
  if constexpr (kBf16Out) {
    for (int c = tid; c < BN / 4; c += NT) {
      const int n = n0 + 4 * c;
      *(f32x4*)&bias_s[4 * c] = n < a.N ? *(const f32x4*)(a.bias + n) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }

  const __amdgpu_buffer_rsrc_t ra_src = buffer_rsrc(a.A, (uint32_t)a.M * a.lda * 2);
  const __amdgpu_buffer_rsrc_t rb_src = buffer_rsrc(a.B, (uint32_t)a.N * a.ldb * 2);
  // load i of a thread fills LDS chunk position i * NT + tid of the A (or B) part of a
  // stage, i.e. tile row p / CPR at chunk position p % CPR, which holds K chunk
  // (p % CPR) ^ swz(row); per load: that K column and the byte offset at k = 0
  int a_off[ACH], b_off[BCH], a_kc[ACH], b_kc[BCH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    const int p = tid + i * NT, row = p / CPR;
    a_kc[i] = ((p % CPR) ^ dma_swz<CPR>(row)) * 8;
    a_off[i] = p < ATOT && m0 + row < a.M ? ((m0 + row) * a.lda + a_kc[i]) * 2 : kOffOOB;
  }
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int p = tid + i * NT, row = p / CPR;
    b_kc[i] = ((p % CPR) ^ dma_swz<CPR>(row)) * 8;
    b_off[i] = p < BTOT && n0 + row < a.N ? ((n0 + row) * a.ldb + b_kc[i]) * 2 : kOffOOB;
  }
  // slice kt into stage buffer sb: every thread issues exactly LPT loads (past the end
  // of K they read zeros), each wavefront's 64 lanes filling one contiguous kilobyte
  // FAST (K a multiple of BK): every slice lies wholly inside K or wholly past it, so
  // the loads go through resources based at the slice's first column and each thread's
  // offsets are the fixed ones of k = 0 (rows past M keep the out-of-range offset); a
  // slice past K gets empty resources and reads zeros without touching memory
  auto issue = [&](auto fast, char* sb, int kt) {
    const int k0 = kt * BK;
    if constexpr (decltype(fast)::value) {
      const bool live = k0 < a.K;
      const __amdgpu_buffer_rsrc_t ra =
          buffer_rsrc((const char*)a.A + 2 * (size_t)k0, live ? (uint32_t)a.M * a.lda * 2 - 2 * k0 : 0u);
      const __amdgpu_buffer_rsrc_t rb =
          buffer_rsrc((const char*)a.B + 2 * (size_t)k0, live ? (uint32_t)a.N * a.ldb * 2 - 2 * k0 : 0u);
#pragma unroll
      for (int i = 0; i < ACH; ++i) {
        const bool in = ATOT % NT == 0 || i * NT + wave * 64 < ATOT;
        buffer_load16_lds(ra, in ? sb + (i * NT + wave * 64) * 16 : spare, a_off[i]);
      }
#pragma unroll
      for (int i = 0; i < BCH; ++i) {
        const bool in = BTOT % NT == 0 || i * NT + wave * 64 < BTOT;
        buffer_load16_lds(rb, in ? sb + ATOT * 16 + (i * NT + wave * 64) * 16 : spare, b_off[i]);
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const bool in = ATOT % NT == 0 || i * NT + wave * 64 < ATOT;
      buffer_load16_lds(ra_src, in ? sb + (i * NT + wave * 64) * 16 : spare,
                        (k0 + a_kc[i] < a.K && a_off[i] != kOffOOB) ? a_off[i] + 2 * k0 : kOffOOB);
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const bool in = BTOT % NT == 0 || i * NT + wave * 64 < BTOT;
      buffer_load16_lds(rb_src, in ? sb + ATOT * 16 + (i * NT + wave * 64) * 16 : spare,
                        (k0 + b_kc[i] < a.K && b_off[i] != kOffOOB) ? b_off[i] + 2 * k0 : kOffOOB);
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // this lane's rows all have the swizzle of row l32 (row blocks are 32 apart); its
  // fragment of MFMA K step kk is K chunk c0 + 2 kk
  const int sw = dma_swz<CPR>(l32);
  const int c0 = 2 * kg * KS + g;
  const int a_row = (wm * TM * 32 + l32) * CPR;
  const int b_row = ATOT + (wn * TN * 32 + l32) * CPR;
  // one K slice: wait for this slice's loads (the later slices' STAGES - 2 stay in
  // flight) and for this thread's LDS accesses, barrier, then the MFMAs on stage S
  // interleaved with the fragment reads and with the loads of slice kt + STAGES - 1
  // into the stage read in the previous step
  constexpr int kWait = waitcnt_vm_lgkm0<(STAGES - 2) * LPT>();
  auto step = [&](auto fast, auto s, int kt) {
    constexpr int S = decltype(s)::value;
    __builtin_amdgcn_s_waitcnt(kWait);
    bare_barrier();
    const char* cur = stage(std::integral_constant<int, S>{});
    bf16x8 af[2][TM], bfr[2][TN];
    auto frag = [&](int row_base, int blk, int kk) {
      return *(const bf16x8*)(cur + (row_base + blk * 32 * CPR + ((c0 + 2 * kk) ^ sw)) * 16);
    };
#pragma unroll
    for (int i = 0; i < TM; ++i) af[0][i] = frag(a_row, i, 0);
#pragma unroll
    for (int j = 0; j < TN; ++j) bfr[0][j] = frag(b_row, j, 0);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int cb = kk & 1;
      if (kk + 1 < KS) {
#pragma unroll
        for (int i = 0; i < TM; ++i) af[cb ^ 1][i] = frag(a_row, i, kk + 1);
#pragma unroll
        for (int j = 0; j < TN; ++j) bfr[cb ^ 1][j] = frag(b_row, j, kk + 1);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[cb][j], af[cb][i], acc[i][j], 0, 0, 0);
    }
    issue(fast, stage(std::integral_constant<int, S + STAGES - 1>{}), kt + STAGES - 1);
    constexpr int H1 = NMFMA / 2, H2 = NMFMA - NMFMA / 2;
#pragma unroll
    for (int i = 0; i < H1; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x100, (NDSR + H1 - 1) / H1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
#pragma unroll
    for (int i = 0; i < H2; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x020, (LPT + H2 - 1) / H2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
  };

  const int nk = (a.K + BK - 1) / BK;
  auto main_loop = [&](auto fast) {
    issue(fast, stage(std::integral_constant<int, 0>{}), 0);
    issue(fast, stage(std::integral_constant<int, 1>{}), 1);
    if constexpr (STAGES > 3) issue(fast, stage(std::integral_constant<int, 2>{}), 2);
    // whole rounds of STAGES steps in a loop with one exit (early exits inside the round
    // would give the loop header a path on which the stage it reads was just issued),
    // then the remaining steps
    int kt = 0;
    for (; kt + STAGES <= nk; kt += STAGES) {
      step(fast, std::integral_constant<int, 0>{}, kt);
      step(fast, std::integral_constant<int, 1>{}, kt + 1);
      step(fast, std::integral_constant<int, 2>{}, kt + 2);
      if constexpr (STAGES > 3) step(fast, std::integral_constant<int, 3>{}, kt + 3);
    }
    if (kt < nk) step(fast, std::integral_constant<int, 0>{}, kt);
    if (kt + 1 < nk) step(fast, std::integral_constant<int, 1>{}, kt + 1);
    if constexpr (STAGES > 3)
      if (kt + 2 < nk) step(fast, std::integral_constant<int, 2>{}, kt + 2);
  };
  if (a.K % BK == 0)
    main_loop(std::true_type{});
  else
    main_loop(std::false_type{});
  // the zero-filling loads past K land before the buffers are reused
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // the residual epilogues' global operands (bias, gate row, residual) for both row
  // halves are loaded now: their latency passes under the K-split merge and the staging
  ResItems<KIND, RP, BN, NT> pre[2];
  if constexpr (!kBf16Out) {
    pre[0].load(a, m0, n0, tid);
    pre[1].load(a, m0 + RP, n0, tid);
  }

  if constexpr (KSPLIT == 2) {
    // the second K half's partial sums go through LDS (lane-major, so each lane reads
    // back exactly what its partner wrote) to the first half's wavefronts: one fixed
    // order (first half + second half) for every element
    auto part = [&](int i, int j, int q) -> f32x4* {
      const int b = i * TN + j;
      const int st = b % STAGES;
      char* base = st == 0 ? st0 : st == 1 ? st1 : st == 2 ? st2 : st3;
      return (f32x4*)(base + (b / STAGES) * PBLK) + (wmn * 4 + q) * 64 + lane;
    };
    if (kg == 1) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *part(i, j, q) = f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
    }
    __syncthreads();
    if (kg == 0) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 v = *part(i, j, q);
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[i][j][4 * q + e] += v[e];
          }
    }
    __syncthreads();
  }
  if constexpr (kBf16Out) {
    bf16_epilogue<KIND, BM, BN, TM, TN, NT>(a, acc, (bf16*)st0, bias_s, m0, n0, wm, wn, l32, g, kg == 0, tid);
  } else {
    // the two row halves of the tile staged in stages 0 and 1 under one barrier
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      float* Cs = (float*)(p == 0 ? st0 : st1);
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int rb0 = (wm * TM + i) * 32;
        if (kg != 0 || rb0 < p * RP || rb0 >= (p + 1) * RP) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
            *(f32x4*)&Cs[(rb0 - p * RP + l32) * CP + (wn * TN + j) * 32 + q * 8 + g * 4] = v;
          }
      }
    }
    __syncthreads();
    pre[0].apply(a, (const float*)st0, CP, m0, n0, tid);
    pre[1].apply(a, (const float*)st1, CP, m0 + RP, n0, tid);
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
  if (!tile_live<KIND, kFT>(a, m0)) return;
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

// Tile shapes (BM x BN x BK, wave grid WM x WN, K split). Per-wave tiles are 64x64,
// 64x96 or 32x96; with a K split of 2 a second set of wavefronts takes the second half
// of every K slice of the same tile. A CU spreads a workgroup's wavefronts round-robin
// over its four SIMDs, so a wavefront count that is a multiple of four keeps them evenly
// loaded (six wavefronts put two on two SIMDs and one on the others).
#define SF_GEMM_TILES(X)          \
  X(0, 128, 128, 64, 2, 2, 1)     \
  X(1, 128, 288, 64, 4, 3, 1)     \
  X(2, 128, 384, 64, 2, 4, 1)     \
  X(3, 256, 192, 64, 4, 2, 1)     \
  X(6, 128, 128, 128, 2, 2, 2)

// Directly staged tiles (as above, plus the number of LDS stages).
#define SF_GEMM_DMA_TILES(X)           \
  X(7, 128, 96, 64, 4, 1, 2, 4)

template <EpiKind KIND>
static hipError_t launch_bf16_tile(int tile, const GemmArgs& a, hipStream_t s) {
  switch (tile) {
#define SF_TILE_CASE(id, bm, bn, bk, wm, wn, ks)                                                   \
  case id:                                                                                         \
    launch((gemm_bf16_sched_kernel<bm, bn, bk, wm, wn, ks, KIND>),                                 \
           dim3(((a.N + bn - 1) / bn) * ((a.M + bm - 1) / bm)), dim3(wm * wn * ks * 64), 0, s, a); \
    break;
    SF_GEMM_TILES(SF_TILE_CASE)
#undef SF_TILE_CASE
#define SF_DMA_TILE_CASE(id, bm, bn, bk, wm, wn, ks, st)                                           \
  case id:                                                                                         \
    launch((gemm_bf16_dma_kernel<bm, bn, bk, wm, wn, ks, st, KIND>),                               \
           dim3(((a.N + bn - 1) / bn) * ((a.M + bm - 1) / bm)), dim3(wm * wn * ks * 64), 0, s, a); \
    break;
    SF_GEMM_DMA_TILES(SF_DMA_TILE_CASE)
#undef SF_DMA_TILE_CASE
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Tiles chosen from measurements on the 512^2 and 1024^2 projection shapes. Narrow
// outputs (N <= 768, e.g. the attention output and MLP down-projections of the width-768
// network) have too few wide tiles to fill the chip, so they take the directly staged
// 128x96 tile (exactly one workgroup per CU at 4096x768) with each 64-wide K slice split
// over two sets of wavefronts (4096x768x3072: 28.2 us, against 29.5 for the
// register-staged 128x128 tile with 128-wide split slices, which remains for other
// multiples of 128 up to 768). (At N = 1152 the 128x128 tiles outnumber the CUs, and a
// split tile, one workgroup per CU, loses to the plain one, two per CU: 72 vs 67 us on
// 4096x1152x4608.) The partial sums of the two halves are added in a fixed order, and
// the choice depends on N and K only, never on M, so a row's result does not depend on
// how many rows are in the batch. Otherwise 128x128 (64x64 per wavefront) is the
// general tile; 128x384 (64x96 per wavefront, 8 wavefronts) and 128x288 (32x96 per
// wavefront, 12 wavefronts: 4096x2304 in 22.5 instead of 23.6 us with 6 wavefronts of
// 64x96) win when they cut the problem into exactly one workgroup per CU (e.g.
// 4096x3072 and 4096x2304), and 256x192 (64x96 per wavefront, 8 wavefronts; 12 % fewer
// operand bytes per CU than 128x384) beats 128x384 where it does so too (4096x3072:
// 25.3 against 26.0 us per launch in the 512^2 step); these accumulate in the same
// order, so switching among them with M changes no result bit.
int choose_gemm_tile(int M, int N, int K) {
  (void)K;
  if (N % 96 == 0 && N <= 768) return 7;
  if (N % 128 == 0 && N <= 768) return 6;
  auto tiles = [&](int bm, int bn) { return ((M + bm - 1) / bm) * ((N + bn - 1) / bn); };
  if (M % 256 == 0 && N % 192 == 0 && tiles(256, 192) == 256) return 3;
  if (M % 128 == 0 && N % 384 == 0 && tiles(128, 384) == 256) return 2;
  if (M % 128 == 0 && N % 288 == 0 && tiles(128, 288) == 256) return 1;
  return 0;
}

template <EpiKind KIND>
static hipError_t launch_kind(bool use_bf16, int tile, const GemmArgs& a, hipStream_t s) {
  if (use_bf16) return launch_bf16_tile<KIND>(tile < 0 ? choose_gemm_tile(a.M, a.N, a.K) : tile, a, s);
  dim3 grid((a.N + kFT - 1) / kFT, (a.M + kFT - 1) / kFT);
  launch(gemm_f32_kernel<KIND>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gemm_tile(bool use_bf16, int tile, EpiKind kind, const GemmArgs& a, hipStream_t s) {
  switch (kind) {
    case EPI_QKV: return launch_kind<EPI_QKV>(use_bf16, tile, a, s);
    case EPI_RES_GATE: return launch_kind<EPI_RES_GATE>(use_bf16, tile, a, s);
    case EPI_GELU: return launch_kind<EPI_GELU>(use_bf16, tile, a, s);
    case EPI_RES: return launch_kind<EPI_RES>(use_bf16, tile, a, s);
    case EPI_RES_GATE_MLP: return launch_kind<EPI_RES_GATE_MLP>(use_bf16, tile, a, s);
    case EPI_KVX: return launch_kind<EPI_KVX>(use_bf16, tile, a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm(bool use_bf16, EpiKind kind, const GemmArgs& a, hipStream_t s) {
  return launch_gemm_tile(use_bf16, -1, kind, a, s);
}

}  // namespace sf
