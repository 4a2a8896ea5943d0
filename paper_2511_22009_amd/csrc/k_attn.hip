// K4: softmax attention softmax(q k^T / sqrt(dh)) v for every (network row, head), no
// mask; each row attends only to its own tokens, so samples never mix.
//
// bf16 path (v_mfma_f32_32x32x16_bf16), online softmax:
//   * a workgroup owns 64 queries of one (row, head) and four wavefronts: two query
//     groups of 32 times two key halves. Each step stages 64 keys; the first 32 go to
//     the key-half-0 wavefronts, the next 32 to key-half-1, and the two halves' partial
//     results (offset, sum, output) are merged at the end. Splitting the keys
//     inside the workgroup gives 4 wavefronts per 64 queries, so a 512^2 layer (49152
//     queries) is 768 workgroups, three per CU on 256 CUs;
//   * scores are computed transposed, S^T = K Q^T, so the MFMA result gives each lane
//     ONE query (column l%32) and 16 of the 32 keys of the block: a step max and the
//     sum are lane-local plus a single cross-half exchange;
//   * q is scaled into exp2 units (times scale * log2 e, rounded to bf16) once per
//     wavefront, and the probabilities 2^(s - m2) are formed against a per-query offset
//     m2 that starts at 0: while it is 0 for the whole wavefront, a probability is one
//     exp2 of the score. The offset only moves when the scores would leave the range
//     where probabilities, sums and outputs keep their precision (softmax_step_lazy,
//     and at head dim 64, where the row sum is kept by vector adds, softmax_step_sum);
//   * the probabilities are rounded to bf16 and used directly as the B operand of
//     O^T = V^T P^T: the MFMA's k-slot order is a permutation of the key order, and V^T
//     is stored in that permuted key order (vt_pos, written so by the QKV projection),
//     so a fragment is one 16-byte LDS read;
//   * K and V^T tiles are double-buffered in LDS and fetched one step ahead through
//     registers with raw buffer loads (keys past the end read as zeros, no branches);
//     rows past dh and keys past Nk are zero, so padding adds nothing.
// fp32 path: one thread per query, keys staged in LDS (parity mode).
#include "sf_device.h"

namespace sf {

constexpr int kKH = 32;    // keys per half per step
constexpr int kQB = 64;    // queries per workgroup
constexpr float kOffSlack = 64.0f;  // scores (exp2 units) may pass the offset by this much

// q fragments scaled into exp2 units: bf16(q * scale * log2 e), once per wavefront, so
// the score MFMA returns the exponents the softmax takes.
__device__ __forceinline__ void scale_q(bf16x8& q, float sl2) {
#pragma unroll
  for (int e = 0; e < 8; ++e) q[e] = (bf16)((float)q[e] * sl2);
}

// The probabilities of one 32-query block's step: 2^(s - m2) for the lane's 16 scores
// (SHIFT false: 2^s, for a block whose offset is 0; s - 0 is s, so both give the same
// bits), added to l (SUM) and rounded to the bf16 P.V operands pf.
template <bool SHIFT, bool SUM>
__device__ __forceinline__ void block_probs(const f32x16& s, float m2, float& l, bf16x8 (&pf)[2]) {
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float x = s[ks * 8 + j];
      const float p = __builtin_amdgcn_exp2f(SHIFT ? x - m2 : x);
      if constexpr (SUM) l += p;
      pf[ks][j] = (bf16)p;
    }
  }
}

// The probabilities of the QB query blocks of a wavefront, without the subtraction when
// every offset of the wavefront is 0 (one uniform branch for all blocks, so the blocks'
// chains stay interleaved).
template <bool SUM, int QB>
__device__ __forceinline__ void wave_probs(const f32x16 (&s)[QB], const float (&m2)[QB], float (&l)[QB],
                                           bf16x8 (&pf)[QB][2]) {
  bool zero = true;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) zero = zero && m2[qb] == 0.0f;
  if (__all(zero)) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) block_probs<false, SUM>(s[qb], m2[qb], l[qb], pf[qb]);
  } else {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) block_probs<true, SUM>(s[qb], m2[qb], l[qb], pf[qb]);
  }
}

// One step of the online softmax for QB 32-query blocks (scores s in exp2 units; a
// lane holds one query and 16 keys of each block). Each block's step max (over both
// lane halves) decides whether its offset m2 moves: up to the max when that passes the
// offset by more than kOffSlack, and, at the wavefront's first step (first: nothing
// accumulated yet), also down to it when it lies more than kOffSlack below. The
// accumulated output (and row sum, SUM) are rescaled when it moves. Then the
// probabilities 2^(s - m2) are formed, added to lsum (SUM; otherwise the ones row of
// V^T sums them in the MFMA) and rounded for P.V. Probabilities stay at most 2^64 and a
// query's largest one at least 2^-64, so everything keeps its relative precision in fp32
// and bf16; the offset is the same on both lane halves of a query at all times.
template <bool SUM, int QB, int DB>
__device__ __forceinline__ void softmax_step_lazy(const f32x16 (&s)[QB], bool first, float (&m2)[QB],
                                                  float (&lsum)[QB], f32x16 (&o)[QB][DB], bf16x8 (&pf)[QB][2]) {
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    float tmax = s[qb][0];
#pragma unroll
    for (int e = 1; e < 16; ++e) tmax = fmaxf(tmax, s[qb][e]);
    tmax = pair32_max(tmax);
    if (__any(tmax > m2[qb] + kOffSlack || (first && tmax < m2[qb] - kOffSlack))) {
      const float mnew = first ? tmax : fmaxf(m2[qb], tmax);
      const float alpha = first ? 0.0f : __builtin_amdgcn_exp2f(m2[qb] - mnew);
      if constexpr (SUM) lsum[qb] *= alpha;
#pragma unroll
      for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[qb][b][e] *= alpha;
      m2[qb] = mnew;
    }
  }
  wave_probs<SUM>(s, m2, lsum, pf);
}

// DHC = ceil(dh/16) contraction chunks, DB = ceil(dh/32) dh blocks. SUMROW (dh not a
// multiple of 32, so the last dh block has zero rows): row DB*32 - 8 of every V^T tile
// is all ones, and the P.V MFMAs then also produce each query's probability sum in that
// output row, which replaces the per-score additions of the row sum.
template <int DHC, int DB, bool SUMROW, int QB>
__global__ __launch_bounds__(256) void attn_bf16_kernel(AttnArgs a) {
  constexpr int KLD = DHC * 16 + 8;     // K tile row pitch (bf16)
  constexpr int VLD = kKH + 8;          // V^T tile row pitch (bf16)
  constexpr int VROWS = DB * 32;
  constexpr int KT = kKH * KLD;         // one half's K tile (bf16 elements)
  constexpr int VT = VROWS * VLD;       // one half's V^T tile
  constexpr int KCHMAX = 2 * kKH * DHC * 2;        // 16-byte K chunks per step (upper bound)
  constexpr int VCHMAX = VROWS * (2 * kKH / 8);    // 16-byte V^T chunks per step (upper bound)
  constexpr int KCH = (KCHMAX + 255) / 256;
  constexpr int VCH = (VCHMAX + 255) / 256;
  constexpr int TILE_BYTES = 2 * 2 * (KT + VT) * 2;             // [buf][half] K and V^T
  constexpr int MERGE_BYTES = 2 * 64 * (DB * 16 + 2) * 4;       // per query group: o, m, l (one block)
  constexpr int SMEM = (TILE_BYTES > MERGE_BYTES ? TILE_BYTES : MERGE_BYTES) + 16;  // + spare slot
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  bf16* const Ks = (bf16*)smem;                  // [buf][half][kKH][KLD]
  bf16* const Vs = Ks + 2 * 2 * KT;              // [buf][half][VROWS][VLD]
  const int SPARE = (TILE_BYTES > MERGE_BYTES ? TILE_BYTES : MERGE_BYTES) / 2;  // bf16 index

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qg = wave & 1, kh = wave >> 1;
  const int l32 = lane & 31, g = lane >> 5;
  // Workgroup b runs on XCD b % 8. Give each XCD a contiguous range of (row, head,
  // query block) triples, query blocks fastest, so the query blocks that stream the same
  // K and V share one L2.
  constexpr int QPW = QB * 64;  // queries per workgroup
  const int nqb = (a.Nq + QPW - 1) / QPW;
  const int T = nqb * a.heads * a.rows;
  const int xcd = blockIdx.x % 8, local = blockIdx.x / 8;
  const int base = T / 8, rem = T % 8;
  const int logical = xcd * base + min(xcd, rem) + local;
  const int qblk = logical % nqb;
  const int rh = logical / nqb;
  const int head = rh % a.heads, r = rh / a.heads;
  const int dh = a.dh;
  const size_t bh = (size_t)r * a.heads + head;
  const size_t kr = a.kv_map ? (size_t)a.kv_map[r] : (size_t)r;  // the row whose keys and values r reads
  const bf16* Q = (const bf16*)a.q + bh * a.Nq * dh;
  const bf16* Kg = (const bf16*)a.k + kr * a.k_rs + (size_t)head * a.k_ld * dh;
  const bf16* Vt = (const bf16*)a.vT + kr * a.v_rs + (size_t)head * dh * a.ldv;
  int qi[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) qi[qb] = qblk * QPW + qg * 32 * QB + qb * 32 + l32;

  // zero the tile buffers once: padding columns (dh..KLD) and rows (dh..VROWS) are
  // never written by the staging
  for (int i = tid; i < TILE_BYTES / 16; i += 256) ((u32x4*)smem)[i] = u32x4{0u, 0u, 0u, 0u};

  const float sl2 = a.scale * 1.4426950408889634f;  // scores -> exp2 units
  bf16x8 qf[QB][DHC];
  const __amdgpu_buffer_rsrc_t q_src = buffer_rsrc(Q, (uint32_t)a.Nq * dh * 2);
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int kk = 0; kk < DHC; ++kk) {
      const int d0 = kk * 16 + g * 8;
      const u32x4 w = buffer_load16(q_src, (qi[qb] < a.Nq && d0 < dh) ? (qi[qb] * dh + d0) * 2 : kOffOOB);
      qf[qb][kk] = __builtin_bit_cast(bf16x8, w);
      scale_q(qf[qb][kk], sl2);
    }

  // staging map, fixed per thread: K chunk c = (key 0..63, 16-byte column); V^T chunk
  // c = (dh row, 8-key column group 0..7). Chunks past the real count read zeros and
  // land in the spare slot. Each step's loads go through buffer resources based at the
  // step's first key, so the offsets stay fixed: keys past Nk fall outside the K
  // resource and read zeros, and the V^T rows (ldv a multiple of 64) hold every key
  // column a step can reach, zero past the last key.
  const int dh8 = dh >> 3;
  const int kchunks = 2 * kKH * dh8;
  const int vchunks = dh * (2 * kKH / 8);
  int k_goff[KCH], k_lds[KCH], v_goff[VCH], v_lds[VCH];
#pragma unroll
  for (int i = 0; i < KCH; ++i) {
    const int c = tid + i * 256;
    const bool in = c < kchunks;
    const int key = in ? c / dh8 : 0, col = in ? (c - key * dh8) * 8 : 0;
    k_goff[i] = in ? (key * dh + col) * 2 : kOffOOB;
    k_lds[i] = in ? (key >> 5) * KT + (key & 31) * KLD + col : -1;
  }
#pragma unroll
  for (int i = 0; i < VCH; ++i) {
    const int c = tid + i * 256;
    const bool in = c < vchunks;
    const int d = in ? c >> 3 : 0, kg = c & 7;
    v_goff[i] = in ? (d * a.ldv + kg * 8) * 2 : kOffOOB;
    v_lds[i] = in ? (kg >> 2) * VT + d * VLD + (kg & 3) * 8 : -1;
  }
  u32x4 rk[KCH], rv[VCH];
  auto gload = [&](int kv0) {
    const __amdgpu_buffer_rsrc_t k_src = buffer_rsrc(Kg + (size_t)kv0 * dh, (uint32_t)max(a.Nk - kv0, 0) * dh * 2);
    const __amdgpu_buffer_rsrc_t v_src = buffer_rsrc(Vt + kv0, (uint32_t)max(dh * a.ldv - kv0, 0) * 2);
#pragma unroll
    for (int i = 0; i < KCH; ++i) rk[i] = buffer_load16(k_src, k_goff[i]);
#pragma unroll
    for (int i = 0; i < VCH; ++i) rv[i] = buffer_load16(v_src, v_goff[i]);
  };
  auto lstore = [&](int buf) {
    // the chunk counts depend on dh at run time, so every chunk checks its slot
#pragma unroll
    for (int i = 0; i < KCH; ++i) *(u32x4*)&Ks[k_lds[i] >= 0 ? buf * 2 * KT + k_lds[i] : SPARE] = rk[i];
#pragma unroll
    for (int i = 0; i < VCH; ++i) *(u32x4*)&Vs[v_lds[i] >= 0 ? buf * 2 * VT + v_lds[i] : SPARE - 4 * KT] = rv[i];
  };

  f32x16 o[QB][DB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int b = 0; b < DB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[qb][b][e] = 0.0f;
  float m2[QB], lsum[QB];                          // offset in exp2 units, partial sum
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m2[qb] = 0.0f;
    lsum[qb] = 0.0f;
  }

  const int nsteps = (a.Nk + 2 * kKH - 1) / (2 * kKH);
  constexpr int kSumRow = DB * 32 - 8;
  __syncthreads();
  if constexpr (SUMROW) {
    // after the zero fill (the barrier above), before the first tile: the ones row of
    // both buffers and key halves (never written by the staging, which fills rows < dh)
    for (int i = tid; i < 2 * 2 * (kKH / 8); i += 256) {
      const int bhalf = i / (kKH / 8), c = i - bhalf * (kKH / 8);
      *(u32x4*)&Vs[bhalf * VT + kSumRow * VLD + c * 8] = u32x4{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
    }
  }
  gload(0);
  lstore(0);
  __syncthreads();
  for (int it = 0; it < nsteps; ++it) {
    const int cur = it & 1;
    const int kv0 = it * 2 * kKH + kh * kKH;      // this wavefront's first key
    if (it + 1 < nsteps) gload((it + 1) * 2 * kKH);
    const bf16* Kb = Ks + (cur * 2 + kh) * KT;
    const bf16* Vb = Vs + (cur * 2 + kh) * VT;
    // a key half that lies wholly past the last key (key half 1 when Nk <= 32, or the
    // tail of the last step) contributes nothing and is skipped: its scores would all be
    // -inf, and its step max would move the offset of a wavefront at its first step
    if (kv0 < a.Nk) {
      // every K and V^T fragment feeds the MFMAs of all QB query blocks
      f32x16 s[QB];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int e = 0; e < 16; ++e) s[qb][e] = 0.0f;
#pragma unroll
      for (int kk = 0; kk < DHC; ++kk) {
        const bf16x8 kf = *(const bf16x8*)&Kb[l32 * KLD + kk * 16 + g * 8];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) s[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[qb][kk], s[qb], 0, 0, 0);
      }
      // s[qb][e]: query l32 of block qb, key kv0 + (e/4)*8 + g*4 + e%4, in exp2 units.
      // Only the last, ragged step needs the key mask.
      if (kv0 + kKH > a.Nk) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (kv0 + (e >> 2) * 8 + g * 4 + (e & 3) >= a.Nk) s[qb][e] = -INFINITY;
      }
      bf16x8 pf[QB][2];
      softmax_step_lazy<!SUMROW>(s, it == 0, m2, lsum, o, pf);
      // V^T fragment of k-slots 8g..8g+7 (keys 16 ks + 4 g + 0..3 and 16 ks + 8 + 4 g + 0..3
      // of this half): one 16-byte read in the permuted key layout (vt_pos)
#pragma unroll
      for (int b = 0; b < DB; ++b) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const bf16x8 vf = *(const bf16x8*)&Vb[(b * 32 + l32) * VLD + ks * 16 + g * 8];
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            o[qb][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[qb][ks], o[qb][b], 0, 0, 0);
        }
      }
    }
    if (it + 1 < nsteps) lstore(cur ^ 1);
    __syncthreads();
  }

  // the ones row's output (row kSumRow of the last block: register 12 of lane half 0;
  // lane half 1 holds row kSumRow + 4, a zero row) is this wavefront's probability sum
  if constexpr (SUMROW) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) lsum[qb] = o[qb][DB - 1][12];
  }
  // merge the key halves one query block at a time: half 1 hands (o, offset, partial sum)
  // to half 0 through LDS
  float* mg = (float*)smem + qg * 64 * (DB * 16 + 2);
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    if (qb > 0) __syncthreads();  // the previous block's values were read
    if (kh == 1) {
#pragma unroll
      for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) mg[(b * 16 + e) * 64 + lane] = o[qb][b][e];
      mg[DB * 16 * 64 + lane] = m2[qb];
      mg[(DB * 16 + 1) * 64 + lane] = lsum[qb];
    }
    __syncthreads();
    if (kh == 1) continue;
    // key half 0 always holds key 0; half 1 saw no key when there are at most 32 (its
    // zeros are then left out by selects, and its offset is not used)
    const bool other = kKH < a.Nk;
    const float m2b = mg[DB * 16 * 64 + lane];
    const float mnew = other ? fmaxf(m2[qb], m2b) : m2[qb];
    const float a0 = __builtin_amdgcn_exp2f(m2[qb] - mnew);
    const float a1 = other ? __builtin_amdgcn_exp2f(m2b - mnew) : 0.0f;
    float ls = lsum[qb] * a0 + (other ? mg[(DB * 16 + 1) * 64 + lane] * a1 : 0.0f);
    ls = pair32_sum(ls);
    const float inv = 1.0f / ls;
    if (qi[qb] < a.Nq) {
      bf16* O = (bf16*)a.o + ((size_t)r * a.Nq + qi[qb]) * a.D + (size_t)head * dh;
#pragma unroll
      for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const int d = b * 32 + e4 * 8 + g * 4;
          float w[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int e = e4 * 4 + q;
            w[q] = (o[qb][b][e] * a0 + (other ? mg[(b * 16 + e) * 64 + lane] * a1 : 0.0f)) * inv;
          }
          if (d < dh) *(bf16x4*)(O + d) = bf16x4{(bf16)w[0], (bf16)w[1], (bf16)w[2], (bf16)w[3]};
        }
    }
  }
}

// One step of the online softmax for QB 32-query blocks at head dim 64, where the row
// sum is kept by vector adds (scores in exp2 units). The probabilities are formed
// against the current offsets first (wave_probs) and added to the row sums; the offsets
// start at 0 and are left alone while every row sum of a block stays in [2^-64, 2^64],
// so the usual step takes no max at all. When a sum leaves the range (scores above
// about 64 or all below about -64 so far, non-finite scores) that block takes the max
// over both lane halves and moves the offset: to the max for a query with nothing
// accumulated yet (which may lower it), else up to the max if that is larger, with the
// output and sum rescaled; then its probabilities are formed again. A softmax does not
// depend on the offset, and inside that range every probability, sum and output keeps
// its relative precision. The offset is the same on both lane halves of a query.
template <int QB, int DB>
__device__ __forceinline__ void softmax_step_sum(const f32x16 (&sc)[QB], float (&m2)[QB], float (&lsum)[QB],
                                                 f32x16 (&o)[QB][DB], bf16x8 (&pf)[QB][2]) {
  float l[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) l[qb] = lsum[qb];
  wave_probs<true>(sc, m2, l, pf);
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    if (__any(!(l[qb] <= 0x1p64f && l[qb] >= 0x1p-64f))) {
      float tmax = sc[qb][0];
#pragma unroll
      for (int e = 1; e < 16; ++e) tmax = fmaxf(tmax, sc[qb][e]);
      tmax = pair32_max(tmax);
      const bool empty = pair32_sum(lsum[qb]) == 0.0f;  // nothing accumulated for this query yet
      const float mnew = empty ? tmax : fmaxf(m2[qb], tmax);
      const float alpha = empty ? 0.0f : __builtin_amdgcn_exp2f(m2[qb] - mnew);
      lsum[qb] *= alpha;
#pragma unroll
      for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[qb][b][e] *= alpha;
      m2[qb] = mnew;
      l[qb] = lsum[qb];
      block_probs<true, true>(sc[qb], m2[qb], l[qb], pf[qb]);
    }
    lsum[qb] = l[qb];
  }
}

// Head dim 64: the same computation with the K and V^T tiles moved by buffer_load ... lds
// straight from global memory into a ring of three LDS stages, two steps ahead (no VGPR
// round trip, no LDS write instructions). Each stage is its own __shared__ variable
// and the key loop is unrolled by three, so the compiler waits only for the stage being
// read; the barrier is a bare s_barrier after an explicit wait for this step's loads.
// A stage holds the step's 64 keys: K as 64 rows x 8 chunks (dh) and V^T as 64 dh rows
// x 8 chunks (keys), both swizzled with dma_swz; 16 KB, so three workgroups of three
// stages fit a CU. V^T comes in the permuted key layout (vt_pos, written so by the QKV
// projection), so each P.V fragment is one 16-byte LDS read instead of two 8-byte ones.
constexpr int kAttnStages = 3;

__global__ __launch_bounds__(256) void attn_bf16_dma64_kernel(AttnArgs a) {
  constexpr int DH = 64, DHC = 4, DB = 2, CPR = 8;
  constexpr int KCHUNKS = 2 * kKH * CPR;  // 512
  constexpr int SB = (KCHUNKS + DH * CPR) * 16;
  constexpr int LPT = SB / 16 / 256;  // loads per thread and step
  constexpr int MERGE = 64 * (DB * 16 + 2) * 4;
  static_assert(MERGE <= SB && LPT == 4, "stage layout");
  __shared__ __attribute__((aligned(16))) char st0[SB];
  __shared__ __attribute__((aligned(16))) char st1[SB];
  __shared__ __attribute__((aligned(16))) char st2[SB];
  auto stage = [&](auto s) -> char* {
    constexpr int S = decltype(s)::value % kAttnStages;
    if constexpr (S == 0) return st0;
    else if constexpr (S == 1) return st1;
    else return st2;
  };

  // the wavefront index is uniform: kept in a scalar register, so the key offsets and
  // step checks derived from it are scalar work
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qg = wave & 1, kh = wave >> 1;
  const int l32 = lane & 31, g = lane >> 5;
  const int nqb = (a.Nq + kQB - 1) / kQB;
  const int T = nqb * a.heads * a.rows;
  const int xcd = blockIdx.x % 8, local = blockIdx.x / 8;
  const int base = T / 8, rem = T % 8;
  const int logical = xcd * base + min(xcd, rem) + local;
  const int qblk = logical % nqb;
  const int rh = logical / nqb;
  const int head = rh % a.heads, r = rh / a.heads;
  const size_t bh = (size_t)r * a.heads + head;
  const size_t kr = a.kv_map ? (size_t)a.kv_map[r] : (size_t)r;  // the row whose keys and values r reads
  const bf16* Q = (const bf16*)a.q + bh * a.Nq * DH;
  const bf16* Kg = (const bf16*)a.k + kr * a.k_rs + (size_t)head * a.k_ld * DH;
  const bf16* Vt = (const bf16*)a.vT + kr * a.v_rs + (size_t)head * DH * a.ldv;
  const int qi = qblk * kQB + qg * 32 + l32;

  const float sl2 = a.scale * 1.4426950408889634f;
  bf16x8 qf[DHC];
  const __amdgpu_buffer_rsrc_t q_src = buffer_rsrc(Q, (uint32_t)a.Nq * DH * 2);
#pragma unroll
  for (int kk = 0; kk < DHC; ++kk) {
    const u32x4 w = buffer_load16(q_src, qi < a.Nq ? (qi * DH + kk * 16 + g * 8) * 2 : kOffOOB);
    qf[kk] = __builtin_bit_cast(bf16x8, w);
    scale_q(qf[kk], sl2);
  }

  // load i of a thread fills chunk position p = i * 256 + tid of a stage: K row (key)
  // p / 8 for i < 2, else V^T row (dh) p / 8 - 64; position p % 8 holds chunk
  // (p % 8) ^ swz(row) of that row (dh columns of K, key columns of V^T). Each step's
  // loads go through buffer resources based at the step's first key, so a thread's
  // offsets are fixed: keys past Nk fall outside the K resource and read zeros, and the
  // V^T rows (ldv a multiple of 64) hold every key column a step can reach, zero past
  // the last key.
  int goff[LPT];
#pragma unroll
  for (int i = 0; i < LPT; ++i) {
    const int p = i * 256 + tid;
    const int row = (p / CPR) % 64;
    const int c = (p % CPR) ^ dma_swz<CPR>(row);
    goff[i] = i < 2 ? (row * DH + c * 8) * 2 : (row * a.ldv + c * 8) * 2;
  }
  auto issue = [&](char* sb, int step) {
    const int kv0 = step * 2 * kKH;
    const __amdgpu_buffer_rsrc_t k_src =
        buffer_rsrc(Kg + (size_t)kv0 * DH, (uint32_t)max(a.Nk - kv0, 0) * DH * 2);
    const __amdgpu_buffer_rsrc_t v_src = buffer_rsrc(Vt + kv0, (uint32_t)max(DH * a.ldv - kv0, 0) * 2);
#pragma unroll
    for (int i = 0; i < LPT; ++i)
      buffer_load16_lds(i < 2 ? k_src : v_src, sb + (i * 256 + wave * 64) * 16, goff[i]);
  };

  // one query block, held as arrays of one for the softmax helpers
  f32x16 o[1][DB];
#pragma unroll
  for (int b = 0; b < DB; ++b)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[0][b][e] = 0.0f;
  float m2[1] = {0.0f}, lsum[1] = {0.0f};
  const int sw = dma_swz<CPR>(l32);  // the swizzle of every row this lane reads
  const int krow = (kh * kKH + l32) * CPR;

  constexpr int kWait = waitcnt_vm_lgkm0<(kAttnStages - 2) * LPT>();
  auto step = [&](auto s, int it) {
    constexpr int S = decltype(s)::value;
    __builtin_amdgcn_s_waitcnt(kWait);
    bare_barrier();
    issue(stage(std::integral_constant<int, S + kAttnStages - 1>{}), it + kAttnStages - 1);
    const char* cur = stage(std::integral_constant<int, S>{});
    const int kv0 = it * 2 * kKH + kh * kKH;
    // a key half wholly past the last key contributes nothing (see attn_bf16_kernel)
    if (kv0 >= a.Nk) return;
    f32x16 sc[1];
#pragma unroll
    for (int e = 0; e < 16; ++e) sc[0][e] = 0.0f;
    // all K fragments are read before the first MFMA, so their LDS latencies overlap
    // (the compiler otherwise waits for each pair in turn)
    bf16x8 kf[DHC];
#pragma unroll
    for (int kk = 0; kk < DHC; ++kk) kf[kk] = *(const bf16x8*)(cur + (krow + ((kk * 2 + g) ^ sw)) * 16);
#pragma unroll
    for (int kk = 0; kk < DHC; ++kk) sc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[kk], sc[0], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, DHC, 0);  // LDS reads
    __builtin_amdgcn_sched_group_barrier(0x008, DHC, 0);  // then the MFMAs
    if (kv0 + kKH > a.Nk) {
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (kv0 + (e >> 2) * 8 + g * 4 + (e & 3) >= a.Nk) sc[0][e] = -INFINITY;
    }
    bf16x8 pf[1][2];
    softmax_step_sum(sc, m2, lsum, o, pf);
    // V^T fragment of k-slots 8g..8g+7: keys 16 ks + 4 g + 0..3 and 16 ks + 8 + 4 g + 0..3
    // of this half, which the permuted layout (vt_pos) keeps in one 16-byte chunk,
    // kh*4 + 2 ks + g
#pragma unroll
    for (int b = 0; b < DB; ++b) {
      const char* vrow = cur + KCHUNKS * 16 + (b * 32 + l32) * CPR * 16;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8 vf = *(const bf16x8*)(vrow + (((kh * 4 + 2 * ks + g) ^ sw) << 4));
        o[0][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[0][ks], o[0][b], 0, 0, 0);
      }
    }
  };

  const int nsteps = (a.Nk + 2 * kKH - 1) / (2 * kKH);
  issue(stage(std::integral_constant<int, 0>{}), 0);
  issue(stage(std::integral_constant<int, 1>{}), 1);
  // whole rounds of three steps in a loop with one exit, then the remaining steps
  int it = 0;
  for (; it + kAttnStages <= nsteps; it += kAttnStages) {
    step(std::integral_constant<int, 0>{}, it);
    step(std::integral_constant<int, 1>{}, it + 1);
    step(std::integral_constant<int, 2>{}, it + 2);
  }
  if (it < nsteps) step(std::integral_constant<int, 0>{}, it);
  if (it + 1 < nsteps) step(std::integral_constant<int, 1>{}, it + 1);
  // the zero-filling loads past the keys land before the stages are reused
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // merge the key halves: half 1 hands (o, offset, partial sum) to half 0 through LDS
  float* mg = (float*)(qg == 0 ? st0 : st1);
  if (kh == 1) {
#pragma unroll
    for (int b = 0; b < DB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) mg[(b * 16 + e) * 64 + lane] = o[0][b][e];
    mg[DB * 16 * 64 + lane] = m2[0];
    mg[(DB * 16 + 1) * 64 + lane] = lsum[0];
  }
  __syncthreads();
  if (kh == 1) return;
  // key half 0 always holds key 0; half 1 saw no key when there are at most 32 (its
  // zeros are then left out by selects, and its offset is not used)
  const bool other = kKH < a.Nk;
  const float m2b = mg[DB * 16 * 64 + lane];
  const float mnew = other ? fmaxf(m2[0], m2b) : m2[0];
  const float a0 = __builtin_amdgcn_exp2f(m2[0] - mnew);
  const float a1 = other ? __builtin_amdgcn_exp2f(m2b - mnew) : 0.0f;
  float ls = lsum[0] * a0 + (other ? mg[(DB * 16 + 1) * 64 + lane] * a1 : 0.0f);
  ls = pair32_sum(ls);
  const float inv = 1.0f / ls;
  if (qi < a.Nq) {
    bf16* O = (bf16*)a.o + ((size_t)r * a.Nq + qi) * a.D + (size_t)head * DH;
#pragma unroll
    for (int b = 0; b < DB; ++b)
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int d = b * 32 + e4 * 8 + g * 4;
        float w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int e = e4 * 4 + q;
          w[q] = (o[0][b][e] * a0 + (other ? mg[(b * 16 + e) * 64 + lane] * a1 : 0.0f)) * inv;
        }
        *(bf16x4*)(O + d) = bf16x4{(bf16)w[0], (bf16)w[1], (bf16)w[2], (bf16)w[3]};
      }
  }
}

// Head dim 64 with two 32-query blocks per wavefront: a workgroup owns 128 queries of
// one (row, head) (two query groups of 64 times two key halves), and every K and V^T
// fragment read from LDS feeds the MFMAs of both query blocks, half the LDS reads per
// FLOP of attn_bf16_dma64_kernel, with two independent score / softmax chains per step
// for the scheduler to interleave. Staging (three DMA stages of 64 keys) and each
// query's arithmetic, in order, are those of attn_bf16_dma64_kernel.
constexpr int kQB2 = 128;  // queries per workgroup

__global__ __launch_bounds__(256, 2) void attn_bf16_dma64x2_kernel(AttnArgs a) {
  constexpr int DH = 64, DHC = 4, DB = 2, CPR = 8, QB = 2;
  constexpr int KCHUNKS = 2 * kKH * CPR;  // 512
  constexpr int SB = (KCHUNKS + DH * CPR) * 16;
  constexpr int LPT = SB / 16 / 256;  // loads per thread and step
  constexpr int MERGE = 64 * (DB * 16 + 2) * 4;  // one query block of one query group
  static_assert(MERGE <= SB && LPT == 4, "stage layout");
  __shared__ __attribute__((aligned(16))) char st0[SB];
  __shared__ __attribute__((aligned(16))) char st1[SB];
  __shared__ __attribute__((aligned(16))) char st2[SB];
  auto stage = [&](auto s) -> char* {
    constexpr int S = decltype(s)::value % kAttnStages;
    if constexpr (S == 0) return st0;
    else if constexpr (S == 1) return st1;
    else return st2;
  };

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qg = wave & 1, kh = wave >> 1;
  const int l32 = lane & 31, g = lane >> 5;
  const int nqb = (a.Nq + kQB2 - 1) / kQB2;
  const int T = nqb * a.heads * a.rows;
  const int xcd = blockIdx.x % 8, local = blockIdx.x / 8;
  const int base = T / 8, rem = T % 8;
  const int logical = xcd * base + min(xcd, rem) + local;
  const int qblk = logical % nqb;
  const int rh = logical / nqb;
  const int head = rh % a.heads, r = rh / a.heads;
  const size_t bh = (size_t)r * a.heads + head;
  const size_t kr = a.kv_map ? (size_t)a.kv_map[r] : (size_t)r;
  const bf16* Q = (const bf16*)a.q + bh * a.Nq * DH;
  const bf16* Kg = (const bf16*)a.k + kr * a.k_rs + (size_t)head * a.k_ld * DH;
  const bf16* Vt = (const bf16*)a.vT + kr * a.v_rs + (size_t)head * DH * a.ldv;
  int qi[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) qi[qb] = qblk * kQB2 + qg * 64 + qb * 32 + l32;

  const float sl2 = a.scale * 1.4426950408889634f;
  bf16x8 qf[QB][DHC];
  const __amdgpu_buffer_rsrc_t q_src = buffer_rsrc(Q, (uint32_t)a.Nq * DH * 2);
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int kk = 0; kk < DHC; ++kk) {
      const u32x4 w = buffer_load16(q_src, qi[qb] < a.Nq ? (qi[qb] * DH + kk * 16 + g * 8) * 2 : kOffOOB);
      qf[qb][kk] = __builtin_bit_cast(bf16x8, w);
      scale_q(qf[qb][kk], sl2);
    }

  int goff[LPT];
#pragma unroll
  for (int i = 0; i < LPT; ++i) {
    const int p = i * 256 + tid;
    const int row = (p / CPR) % 64;
    const int c = (p % CPR) ^ dma_swz<CPR>(row);
    goff[i] = i < 2 ? (row * DH + c * 8) * 2 : (row * a.ldv + c * 8) * 2;
  }
  auto issue = [&](char* sb, int step) {
    const int kv0 = step * 2 * kKH;
    const __amdgpu_buffer_rsrc_t k_src =
        buffer_rsrc(Kg + (size_t)kv0 * DH, (uint32_t)max(a.Nk - kv0, 0) * DH * 2);
    const __amdgpu_buffer_rsrc_t v_src = buffer_rsrc(Vt + kv0, (uint32_t)max(DH * a.ldv - kv0, 0) * 2);
#pragma unroll
    for (int i = 0; i < LPT; ++i)
      buffer_load16_lds(i < 2 ? k_src : v_src, sb + (i * 256 + wave * 64) * 16, goff[i]);
  };

  f32x16 o[QB][DB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int b = 0; b < DB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[qb][b][e] = 0.0f;
  float m2[QB], lsum[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m2[qb] = 0.0f;
    lsum[qb] = 0.0f;
  }
  const int sw = dma_swz<CPR>(l32);
  const int krow = (kh * kKH + l32) * CPR;

  constexpr int kWait = waitcnt_vm_lgkm0<(kAttnStages - 2) * LPT>();
  auto step = [&](auto s, int it) {
    constexpr int S = decltype(s)::value;
    __builtin_amdgcn_s_waitcnt(kWait);
    bare_barrier();
    issue(stage(std::integral_constant<int, S + kAttnStages - 1>{}), it + kAttnStages - 1);
    const char* cur = stage(std::integral_constant<int, S>{});
    const int kv0 = it * 2 * kKH + kh * kKH;
    if (kv0 >= a.Nk) return;
    f32x16 sc[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[qb][e] = 0.0f;
    bf16x8 kf[DHC];
#pragma unroll
    for (int kk = 0; kk < DHC; ++kk) kf[kk] = *(const bf16x8*)(cur + (krow + ((kk * 2 + g) ^ sw)) * 16);
#pragma unroll
    for (int kk = 0; kk < DHC; ++kk)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) sc[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[qb][kk], sc[qb], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, DHC, 0);       // LDS reads
    __builtin_amdgcn_sched_group_barrier(0x008, DHC * QB, 0);  // then the MFMAs
    if (kv0 + kKH > a.Nk) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (kv0 + (e >> 2) * 8 + g * 4 + (e & 3) >= a.Nk) sc[qb][e] = -INFINITY;
    }
    bf16x8 pf[QB][2];
    softmax_step_sum(sc, m2, lsum, o, pf);
#pragma unroll
    for (int b = 0; b < DB; ++b) {
      const char* vrow = cur + KCHUNKS * 16 + (b * 32 + l32) * CPR * 16;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8 vf = *(const bf16x8*)(vrow + (((kh * 4 + 2 * ks + g) ^ sw) << 4));
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          o[qb][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[qb][ks], o[qb][b], 0, 0, 0);
      }
    }
  };

  const int nsteps = (a.Nk + 2 * kKH - 1) / (2 * kKH);
  issue(stage(std::integral_constant<int, 0>{}), 0);
  issue(stage(std::integral_constant<int, 1>{}), 1);
  int it = 0;
  for (; it + kAttnStages <= nsteps; it += kAttnStages) {
    step(std::integral_constant<int, 0>{}, it);
    step(std::integral_constant<int, 1>{}, it + 1);
    step(std::integral_constant<int, 2>{}, it + 2);
  }
  if (it < nsteps) step(std::integral_constant<int, 0>{}, it);
  if (it + 1 < nsteps) step(std::integral_constant<int, 1>{}, it + 1);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // merge the key halves one query block at a time: half 1 hands (o, offset, partial sum)
  // to half 0 through LDS (stage 0 for query group 0, stage 1 for query group 1)
  float* mg = (float*)(qg == 0 ? st0 : st1);
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    if (qb > 0) __syncthreads();  // the previous block's values were read
    if (kh == 1) {
#pragma unroll
      for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) mg[(b * 16 + e) * 64 + lane] = o[qb][b][e];
      mg[DB * 16 * 64 + lane] = m2[qb];
      mg[(DB * 16 + 1) * 64 + lane] = lsum[qb];
    }
    __syncthreads();
    if (kh == 0) {
      // as in attn_bf16_dma64_kernel: half 1 saw keys only when there are more than 32
      const bool other = kKH < a.Nk;
      const float m2b = mg[DB * 16 * 64 + lane];
      const float mnew = other ? fmaxf(m2[qb], m2b) : m2[qb];
      const float a0 = __builtin_amdgcn_exp2f(m2[qb] - mnew);
      const float a1 = other ? __builtin_amdgcn_exp2f(m2b - mnew) : 0.0f;
      float ls = lsum[qb] * a0 + (other ? mg[(DB * 16 + 1) * 64 + lane] * a1 : 0.0f);
      ls = pair32_sum(ls);
      const float inv = 1.0f / ls;
      if (qi[qb] < a.Nq) {
        bf16* O = (bf16*)a.o + ((size_t)r * a.Nq + qi[qb]) * a.D + (size_t)head * DH;
#pragma unroll
        for (int b = 0; b < DB; ++b)
#pragma unroll
          for (int e4 = 0; e4 < 4; ++e4) {
            const int d = b * 32 + e4 * 8 + g * 4;
            float w[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int e = e4 * 4 + q;
              w[q] = (o[qb][b][e] * a0 + (other ? mg[(b * 16 + e) * 64 + lane] * a1 : 0.0f)) * inv;
            }
            *(bf16x4*)(O + d) = bf16x4{(bf16)w[0], (bf16)w[1], (bf16)w[2], (bf16)w[3]};
          }
      }
    }
  }
}

// Head dim 72 with two 32-query blocks per wavefront, K and V^T moved by buffer_load ...
// lds into a ring of three LDS stages two steps ahead, as attn_bf16_dma64_kernel does for
// head dim 64. A stage holds the step's 64 keys:
//  * K as 64 rows of 144 bytes (9 chunks). Consecutive rows then start 16 bytes apart
//    modulo 128, so the fragment reads are conflict-free without a swizzle, and the
//    stage is a byte copy of the step's contiguous K block.
//  * V^T as 72 dh rows x 8 chunks (keys, permuted layout), swizzled with dma_swz.
//  * 24 constant rows up to the 96 rows of the three dh blocks: zeros, and the ones row
//    (row 88) whose P.V output is each query's probability sum. They are written once,
//    before the first step; the loads never touch them.
// The K fragment of dh 72..79 (the second half of the fifth 16-wide chunk) is a zero
// register, like the zero padding of attn_bf16_kernel's K tile, and the queries' dh
// 72..79 are zero too. Every query's arithmetic, in order, is that of
// attn_bf16_kernel<5, 3, true, 2>, so both return the same bits.
constexpr int kD72K = 64 * 9;                    // 16-byte K chunks per stage
constexpr int kD72V = 72 * 8;                    // 16-byte V^T chunks per stage
constexpr int kD72Stage = (kD72K + 96 * 8) * 16;  // + the constant rows: 21 KB
__shared__ __attribute__((aligned(16))) char g_attn72_st0[kD72Stage];
__shared__ __attribute__((aligned(16))) char g_attn72_st1[kD72Stage];
__shared__ __attribute__((aligned(16))) char g_attn72_st2[kD72Stage];
__shared__ __attribute__((aligned(16))) char g_attn72_spare[1024];

__global__ __launch_bounds__(256, 2) void attn_bf16_dma72x2_kernel(AttnArgs a) {
  constexpr int DH = 72, DHC = 5, DB = 3, QB = 2;
  constexpr int NCH = kD72K + kD72V;         // 1152 chunks per step
  constexpr int LPT = (NCH + 255) / 256;     // 5 loads per thread (128 of them spare)
  constexpr int V_OFF = kD72K * 16;          // byte offset of V^T in a stage
  constexpr int MERGE = 64 * (DB * 16 + 2) * 4;
  static_assert(MERGE <= kD72Stage && NCH % 64 == 0, "stage layout");
  constexpr int kSumRow = DB * 32 - 8;
  char* const st0 = g_attn72_st0;
  char* const st1 = g_attn72_st1;
  char* const st2 = g_attn72_st2;
  auto stage = [&](auto s) -> char* {
    constexpr int S = decltype(s)::value % kAttnStages;
    if constexpr (S == 0) return st0;
    else if constexpr (S == 1) return st1;
    else return st2;
  };

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qg = wave & 1, kh = wave >> 1;
  const int l32 = lane & 31, g = lane >> 5;
  // each XCD (workgroup b runs on XCD b % 8) takes a contiguous range of (row, head,
  // query block) triples, query blocks fastest, so the blocks of one (row, head) share
  // an L2
  const int nqb = (a.Nq + kQB2 - 1) / kQB2;
  const int T = nqb * a.heads * a.rows;
  const int xcd = blockIdx.x % 8, local = blockIdx.x / 8;
  const int base = T / 8, rem = T % 8;
  const int logical = xcd * base + min(xcd, rem) + local;
  const int qblk = logical % nqb;
  const int rh = logical / nqb;
  const int head = rh % a.heads, r = rh / a.heads;
  const size_t bh = (size_t)r * a.heads + head;
  const size_t kr = a.kv_map ? (size_t)a.kv_map[r] : (size_t)r;
  const bf16* Q = (const bf16*)a.q + bh * a.Nq * DH;
  const bf16* Kg = (const bf16*)a.k + kr * a.k_rs + (size_t)head * a.k_ld * DH;
  const bf16* Vt = (const bf16*)a.vT + kr * a.v_rs + (size_t)head * DH * a.ldv;
  int qi[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) qi[qb] = qblk * kQB2 + qg * 64 + qb * 32 + l32;

  // the constant rows 72..95 of every stage's V^T: zeros, ones in row kSumRow
  for (int i = tid; i < kAttnStages * 24 * 8; i += 256) {
    const int st = i / (24 * 8), c = i - st * (24 * 8), row = 72 + c / 8;
    char* base = st == 0 ? st0 : st == 1 ? st1 : st2;
    const uint32_t w = row == kSumRow ? 0x3F803F80u : 0u;
    *(u32x4*)(base + V_OFF + (row * 8 + c % 8) * 16) = u32x4{w, w, w, w};
  }

  const float sl2 = a.scale * 1.4426950408889634f;
  bf16x8 qf[QB][DHC];
  const __amdgpu_buffer_rsrc_t q_src = buffer_rsrc(Q, (uint32_t)a.Nq * DH * 2);
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int kk = 0; kk < DHC; ++kk) {
      const int d0 = kk * 16 + g * 8;
      const u32x4 w = buffer_load16(q_src, (qi[qb] < a.Nq && d0 < DH) ? (qi[qb] * DH + d0) * 2 : kOffOOB);
      qf[qb][kk] = __builtin_bit_cast(bf16x8, w);
      scale_q(qf[qb][kk], sl2);
    }

  // load i of a thread fills chunk position p = i * 256 + tid of a stage: K chunk p
  // (bytes 16 p of the step's K block) for p < 576, V^T chunk p - 576 (dh row
  // (p - 576) / 8, chunk position (p - 576) % 8 holding key chunk position ^ swz(row))
  // below 1152, else nothing (the load reads zeros into the spare slot). Whole
  // wavefronts fall in one part, since both parts are multiples of 64 chunks.
  int goff[LPT];
  bool isk[LPT], inr[LPT];
#pragma unroll
  for (int i = 0; i < LPT; ++i) {
    const int p = i * 256 + tid;
    isk[i] = p < kD72K;
    inr[i] = p < NCH;
    if (p < kD72K) {
      goff[i] = p * 16;
    } else if (p < NCH) {
      const int pv = p - kD72K, row = pv / 8;
      goff[i] = (row * a.ldv + (((pv % 8) ^ dma_swz<8>(row)) * 8)) * 2;
    } else {
      goff[i] = kOffOOB;
    }
  }
  auto issue = [&](char* sb, int step) {
    const int kv0 = step * 2 * kKH;
    const __amdgpu_buffer_rsrc_t k_src =
        buffer_rsrc(Kg + (size_t)kv0 * DH, (uint32_t)max(a.Nk - kv0, 0) * DH * 2);
    const __amdgpu_buffer_rsrc_t v_src = buffer_rsrc(Vt + kv0, (uint32_t)max(DH * a.ldv - kv0, 0) * 2);
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      // the wavefront's part is uniform (the parts are whole wavefronts)
      char* dst = inr[i] ? sb + (isk[i] ? (i * 256 + wave * 64) * 16 : V_OFF + (i * 256 + wave * 64 - kD72K) * 16)
                         : g_attn72_spare;
      buffer_load16_lds(isk[i] ? k_src : v_src, dst, goff[i]);
    }
  };

  f32x16 o[QB][DB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int b = 0; b < DB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[qb][b][e] = 0.0f;
  float m2[QB], unused[QB];  // offsets; the row sums come from the ones row
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) m2[qb] = unused[qb] = 0.0f;
  const int sw = dma_swz<8>(l32);
  const int krow = (kh * kKH + l32) * 9;

  constexpr int kWait = waitcnt_vm_lgkm0<(kAttnStages - 2) * LPT>();
  auto step = [&](auto s, int it) {
    constexpr int S = decltype(s)::value;
    __builtin_amdgcn_s_waitcnt(kWait);
    bare_barrier();
    issue(stage(std::integral_constant<int, S + kAttnStages - 1>{}), it + kAttnStages - 1);
    const char* cur = stage(std::integral_constant<int, S>{});
    const int kv0 = it * 2 * kKH + kh * kKH;
    if (kv0 >= a.Nk) return;
    f32x16 sc[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[qb][e] = 0.0f;
    bf16x8 kf[DHC];
#pragma unroll
    for (int kk = 0; kk < DHC; ++kk) kf[kk] = *(const bf16x8*)(cur + (krow + kk * 2 + g) * 16);
    if (g == 1) kf[DHC - 1] = bf16x8{};  // dh 72..79
#pragma unroll
    for (int kk = 0; kk < DHC; ++kk)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) sc[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[qb][kk], sc[qb], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, DHC, 0);       // LDS reads
    __builtin_amdgcn_sched_group_barrier(0x008, DHC * QB, 0);  // then the MFMAs
    if (kv0 + kKH > a.Nk) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (kv0 + (e >> 2) * 8 + g * 4 + (e & 3) >= a.Nk) sc[qb][e] = -INFINITY;
    }
    bf16x8 pf[QB][2];
    softmax_step_lazy<false>(sc, it == 0, m2, unused, o, pf);
#pragma unroll
    for (int b = 0; b < DB; ++b) {
      const char* vrow = cur + V_OFF + (b * 32 + l32) * 8 * 16;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8 vf = *(const bf16x8*)(vrow + (((kh * 4 + 2 * ks + g) ^ sw) << 4));
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          o[qb][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[qb][ks], o[qb][b], 0, 0, 0);
      }
    }
  };

  const int nsteps = (a.Nk + 2 * kKH - 1) / (2 * kKH);
  // the constant rows are in place before any stage is read
  __syncthreads();
  issue(stage(std::integral_constant<int, 0>{}), 0);
  issue(stage(std::integral_constant<int, 1>{}), 1);
  int it = 0;
  for (; it + kAttnStages <= nsteps; it += kAttnStages) {
    step(std::integral_constant<int, 0>{}, it);
    step(std::integral_constant<int, 1>{}, it + 1);
    step(std::integral_constant<int, 2>{}, it + 2);
  }
  if (it < nsteps) step(std::integral_constant<int, 0>{}, it);
  if (it + 1 < nsteps) step(std::integral_constant<int, 1>{}, it + 1);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // the ones row's output (row kSumRow of the last block: register 12 of lane half 0;
  // lane half 1 holds row kSumRow + 4, a zero row) is this wavefront's probability sum
  float lsum[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) lsum[qb] = o[qb][DB - 1][12];
  float* mg = (float*)(qg == 0 ? st0 : st1);
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    if (qb > 0) __syncthreads();  // the previous block's values were read
    if (kh == 1) {
#pragma unroll
      for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) mg[(b * 16 + e) * 64 + lane] = o[qb][b][e];
      mg[DB * 16 * 64 + lane] = m2[qb];
      mg[(DB * 16 + 1) * 64 + lane] = lsum[qb];
    }
    __syncthreads();
    if (kh == 1) continue;
    // as in attn_bf16_kernel: half 1 saw keys only when there are more than 32
    const bool other = kKH < a.Nk;
    const float m2b = mg[DB * 16 * 64 + lane];
    const float mnew = other ? fmaxf(m2[qb], m2b) : m2[qb];
    const float a0 = __builtin_amdgcn_exp2f(m2[qb] - mnew);
    const float a1 = other ? __builtin_amdgcn_exp2f(m2b - mnew) : 0.0f;
    float ls = lsum[qb] * a0 + (other ? mg[(DB * 16 + 1) * 64 + lane] * a1 : 0.0f);
    ls = pair32_sum(ls);
    const float inv = 1.0f / ls;
    if (qi[qb] < a.Nq) {
      bf16* O = (bf16*)a.o + ((size_t)r * a.Nq + qi[qb]) * a.D + (size_t)head * DH;
#pragma unroll
      for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const int d = b * 32 + e4 * 8 + g * 4;
          float w[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int e = e4 * 4 + q;
            w[q] = (o[qb][b][e] * a0 + (other ? mg[(b * 16 + e) * 64 + lane] * a1 : 0.0f)) * inv;
          }
          if (d < DH) *(bf16x4*)(O + d) = bf16x4{(bf16)w[0], (bf16)w[1], (bf16)w[2], (bf16)w[3]};
        }
    }
  }
}

// ------------------------------------------------------------------ fp32
constexpr int kFKV = 32;

template <int DHMAX>
__global__ __launch_bounds__(128) void attn_f32_kernel(AttnArgs a) {
  __shared__ float Ks[kFKV][DHMAX];
  __shared__ float Vs[kFKV][DHMAX];
  const int head = blockIdx.y, r = blockIdx.z;
  const int dh = a.dh;
  const size_t bh = (size_t)r * a.heads + head;
  const size_t kr = a.kv_map ? (size_t)a.kv_map[r] : (size_t)r;  // the row whose keys and values r reads
  const float* Q = (const float*)a.q + bh * a.Nq * dh;
  const float* Kg = (const float*)a.k + kr * a.k_rs + (size_t)head * a.k_ld * dh;
  const float* Vt = (const float*)a.vT + kr * a.v_rs + (size_t)head * dh * a.ldv;
  const int qi = blockIdx.x * blockDim.x + threadIdx.x;
  float q[DHMAX], o[DHMAX];
#pragma unroll
  for (int d = 0; d < DHMAX; ++d) {
    q[d] = (qi < a.Nq && d < dh) ? Q[(size_t)qi * dh + d] * a.scale : 0.0f;
    o[d] = 0.0f;
  }
  float m = -INFINITY, l = 0.0f;
  for (int kv0 = 0; kv0 < a.Nk; kv0 += kFKV) {
    for (int i = threadIdx.x; i < kFKV * dh; i += blockDim.x) {
      const int j = i / dh, d = i - j * dh;
      const bool ok = kv0 + j < a.Nk;
      Ks[j][d] = ok ? Kg[(size_t)(kv0 + j) * dh + d] : 0.0f;
      Vs[j][d] = ok ? Vt[(size_t)d * a.ldv + kv0 + j] : 0.0f;
    }
    __syncthreads();
    const int nj = min(kFKV, a.Nk - kv0);
    for (int j = 0; j < nj; ++j) {
      float sc = 0.0f;
#pragma unroll
      for (int d = 0; d < DHMAX; ++d)
        if (d < dh) sc += q[d] * Ks[j][d];
      const float mn = fmaxf(m, sc);
      const float corr = expf(m - mn);
      const float p = expf(sc - mn);
      l = l * corr + p;
#pragma unroll
      for (int d = 0; d < DHMAX; ++d)
        if (d < dh) o[d] = o[d] * corr + p * Vs[j][d];
      m = mn;
    }
    __syncthreads();
  }
  if (qi < a.Nq) {
    float* O = (float*)a.o + ((size_t)r * a.Nq + qi) * a.D + (size_t)head * dh;
#pragma unroll
    for (int d = 0; d < DHMAX; ++d)
      if (d < dh) O[d] = o[d] / l;
  }
}

bool attention_supports(int dh) { return dh >= 8 && dh <= 128 && dh % 8 == 0; }

template <int DHC, int DB>
static void launch_bf16_inst(const AttnArgs& a, bool two_blocks, hipStream_t s) {
  if (two_blocks) {
    dim3 grid(((a.Nq + 2 * kQB - 1) / (2 * kQB)) * a.heads * a.rows);
    if (a.dh % 32 != 0)
      launch((attn_bf16_kernel<DHC, DB, true, 2>), grid, dim3(256), 0, s, a);
    else
      launch((attn_bf16_kernel<DHC, DB, false, 2>), grid, dim3(256), 0, s, a);
    return;
  }
  dim3 grid(((a.Nq + kQB - 1) / kQB) * a.heads * a.rows);
  if (a.dh % 32 != 0)
    launch((attn_bf16_kernel<DHC, DB, true, 1>), grid, dim3(256), 0, s, a);
  else
    launch((attn_bf16_kernel<DHC, DB, false, 1>), grid, dim3(256), 0, s, a);
}

hipError_t launch_attention(bool use_bf16, const AttnArgs& args, hipStream_t s) {
  AttnArgs a = args;
  if (!a.k_ld) a.k_ld = a.Nk;
  if (!a.k_rs) a.k_rs = (size_t)a.heads * a.k_ld * a.dh;
  if (!a.v_rs) a.v_rs = (size_t)a.heads * a.dh * a.ldv;
  if (!attention_supports(a.dh)) return hipErrorInvalidValue;
  // the bf16 kernels read transposed v in the permuted key layout only, with rows of
  // whole 64-key steps; the fp32 kernel reads the plain layout
  if ((a.vperm != 0) != use_bf16 || (a.vperm && a.ldv % 64 != 0)) return hipErrorInvalidValue;
  if (use_bf16) {
    // Two query blocks per wavefront (128 queries per workgroup) halve the LDS reads per
    // FLOP but need two such workgroups per CU to fill the chip: taken when the layer
    // has at least 512 of them. Both forms compute every query in the same order (the
    // same bits), so the choice changes no result.
    const bool two = (size_t)((a.Nq + 2 * kQB - 1) / (2 * kQB)) * a.heads * a.rows >= 512;
    const int dhc = (a.dh + 15) / 16;
    switch (dhc) {
      case 1: launch_bf16_inst<1, 1>(a, two, s); break;
      case 2: launch_bf16_inst<2, 1>(a, two, s); break;
      case 3: launch_bf16_inst<3, 2>(a, two, s); break;
      case 4:
        if (a.dh == 64 && two)
          launch(attn_bf16_dma64x2_kernel, dim3(((a.Nq + kQB2 - 1) / kQB2) * a.heads * a.rows), dim3(256), 0, s, a);
        else if (a.dh == 64)
          launch(attn_bf16_dma64_kernel, dim3(((a.Nq + kQB - 1) / kQB) * a.heads * a.rows), dim3(256), 0, s, a);
        else
          launch_bf16_inst<4, 2>(a, two, s);
        break;
      case 5:
        if (a.dh == 72 && two)
          launch(attn_bf16_dma72x2_kernel, dim3(((a.Nq + kQB2 - 1) / kQB2) * a.heads * a.rows), dim3(256), 0, s, a);
        else
          launch_bf16_inst<5, 3>(a, two, s);
        break;
      case 6: launch_bf16_inst<6, 3>(a, two, s); break;
      case 7: launch_bf16_inst<7, 4>(a, two, s); break;
      case 8: launch_bf16_inst<8, 4>(a, two, s); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    dim3 grid((a.Nq + 127) / 128, a.heads, a.rows);
    if (a.dh <= 32)
      launch(attn_f32_kernel<32>, grid, dim3(128), 0, s, a);
    else if (a.dh <= 64)
      launch(attn_f32_kernel<64>, grid, dim3(128), 0, s, a);
    else
      launch(attn_f32_kernel<128>, grid, dim3(128), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace sf
