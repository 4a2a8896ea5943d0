// K4: softmax attention softmax(q k^T / sqrt(dh)) v for every (network row, head), no
// mask; each row attends only to its own tokens, so samples never mix.
//
// bf16 path (v_mfma_f32_32x32x16_bf16), online softmax over 64-key tiles:
//   * a workgroup owns 128 queries of one (row, head); each of its 4 wavefronts owns 32;
//   * scores are computed transposed, S^T = K Q^T, so the MFMA result gives each lane
//     ONE query (column l%32) and 16 of the 32 keys of a 32-key block: the running max
//     and sum are lane-local plus a single cross-half shuffle;
//   * the probabilities are rounded to bf16 and used directly as the B operand of
//     O^T = V^T P^T: the MFMA's k-slot order is a permutation of the key order, and V^T
//     is read from LDS under the same permutation (two 8-byte reads per fragment);
//   * K and V^T tiles are double-buffered in LDS and fetched one tile ahead through
//     registers; rows past dh and keys past Nk are zero, so padding adds nothing.
// fp32 path: one thread per query, keys staged in LDS (parity mode).
#include "sf_device.h"

namespace sf {

constexpr int kBKV = 64;   // keys per tile
constexpr int kQB = 128;   // queries per workgroup

template <int DHC, int DB>  // DHC = ceil(dh/16) contraction chunks, DB = ceil(dh/32) dh blocks
__global__ __launch_bounds__(256) void attn_bf16_kernel(AttnArgs a) {
  constexpr int KLD = DHC * 16 + 8;     // K tile row pitch (bf16)
  constexpr int VLD = kBKV + 8;         // V^T tile row pitch (bf16)
  constexpr int VROWS = DB * 32;
  constexpr int KCH = (kBKV * DHC * 2 + 255) / 256;   // 16-byte K chunks per thread (upper bound)
  constexpr int VCH = (VROWS * (kBKV / 8) + 255) / 256;
  __shared__ bf16 Ks[2][kBKV * KLD];
  __shared__ bf16 Vs[2][VROWS * VLD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, g = lane >> 5;
  // Workgroup b runs on XCD b % 8. Give each XCD a contiguous range of (row, head,
  // query block) triples, query blocks fastest, so the query blocks that stream the same
  // K and V share one L2.
  const int nqb = (a.Nq + kQB - 1) / kQB;
  const int T = nqb * a.heads * a.rows;
  const int xcd = blockIdx.x % 8, local = blockIdx.x / 8;
  const int base = T / 8, rem = T % 8;
  const int logical = xcd * base + min(xcd, rem) + local;
  const int qblk = logical % nqb;
  const int rh = logical / nqb;
  const int head = rh % a.heads, r = rh / a.heads;
  const int dh = a.dh;
  const size_t bh = (size_t)r * a.heads + head;
  const bf16* Q = (const bf16*)a.q + bh * a.Nq * dh;
  const bf16* Kg = (const bf16*)a.k + bh * a.Nk * dh;
  const bf16* Vt = (const bf16*)a.vT + bh * dh * a.ldv;
  const int qi = qblk * kQB + wave * 32 + l32;

  // zero both buffers once: padding columns/rows are never written by the staging
  for (int i = tid; i < 2 * kBKV * KLD; i += 256) (&Ks[0][0])[i] = (bf16)0.0f;
  for (int i = tid; i < 2 * VROWS * VLD; i += 256) (&Vs[0][0])[i] = (bf16)0.0f;

  bf16x8 qf[DHC];
#pragma unroll
  for (int kk = 0; kk < DHC; ++kk) {
    const int d0 = kk * 16 + g * 8;
    if (qi < a.Nq && d0 < dh) {
      qf[kk] = *(const bf16x8*)(Q + (size_t)qi * dh + d0);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[kk][e] = (bf16)0.0f;
    }
  }

  const int kchunks = kBKV * (dh >> 3);       // K tile: kBKV rows x dh/8 chunks
  const int vchunks = dh * (kBKV / 8);        // V^T tile: dh rows x 8 chunks
  // K and V^T come in through raw buffer loads: keys past Nk (K) and columns past the
  // padded row (V^T) get an out-of-range offset and read as zeros, without branches.
  const __amdgpu_buffer_rsrc_t k_src = buffer_rsrc(Kg, (uint32_t)a.Nk * dh * 2);
  const __amdgpu_buffer_rsrc_t v_src = buffer_rsrc(Vt, (uint32_t)dh * a.ldv * 2);
  int k_row[KCH], k_col[KCH], v_off[VCH], v_kv[VCH];
#pragma unroll
  for (int i = 0; i < KCH; ++i) {
    const int c = tid + i * 256;
    k_row[i] = c < kchunks ? c / (dh >> 3) : 1 << 20;
    k_col[i] = c < kchunks ? (c - (c / (dh >> 3)) * (dh >> 3)) * 8 : 0;
  }
#pragma unroll
  for (int i = 0; i < VCH; ++i) {
    const int c = tid + i * 256;
    v_kv[i] = (c & 7) * 8;
    v_off[i] = c < vchunks ? ((c >> 3) * a.ldv + v_kv[i]) * 2 : kOffOOB;
  }
  u32x4 rk[KCH], rv[VCH];
  auto gload = [&](int kv0) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int row = kv0 + k_row[i];
      rk[i] = buffer_load16(k_src, row < a.Nk ? (row * dh + k_col[i]) * 2 : kOffOOB);
    }
#pragma unroll
    for (int i = 0; i < VCH; ++i)
      rv[i] = buffer_load16(v_src, (v_off[i] != kOffOOB && kv0 + v_kv[i] < a.ldv) ? v_off[i] + 2 * kv0 : kOffOOB);
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KCH; ++i)
      if (tid + i * 256 < kchunks) *(u32x4*)&Ks[buf][k_row[i] * KLD + k_col[i]] = rk[i];
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int c = tid + i * 256;
      if (c < vchunks) *(u32x4*)&Vs[buf][(c >> 3) * VLD + (c & 7) * 8] = rv[i];
    }
  };

  f32x16 o[DB];
#pragma unroll
  for (int b = 0; b < DB; ++b)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[b][e] = 0.0f;
  float mrow = -INFINITY, lsum = 0.0f;
  const float sl2 = a.scale * 1.4426950408889634f;  // scores in log2 units

  const int ntiles = (a.Nk + kBKV - 1) / kBKV;
  __syncthreads();
  gload(0);
  lstore(0);
  __syncthreads();
  for (int it = 0; it < ntiles; ++it) {
    const int cur = it & 1;
    const int kv0 = it * kBKV;
    if (it + 1 < ntiles) gload(kv0 + kBKV);

    f32x16 s[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s[c][e] = 0.0f;
#pragma unroll
      for (int kk = 0; kk < DHC; ++kk) {
        const bf16x8 kf = *(const bf16x8*)&Ks[cur][(c * 32 + l32) * KLD + kk * 16 + g * 8];
        s[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], s[c], 0, 0, 0);
      }
    }
    // s[c][e]: query l32, key kv0 + c*32 + (e/4)*8 + g*4 + e%4. Raw scores; the
    // scale (log2 e / sqrt(dh)) is folded into the exp2 argument. Only the last,
    // ragged tile needs the key mask.
    if (kv0 + kBKV > a.Nk) {
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kv = kv0 + c * 32 + (e >> 2) * 8 + g * 4 + (e & 3);
          if (kv >= a.Nk) s[c][e] = -INFINITY;
        }
    }
    float tmax = s[0][0];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int e = 0; e < 16; ++e) tmax = fmaxf(tmax, s[c][e]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float mnew = fmaxf(mrow, tmax);
    // rescale the running output and sum only when some query's max moved
    if (__any(mnew != mrow)) {
      const float alpha = __builtin_amdgcn_exp2f((mrow - mnew) * sl2);
      lsum *= alpha;
#pragma unroll
      for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[b][e] *= alpha;
    }
    mrow = mnew;
    const float moff = -mnew * sl2;

    bf16x8 pf[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[ks >> 1][(ks & 1) * 8 + j], sl2, moff));
        lsum += p;
        pf[ks][j] = (bf16)p;
      }
    }
#pragma unroll
    for (int b = 0; b < DB; ++b) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const bf16* vr = &Vs[cur][(b * 32 + l32) * VLD + ks * 16 + g * 4];
        const bf16x4 lo = *(const bf16x4*)vr;
        const bf16x4 hi = *(const bf16x4*)(vr + 8);
        const bf16x8 vf = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        o[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[ks], o[b], 0, 0, 0);
      }
    }
    if (it + 1 < ntiles) lstore(cur ^ 1);
    __syncthreads();
  }

  lsum += __shfl_xor(lsum, 32);
  const float inv = 1.0f / lsum;
  if (qi < a.Nq) {
    bf16* O = (bf16*)a.o + ((size_t)r * a.Nq + qi) * a.D + (size_t)head * dh;
#pragma unroll
    for (int b = 0; b < DB; ++b)
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int d = b * 32 + e4 * 8 + g * 4;
        if (d < dh) {
          const bf16x4 w = {(bf16)(o[b][e4 * 4 + 0] * inv), (bf16)(o[b][e4 * 4 + 1] * inv),
                            (bf16)(o[b][e4 * 4 + 2] * inv), (bf16)(o[b][e4 * 4 + 3] * inv)};
          *(bf16x4*)(O + d) = w;
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
  const float* Q = (const float*)a.q + bh * a.Nq * dh;
  const float* Kg = (const float*)a.k + bh * a.Nk * dh;
  const float* Vt = (const float*)a.vT + bh * dh * a.ldv;
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
static void launch_bf16_inst(const AttnArgs& a, hipStream_t s) {
  dim3 grid(((a.Nq + kQB - 1) / kQB) * a.heads * a.rows);
  launch((attn_bf16_kernel<DHC, DB>), grid, dim3(256), 0, s, a);
}

hipError_t launch_attention(bool use_bf16, const AttnArgs& a, hipStream_t s) {
  if (!attention_supports(a.dh)) return hipErrorInvalidValue;
  if (use_bf16) {
    const int dhc = (a.dh + 15) / 16;
    switch (dhc) {
      case 1: launch_bf16_inst<1, 1>(a, s); break;
      case 2: launch_bf16_inst<2, 1>(a, s); break;
      case 3: launch_bf16_inst<3, 2>(a, s); break;
      case 4: launch_bf16_inst<4, 2>(a, s); break;
      case 5: launch_bf16_inst<5, 3>(a, s); break;
      case 6: launch_bf16_inst<6, 3>(a, s); break;
      case 7: launch_bf16_inst<7, 4>(a, s); break;
      case 8: launch_bf16_inst<8, 4>(a, s); break;
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
