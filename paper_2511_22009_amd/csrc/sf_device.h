// Device-side helpers shared by the gfx950 kernels: vector types for the MFMA
// builtins, wavefront (64-lane) reductions, invariant-divisor division, bf16 I/O.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sf_launch.h"

namespace sf {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// n / d for a divisor fixed at launch: q = (umulhi(n, magic) + n) >> shift.
__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv& f) {
  return (uint32_t)(((uint64_t)__umulhi(n, f.magic) + n) >> f.shift);
}

// The value that lane l ^ M holds, moved in vector registers without the LDS crossbar
// that __shfl_xor (ds_bpermute) goes through, where each exchange waits a full LDS round
// trip, behind any other LDS traffic of the CU:
//   M = 1, 2: DPP quad_perm [1,0,3,2] and [2,3,0,1];
//   M = 4: DPP row_shl:4 written to lanes 0-3 and 8-11 of each 16-lane row (bank mask
//          0101), then row_shr:4 to lanes 4-7 and 12-15 (bank mask 1010);
//   M = 8: DPP row_ror:8 (rotation by 8 within a 16-lane row);
//   M = 16, 32: v_permlane16_swap / v_permlane32_swap with v as both operands, which
//          return (r0, r1) with r1 = v[l + M] in the lanes whose bit M is clear and
//          r0 = v[l - M] in the others.
// (Lane layouts of all six checked on the GPU against l ^ M.)
template <int M>
__device__ __forceinline__ float lane_xor(float v) {
  const int x = __float_as_int(v);
  if constexpr (M == 1) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, true));
  } else if constexpr (M == 2) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, true));
  } else if constexpr (M == 4) {
    const int y = __builtin_amdgcn_update_dpp(x, x, 0x104, 0xF, 0x5, false);
    return __int_as_float(__builtin_amdgcn_update_dpp(y, x, 0x114, 0xF, 0xA, false));
  } else if constexpr (M == 8) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0x128, 0xF, 0xF, true));
  } else if constexpr (M == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap((unsigned)x, (unsigned)x, false, false);
    return __uint_as_float((threadIdx.x & 16) ? r[0] : r[1]);
  } else {
    static_assert(M == 32, "lane_xor: M is 1, 2, 4, 8, 16 or 32");
    const auto r = __builtin_amdgcn_permlane32_swap((unsigned)x, (unsigned)x, false, false);
    return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
  }
}

// Butterfly over lane xor 32, 16, 8, 4, 2, 1 (each lane adds its partner's value to
// its own, so every lane ends with the same bits).
__device__ __forceinline__ float wave_sum(float v) {
  v += lane_xor<32>(v);
  v += lane_xor<16>(v);
  v += lane_xor<8>(v);
  v += lane_xor<4>(v);
  v += lane_xor<2>(v);
  v += lane_xor<1>(v);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, lane_xor<32>(v));
  v = fmaxf(v, lane_xor<16>(v));
  v = fmaxf(v, lane_xor<8>(v));
  v = fmaxf(v, lane_xor<4>(v));
  v = fmaxf(v, lane_xor<2>(v));
  v = fmaxf(v, lane_xor<1>(v));
  return v;
}

// Max and sum of v over the lane pair (l, l ^ 32), in vector registers.
// v_permlane32_swap with v as both operands returns (r0, r1) where lane l < 32 holds
// (v[l], v[l + 32]) and lane l >= 32 holds (v[l - 32], v[l]). So max(r0, r1) and r0 + r1
// are the pair's max and sum in every lane. Both operations commute, so the bits equal
// those of v op __shfl_xor(v, 32), which goes through the LDS crossbar (ds_bpermute)
// and waits behind any LDS traffic.
__device__ __forceinline__ float pair32_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float pair32_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Sums each of 16 per-lane values over the 64 lanes of a wavefront and returns, in
// lane l, the total of index (l >> 2) & 15 (lanes 4i..4i+3 all hold total i). Butterfly
// reduce-scatter: four halving exchanges (lane xor 32, 16, 8, 4) then two plain ones
// (xor 2, 1). In a halving exchange over bit M a lane keeps half of its values ("mine")
// and receives its partner's copy of that half. For M = 32 and 16 one lane swap moves
// both halves at once: with X = the lower half and Y = the upper half as operands, a
// lane whose bit M is clear reads its partner's X in r1, the others their partner's Y
// in r0.
__device__ __forceinline__ float wave_reduce16(float (&v)[16]) {
  const int lane = threadIdx.x & 63;
  float a8[8], a4[4], a2[2];
  {
    const bool hi = lane & 32;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[i]), __float_as_uint(v[8 + i]), false, false);
      a8[i] = hi ? v[8 + i] + __uint_as_float(r[0]) : v[i] + __uint_as_float(r[1]);
    }
  }
  {
    const bool hi = lane & 16;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a8[i]), __float_as_uint(a8[4 + i]), false, false);
      a4[i] = hi ? a8[4 + i] + __uint_as_float(r[0]) : a8[i] + __uint_as_float(r[1]);
    }
  }
  {
    const bool hi = lane & 8;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const float mine = hi ? a4[2 + i] : a4[i];
      const float give = hi ? a4[i] : a4[2 + i];
      a2[i] = mine + lane_xor<8>(give);
    }
  }
  const bool hi = lane & 4;
  float r = (hi ? a2[1] : a2[0]) + lane_xor<4>(hi ? a2[0] : a2[1]);
  r += lane_xor<2>(r);
  r += lane_xor<1>(r);
  return r;
}

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }  // RNE

template <typename T> __device__ __forceinline__ float to_f32(T v) { return (float)v; }

// tanh-form GELU written as z * sigmoid(2u), u = sqrt(2/pi) (z + 0.044715 z^3), since
// 0.5 (1 + tanh(u)) = 1 / (1 + exp(-2u)); with exp(-2u) = 2^y, y = z (c0 + c1 z^2)
// (log2(e) folded into the constants) it is five plain operations plus the hardware
// exp2 and reciprocal (each within about 1 ulp). Both limits are exact: 2^y overflows to
// inf for very negative z (result -0) and underflows to 0 for large z (result z).
__device__ __forceinline__ float gelu_tanh(float z) {
  constexpr float c0 = -2.0f * 0.7978845608028654f * 1.4426950408889634f;
  constexpr float c1 = c0 * 0.044715f;
  const float y = z * __builtin_fmaf(c1, z * z, c0);
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(y));
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

// Raw buffer resource over [base, base + bytes): a load whose byte offset is at or
// past `bytes` returns zeros in hardware, so tile loads need no branches.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kOffOOB = kOffOOBHost;  // any offset >= every buffer size used here (the
                                      // loader bounds each operand below it)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ u32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
// The same load marked non-temporal (nt): for data read once per call, such as the
// adaLN projection weights, so that streaming them does not push the projection GEMMs'
// weights and activations out of the caches.
__device__ __forceinline__ u32x4 buffer_load16_stream(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2);
}

// ---- direct global -> LDS staging (buffer_load ... lds) ---------------------------
// Unpadded LDS tiles of 8 or 16 16-byte chunks per row: chunk c of row r sits at chunk
// position c ^ dma_swz(r), which keeps 16-byte fragment reads (one row per lane, lanes
// 0-15 and 16-31 each reading one chunk column of 16 consecutive rows) free of bank
// conflicts whether the LDS serves 8 or 16 lanes of a 16-byte read per cycle. The
// swizzle depends on r % 16 only, so rows 32 apart share it.
template <int CPR>
__device__ __forceinline__ int dma_swz(int r) {
  static_assert(CPR == 8 || CPR == 16, "8 or 16 chunks per row");
  if constexpr (CPR == 8)
    return (r & 7) ^ ((r >> 3) & 1);
  else
    return r & 15;
}

// A non-template wrapper: with the builtin written inside the kernel template the
// host-side pass of this compiler dropped the kernels' launch stubs.
__device__ __forceinline__ void buffer_load16_lds(__amdgpu_buffer_rsrc_t r, char* lds, int off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, off, 0, 0, 0);
}


// Workgroup barrier without a memory fence; the signal fences keep the compiler from
// moving LDS accesses across it. Callers wait for what the barrier must cover first.
__device__ __forceinline__ void bare_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// s_waitcnt immediate: at most N vector-memory operations outstanding, no LDS ones.
template <int N>
__device__ __forceinline__ constexpr int waitcnt_vm_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt holds 6 bits");
  return (N & 15) | ((N >> 4) << 14) | (7 << 4);
}

}  // namespace sf
