// Shared device helpers for the gfx950 kernels (wave64, CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace metro {

constexpr int kWave = 64;
constexpr int kPage = 16;  // tokens per KV page

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// float32 -> bfloat16 bits, round to nearest even (subnormals kept); a NaN
// stays a NaN.  One v_cvt_pk_bf16_f32 for two values.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{lo, hi}), bf16x2));
}

__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return static_cast<uint16_t>(pack_bf16x2(f, 0.f)); }

// The two bf16 values of a 32-bit word as floats (exact).
__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Reductions over lane pairs (l, l^16) and (l, l^32): gfx950's row-swap
// instructions hand every lane its own value and its partner's, in VALU
// registers (no LDS round trip as for a general shuffle).
__device__ __forceinline__ float max_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

__device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Element offset of (page, K|V, kv_head, slot, dim) inside one layer's slab of
// the KV pool, laid out as [layer][page][2][n_kv_heads][kPage][head_dim].
__device__ __forceinline__ size_t kv_offset(int page, int kv, int n_kv_heads, int head, int slot, int head_dim,
                                            int dim) {
  return static_cast<size_t>(page) * (2 * n_kv_heads * kPage * head_dim) +
         static_cast<size_t>((kv * n_kv_heads + head) * kPage + slot) * head_dim + dim;
}

// Element offsets inside one (page, kv head) tile of 16 keys x hd dims, laid
// out so that every matrix-core operand of the attention kernels is one
// 16-byte load per lane, lane l = 16g + r reading bytes 16l .. 16l+15 of a
// 1 KiB block (g = l/16, r = l%16):
//   K:   block i = dims 32i .. 32i+31, element (key r, dim 32i + 8g + e) at
//        ((i*4 + g)*16 + r)*8 + e
//   V^T: block c = dims 32c .. 32c+31, element (dim 32c + 16u + r, key 4g + j)
//        at ((c*4 + g)*16 + r)*8 + 4u + j: one load gives lane (r, g) the 4
//        keys of dims 32c + r and 32c + 16 + r.
__device__ __forceinline__ int k_tile_offset(int key, int d) {
  return (((d >> 5) * 4 + ((d >> 3) & 3)) * 16 + key) * 8 + (d & 7);
}
__device__ __forceinline__ int vt_tile_offset(int d, int key) {
  return (((d >> 5) * 4 + (key >> 2)) * 16 + (d & 15)) * 8 + ((d >> 4) & 1) * 4 + (key & 3);
}

// Projection weights W [N][Kp] (bf16, Kp % 128 == 0, N % 16 == 0) are stored in
// the operand order of v_mfma_f32_16x16x32_bf16: W is cut into 16 x 32 tiles
// (16 rows n, 32 reduction indices k), tiles row-major over (n/16, k/32), and
// tile (tn, tk) is 64 chunks of 16 bytes in lane order, the chunk of lane
// l = 16g + r holding W[16tn + r][32tk + 8g .. 8g + 7].  One wave reading one
// tile (lane l the bytes 16l .. 16l+15) is a single contiguous 1 KiB request,
// and a row tile's successive k tiles are contiguous.
__host__ __device__ __forceinline__ int64_t packed_offset(int64_t n, int64_t k, int64_t Kp) {
  return ((((n >> 4) * (Kp >> 5) + (k >> 5)) * 64 + (n & 15) + 16 * ((k >> 3) & 3)) << 3) + (k & 7);
}

// --- direct loads into LDS ---------------------------------------------------
// global_load_lds_dwordx4 writes each lane's 16 bytes at LDS base + 16 * lane
// (base in M0, wave-uniform) and counts in vmcnt like any vector load.  The
// loads and their waits are issued as inline assembly so that the compiler,
// which cannot tell which LDS bytes they write, does not guard every later
// LDS read with a wait for all of them; code using them waits explicitly
// (wait_vmcnt) and synchronises the workgroup with lds_barrier.  Waits the
// compiler inserts for its own loads can only wait longer, never shorter.

template <int N_>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N_) : "memory");
}

__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// 16 bytes per lane from gptr into LDS bytes lds_base + 16 * lane; one wait
// state separates the M0 write from the load that reads it
__device__ __forceinline__ void lds_load16(const void* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(gptr), "s"(lds_base)
               : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const void*)p));
}

}  // namespace metro
