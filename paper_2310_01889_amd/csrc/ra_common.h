// Internal helpers shared by the gfx950 kernels and the host scheduler.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace ra {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

typedef __attribute__((address_space(3))) void lds_void;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// ---------------------------------------------------------------------------------
// Matrix-core helpers (gfx950).  Lane layouts, verified on the device:
//   32x32x16 bf16:  A[m][k]: lane l holds m = l%32, k = 8*(l/32) + 0..7
//                   B[k][n]: lane l holds n = l%32, k = 8*(l/32) + 0..7
//                   C[m][n]: lane l, reg i holds n = l%32, m = 8*(i/4) + 4*(l/32) + i%4
//   16x16x32 bf16:  A: m = l%16, k = 8*(l/16) + 0..7;  B: n = l%16, same k;
//                   C: reg i holds n = l%16, m = 4*(l/16) + i
// Any permutation of k applied to both operands leaves the product unchanged.
// ---------------------------------------------------------------------------------
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// LDS transpose read (ds_read_b64_tr_b16).  Within each group of 16 lanes, lane L
// supplies the address of 4 consecutive 16-bit values M[L][0..3]; lane i receives
// element j = M[4j + i/4][i%4].  Used to feed a row-major [k][n] tile as an operand
// whose lanes run along n and registers along k.
__device__ __forceinline__ bf16x4 lds_read_tr16(const bf16* lds_ptr) {
  s16x4 t = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)((lds_void*)lds_ptr));
  return __builtin_bit_cast(bf16x4, t);
}

// Direct-to-LDS load of 16 bytes per lane through a buffer descriptor: lane i reads
// base + voff_bytes (reads at or past num_bytes return zero) and its data lands at byte
// 16 i of lds_dst, which must be wave-uniform.  The descriptor is scalar, so moving base
// from tile to tile costs no vector instructions.
__device__ __forceinline__ void buffer_load_lds16(const void* base, int num_bytes, void* lds_dst, int voff_bytes) {
#if __HIP_DEVICE_COMPILE__
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, num_bytes, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void*)lds_dst, 16, voff_bytes, 0, 0, 0);
#endif
}

// As buffer_load_lds16, the read address being base + voff_bytes + soff_bytes with soff_bytes
// wave-uniform (a scalar register: no vector register per load).
__device__ __forceinline__ void buffer_load_lds16_so(const void* base, int num_bytes, void* lds_dst, int voff_bytes,
                                                     int soff_bytes) {
#if __HIP_DEVICE_COMPILE__
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, num_bytes, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void*)lds_dst, 16, voff_bytes, soff_bytes, 0, 0);
#endif
}

// As buffer_load_lds16 with 4 bytes per lane (lane i lands at byte 4 i of lds_dst).
__device__ __forceinline__ void buffer_load_lds4(const void* base, int num_bytes, void* lds_dst, int voff_bytes) {
#if __HIP_DEVICE_COMPILE__
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, num_bytes, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void*)lds_dst, 4, voff_bytes, 0, 0, 0);
#endif
}

// Max / sum of a value with the same value in lane l ^ 32 (v_permlane32_swap).
__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// acc + lo + hi of a packed bf16 pair (v_dot2c_f32_bf16 against (1, 1)); exact products.
__device__ __forceinline__ float dot2_bf16_ones(uint32_t packed, float acc) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t ones = {(__bf16)1.0f, (__bf16)1.0f};
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, packed), ones, acc, false);
}

// Two float -> packed bf16 pair, round-to-nearest-even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// Map a linear workgroup id so that each XCD (workgroups are dispatched round-robin
// over the 8 XCDs) receives a contiguous range of logical tiles: tiles that share
// key/value data then share one L2.
__device__ __forceinline__ int xcd_swizzle(int id, int total) {
  const int nx = 8;
  const int per = total / nx, rem = total % nx;
  const int xcd = id % nx, n = id / nx;
  return xcd * per + (xcd < rem ? xcd : rem) + n;
}

// Row index with bits 2 and 3 swapped.  Loading the A operand of a 32x32x16 MFMA from
// row swap_bits23(l % 32) puts, in each lane half h, the 8 consecutive rows 8h..8h+7 of
// every 16-row group into registers 0..7 and 8..15 of the result -- the k layout of a
// B operand -- so a transposed product can feed the next MFMA without a shuffle.
__device__ __forceinline__ int swap_bits23(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

template <int I, int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// XOR swizzle of the 16-byte chunks of an unpadded LDS tile row of D bf16 elements:
// logical chunk c of row r is stored at chunk c ^ swz<D>(r).  For D = 128 (16 chunks)
// both 16 consecutive rows read at one chunk and 4 consecutive rows read across 4
// consecutive chunks touch 16 distinct chunk positions (no bank conflicts); for D = 64
// (8 chunks, two rows per 256-byte bank sweep) rows of equal parity are spread.
template <int D>
__device__ __forceinline__ int swz(int r) {
  if constexpr (D == 128) {
    return 4 * (r & 3) + ((r >> 2) & 3);
  } else {
    const int s = (r >> 1) & 7;
    return s ^ ((s & 1) << 2);
  }
}

}  // namespace ra
