// Device helpers for the gfx950 (CDNA4) SRA kernels: MFMA, LDS transpose reads, wave64
// lane-pair reductions and the LDS swizzles.
//
// Lane layouts of V_MFMA_F32_32X32X16_BF16 used throughout (lane l of a wave64):
//   A (32 x 16): lane l holds A[l%32][8*(l/32) + j], j = 0..7
//   B (16 x 32): lane l holds B[8*(l/32) + j][l%32]
//   C (32 x 32): register i of lane l holds C[8*(i/4) + 4*(l/32) + i%4][l%32]
// So lanes l and l+32 share one output column and split its 32 rows between them.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sra {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

typedef bf16x4 __attribute__((address_space(3))) lds_bf16x4;

__device__ __forceinline__ floatx16 mfma32(bf16x8 a, bf16x8 b, floatx16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// acc += A B with the accumulator pinned to AGPRs. For kernels whose accumulators fill the
// AGPR file for their whole run while the VGPRs hold the other MFMA operands and results; the
// compiler sees no MFMA here, so the two wait states cover a VALU write of A or B just
// before, and readers of acc must wait out the MFMA latency themselves.
__device__ __forceinline__ void mfma32_agpr(floatx16& acc, bf16x8 a, bf16x8 b) {
  asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}

// Waits out the latency of MFMAs issued by mfma32_agpr: the compiler does not see those, so
// it inserts no wait states of its own before an accumulator is read. The kernels issue it
// inside their step loop, after the last step, so that no accumulator read (all of which
// follow the loop) can be scheduled above it.
__device__ __forceinline__ void mfma_drain() { asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory"); }

__device__ __forceinline__ bf16x8 ld8(const __bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Combine a value held by lanes l and l^32 (the two halves of one MFMA output column).
__device__ __forceinline__ float pair_max(float x) {
  auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __builtin_elementwise_maximum(__uint_as_float(s[0]), __uint_as_float(s[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

// DS_READ_B64_TR_B16: within each 16-lane group, lane j addresses row j/4, columns
// 4*(j%4)..+3 of a 4 x 16 block of 16-bit values; lane i receives column i (4 rows).
__device__ __forceinline__ bf16x4 lds_read_tr(const __bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p);
}

__device__ __forceinline__ bf16x8 cat8(bf16x4 lo, bf16x4 hi) {
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// IEEE-2019 maximum (V_MAXIMUM3_F32 on gfx950): needs no NaN canonicalisation of MFMA results.
__device__ __forceinline__ float max2f(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float max3f(float a, float b, float c) { return max2f(a, max2f(b, c)); }

// Eight consecutive accumulator registers -> bf16 (round to nearest even).
__device__ __forceinline__ bf16x8 to_bf16x8(const floatx16& v, int base) {
  bf16x8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = (__bf16)v[base + j];
  return r;
}

}  // namespace sra
