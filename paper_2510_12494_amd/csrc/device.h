// Device helpers shared by the gfx950 kernel files: vector types, bf16
// conversion, element loads/stores, wavefront reductions, the Philox4x32-10
// counter generator with its Box-Muller Gaussian pairs, and register
// transposes between row-major tiles and the row-chunked (RC) layout.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vfl {
namespace dev {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

// Global-memory view of a pointer read from a job descriptor: without it
// the compiler emits flat accesses, which wait on both the vector-memory and
// the LDS counters and so serialise loads with LDS work.
#define VFL_GLOBAL __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ VFL_GLOBAL T* glb(T* p) { return (VFL_GLOBAL T*)p; }
template <typename T>
__device__ __forceinline__ const VFL_GLOBAL T* glb(const T* p) { return (const VFL_GLOBAL T*)p; }

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// two floats -> packed bf16 (low half first), round to nearest even: one
// v_cvt_pk_bf16_f32 on gfx950
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){a, b}, bf16x2));
}

template <typename T>
__device__ __forceinline__ float ld1(const T* p) {
  if constexpr (sizeof(T) == 4) return *p;
  else return bf2f(*p);
}

template <typename T>
__device__ __forceinline__ void st1(T* p, float v) {
  if constexpr (sizeof(T) == 4) *p = v;
  else *p = (uint16_t)pack_bf16(v, 0.f);
}

// four consecutive elements (8 bytes of bf16 or 16 bytes of float32)
template <typename T>
__device__ __forceinline__ void ld4(const void* p, float (&v)[4]) {
  if constexpr (sizeof(T) == 4) {
    const f32x4 x = *(const f32x4*)p;
    v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
  } else {
    const u32x2 x = *(const u32x2*)p;
    v[0] = __uint_as_float(x[0] << 16); v[1] = __uint_as_float(x[0] & 0xffff0000u);
    v[2] = __uint_as_float(x[1] << 16); v[3] = __uint_as_float(x[1] & 0xffff0000u);
  }
}

template <typename T>
__device__ __forceinline__ void st4(void* p, const float (&v)[4]) {
  if constexpr (sizeof(T) == 4) {
    *(f32x4*)p = f32x4{v[0], v[1], v[2], v[3]};
  } else {
    u32x2 x;
    x[0] = pack_bf16(v[0], v[1]);
    x[1] = pack_bf16(v[2], v[3]);
    *(u32x2*)p = x;
  }
}

// zero the elements of a 16-byte chunk at and beyond `valid`
template <typename T>
__device__ __forceinline__ u32x4 mask_tail(u32x4 v, int valid) {
  constexpr int CE = 16 / sizeof(T);
  if (valid >= CE) return v;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if constexpr (sizeof(T) == 4) {
      if (i >= valid) v[i] = 0u;
    } else {
      if (2 * i >= valid) v[i] = 0u;
      else if (2 * i + 1 >= valid) v[i] &= 0xffffu;
    }
  }
  return v;
}

// Packed MFMA operand of a chain product [N x K]: stored fragment by
// fragment, fragment (tile, ks) = rows 16*tile .. +16, columns KS*ks .. +KS
// (KS = 4 * CE: one MFMA step), lane l holding row 16*tile + l % 16 and
// columns KS*ks + CE*(l / 16) .. +CE in 16 bytes, fragments of a tile
// consecutive in ks; kst = steps per tile.  A wavefront's fragment load is
// then one contiguous 1 KB block.  Element index of (n, k):
template <typename T>
__device__ __forceinline__ int64_t pk_index(int n, int k, int kst) {
  constexpr int CE = 16 / (int)sizeof(T), KS = 4 * CE;
  const int lane = (n & 15) + 16 * ((k % KS) / CE);
  return ((((int64_t)(n >> 4) * kst + k / KS) * 64 + lane) * CE) + k % CE;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Philox4x32-10 (Salmon et al., SC'11): 10 rounds of the 4x32 bijection
// with Weyl-sequence key increments.
__device__ __forceinline__ void philox4x32_10(uint32_t (&c)[4], uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    const uint32_t hi0 = __umulhi(0xD2511F53u, c[0]), lo0 = 0xD2511F53u * c[0];
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c[2]), lo1 = 0xCD9E8D57u * c[2];
    const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0; c[1] = lo1; c[2] = n2; c[3] = lo0;
  }
}

__device__ __forceinline__ float word_uniform(uint32_t w) {  // (0, 1], exact
  return (float)((w >> 8) + 1u) * 5.9604644775390625e-8f;
}

// four standard normals for columns 4q .. 4q+3 of (step, row, tag):
// Box-Muller on the word pairs (0, 1) and (2, 3) of one Philox block, with
// the hardware's single-instruction transcendentals: -2 ln u = -2 ln 2 *
// log2 u (v_log_f32), v_sqrt_f32, and v_sin_f32 / v_cos_f32, whose argument
// is in revolutions, so sin(2 pi u) is one instruction
__device__ __forceinline__ void gauss4(uint64_t seed, uint32_t step, uint32_t row, uint32_t q,
                                       uint32_t tag, float (&n)[4]) {
  uint32_t c[4] = {step, row, q, tag};
  philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const float ua = word_uniform(c[2 * p]), ub = word_uniform(c[2 * p + 1]);
    const float rad = __builtin_amdgcn_sqrtf(-1.3862943611198906f * __builtin_amdgcn_logf(ua));
    n[2 * p] = rad * __builtin_amdgcn_cosf(ub);
    n[2 * p + 1] = rad * __builtin_amdgcn_sinf(ub);
  }
}

// 8 x 8 transpose of 16-bit elements: in[i] holds row i (columns 0..7, two
// per word, low half first); out[j] receives column j (rows 0..7).
__device__ __forceinline__ void transpose8x8_u16(const u32x4 (&in)[8], u32x4 (&out)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t a = in[2 * w][j >> 1], b = in[2 * w + 1][j >> 1];
      out[j][w] = (j & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
    }
  }
}

// 4 x 4 transpose of 32-bit elements
__device__ __forceinline__ void transpose4x4_u32(const u32x4 (&in)[4], u32x4 (&out)[4]) {
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) out[j][i] = in[i][j];
}

}  // namespace dev
}  // namespace vfl
