// MFMA matrix products of the split-learning step on gfx950.
//
// Every dense layer of the bottom and top models is y = x W^T + b (W stored
// [out x in]).  Forward, input-gradient and weight-gradient products are the
// three contractions of that layer:
//   forward  Y  = act(X W^T + b)              "NT": both operands K-contiguous
//   input    dX = (dY W) * relu'(X)            NT against the transposed
//                                              weight copy W^T [in x out]
//   weight   dW = dY^T X, db = colsum(dY)      reduction over rows: both
//                                              operands are transposed while
//                                              staged through LDS; the SGD
//                                              step is fused into it
// Tiles: 256 threads = 4 wavefronts in a 2 x 2 grid, each wavefront owning a
// (BM/2) x (BN/2) block of 16 x 16 MFMA tiles (v_mfma_f32_16x16x32_bf16 for
// bf16 operands, v_mfma_f32_16x16x4_f32 for float32), float32 accumulation.
// LDS holds one 128-byte K stage per operand row; 16-byte chunks of a row
// are XOR-swizzled by the row index so that both the MFMA fragment reads
// (16 rows, same chunk) and the transposing writes of the weight-gradient
// kernel (8 rows 8 apart, same chunk) hit distinct banks.
#include "kernels.h"

namespace vfl {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

// byte offset of 16-byte chunk `ch` (0..7) of LDS row `row` (128-byte rows)
__device__ __forceinline__ int swz(int row, int ch) {
  return row * 128 + ((ch ^ (row & 7) ^ ((row >> 3) & 7)) << 4);
}

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {  // round to nearest even
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
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

template <typename T, int BM, int BN>
__device__ __forceinline__ void mma_stage(const char* sP, const char* sQ,
                                          f32x4 (&acc)[BN / 32][BM / 32], int lane,
                                          int wm, int wn) {
  constexpr int TM = BM / 32, TN = BN / 32;
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const int ch = ks * 4 + (lane >> 4);
    u32x4 pf[TM], qf[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
      pf[i] = *(const u32x4*)(sP + swz(wm * (BM / 2) + i * 16 + (lane & 15), ch));
#pragma unroll
    for (int j = 0; j < TN; ++j)
      qf[j] = *(const u32x4*)(sQ + swz(wn * (BN / 2) + j * 16 + (lane & 15), ch));
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        if constexpr (sizeof(T) == 2) {
          acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, qf[j]), __builtin_bit_cast(bf16x8, pf[i]),
              acc[j][i], 0, 0, 0);
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                __uint_as_float(qf[j][q]), __uint_as_float(pf[i][q]), acc[j][i], 0, 0, 0);
        }
      }
    }
  }
}

template <typename T>
__device__ __forceinline__ void load4(const T* p, float (&v)[4]) {
  if constexpr (sizeof(T) == 4) {
    f32x4 x = *(const f32x4*)p;
    v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
  } else {
    u32x2 x = *(const u32x2*)p;
    v[0] = __uint_as_float(x[0] << 16); v[1] = __uint_as_float(x[0] & 0xffff0000u);
    v[2] = __uint_as_float(x[1] << 16); v[3] = __uint_as_float(x[1] & 0xffff0000u);
  }
}

template <typename T>
__device__ __forceinline__ void store4(T* p, const float (&v)[4]) {
  if constexpr (sizeof(T) == 4) {
    *(f32x4*)p = f32x4{v[0], v[1], v[2], v[3]};
  } else {
    u32x2 x;
    x[0] = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
    x[1] = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
    *(u32x2*)p = x;
  }
}

template <typename T>
__device__ __forceinline__ float load1(const T* p) {
  if constexpr (sizeof(T) == 4) return *p;
  else return bf2f(*p);
}

template <typename T>
__device__ __forceinline__ void store1(T* p, float v) {
  if constexpr (sizeof(T) == 4) *p = v;
  else *p = f2bf(v);
}

template <typename T, int BM, int BN>
__global__ __launch_bounds__(256) void k_gemm_nt(GemmNT g) {
  constexpr int CE = 16 / (int)sizeof(T);
  constexpr int KE = 128 / (int)sizeof(T);
  constexpr int PC = BM / 32, QC = BN / 32;   // 16-byte chunks per thread
  __shared__ __attribute__((aligned(16))) char sP[BM * 128];
  __shared__ __attribute__((aligned(16))) char sQ[BN * 128];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM;
  const T* A1 = (const T*)g.A1;
  const T* A2 = (const T*)g.A2;
  const T* Bm = (const T*)g.B;

  f32x4 acc[BN / 32][BM / 32];
#pragma unroll
  for (int j = 0; j < BN / 32; ++j)
#pragma unroll
    for (int i = 0; i < BM / 32; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 rp[PC], rq[QC];
  auto gload = [&](int k0) {
#pragma unroll
    for (int j = 0; j < PC; ++j) {
      const int c = tid + 256 * j, row = c >> 3, ch = c & 7;
      const int m = m0 + row, k = k0 + ch * CE;
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (m < g.M && k < g.K) {
        const T* src = k < g.ksplit ? A1 + (int64_t)m * g.lda1 + k
                                    : A2 + (int64_t)m * g.lda2 + (k - g.ksplit);
        v = mask_tail<T>(*(const u32x4*)src, g.K - k);
      }
      rp[j] = v;
    }
#pragma unroll
    for (int j = 0; j < QC; ++j) {
      const int c = tid + 256 * j, row = c >> 3, ch = c & 7;
      const int n = n0 + row, k = k0 + ch * CE;
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (n < g.N && k < g.K) v = mask_tail<T>(*(const u32x4*)(Bm + (int64_t)n * g.ldb + k), g.K - k);
      rq[j] = v;
    }
  };
  auto lstore = [&]() {
#pragma unroll
    for (int j = 0; j < PC; ++j) {
      const int c = tid + 256 * j;
      *(u32x4*)(sP + swz(c >> 3, c & 7)) = rp[j];
    }
#pragma unroll
    for (int j = 0; j < QC; ++j) {
      const int c = tid + 256 * j;
      *(u32x4*)(sQ + swz(c >> 3, c & 7)) = rq[j];
    }
  };

  const int nk = (g.K + KE - 1) / KE;
  gload(0);
  for (int kt = 0; kt < nk; ++kt) {
    lstore();
    __syncthreads();
    if (kt + 1 < nk) gload((kt + 1) * KE);
    mma_stage<T, BM, BN>(sP, sQ, acc, lane, wm, wn);
    __syncthreads();
  }

  if (blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) {
    if (g.hdr_out) { g.hdr_out[0] = g.hdr[0]; g.hdr_out[1] = g.hdr[1]; g.hdr_out[2] = g.hdr[2]; }
    if (g.hdr_chk && g.hdr_chk[0] != g.chk_seq) atomicAdd(g.err, 1);
  }

  T* C1 = (T*)g.C1;
  const T* Mk = (const T*)g.mask;
#pragma unroll
  for (int j = 0; j < BN / 32; ++j) {
#pragma unroll
    for (int i = 0; i < BM / 32; ++i) {
      const int m = m0 + wm * (BM / 2) + i * 16 + (lane & 15);
      const int nb = n0 + wn * (BN / 2) + j * 16 + (lane >> 4) * 4;
      if (m >= g.M || nb >= g.N) continue;
      float v[4] = {acc[j][i][0], acc[j][i][1], acc[j][i][2], acc[j][i][3]};
      const bool full = nb + 4 <= g.N && (nb + 4 <= g.nsplit || nb >= g.nsplit);
      if (full) {
        if (g.bias) {
          f32x4 b = *(const f32x4*)(g.bias + nb);
          v[0] += b[0]; v[1] += b[1]; v[2] += b[2]; v[3] += b[3];
        }
        if (g.relu) {
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] = fmaxf(v[r], 0.f);
        }
        if (nb < g.nsplit) {
          if (Mk) {
            float mk[4];
            load4<T>(Mk + (int64_t)m * g.ldm + nb, mk);
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = mk[r] > 0.f ? v[r] : 0.f;
          }
          store4<T>(C1 + (int64_t)m * g.ldc1 + nb, v);
        } else if (g.c2_f32) {
          store4<float>((float*)g.C2 + (int64_t)m * g.ldc2 + (nb - g.nsplit), v);
        } else {
          store4<T>((T*)g.C2 + (int64_t)m * g.ldc2 + (nb - g.nsplit), v);
        }
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = nb + r;
          if (n >= g.N) break;
          float x = v[r];
          if (g.bias) x += g.bias[n];
          if (g.relu) x = fmaxf(x, 0.f);
          if (n < g.nsplit) {
            if (Mk && !(load1<T>(Mk + (int64_t)m * g.ldm + n) > 0.f)) x = 0.f;
            store1<T>(C1 + (int64_t)m * g.ldc1 + n, x);
          } else if (g.c2_f32) {
            ((float*)g.C2)[(int64_t)m * g.ldc2 + (n - g.nsplit)] = x;
          } else {
            store1<T>((T*)g.C2 + (int64_t)m * g.ldc2 + (n - g.nsplit), x);
          }
        }
      }
    }
  }
}

// Weight gradient.  LDS rows: sQ row n holds D[r][n] for the stage's rows,
// sP row k holds X[r][k]; both are written transposed from row-major loads.
template <typename T, int BN, int BK>
__global__ __launch_bounds__(256) void k_gemm_dw(GemmDW g) {
  constexpr int CE = 16 / (int)sizeof(T);
  constexpr int RE = 128 / (int)sizeof(T);       // rows per stage
  constexpr int RH = RE / 8;
  constexpr int QC = BN / 32, PC = BK / 32;
  __shared__ __attribute__((aligned(16))) char sQ[BN * 128];
  __shared__ __attribute__((aligned(16))) char sP[BK * 128];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int tiles_k = (g.K + BK - 1) / BK;
  const int n0 = (blockIdx.x / tiles_k) * BN, k0 = (blockIdx.x % tiles_k) * BK;
  const int split = blockIdx.y;
  const int rb = split * g.rows_per_split;
  const int re = min(g.R, rb + g.rows_per_split);
  const T* D = (const T*)g.D;
  const T* X1 = (const T*)g.X1;
  const T* X2 = (const T*)g.X2;
  const bool do_bias = g.partb && (blockIdx.x % tiles_k) == 0;

  f32x4 acc[BN / 32][BK / 32];
#pragma unroll
  for (int j = 0; j < BN / 32; ++j)
#pragma unroll
    for (int i = 0; i < BK / 32; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float accb = 0.f;

  u32x4 rq[QC], rp[PC];
  // chunk c -> (row r in stage, chunk column); 8 rows x 8 chunks per wavefront
  auto crow = [](int c) { return (c & 7) | (((c >> 6) % RH) << 3); };
  auto ccol = [](int c) { return ((c >> 3) & 7) | (((c >> 6) / RH) << 3); };
  auto gload = [&](int r0) {
#pragma unroll
    for (int j = 0; j < QC; ++j) {
      const int c = tid + 256 * j, r = r0 + crow(c), n = n0 + ccol(c) * CE;
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (r < re && n < g.N) v = mask_tail<T>(*(const u32x4*)(D + (int64_t)r * g.ldd + n), g.N - n);
      rq[j] = v;
    }
#pragma unroll
    for (int j = 0; j < PC; ++j) {
      const int c = tid + 256 * j, r = r0 + crow(c), k = k0 + ccol(c) * CE;
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (r < re && k < g.K) {
        const T* src = k < g.ksplit ? X1 + (int64_t)r * g.ldx1 + k
                                    : X2 + (int64_t)r * g.ldx2 + (k - g.ksplit);
        v = mask_tail<T>(*(const u32x4*)src, g.K - k);
      }
      rp[j] = v;
    }
  };
  auto tstore = [&](char* s, const u32x4& v, int c) {
    const int r = crow(c), col0 = ccol(c) * CE;
    const int off = (r % CE) * (int)sizeof(T);
#pragma unroll
    for (int e = 0; e < CE; ++e) {
      char* p = s + swz(col0 + e, r / CE) + off;
      if constexpr (sizeof(T) == 4) {
        *(uint32_t*)p = v[e];
      } else {
        *(uint16_t*)p = (uint16_t)((e & 1) ? (v[e >> 1] >> 16) : (v[e >> 1] & 0xffffu));
      }
    }
  };

  gload(rb);
  for (int r0 = rb; r0 < re; r0 += RE) {
#pragma unroll
    for (int j = 0; j < QC; ++j) tstore(sQ, rq[j], tid + 256 * j);
#pragma unroll
    for (int j = 0; j < PC; ++j) tstore(sP, rp[j], tid + 256 * j);
    __syncthreads();
    if (r0 + RE < re) gload(r0 + RE);
    if (do_bias && tid < BN) {
#pragma unroll
      for (int ch = 0; ch < 8; ++ch) {
        u32x4 v = *(const u32x4*)(sQ + swz(tid, ch));
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if constexpr (sizeof(T) == 4) accb += __uint_as_float(v[q]);
          else accb += __uint_as_float(v[q] << 16) + __uint_as_float(v[q] & 0xffff0000u);
        }
      }
    }
    mma_stage<T, BK, BN>(sP, sQ, acc, lane, wm, wn);
    __syncthreads();
  }

  if (g.splits == 1) {
    // the block holds the whole row sum: SGD straight from the accumulators
#pragma unroll
    for (int j = 0; j < BN / 32; ++j) {
#pragma unroll
      for (int i = 0; i < BK / 32; ++i) {
        const int k = k0 + wm * (BK / 2) + i * 16 + (lane & 15);
        const int nb = n0 + wn * (BN / 2) + j * 16 + (lane >> 4) * 4;
        if (k >= g.K) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (nb + r < g.N) g.W[(int64_t)(nb + r) * g.K + k] -= g.scale * acc[j][i][r];
      }
    }
    if (do_bias && tid < BN && n0 + tid < g.N) g.bias[n0 + tid] -= g.scale * accb;
    return;
  }
  float* part = g.part + (int64_t)split * g.N * g.K;
#pragma unroll
  for (int j = 0; j < BN / 32; ++j) {
#pragma unroll
    for (int i = 0; i < BK / 32; ++i) {
      const int k = k0 + wm * (BK / 2) + i * 16 + (lane & 15);
      const int nb = n0 + wn * (BN / 2) + j * 16 + (lane >> 4) * 4;
      if (k >= g.K) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (nb + r < g.N) part[(int64_t)(nb + r) * g.K + k] = acc[j][i][r];
    }
  }
  if (do_bias && tid < BN && n0 + tid < g.N) g.partb[(int64_t)split * g.N + n0 + tid] = accb;
}

// Sum of the split partials in split order + SGD: four consecutive
// elements per thread (weights first, then bias), eight splits' loads in
// flight at a time.
__global__ __launch_bounds__(256) void k_dw_reduce(GemmDW g) {
  const int64_t NK = (int64_t)g.N * g.K;
  const int64_t qw = (NK + 3) / 4, qb = (g.N + 3) / 4;
  const int64_t t = blockIdx.x * (int64_t)256 + threadIdx.x;
  if (t >= qw + qb) return;
  const bool is_w = t < qw;
  const float* src = is_w ? g.part : g.partb;
  const int64_t stride = is_w ? NK : g.N;
  const int64_t base = 4 * (is_w ? t : t - qw);
  float* dst = (is_w ? g.W : g.bias) + base;
  const int n = (int)std::min<int64_t>(4, stride - base);
  float sum[4] = {0.f, 0.f, 0.f, 0.f};
  int q = 0;
  for (; q + 8 <= g.splits; q += 8) {
    float v[8][4];
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) v[u][e] = e < n ? src[(q + u) * stride + base + e] : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) sum[e] += v[u][e];
  }
  for (; q < g.splits; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) sum[e] += e < n ? src[q * stride + base + e] : 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (e < n) dst[e] -= g.scale * sum[e];
}

template <typename T, int BM, int BN>
hipError_t nt_launch(const GemmNT& g, hipStream_t st) {
  dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM);
  hipLaunchKernelGGL((k_gemm_nt<T, BM, BN>), grid, dim3(256), 0, st, g);
  return hipGetLastError();
}

template <typename T, int BN, int BK>
hipError_t dw_launch(const GemmDW& g, hipStream_t st) {
  dim3 grid(((g.N + BN - 1) / BN) * ((g.K + BK - 1) / BK), g.splits);
  hipLaunchKernelGGL((k_gemm_dw<T, BN, BK>), grid, dim3(256), 0, st, g);
  return hipGetLastError();
}

}  // namespace

int dw_stage_rows(Elt e) { return 128 / elt_size(e); }
int dw_tile(Elt) { return 64; }
int dw_tiles(int N, int K) { return ((N + 63) / 64) * ((K + 63) / 64); }

hipError_t launch_gemm_nt(Elt e, const GemmNT& g, hipStream_t st) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  const int64_t big = (int64_t)((g.M + 127) / 128) * ((g.N + 127) / 128);
  if (e == BF16) {
    if (big >= 512) return nt_launch<uint16_t, 128, 128>(g, st);
    return nt_launch<uint16_t, 64, 64>(g, st);
  }
  if (big >= 512) return nt_launch<float, 128, 128>(g, st);
  return nt_launch<float, 64, 64>(g, st);
}

hipError_t launch_dw_reduce(const GemmDW& g, hipStream_t st) {
  if (g.splits <= 1 || g.N <= 0 || g.K <= 0) return hipSuccess;
  const int64_t quads = ((int64_t)g.N * g.K + 3) / 4 + (g.N + 3) / 4;
  hipLaunchKernelGGL(k_dw_reduce, dim3((unsigned)((quads + 255) / 256)), dim3(256), 0, st, g);
  return hipGetLastError();
}

hipError_t launch_gemm_dw(Elt e, const GemmDW& g, hipStream_t st) {
  if (g.N <= 0 || g.K <= 0 || g.splits <= 0) return hipSuccess;
  if (e == BF16) return dw_launch<uint16_t, 64, 64>(g, st);
  return dw_launch<float, 64, 64>(g, st);
}

}  // namespace vfl
