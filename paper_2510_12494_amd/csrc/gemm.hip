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
  int M = g.M;
  if (g.ta) {
    M = g.ta->rows;
    if (g.ta_in) A1 += g.ta->row0 * g.lda1;
  }
  if (m0 >= M) return;

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
      if (m < M && k < g.K) {
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
    const int32_t* hv = g.ta ? g.ta->hdr : g.hdr;
    if (g.hdr_out) { g.hdr_out[0] = hv[0]; g.hdr_out[1] = hv[1]; g.hdr_out[2] = hv[2]; }
    if (g.hdr_chk && g.hdr_chk[0] != (g.ta ? g.ta->chk : g.chk_seq)) atomicAdd(g.err, 1);
  }

  T* C1 = (T*)g.C1;
  const T* Mk = (const T*)g.mask;
#pragma unroll
  for (int j = 0; j < BN / 32; ++j) {
#pragma unroll
    for (int i = 0; i < BM / 32; ++i) {
      const int m = m0 + wm * (BM / 2) + i * 16 + (lane & 15);
      const int nb = n0 + wn * (BN / 2) + j * 16 + (lane >> 4) * 4;
      if (m >= M || nb >= g.N) continue;
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

// Weight gradients of several layers in one launch.  Block -> (layer,
// output tile, row chunk).  LDS rows: sQ row n holds D[r][n] for the stage's
// rows, sP row k holds X[r][k]; both are written transposed from row-major
// loads.  An unsplit tile applies SGD in its epilogue and refreshes the
// layer's operand copies; a split tile writes float32 partials for
// k_multi_reduce.
template <typename T>
__device__ __forceinline__ void copy_out(void* Wq, int64_t ldq, void* Wtq, int64_t ldt, int n,
                                         int k, float w) {
  if (Wq) store1<T>((T*)Wq + (int64_t)n * ldq + k, w);
  if (Wtq) store1<T>((T*)Wtq + (int64_t)k * ldt + n, w);
}

template <typename T, int BN, int BK>
__global__ __launch_bounds__(256) void k_multi_dw(MultiDW m) {
  constexpr int CE = 16 / (int)sizeof(T);
  constexpr int RE = 128 / (int)sizeof(T);       // rows per stage
  constexpr int RH = RE / 8;
  constexpr int QC = BN / 32, PC = BK / 32;
  __shared__ __attribute__((aligned(16))) char sQ[BN * 128];
  __shared__ __attribute__((aligned(16))) char sP[BK * 128];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  int q = 0;
#pragma unroll 1
  while (q + 1 < m.n && (int)blockIdx.x >= m.first_block[q + 1]) ++q;
  const GemmDW& g = m.p[q];
  const int lb = blockIdx.x - m.first_block[q];
  const int tiles_k = (g.K + BK - 1) / BK;
  const int tile = lb / g.splits, split = lb % g.splits;
  const int n0 = (tile / tiles_k) * BN, k0 = (tile % tiles_k) * BK;
  const int rows = m.ta ? m.ta->rows : m.R;
  const float scale = m.ta ? m.ta->scale : m.scale;
  const int rb = split * g.rows_per_split;
  const int re = min(rows, rb + g.rows_per_split);
  const T* D = (const T*)g.D;
  const T* X1 = (const T*)g.X1;
  if (g.x_ta) X1 += m.ta->row0 * g.ldx1;
  const T* X2 = (const T*)g.X2;
  const bool do_bias = (tile % tiles_k) == 0;

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
  auto tstore = [&](char* sm, const u32x4& v, int c) {
    const int r = crow(c), col0 = ccol(c) * CE;
    const int off = (r % CE) * (int)sizeof(T);
#pragma unroll
    for (int e = 0; e < CE; ++e) {
      char* ptr = sm + swz(col0 + e, r / CE) + off;
      if constexpr (sizeof(T) == 4) {
        *(uint32_t*)ptr = v[e];
      } else {
        *(uint16_t*)ptr = (uint16_t)((e & 1) ? (v[e >> 1] >> 16) : (v[e >> 1] & 0xffffu));
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
        for (int u = 0; u < 4; ++u) {
          if constexpr (sizeof(T) == 4) accb += __uint_as_float(v[u]);
          else accb += __uint_as_float(v[u] << 16) + __uint_as_float(v[u] & 0xffff0000u);
        }
      }
    }
    mma_stage<T, BK, BN>(sP, sQ, acc, lane, wm, wn);
    __syncthreads();
  }

  if (g.splits == 1) {
    // the block holds the whole row sum: SGD from the accumulators, then the
    // operand copies of the updated weights
#pragma unroll
    for (int j = 0; j < BN / 32; ++j) {
#pragma unroll
      for (int i = 0; i < BK / 32; ++i) {
        const int k = k0 + wm * (BK / 2) + i * 16 + (lane & 15);
        const int nb = n0 + wn * (BN / 2) + j * 16 + (lane >> 4) * 4;
        if (k >= g.K) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = nb + r;
          if (n < g.N) {
            float* wp = g.W + (int64_t)n * g.K + k;
            const float w = *wp - scale * acc[j][i][r];
            *wp = w;
            copy_out<T>(g.Wq, g.ldq, g.Wtq, g.ldt, n, k, w);
          }
        }
      }
    }
    if (do_bias && tid < BN && n0 + tid < g.N) g.bias[n0 + tid] -= scale * accb;
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

// Second stage: sum the split partials of every split layer in split order,
// apply SGD and refresh the operand copies; optionally the logit kernel's
// block partials (loss, logit weight and bias gradients).  Thread ranges:
// [layers' weight quads | layers' bias quads | logit columns].
template <typename T>
__global__ __launch_bounds__(256) void k_multi_reduce(MultiDW m, LogitJob lj, int with_logit) {
  int64_t t = blockIdx.x * (int64_t)256 + threadIdx.x;
  const float scale = m.ta ? m.ta->scale : m.scale;
  for (int q = 0; q < m.n; ++q) {
    const GemmDW& g = m.p[q];
    if (g.splits <= 1) continue;
    const int64_t NK = (int64_t)g.N * g.K;
    const int64_t qw = (NK + 3) / 4, qb = (g.N + 3) / 4;
    if (t >= qw + qb) { t -= qw + qb; continue; }
    const bool is_w = t < qw;
    const float* src = is_w ? g.part : g.partb;
    const int64_t stride = is_w ? NK : g.N;
    const int64_t base = 4 * (is_w ? t : t - qw);
    const int n_el = (int)min((int64_t)4, stride - base);
    float sum[4] = {0.f, 0.f, 0.f, 0.f};
    int s = 0;
    for (; s + 8 <= g.splits; s += 8) {
      float v[8][4];
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) v[u][e] = e < n_el ? src[(s + u) * stride + base + e] : 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) sum[e] += v[u][e];
    }
    for (; s < g.splits; ++s)
#pragma unroll
      for (int e = 0; e < 4; ++e) sum[e] += e < n_el ? src[s * stride + base + e] : 0.f;
    for (int e = 0; e < n_el; ++e) {
      const int64_t idx = base + e;
      if (is_w) {
        const float w = g.W[idx] - scale * sum[e];
        g.W[idx] = w;
        copy_out<T>(g.Wq, g.ldq, g.Wtq, g.ldt, (int)(idx / g.K), (int)(idx % g.K), w);
      } else {
        g.bias[idx] -= scale * sum[e];
      }
    }
    return;
  }
  if (!with_logit) return;
  const int W = lj.Hd + 2;
  if (t >= W) return;
  const int c = (int)t;
  float sum = 0.f;
  int b = 0;
  for (; b + 8 <= lj.blocks; b += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = lj.part[(int64_t)(b + u) * W + c];
#pragma unroll
    for (int u = 0; u < 8; ++u) sum += v[u];
  }
  for (; b < lj.blocks; ++b) sum += lj.part[(int64_t)b * W + c];
  const float ls = lj.ta ? lj.ta->scale : lj.scale;
  if (c == 0) {
    float* lo = lj.ta ? (lj.loss_base ? lj.loss_base + lj.ta->loss_idx : nullptr) : lj.loss_out;
    if (lo) *lo = sum / (float)(lj.ta ? lj.ta->rows : lj.R);
  } else if (c == 1) {
    lj.b[0] -= ls * sum;
  } else {
    lj.w[c - 2] -= ls * sum;
  }
}

template <typename T, int BM, int BN>
hipError_t nt_launch(const GemmNT& g, hipStream_t st) {
  dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM);
  hipLaunchKernelGGL((k_gemm_nt<T, BM, BN>), grid, dim3(256), 0, st, g);
  return hipGetLastError();
}

}  // namespace

int dw_stage_rows(Elt e) { return 128 / elt_size(e); }
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

hipError_t launch_multi_dw(Elt e, MultiDW& m, hipStream_t st) {
  if (m.n <= 0 || m.n > kMaxDw || m.R <= 0) return m.n == 0 ? hipSuccess : hipErrorInvalidValue;
  int blocks = 0;
  for (int q = 0; q < m.n; ++q) {
    m.first_block[q] = blocks;
    blocks += dw_tiles(m.p[q].N, m.p[q].K) * m.p[q].splits;
  }
  m.first_block[m.n] = blocks;
  if (e == BF16) hipLaunchKernelGGL((k_multi_dw<uint16_t, 64, 64>), dim3(blocks), dim3(256), 0, st, m);
  else hipLaunchKernelGGL((k_multi_dw<float, 64, 64>), dim3(blocks), dim3(256), 0, st, m);
  return hipGetLastError();
}

hipError_t launch_multi_reduce(Elt e, const MultiDW& m, const LogitJob* lj, hipStream_t st) {
  int64_t threads = 0;
  for (int q = 0; q < m.n; ++q)
    if (m.p[q].splits > 1)
      threads += ((int64_t)m.p[q].N * m.p[q].K + 3) / 4 + (m.p[q].N + 3) / 4;
  if (lj) threads += lj->Hd + 2;
  if (threads == 0) return hipSuccess;
  LogitJob none{};
  const int blocks = (int)((threads + 255) / 256);
  if (e == BF16)
    hipLaunchKernelGGL(k_multi_reduce<uint16_t>, dim3(blocks), dim3(256), 0, st, m, lj ? *lj : none, lj ? 1 : 0);
  else
    hipLaunchKernelGGL(k_multi_reduce<float>, dim3(blocks), dim3(256), 0, st, m, lj ? *lj : none, lj ? 1 : 0);
  return hipGetLastError();
}

}  // namespace vfl
