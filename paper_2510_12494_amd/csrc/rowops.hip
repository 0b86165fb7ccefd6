// Row-wise kernels of the split-learning step on gfx950: the logit layer +
// binary cross-entropy (Eq. 1) with its gradient, per-row clip + Philox
// Gaussian noise of the exchanged messages, the cut-layer backward of the
// passive party and the weight operand copies.
// One 64-lane wavefront owns one row at a time; row reductions (dot
// products, norms) use cross-lane shuffles.
#include <algorithm>

#include "kernels.h"

namespace vfl {
namespace {

typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T>
__device__ __forceinline__ float ld1(const T* p) {
  if constexpr (sizeof(T) == 4) return *p;
  else return bf2f(*p);
}

template <typename T>
__device__ __forceinline__ void st1(T* p, float v) {
  if constexpr (sizeof(T) == 4) *p = v;
  else *p = f2bf(v);
}

// one 16-byte chunk <-> CE floats
template <typename T>
__device__ __forceinline__ void load8(const T* p, float (&v)[16 / sizeof(T)]) {
  typedef __attribute__((ext_vector_type(4))) uint32_t u4;
  const u4 x = *(const u4*)p;
  if constexpr (sizeof(T) == 4) {
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = __uint_as_float(x[i]);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(x[i] << 16);
      v[2 * i + 1] = __uint_as_float(x[i] & 0xffff0000u);
    }
  }
}

template <typename T>
__device__ __forceinline__ void store8(T* p, const float (&v)[16 / sizeof(T)]) {
  typedef __attribute__((ext_vector_type(4))) uint32_t u4;
  u4 x;
  if constexpr (sizeof(T) == 4) {
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = __float_as_uint(v[i]);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = (uint32_t)f2bf(v[2 * i]) | ((uint32_t)f2bf(v[2 * i + 1]) << 16);
  }
  *(u4*)p = x;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// ---------------------------------------------------------------- logit + BCE
// A row is owned by a group of lpr lanes (a power of two <= 64), each lane
// holding up to two 16-byte chunks of the row, so a wavefront works on
// 64 / lpr rows at once; the dot product is a shuffle reduction inside the
// group.  Block partials are summed by k_multi_reduce.
template <typename T>
__global__ __launch_bounds__(256) void k_logit_bce(LogitJob j) {
  constexpr int CE = 16 / (int)sizeof(T);
  constexpr int MAXC = 2;
  __shared__ float red[256 * CE * MAXC];
  __shared__ float redl[256], redb[256];
  const int nch = (j.Hd + CE - 1) / CE;
  int lpr = 1;
  while (lpr < nch && lpr < 64) lpr <<= 1;
  const int cpl = (nch + lpr - 1) / lpr;
  const int G = 256 / lpr;
  const int grp = threadIdx.x / lpr, li = threadIdx.x % lpr;
  const T* H = (const T*)j.H;
  T* Dl = (T*)j.delta;
  float wv[MAXC][CE], gw[MAXC][CE];
#pragma unroll
  for (int c = 0; c < MAXC; ++c)
#pragma unroll
    for (int e = 0; e < CE; ++e) {
      const int col = (li + c * lpr) * CE + e;
      wv[c][e] = (c < cpl && col < j.Hd) ? j.w[col] : 0.f;
      gw[c][e] = 0.f;
    }
  const float bias = j.b[0];
  float gb = 0.f, lsum = 0.f;
  const int R = j.ta ? j.ta->rows : j.R;
  const float* Y = j.ta ? j.y + j.ta->row0 : j.y;
  const int per = (R + gridDim.x - 1) / gridDim.x;
  const int rb = blockIdx.x * per, re = min(R, rb + per);
  for (int r = rb + grp; r < re; r += G) {
    float h[MAXC][CE];
    float dot = 0.f;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      const int col0 = (li + c * lpr) * CE;
      if (c < cpl && col0 < j.Hd) {
        load8<T>(H + (int64_t)r * j.ldh + col0, h[c]);
#pragma unroll
        for (int e = 0; e < CE; ++e)
          if (col0 + e >= j.Hd) h[c][e] = 0.f;
      } else {
#pragma unroll
        for (int e = 0; e < CE; ++e) h[c][e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < CE; ++e) dot += h[c][e] * wv[c][e];
    }
    for (int o = lpr >> 1; o > 0; o >>= 1) dot += __shfl_xor(dot, o, 64);
    const float l = dot + bias;
    const float y = Y[r];
    const float ex = expf(-fabsf(l));
    const float loss = fmaxf(l, 0.f) - y * l + log1pf(ex);
    const float sig = l >= 0.f ? 1.f / (1.f + ex) : ex / (1.f + ex);
    const float dl = sig - y;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      const int col0 = (li + c * lpr) * CE;
      if (c < cpl && col0 < j.Hd) {
        float d[CE];
#pragma unroll
        for (int e = 0; e < CE; ++e) {
          d[e] = dl * wv[c][e];
          if (j.relu && !(h[c][e] > 0.f)) d[e] = 0.f;
          gw[c][e] += dl * h[c][e];
        }
        store8<T>(Dl + (int64_t)r * j.ldd + col0, d);
      }
    }
    if (li == 0) { gb += dl; lsum += loss; }
  }
#pragma unroll
  for (int c = 0; c < MAXC; ++c)
#pragma unroll
    for (int e = 0; e < CE; ++e) {
      const int col = (li + c * lpr) * CE + e;
      if (c < cpl && col < j.Hd) red[grp * j.Hd + col] = gw[c][e];
    }
  if (li == 0) { redl[grp] = lsum; redb[grp] = gb; }
  __syncthreads();
  const int W = j.Hd + 2;
  for (int col = threadIdx.x; col < j.Hd; col += 256) {
    float acc = 0.f;
    for (int g = 0; g < G; ++g) acc += red[g * j.Hd + col];
    j.part[(int64_t)blockIdx.x * W + 2 + col] = acc;
  }
  if (threadIdx.x == 0) {
    float a = 0.f, b2 = 0.f;
    for (int g = 0; g < G; ++g) { a += redl[g]; b2 += redb[g]; }
    j.part[(int64_t)blockIdx.x * W] = a;
    j.part[(int64_t)blockIdx.x * W + 1] = b2;
  }
}

// ---------------------------------------------------- Philox4x32-10 + noise
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

// four standard normals for columns 4q .. 4q+3 of (step, row, tag)
__device__ __forceinline__ void gauss4(uint64_t seed, uint32_t step, uint32_t row, uint32_t q,
                                       uint32_t tag, float (&n)[4]) {
  uint32_t c[4] = {step, row, q, tag};
  philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const float ua = word_uniform(c[2 * p]), ub = word_uniform(c[2 * p + 1]);
    const float rad = sqrtf(-2.f * logf(ua));
    float s, co;
    sincospif(2.f * ub, &s, &co);
    n[2 * p] = rad * co;
    n[2 * p + 1] = rad * s;
  }
}

__device__ __forceinline__ uint32_t global_row(const RowMap& m, int r) {
  int s = 0;
#pragma unroll
  for (int i = 1; i < 8; ++i)
    if (i < m.n && r >= m.start[i]) s = i;
  return (uint32_t)(m.row0[s] + (r - m.start[s]));
}

template <typename T, typename V>
__global__ __launch_bounds__(256) void k_clip_noise(ClipNoiseJob j) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (j.ta) {
    j.R = j.ta->rows;
    j.step = (uint32_t)j.ta->group;
    j.rows.n = 1;
    j.rows.start[0] = 0;
    j.rows.row0[0] = j.ta->row0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0 && j.hdr_out) {
    const int32_t* hv = j.ta ? j.ta->hdr : j.hdr;
    j.hdr_out[0] = hv[0]; j.hdr_out[1] = hv[1]; j.hdr_out[2] = hv[2];
  }
  const V* v = (const V*)j.v;
  T* out = (T*)j.out;
  const int ngrp = (j.D + 3) >> 2;
  for (int r = blockIdx.x * 4 + wave; r < j.R; r += gridDim.x * 4) {
    float ss = 0.f;
    for (int g = lane; g < ngrp; g += 64) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = 4 * g + e;
        if (c < j.D) { const float x = ld1<V>(v + (int64_t)r * j.ldv + c); ss += x * x; }
      }
    }
    const float n = sqrtf(wave_sum(ss));
    const float cf = (j.clip && n > j.C) ? j.C / n : 1.f;
    if (lane == 0) {
      if (j.norm) j.norm[r] = n;
      if (j.cfac) j.cfac[r] = cf;
    }
    const uint32_t grow = j.noise ? global_row(j.rows, r) : 0u;
    for (int g = lane; g < ngrp; g += 64) {
      float xi[4] = {0.f, 0.f, 0.f, 0.f};
      if (j.noise) gauss4(j.seed, j.step, grow, (uint32_t)g, j.tag, xi);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = 4 * g + e;
        if (c < j.D) {
          const float x = ld1<V>(v + (int64_t)r * j.ldv + c);
          st1<T>(out + (int64_t)r * j.ldo + c, cf * x + j.stdv * xi[e]);
        }
      }
    }
  }
}

__global__ __launch_bounds__(256) void k_philox_words(uint64_t seed, uint32_t step, uint32_t tag,
                                                      uint32_t row0, int rows, int groups,
                                                      uint32_t* out) {
  const int64_t total = (int64_t)rows * groups;
  for (int64_t i = blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int q = (int)(i % groups);
    const uint32_t row = row0 + (uint32_t)(i / groups);
    uint32_t c[4] = {step, row, (uint32_t)q, tag};
    philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
#pragma unroll
    for (int k = 0; k < 4; ++k) out[4 * i + k] = c[k];
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_cut_backward(CutBwdJob j) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (j.ta) {
    j.R = j.ta->rows;
    j.chk_seq = j.ta->chk;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0 && j.hdr_chk && j.hdr_chk[0] != j.chk_seq)
    atomicAdd(j.err, 1);
  const T* G = (const T*)j.g;
  const T* Z = (const T*)j.z;
  T* Dl = (T*)j.delta;
  for (int r = blockIdx.x * 4 + wave; r < j.R; r += gridDim.x * 4) {
    const bool clipped = j.clip && j.norm[r] > j.C;
    float dot = 0.f, inv = 0.f, cf = 1.f;
    if (clipped) {
      inv = 1.f / j.norm[r];
      cf = j.cfac[r];
      for (int c = lane; c < j.D; c += 64)
        dot += ld1<T>(Z + (int64_t)r * j.ldz + c) * inv * ld1<T>(G + (int64_t)r * j.ldg + c);
      dot = wave_sum(dot);
    }
    for (int c = lane; c < j.D; c += 64) {
      const float z = ld1<T>(Z + (int64_t)r * j.ldz + c);
      float g = ld1<T>(G + (int64_t)r * j.ldg + c);
      if (clipped) g = cf * (g - z * inv * dot);
      if (j.relu && !(z > 0.f)) g = 0.f;
      st1<T>(Dl + (int64_t)r * j.ldd + c, g);
    }
  }
}

// ------------------------------------------------------------ weight copies
struct CastJobs { CastJob j[2 * 8 + 2]; int n; };

template <typename T>
__global__ __launch_bounds__(256) void k_cast(CastJobs js) {
  const CastJob& j = js.j[blockIdx.y];
  const int64_t total = (int64_t)j.out * j.in;
  T* Wq = (T*)j.Wq;
  T* Wt = (T*)j.Wtq;
  for (int64_t i = blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int o = (int)(i / j.in), k = (int)(i % j.in);
    const float w = j.W[i];
    st1<T>(Wq + (int64_t)o * j.ldq + k, w);
    st1<T>(Wt + (int64_t)k * j.ldt + o, w);
  }
}

__device__ void fill_tick(const AdvanceJob& j, TickArgs* o, int64_t g) {
  const int64_t E = (j.n_rows + j.R - 1) / j.R;
  const int64_t start = (g % E) * j.R;
  const int64_t rows = j.n_rows - start < j.R ? j.n_rows - start : j.R;
  o->rows = (int32_t)rows;
  o->group = (int32_t)g;
  o->row0 = start;
  o->scale = j.lr / (float)rows;
  o->loss_idx = g % j.loss_len;
  o->chk = (int32_t)g;
}

__global__ void k_advance(AdvanceJob j) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const int64_t t = *j.counter;
  *j.counter = t + 1;
  const int64_t u = t - j.s;
  if (j.kind == 0) {
    // party A consumes group u and writes the header of its gradient slot
    fill_tick(j, j.out[0], u);
    j.out[0]->hdr[0] = (int32_t)u;
    j.out[0]->hdr[1] = (int32_t)t;
    j.out[0]->hdr[2] = (int32_t)(u - j.s > 0 ? u - j.s : 0);
  } else {
    // party B publishes group t (version max(0, t - s)) and back-propagates u
    fill_tick(j, j.out[0], t);
    j.out[0]->hdr[0] = (int32_t)t;
    j.out[0]->hdr[1] = (int32_t)t;
    j.out[0]->hdr[2] = (int32_t)(t - j.s > 0 ? t - j.s : 0);
    fill_tick(j, j.out[1], u);
  }
}

int grid_for(int64_t work, int per_block, int cap) {
  return (int)std::max<int64_t>(1, std::min<int64_t>((work + per_block - 1) / per_block, cap));
}

}  // namespace

hipError_t launch_logit_bce(Elt e, const LogitJob& j, hipStream_t st) {
  if (j.Hd > kMaxLogitCols) return hipErrorInvalidValue;
  if (e == BF16) hipLaunchKernelGGL(k_logit_bce<uint16_t>, dim3(j.blocks), dim3(256), 0, st, j);
  else hipLaunchKernelGGL(k_logit_bce<float>, dim3(j.blocks), dim3(256), 0, st, j);
  return hipGetLastError();
}

hipError_t launch_advance(const AdvanceJob& j, hipStream_t st) {
  hipLaunchKernelGGL(k_advance, dim3(1), dim3(64), 0, st, j);
  return hipGetLastError();
}

hipError_t launch_philox_words(uint64_t seed, uint32_t step, uint32_t tag, uint32_t row0,
                               int rows, int groups, uint32_t* out, hipStream_t st) {
  const int64_t total = (int64_t)rows * groups;
  hipLaunchKernelGGL(k_philox_words, dim3(grid_for(total, 256, 4096)), dim3(256), 0, st, seed,
                     step, tag, row0, rows, groups, out);
  return hipGetLastError();
}

hipError_t launch_clip_noise(Elt e, const ClipNoiseJob& j, hipStream_t st) {
  const int blocks = grid_for(j.R, 4, 4096);
  if (e == BF16) {
    if (j.v_f32) hipLaunchKernelGGL((k_clip_noise<uint16_t, float>), dim3(blocks), dim3(256), 0, st, j);
    else hipLaunchKernelGGL((k_clip_noise<uint16_t, uint16_t>), dim3(blocks), dim3(256), 0, st, j);
  } else {
    hipLaunchKernelGGL((k_clip_noise<float, float>), dim3(blocks), dim3(256), 0, st, j);
  }
  return hipGetLastError();
}

hipError_t launch_cut_backward(Elt e, const CutBwdJob& j, hipStream_t st) {
  const int blocks = grid_for(j.R, 4, 4096);
  if (e == BF16) hipLaunchKernelGGL(k_cut_backward<uint16_t>, dim3(blocks), dim3(256), 0, st, j);
  else hipLaunchKernelGGL(k_cut_backward<float>, dim3(blocks), dim3(256), 0, st, j);
  return hipGetLastError();
}

hipError_t launch_cast(Elt e, const CastJob* jobs, int n_jobs, hipStream_t st) {
  if (n_jobs <= 0) return hipSuccess;
  CastJobs js;
  if (n_jobs > (int)(sizeof(js.j) / sizeof(js.j[0]))) return hipErrorInvalidValue;
  int64_t maxw = 0;
  for (int i = 0; i < n_jobs; ++i) {
    js.j[i] = jobs[i];
    maxw = std::max<int64_t>(maxw, (int64_t)jobs[i].out * jobs[i].in);
  }
  js.n = n_jobs;
  dim3 grid(grid_for(maxw, 256, 1024), n_jobs);
  if (e == BF16) hipLaunchKernelGGL(k_cast<uint16_t>, grid, dim3(256), 0, st, js);
  else hipLaunchKernelGGL(k_cast<float>, grid, dim3(256), 0, st, js);
  return hipGetLastError();
}

}  // namespace vfl
