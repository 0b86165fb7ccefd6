// Small kernels of the split-learning step on gfx950: the weight operand
// copies, the replicas' parameter averaging, the tick base of a replayed
// graph, and the raw Philox4x32-10 words of the noise generator.
#include <algorithm>

#include "device.h"
#include "kernels.h"

namespace vfl {
namespace {

using namespace dev;

// ------------------------------------------------------------ weight copies
struct CastJobs { CastJob j[2 * kMaxChain + 2]; int n; };

template <typename T>
__global__ __launch_bounds__(256) void k_cast(CastJobs js) {
  const CastJob& j = js.j[blockIdx.y];
  const int64_t total = (int64_t)j.out * j.in;
  T* Wq = (T*)j.Wq;
  T* Wt = (T*)j.Wtq;
  for (int64_t i = blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int o = (int)(i / j.in), k = (int)(i % j.in);
    const float w = j.W[i];
    st1<T>(Wq + pk_index<T>(o, k, j.kq), w);
    st1<T>(Wt + pk_index<T>(k, o, j.kt), w);
  }
}

__global__ void k_tick_base(TickSrc* src, int cyc) {
  if (threadIdx.x == 0 && blockIdx.x == 0) src->base += cyc;
}

__global__ void k_tick_set(TickSrc* dst, TickSrc v) {
  if (threadIdx.x == 0 && blockIdx.x == 0) *dst = v;
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

// ------------------------------------------------------- replica averaging
// One thread per float4 unit of the segment list (a scalar tail where a
// segment's length is not a multiple of 4): loads the unit from all N sets,
// forms the weighted sum in a fixed order and writes it to every set.
template <int N>
__global__ __launch_bounds__(256) void k_avg(AvgJob j) {
  const int64_t total = j.first[j.nseg];
  for (int64_t u = blockIdx.x * 256 + threadIdx.x; u < total; u += (int64_t)gridDim.x * 256) {
    int lo = 0, hi = j.nseg - 1;                  // last segment with first <= u
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (j.first[mid] <= u) lo = mid;
      else hi = mid - 1;
    }
    const int64_t e = (u - j.first[lo]) * 4;      // first float of the unit
    const int64_t cnt = j.cnt[lo];
    const int64_t off = j.off[lo] + e * 4;
    const float* w = j.w[j.wsel[lo]];
    if (e + 4 <= cnt) {
      float4 v[N];
#pragma unroll
      for (int i = 0; i < N; ++i) v[i] = *(const float4*)(j.base[i] + off);
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int i = 0; i < N; ++i) {
        acc.x = fmaf(w[i], v[i].x, acc.x);
        acc.y = fmaf(w[i], v[i].y, acc.y);
        acc.z = fmaf(w[i], v[i].z, acc.z);
        acc.w = fmaf(w[i], v[i].w, acc.w);
      }
#pragma unroll
      for (int i = 0; i < N; ++i) *(float4*)(j.base[i] + off) = acc;
    } else {
      for (int64_t q = 0; q < cnt - e; ++q) {
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < N; ++i) acc = fmaf(w[i], ((const float*)(j.base[i] + off))[q], acc);
#pragma unroll
        for (int i = 0; i < N; ++i) ((float*)(j.base[i] + off))[q] = acc;
      }
    }
  }
}

template <int N>
void launch_avg_n(const AvgJob& j, int grid, hipStream_t st) {
  hipLaunchKernelGGL(k_avg<N>, dim3(grid), dim3(256), 0, st, j);
}

int grid_for(int64_t work, int per_block, int cap) {
  return (int)std::max<int64_t>(1, std::min<int64_t>((work + per_block - 1) / per_block, cap));
}

}  // namespace

hipError_t launch_tick_base(TickSrc* src, int cyc, hipStream_t st) {
  hipLaunchKernelGGL(k_tick_base, dim3(1), dim3(64), 0, st, src, cyc);
  return hipGetLastError();
}

hipError_t launch_tick_set(TickSrc* dst, const TickSrc& v, hipStream_t st) {
  hipLaunchKernelGGL(k_tick_set, dim3(1), dim3(64), 0, st, dst, v);
  return hipGetLastError();
}

hipError_t launch_philox_words(uint64_t seed, uint32_t step, uint32_t tag, uint32_t row0,
                               int rows, int groups, uint32_t* out, hipStream_t st) {
  const int64_t total = (int64_t)rows * groups;
  hipLaunchKernelGGL(k_philox_words, dim3(grid_for(total, 256, 4096)), dim3(256), 0, st, seed,
                     step, tag, row0, rows, groups, out);
  return hipGetLastError();
}

hipError_t launch_avg(const AvgJob& j, hipStream_t st) {
  if (j.n < 1 || j.n > kMaxAvgSets || j.nseg < 1 || j.nseg > kMaxAvgSegs) return hipErrorInvalidValue;
  const int64_t total = j.first[j.nseg];
  if (total == 0) return hipSuccess;
  const int g = grid_for(total, 256, 4096);
  switch (j.n) {
    case 1: launch_avg_n<1>(j, g, st); break;
    case 2: launch_avg_n<2>(j, g, st); break;
    case 3: launch_avg_n<3>(j, g, st); break;
    case 4: launch_avg_n<4>(j, g, st); break;
    case 5: launch_avg_n<5>(j, g, st); break;
    case 6: launch_avg_n<6>(j, g, st); break;
    case 7: launch_avg_n<7>(j, g, st); break;
    case 8: launch_avg_n<8>(j, g, st); break;
    case 9: launch_avg_n<9>(j, g, st); break;
    case 10: launch_avg_n<10>(j, g, st); break;
    case 11: launch_avg_n<11>(j, g, st); break;
    case 12: launch_avg_n<12>(j, g, st); break;
    case 13: launch_avg_n<13>(j, g, st); break;
    case 14: launch_avg_n<14>(j, g, st); break;
    case 15: launch_avg_n<15>(j, g, st); break;
    default: launch_avg_n<16>(j, g, st); break;
  }
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
