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
// segment's length is not a multiple of 4): reads the unit from every set,
// forms the weighted sum in a fixed order and writes it to every set.
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
    if (e + 4 <= cnt) {
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int i = 0; i < j.n; ++i) {
        const float4 v = *(const float4*)(j.base[i] + off);
        const float w = j.w[i];
        acc.x = fmaf(w, v.x, acc.x);
        acc.y = fmaf(w, v.y, acc.y);
        acc.z = fmaf(w, v.z, acc.z);
        acc.w = fmaf(w, v.w, acc.w);
      }
      for (int i = 0; i < j.n; ++i) *(float4*)(j.base[i] + off) = acc;
    } else {
      for (int64_t q = 0; q < cnt - e; ++q) {
        float acc = 0.f;
        for (int i = 0; i < j.n; ++i) acc = fmaf(j.w[i], ((const float*)(j.base[i] + off))[q], acc);
        for (int i = 0; i < j.n; ++i) ((float*)(j.base[i] + off))[q] = acc;
      }
    }
  }
}

int grid_for(int64_t work, int per_block, int cap) {
  return (int)std::max<int64_t>(1, std::min<int64_t>((work + per_block - 1) / per_block, cap));
}

}  // namespace

hipError_t launch_tick_base(TickSrc* src, int cyc, hipStream_t st) {
  hipLaunchKernelGGL(k_tick_base, dim3(1), dim3(64), 0, st, src, cyc);
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
  hipLaunchKernelGGL(k_avg, dim3(grid_for(total, 256, 2048)), dim3(256), 0, st, j);
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
