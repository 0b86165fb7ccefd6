// Sparse SGD step on the embedding tables of the categorical bottoms on
// gfx950 (the gather of the looked-up rows is part of the chain kernels'
// input stage).
//
// The sparse step sums, for every table row a batch touches, the gradient
// rows of all samples that looked it up, and applies SGD once per touched
// row.  One workgroup owns one field: it sorts the (id, row) keys of up to
// 8192 samples in LDS (bitonic network over unique 32-bit keys, so the order
// is deterministic), walks the sorted keys in 16-key pieces per thread,
// and combines the pieces of each id in sample order; the table row is then
// updated with a single rounding.  Fields own disjoint table rows, so the
// workgroups never write the same address.
#include <algorithm>

#include "kernels.h"

namespace vfl {
namespace {

constexpr int kSortN = 8192;               // samples sorted per pass
constexpr int kThreads = 512;
constexpr int kPer = kSortN / kThreads;    // sorted keys walked per thread
constexpr int kRowBits = 13;               // kSortN == 1 << kRowBits
constexpr uint32_t kNone = 0xFFFFFFFFu;

__global__ __launch_bounds__(kThreads) void k_embed_sgd(ScatterJob j) {
  __shared__ uint32_t keys[kSortN];
  __shared__ float facc[kThreads][kMaxEmbDim], lacc[kThreads][kMaxEmbDim];
  __shared__ uint32_t fid[kThreads], lid[kThreads];
  __shared__ uint8_t single[kThreads];
  const int tid = threadIdx.x;
  const int f = blockIdx.x;
  const int E = j.E;
  if (j.tr.src) {
    const TickArgs ta = tick_args(j.tr);
    j.R = ta.rows;
    j.scale = ta.scale;
    j.ids += ta.row0 * j.n_cat;
  }
  float* table = j.T + (int64_t)f * j.V * E;

  auto apply = [&](uint32_t id, const float (&s)[kMaxEmbDim]) {
    float* row = table + (int64_t)id * E;
    for (int e = 0; e < E; ++e) row[e] -= j.scale * s[e];
  };

  for (int c0 = 0; c0 < j.R; c0 += kSortN) {
    const int n = min(kSortN, j.R - c0);
    for (int i = tid; i < kSortN; i += kThreads)
      keys[i] = i < n ? ((uint32_t)j.ids[(int64_t)(c0 + i) * j.n_cat + f] << kRowBits) | (uint32_t)i
                      : kNone;
    __syncthreads();
    for (int k = 2; k <= kSortN; k <<= 1) {
      for (int h = k >> 1; h > 0; h >>= 1) {
        for (int i = tid; i < kSortN; i += kThreads) {
          const int l = i ^ h;
          if (l > i) {
            const uint32_t a = keys[i], b = keys[l];
            const bool up = (i & k) == 0;
            if (up ? (a > b) : (a < b)) { keys[i] = b; keys[l] = a; }
          }
        }
        __syncthreads();
      }
    }
    // walk this thread's sorted keys; pieces strictly inside are complete ids
    uint32_t cur = kNone, first = kNone;
    float acc[kMaxEmbDim];
    for (int e = 0; e < kMaxEmbDim; ++e) acc[e] = 0.f;
    int pieces = 0;
    for (int p = 0; p < kPer; ++p) {
      const uint32_t key = keys[tid * kPer + p];
      if (key == kNone) break;
      const uint32_t id = key >> kRowBits;
      const int r = (int)(key & (kSortN - 1));
      if (id != cur) {
        if (cur != kNone) {
          if (pieces == 1) {
            for (int e = 0; e < E; ++e) facc[tid][e] = acc[e];
          } else {
            apply(cur, acc);
          }
        }
        if (pieces == 0) first = id;
        cur = id;
        ++pieces;
        for (int e = 0; e < E; ++e) acc[e] = 0.f;
      }
      const float* g = j.G + (int64_t)(c0 + r) * j.ldg + f * E;
      for (int e = 0; e < E; ++e) acc[e] += g[e];
    }
    fid[tid] = first;
    lid[tid] = cur;
    single[tid] = pieces == 1;
    if (pieces >= 1) {
      if (pieces == 1) {
        for (int e = 0; e < E; ++e) facc[tid][e] = acc[e];
      } else {
        for (int e = 0; e < E; ++e) lacc[tid][e] = acc[e];
      }
    }
    __syncthreads();
    // an id's pieces lie in consecutive threads; its first piece's owner sums
    // them in thread (= sample) order and applies the update once
    float tot[kMaxEmbDim];
    auto gather_from = [&](uint32_t id, int t0) {
      for (int t = t0; t < kThreads && fid[t] == id; ++t) {
        for (int e = 0; e < E; ++e) tot[e] += facc[t][e];
        if (!single[t]) break;
      }
    };
    if (fid[tid] != kNone && (tid == 0 || lid[tid - 1] != fid[tid])) {
      for (int e = 0; e < E; ++e) tot[e] = facc[tid][e];
      if (single[tid]) gather_from(fid[tid], tid + 1);
      apply(fid[tid], tot);
    }
    if (lid[tid] != kNone && !single[tid]) {
      for (int e = 0; e < E; ++e) tot[e] = lacc[tid][e];
      gather_from(lid[tid], tid + 1);
      apply(lid[tid], tot);
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_scatter_sgd(const ScatterJob& j, hipStream_t st) {
  if (j.E > kMaxEmbDim || j.V > (1 << (32 - kRowBits))) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_embed_sgd, dim3(j.n_cat), dim3(kThreads), 0, st, j);
  return hipGetLastError();
}

}  // namespace vfl
