// Sparse SGD step on the embedding tables of the categorical bottoms on
// gfx950 (the gather of the looked-up rows is part of the chain kernels'
// input stage).
//
// The sparse step (Eq. 2 restricted to the table rows a batch touches) sums,
// for every touched table row, the gradient rows of all samples that looked
// it up, and applies SGD once per touched row.
//
// Work split: no two workgroups ever write the same table row.  Workgroup
// (field f, hot id h), h < H = 16, owns id h alone; workgroup (field f,
// part p) owns the ids >= H with id mod P == p (P = 16).  With Zipf-like
// fields the small ids carry a large share of the samples (ids 0..15 about
// 40 % at exponent 1.1 over 100k ids, id 0 alone 13 %): alone in a
// workgroup each, their rows are summed without a sort, and the parts
// left to sort stay small.  A hot-id workgroup collects the rows of its id
// per pass (block scan, order fixed by the data), sums their gradient rows
// with 64 scanners per 4-column chunk (each over every 64th listed row, in
// list order) and a fixed-order tree over the scanners, and updates the
// row once.  Per pass of up to 8192 samples a part workgroup
//   1. collects its (id / P, row) keys into LDS from the field's row of the
//      field-major id copy (a block scan of per-thread match counts places
//      them; the keys are unique, so their order does not matter),
//   2. sorts them (bitonic network over 2, 8 or 32 keys per thread held in
//      registers, so the order is deterministic: by id, then by sample),
//   3. stages the gradient rows of the sorted keys and the table rows of
//      their ids in LDS, 256 positions at a time (every global load of a
//      stage issued together, while the previous stage is scanned), and forms segmented
//      sums per id with a fixed-shape scan: 64 scanners per 4-column chunk
//      each reduce 8 consecutive positions, an exclusive segmented scan
//      combines the scanners (lanes in order, then wavefronts in order),
//      and each scanner walks its positions again, storing the updated
//      table row where its id's segment ends.
// The summation order depends only on the sorted positions, so two runs
// give bitwise the same tables.
#include <algorithm>

#include "device.h"
#include "kernels.h"

namespace vfl {
namespace {
using namespace dev;

constexpr int kThreads = 256;
constexpr int kRowBits = 13;
constexpr int kPass = 1 << kRowBits;           // samples per pass
constexpr uint32_t kRowMask = kPass - 1;
constexpr int kStage = 256;                    // sorted positions staged at a time (64 KB of
                                               // LDS in all: two workgroups per CU)
constexpr int kScanners = kThreads / 4;        // per 4-column chunk
constexpr int kSpan = kStage / kScanners;      // positions per scanner
constexpr int kRowsPerThread = kPass / kThreads;     // rows a thread tests per pass
constexpr int kParts = 16;                     // id parts per field (id mod kParts)
constexpr int kHot = 16;                       // ids 0 .. kHot-1: a workgroup each
constexpr int kStageLoads = kStage * 4 / kThreads;   // (gradient, table) pairs per thread and stage
constexpr uint32_t kNone = 0xFFFFFFFFu;

// segmented-scan operator on (head seen, value): a later head restarts the sum
__device__ __forceinline__ void seg_combine(bool& F, f32x4& V, bool f2, const f32x4& v2) {
  V = f2 ? v2 : V + v2;
  F = F || f2;
}

__device__ __forceinline__ f32x4 shfl_up4(const f32x4& v, int d) {
  f32x4 r;
#pragma unroll
  for (int e = 0; e < 4; ++e) r[e] = __shfl_up(v[e], d, 64);
  return r;
}

// Bitonic sort of a[0, n) (n <= kThreads * KPT) into ascending order over
// N = kThreads * KPT slots, a[n, N) padded with kNone.  Thread t holds the
// slots [t * KPT, t * KPT + KPT) in registers: compare-exchange distances
// below KPT stay in the thread, those below 64 * KPT go through wavefront
// shuffles, and only the longer ones through LDS.  Ends with a[0, N)
// written back and a barrier.
template <int KPT>
__device__ __forceinline__ void bitonic(uint32_t* a, int n) {
  constexpr int N = kThreads * KPT;
  const int t = threadIdx.x;
  uint32_t x[KPT];
#pragma unroll
  for (int e = 0; e < KPT; ++e) x[e] = t * KPT + e < n ? a[t * KPT + e] : kNone;
  for (int k = 2; k <= N; k <<= 1) {
    for (int h = k >> 1; h >= KPT; h >>= 1) {
      // bit k of a slot index lies in t * KPT (k > h >= KPT)
      const bool asc = ((t * KPT) & k) == 0;
      const bool lower = ((t * KPT) & h) == 0;
      const bool keep_min = asc == lower;
      if (h < 64 * KPT) {
        const int m = h / KPT;
#pragma unroll
        for (int e = 0; e < KPT; ++e) {
          const uint32_t o = (uint32_t)__shfl_xor((int)x[e], m, 64);
          x[e] = keep_min ? min(x[e], o) : max(x[e], o);
        }
      } else {
#pragma unroll
        for (int e = 0; e < KPT; ++e) a[t * KPT + e] = x[e];
        __syncthreads();
#pragma unroll
        for (int e = 0; e < KPT; ++e) {
          const uint32_t o = a[(t * KPT + e) ^ h];
          x[e] = keep_min ? min(x[e], o) : max(x[e], o);
        }
        __syncthreads();
      }
    }
    // distances below KPT: inside the thread
#pragma unroll
    for (int h = KPT / 2; h >= 1; h >>= 1) {
      if (h >= k) continue;
#pragma unroll
      for (int e = 0; e < KPT; ++e) {
        if (e & h) continue;
        const bool asc = ((t * KPT + e) & k) == 0;
        const uint32_t lo = min(x[e], x[e + h]), hi = max(x[e], x[e + h]);
        x[e] = asc ? lo : hi;
        x[e + h] = asc ? hi : lo;
      }
    }
  }
#pragma unroll
  for (int e = 0; e < KPT; ++e) a[t * KPT + e] = x[e];
  __syncthreads();
}

// Block-wide placement of this thread's flagged rows (bit i of take: row
// i * kThreads + tid of the pass) into keys[], key(i) each, in thread order;
// returns the number of keys.  Ends with a barrier.
template <typename KeyOf>
__device__ __forceinline__ int place_keys(uint32_t take, uint32_t* keys, int* wcnt, KeyOf&& key) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = __builtin_popcount(take);
  int incl = c;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int v = __shfl_up(incl, d, 64);
    if (lane >= d) incl += v;
  }
  if (lane == 63) wcnt[wave] = incl;
  __syncthreads();
  int pos = incl - c, total = 0;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) {
    const int x = wcnt[w];
    pos += w < wave ? x : 0;
    total += x;
  }
#pragma unroll
  for (int i = 0; i < kRowsPerThread; ++i)
    if ((take >> i) & 1u) keys[pos++] = key(i);
  __syncthreads();
  return total;
}

__global__ __launch_bounds__(kThreads) void k_embed_sgd(ScatterJob j) {
  __shared__ uint32_t keys[kPass];
  __shared__ f32x4 gs[kStage][4], ts[kStage][4];
  __shared__ f32x4 wv[kThreads / 64][4];
  __shared__ int wf[kThreads / 64][4];
  __shared__ int wcnt[kThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // part workgroups first (the longer work is dispatched first), then the
  // hot ids
  const int nparts = j.n_cat * kParts;
  const bool hot = (int)blockIdx.x >= nparts;
  const int b = hot ? (int)blockIdx.x - nparts : (int)blockIdx.x;
  const int f = hot ? b / kHot : b / kParts, part = hot ? b % kHot : b % kParts;
  int R = j.R;
  float scale = j.scale;
  if (j.tr.src) {
    const TickArgs ta = tick_args(j.tr);
    R = ta.rows;
    scale = ta.scale;
  }
  const int EC = j.E / 4;                       // 4-column chunks per table row
  const VFL_GLOBAL int32_t* ids = glb(j.idt) + (int64_t)f * j.ldi;
  const VFL_GLOBAL f32x4* G = glb((const f32x4*)j.G);
  const int64_t ldg4 = j.ldg / 4;
  VFL_GLOBAL f32x4* Tf = glb((f32x4*)(j.T + (int64_t)f * j.V * j.E));
  const int q = tid >> 2, ch = tid & 3;         // scanner, chunk

  for (int c0 = 0; c0 < R; c0 += kPass) {
    const int n = min(kPass, R - c0);
    // 1. the workgroup's keys: every thread tests kPass / kThreads rows
    // (strided, so each load instruction of a wavefront is contiguous), then
    // a block scan of the per-thread counts places them
    uint32_t idv[kRowsPerThread];
#pragma unroll
    for (int i = 0; i < kRowsPerThread; ++i) idv[i] = (uint32_t)ids[c0 + min(i * kThreads + tid, n - 1)];
    uint32_t take = 0u;
#pragma unroll
    for (int i = 0; i < kRowsPerThread; ++i) {
      const uint32_t id = idv[i];
      const bool mine = hot ? id == (uint32_t)part : id >= (uint32_t)kHot && (id & (kParts - 1)) == (uint32_t)part;
      take |= (uint32_t)(i * kThreads + tid < n && mine) << i;
    }
    if (hot) {
      // rows of id `part`, in thread order; scanner q sums listed rows q,
      // q + 64, ... of its chunk in list order (eight loads in flight)
      const int np = place_keys(take, keys, wcnt, [&](int i) { return (uint32_t)(i * kThreads + tid); });
      if (np == 0) continue;   // uniform: no barrier skipped by part of the block
      const int cq = min(ch, EC - 1);
      const VFL_GLOBAL f32x4* Gc = G + (int64_t)c0 * ldg4 + f * EC + cq;
      f32x4 sum = f32x4{0.f, 0.f, 0.f, 0.f};
      int p = q;
      for (; p + 7 * kScanners < np; p += 8 * kScanners) {
        f32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = Gc[(int64_t)keys[p + u * kScanners] * ldg4];
#pragma unroll
        for (int u = 0; u < 8; ++u) sum += v[u];
      }
      for (; p < np; p += kScanners) sum += Gc[(int64_t)keys[p] * ldg4];
      // the 16 scanners of a wavefront (lanes 4 apart), a fixed tree
#pragma unroll
      for (int d = 32; d >= 4; d >>= 1) {
        const f32x4 o = f32x4{__shfl_down(sum[0], d, 64), __shfl_down(sum[1], d, 64),
                              __shfl_down(sum[2], d, 64), __shfl_down(sum[3], d, 64)};
        sum += o;
      }
      if (lane < 4) wv[wave][lane] = sum;
      __syncthreads();
      if (tid < EC) {
        const f32x4 tot = ((wv[0][tid] + wv[1][tid]) + wv[2][tid]) + wv[3][tid];
        VFL_GLOBAL f32x4* row = Tf + (int64_t)part * EC + tid;
        *row = *row - scale * tot;
      }
      __syncthreads();
      continue;
    }
    const int np = place_keys(take, keys, wcnt, [&](int i) {
      return ((idv[i] / kParts) << kRowBits) | (uint32_t)(i * kThreads + tid);
    });
    // 2. sort keys[0, np) ascending (padding kNone sorts last)
    if (np <= 2 * kThreads) bitonic<2>(keys, np);
    else if (np <= 8 * kThreads) bitonic<8>(keys, np);
    else bitonic<32>(keys, np);
    // 3. segmented sums, kStage sorted positions at a time; the gradient and
    // table rows of the next stage are loaded while this one is scanned
    f32x4 carry = f32x4{0.f, 0.f, 0.f, 0.f};    // the open segment entering the stage
    f32x4 gv[kStageLoads], tv[kStageLoads];
    // loads clamped into range, so all are unconditional and in flight
    // together; chunks past E repeat the last one (never stored back)
    auto issue = [&](int s0) {
#pragma unroll
      for (int u = 0; u < kStageLoads; ++u) {
        const int i = min(s0 * 4 + u * kThreads + tid, np * 4 - 1);
        const int c = min(i & 3, EC - 1);
        const uint32_t key = keys[i >> 2];
        gv[u] = G[(int64_t)(c0 + (key & kRowMask)) * ldg4 + f * EC + c];
        tv[u] = Tf[(int64_t)((key >> kRowBits) * (uint32_t)kParts + (uint32_t)part) * EC + c];
      }
    };
    if (np > 0) issue(0);
    for (int s0 = 0; s0 < np; s0 += kStage) {
      const int ns = min(kStage, np - s0);
#pragma unroll
      for (int u = 0; u < kStageLoads; ++u) {
        const int i = u * kThreads + tid;
        if (i < ns * 4) { gs[i >> 2][i & 3] = gv[u]; ts[i >> 2][i & 3] = tv[u]; }
      }
      __syncthreads();
      issue(s0 + kStage);   // past the last stage: clamped repeats, never stored
      auto head = [&](int a) { return a == 0 || (keys[a] >> kRowBits) != (keys[a - 1] >> kRowBits); };
      const int p0 = q * kSpan, p1 = min(p0 + kSpan, ns);
      // (a) the scanner's aggregate
      bool F = false;
      f32x4 V = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int i = p0; i < p1; ++i) seg_combine(F, V, head(s0 + i), gs[i][ch]);
      // (b) inclusive scan over the 16 scanners of the wavefront (lanes 4 apart)
      bool Fi = F;
      f32x4 Vi = V;
#pragma unroll
      for (int d = 1; d < 16; d <<= 1) {
        const f32x4 vu = shfl_up4(Vi, 4 * d);
        const bool fu = __shfl_up((int)Fi, 4 * d, 64) != 0;
        if ((lane >> 2) >= d) {
          // (fu, vu) comes first: (fu, vu) then (Fi, Vi)
          Vi = Fi ? Vi : vu + Vi;
          Fi = Fi || fu;
        }
      }
      if ((lane >> 2) == 15) { wv[wave][ch] = Vi; wf[wave][ch] = Fi; }
      // exclusive prefix within the wavefront
      f32x4 Ve = shfl_up4(Vi, 4);
      bool Fe = __shfl_up((int)Fi, 4, 64) != 0;
      if ((lane >> 2) == 0) { Ve = f32x4{0.f, 0.f, 0.f, 0.f}; Fe = false; }
      __syncthreads();
      // carry-in: stage carry, then the earlier wavefronts in order, then
      // the earlier scanners of this wavefront
      bool Fc = false;
      f32x4 Vc = carry;
      for (int w = 0; w < wave; ++w) seg_combine(Fc, Vc, wf[w][ch] != 0, wv[w][ch]);
      seg_combine(Fc, Vc, Fe, Ve);
      // (c) walk again; update where a segment ends
      f32x4 run = Vc;
      for (int i = p0; i < p1; ++i) {
        const int a = s0 + i;
        const f32x4 g = gs[i][ch];
        run = head(a) ? g : run + g;
        const bool last = a + 1 == np || (keys[a + 1] >> kRowBits) != (keys[a] >> kRowBits);
        if (last && ch < EC) {
          const uint32_t id = (keys[a] >> kRowBits) * (uint32_t)kParts + (uint32_t)part;
          Tf[(int64_t)id * EC + ch] = ts[i][ch] - scale * run;
        }
      }
      // the open segment after the whole stage
      bool Ft = false;
      for (int w = 0; w < kThreads / 64; ++w) seg_combine(Ft, carry, wf[w][ch] != 0, wv[w][ch]);
      __syncthreads();
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_scatter_sgd(const ScatterJob& j, hipStream_t st) {
  if (j.E > kMaxEmbDim || j.E % 4 || j.ldg % 4 || j.V > (1 << (32 - kRowBits))) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_embed_sgd, dim3(j.n_cat * (kParts + kHot)), dim3(kThreads), 0, st, j);
  return hipGetLastError();
}

}  // namespace vfl
