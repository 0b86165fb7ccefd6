// Weight gradients and SGD of the split-learning step on gfx950 (k_dw,
// k_dw_reduce; see kernels.h).
//
// G = D^T X contracts over the rows of the group.  Both operands are in the
// row-chunked layout, so every MFMA fragment is one 16-byte load per lane
// straight from global memory: lane group g (lane / 16) takes the chunk of
// rows [8g, 8g + 8) of the step (4 rows for float32), lane % 16 the column.
// The input X is the MFMA's A operand and the delta D its B operand, so a
// lane accumulates four consecutive k of one output row n: partials and SGD
// updates are 16-byte row segments.  A block owns a 64 x 64 output tile (2 x
// 2 wavefronts of 32 x 32) and one chunk of rows, loads the fragments of
// four MFMA steps as one group while multiplying the previous group, and
// sums the bias gradient from the D fragments it already holds.
//
// Split chunks are summed by k_dw_reduce in chunk order, as are the logit
// layer's per-block partials, so every result is deterministic.  SGD (Eq. 2)
// updates the float32 master weights; the element-type operand copies the
// next forward (W) and input-gradient (W^T) products read are rewritten from
// the new weights in the same pass.
#include "device.h"
#include "kernels.h"

namespace vfl {
namespace {
using namespace dev;

// SGD of the master weights W[n][kb .. kb+3] (those below K) with the
// gradient g, and the new values into the packed operand copies.  The four
// master values are loaded first, unconditionally (clamped), so that their
// loads are in flight together.
template <typename T>
__device__ __forceinline__ void sgd_load4(const DwProb& P, int n, int kb, float (&w)[4]) {
  const int K = P.K;
  const VFL_GLOBAL float* W = glb(P.W) + (int64_t)min(n, P.N - 1) * K;
#pragma unroll
  for (int e = 0; e < 4; ++e) w[e] = W[min(kb + e, K - 1)];
}
template <typename T>
__device__ __forceinline__ void sgd_store4(const DwProb& P, int n, int kb, const float (&w)[4], const f32x4& g,
                                           float scale) {
  const int K = P.K;
  VFL_GLOBAL float* W = glb(P.W) + (int64_t)n * K;
  float v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = w[e] - scale * g[e];   // unconditional: keeps the loads unsunk
  if (n >= P.N) return;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int k = kb + e;
    if (k >= K) continue;
    W[k] = v[e];
    if (P.Wq) st1<T>((T*)(glb((T*)P.Wq) + pk_index<T>(n, k, P.kq)), v[e]);
    if (P.Wtq) st1<T>((T*)(glb((T*)P.Wtq) + pk_index<T>(k, n, P.kt)), v[e]);
  }
}

// The problem, output tile and row chunk of this block (tile_w: the square
// tile width).  Workgroups are dealt to the 8 XCDs round-robin (block b on
// XCD b mod 8); XCD x takes the contiguous range [x * per, (x + 1) * per)
// of the job's work items, ordered problem by problem and chunk by chunk
// with the chunk's tiles innermost, so that the tiles reading the same rows
// of the same operands run at the same time on one XCD and share its L2.
// False for the blocks that round the grid up to a multiple of 8.
__device__ __forceinline__ bool dw_item(const DwJob& J, int tile_w, int& q, int& tile, int& split) {
  const int per = (J.blocks + 7) / 8;
  const int v = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (v >= J.blocks) return false;
  q = 0;
#pragma unroll 1
  while (q + 1 < J.n && v >= J.p[q + 1].first_block) ++q;
  const DwProb& P = J.p[q];
  const int tiles = ((P.N + tile_w - 1) / tile_w) * ((P.K + tile_w - 1) / tile_w);
  const int lb = v - P.first_block;
  split = lb / tiles;
  tile = lb % tiles;
  return true;
}

template <typename T>
__global__ __launch_bounds__(256) void k_dw(const DwJob* __restrict__ jp, int Rarg, float scale_arg,
                                            TickRef tr) {
  constexpr int RR = 16 / (int)sizeof(T);   // rows per chunk
  constexpr int KR = 4 * RR;                // rows per MFMA step
  constexpr int PF = 4;                     // MFMA steps per load group
  const DwJob& J = *jp;
  int q, tile, split;
  if (!dw_item(J, 64, q, tile, split)) return;
  const DwProb& P = J.p[q];
  const int tiles_k = (P.K + 63) / 64;
  const int n0 = (tile / tiles_k) * 64, k0 = (tile % tiles_k) * 64;
  float scale = scale_arg;
  if (tr.src) scale = tick_args(tr).scale;
  (void)Rarg;   // every chunk is contracted whole: the group's row count is not needed
  const int rb = split * P.rps;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int wm = wave >> 1, wn = wave & 1, kc = lane >> 4, lr = lane & 15;
  const VFL_GLOBAL char* Dp = glb((const char*)P.D.p);
  const VFL_GLOBAL char* Xp = glb((const char*)P.X.p);
  const int64_t dcp = P.D.cp, xcp = P.X.cp;
  const int N = P.N, K = P.K;
  int nd[2], kx[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    nd[i] = n0 + 32 * wm + 16 * i + lr;
    kx[i] = k0 + 32 * wn + 16 * i + lr;
  }
  const bool do_bias = (tile % tiles_k) == 0 && wn == 0;

  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jn = 0; jn < 2; ++jn) acc[i][jn] = f32x4{0.f, 0.f, 0.f, 0.f};
  float bsum[2] = {0.f, 0.f};

  // group g: MFMA steps at rows rb + (g * PF + st) * KR.  Loads are
  // unconditional: rps is a multiple of PF * KR, so a group never reaches
  // into the next chunk, and the delta rows from the group's end up to the
  // group's last step are zero (chain blocks zero them); columns are
  // clamped, their outputs discarded.
  const VFL_GLOBAL char* dcol[2];
  const VFL_GLOBAL char* xcol[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    dcol[i] = Dp + (int64_t)min(nd[i], N - 1) * 16;
    xcol[i] = Xp + (int64_t)min(kx[i], K - 1) * 16;
  }
  auto load = [&](int g, u32x4 (&df)[PF][2], u32x4 (&xf)[PF][2]) {
#pragma unroll
    for (int st = 0; st < PF; ++st) {
      const int64_t rg = (rb + (g * PF + st) * KR) / RR + kc;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        df[st][i] = *(const VFL_GLOBAL u32x4*)(dcol[i] + rg * dcp * 16);
        xf[st][i] = *(const VFL_GLOBAL u32x4*)(xcol[i] + rg * xcp * 16);
      }
    }
  };
  // every chunk is contracted whole (rps rows, a multiple of two load
  // groups; the delta rows past the group are zero)
  const int ngr = P.rps / (PF * KR);
  u32x4 dA[PF][2], xA[PF][2], dB[PF][2], xB[PF][2];
  auto group = [&](const u32x4 (&df)[PF][2], const u32x4 (&xf)[PF][2]) {
#pragma unroll
    for (int st = 0; st < PF; ++st) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int jn = 0; jn < 2; ++jn) {
          if constexpr (sizeof(T) == 2) {
            acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, xf[st][i]), __builtin_bit_cast(bf16x8, df[st][jn]), acc[i][jn], 0, 0, 0);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                  __uint_as_float(xf[st][i][e]), __uint_as_float(df[st][jn][e]), acc[i][jn], 0, 0, 0);
          }
        }
      }
      if (do_bias) {
#pragma unroll
        for (int jn = 0; jn < 2; ++jn) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if constexpr (sizeof(T) == 2) {
              bsum[jn] += __uint_as_float(df[st][jn][e] << 16) + __uint_as_float(df[st][jn][e] & 0xffff0000u);
            } else {
              bsum[jn] += __uint_as_float(df[st][jn][e]);
            }
          }
        }
      }
    }
  };
  // two groups in flight at the top of every iteration (A: group g, B:
  // group g + 1), each refilled as soon as its MFMAs have read it; every
  // load is unconditional (past the end it reloads the last group), and
  // the first iteration is peeled, so that the loop is entered with the
  // loads in flight exactly as at its back edge (exact wait counts)
  load(0, dA, xA);
  load(min(1, ngr - 1), dB, xB);
  group(dA, xA);
  load(min(2, ngr - 1), dA, xA);
  group(dB, xB);
  load(min(3, ngr - 1), dB, xB);
#pragma unroll 1
  for (int g = 2; g < ngr; g += 2) {
    group(dA, xA);
    load(min(g + 2, ngr - 1), dA, xA);
    group(dB, xB);
    load(min(g + 3, ngr - 1), dB, xB);
  }

  // bias: sum the four lane groups of each column
  if (do_bias) {
#pragma unroll
    for (int jn = 0; jn < 2; ++jn) {
      bsum[jn] += __shfl_xor(bsum[jn], 16, 64);
      bsum[jn] += __shfl_xor(bsum[jn], 32, 64);
    }
    if (kc == 0) {
#pragma unroll
      for (int jn = 0; jn < 2; ++jn) {
        const int n = nd[jn];
        if (n >= N) continue;
        if (P.splits == 1) glb(P.bias)[n] -= scale * bsum[jn];
        else glb(P.partb)[(int64_t)split * N + n] = bsum[jn];
      }
    }
  }
  // weights: lane holds G[n][kb .. kb+3]
  if (P.splits > 1) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int jn = 0; jn < 2; ++jn) {
        const int n = nd[jn];
        const int kb = k0 + 32 * wn + 16 * i + 4 * kc;
        if (n >= N || kb >= K) continue;
        *(VFL_GLOBAL f32x4*)(glb(P.part) + ((int64_t)split * N + n) * P.kp + kb) = acc[i][jn];
      }
    }
  } else {
    // every master value first (one wait), then the updates
    float w[2][2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int jn = 0; jn < 2; ++jn) sgd_load4<T>(P, nd[jn], k0 + 32 * wn + 16 * i + 4 * kc, w[i][jn]);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int jn = 0; jn < 2; ++jn)
        sgd_store4<T>(P, nd[jn], k0 + 32 * wn + 16 * i + 4 * kc, w[i][jn], acc[i][jn], scale);
  }
}

// Large-tile weight gradient for bf16 operands and long groups: a block of
// 256 threads owns a kDwtN x kDwtK (256 x 256) output tile of one problem
// and one row chunk.  Rows go through LDS in stages of 32 (five 32 KB
// buffers, one barrier per stage), copied from
// global memory straight into LDS (global_load_lds_dwordx4) in the order
// the matrix cores read them: one 1 KB block per 32 x 16 operand fragment of
// v_mfma_f32_32x32x16_bf16, which in the row-chunked layout is 32
// consecutive chunks (columns) of one 8-row group for each half-wavefront.
// Waves 0 and 1 copy the X fragments (32-input slabs 0-3 and 4-7), waves 2
// and 3 the D fragments.  Wavefront (wn, wk) of the 2 x 2 grid computes 128
// outputs x 128 inputs: X fragments as the A operand (32 inputs x 16 rows),
// D fragments as the B operand (16 rows x 32 outputs), so a lane
// accumulates four runs of four consecutive inputs k of one output n; per
// 16-row step 4 X and 4 D fragments feed 16 MFMAs, and the next stage's
// fragment reads are issued between the two steps of a stage.  The bias
// gradient is summed from the D fragments of the wavefronts with wk == 0 in the tiles at k0 == 0 (one
// v_dot2_f32_bf16 against (1, 1) per two rows).  The row chunks always
// write float32 partials (as k_dw's split problems; tiles counted 256 x
// 256): k_dw_reduce sums them and makes the SGD step.
constexpr int kDwtN = 256, kDwtK = 256;
constexpr int kDwtStageRows = 32;
constexpr int kDwtFrag = 1024;                              // one 32 x 16 bf16 fragment
constexpr int kDwtStageBytes = 2 * (kDwtN / 32) * 2 * kDwtFrag;   // 16 X + 16 D fragments
constexpr int kDwtBufs = 5;                                 // up to four stages in flight
constexpr int kDwtLds = kDwtBufs * kDwtStageBytes;

typedef __attribute__((address_space(3))) void lds_void;

// wait until at most n (0, 8, 16 or 24) of this wave's vector-memory operations
// are outstanding (expcnt and lgkmcnt unconstrained)
__device__ __forceinline__ void wait_vm(int n) {
  if (n >= 24) __builtin_amdgcn_s_waitcnt((1 << 14) | (15 << 8) | (7 << 4) | 8);
  else if (n >= 16) __builtin_amdgcn_s_waitcnt((1 << 14) | (15 << 8) | (7 << 4));
  else if (n >= 8) __builtin_amdgcn_s_waitcnt((15 << 8) | (7 << 4) | 8);
  else __builtin_amdgcn_s_waitcnt((15 << 8) | (7 << 4));
}

__global__ __launch_bounds__(256) void k_dwt(const DwJob* __restrict__ jp) {
  typedef __attribute__((ext_vector_type(16))) float f32x16;
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const DwJob& J = *jp;
  int q, tile, split;
  if (!dw_item(J, kDwtK, q, tile, split)) return;
  const DwProb& P = J.p[q];
  const int tiles_k = (P.K + kDwtK - 1) / kDwtK;
  const int n0 = (tile / tiles_k) * kDwtN, k0 = (tile % tiles_k) * kDwtK;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wn = wave >> 1, wk = wave & 1;
  const int col = lane & 31, hi = lane >> 5;
  const int N = P.N, K = P.K;
  const bool do_bias = k0 == 0 && wk == 0;

  // the lane's source column of the four slabs this wave copies (clamped
  // into the operand: those outputs are discarded); the chunk of 16-row
  // step k16 of stage s is 8-row group rb / 8 + 4 s + 2 k16 + hi
  const bool copies_x = wave < 2;
  const int wq = copies_x ? wave : wave - 2;
  const VFL_GLOBAL char* base = glb((const char*)(copies_x ? P.X.p : P.D.p));
  const int64_t unit = (int64_t)(copies_x ? P.X.cp : P.D.cp) * 16;   // bytes per 8-row group
  const int lim = copies_x ? K - 1 : N - 1;
  const int c0 = copies_x ? k0 : n0;
  const VFL_GLOBAL char* src[4];
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) src[s4] = base + (int64_t)min(c0 + 32 * (4 * wq + s4) + col, lim) * 16;
  const int64_t rg0 = (int64_t)split * P.rps / 8;
  auto issue = [&](int s) {
    char* dst = smem + (s % kDwtBufs) * kDwtStageBytes + (copies_x ? 0 : kDwtStageBytes / 2) + wq * 8 * kDwtFrag;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int s4 = i >> 1, k16 = i & 1;
      __builtin_amdgcn_global_load_lds((VFL_GLOBAL void*)(src[s4] + (rg0 + 4 * s + 2 * k16 + hi) * unit),
                                       (lds_void*)(dst + i * kDwtFrag), 16, 0, 0);
    }
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[kb][nb][e] = 0.f;
  float bsum[4] = {0.f, 0.f, 0.f, 0.f};
  const bf16x2 kOnes2 = __builtin_bit_cast(bf16x2, 0x3F803F80u);

  auto frags = [&](const char* S, int k16, u32x4 (&xa)[4], u32x4 (&db)[4]) {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) xa[kb] = *(const u32x4*)(S + ((4 * wk + kb) * 2 + k16) * kDwtFrag + lane * 16);
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
      db[nb] = *(const u32x4*)(S + kDwtStageBytes / 2 + ((4 * wn + nb) * 2 + k16) * kDwtFrag + lane * 16);
  };
  auto mma = [&](const u32x4 (&xa)[4], const u32x4 (&db)[4]) {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
        acc[kb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8, xa[kb]), __builtin_bit_cast(bf16x8, db[nb]), acc[kb][nb], 0, 0, 0);
  };
  auto bias_sums = [&](const u32x4 (&db)[4]) {
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      const bf16x8 v = __builtin_bit_cast(bf16x8, db[nb]);
      bsum[nb] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 0, 1), kOnes2, bsum[nb], false);
      bsum[nb] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 2, 3), kOnes2, bsum[nb], false);
      bsum[nb] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 4, 5), kOnes2, bsum[nb], false);
      bsum[nb] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, 6, 7), kOnes2, bsum[nb], false);
    }
  };

  // the chunk is contracted whole (rps rows, a multiple of the stage; the
  // delta rows past the group are zero).  Software pipeline: the fragment
  // reads of stage s + 1 are issued between the two halves of the products
  // of stage s (two register sets), after the barrier that makes stage s + 1
  // visible; that
  // barrier also retires the buffer of stage s - 1, which then takes the
  // copies of stage s + kDwtBufs - 1.
  struct Frags { u32x4 xa0[4], db0[4], xa1[4], db1[4]; };
  const int nst = P.rps / kDwtStageRows;
  auto read_stage = [&](int s, Frags& f) {
    const char* S = smem + (s % kDwtBufs) * kDwtStageBytes;
    frags(S, 0, f.xa0, f.db0);
    frags(S, 1, f.xa1, f.db1);
  };
  auto step = [&](int s, const Frags& x, Frags& y) {
    if (s + 1 < nst) {
      // this wave's copies of stage s + 1 have landed (later stages may be
      // in flight); after the unfenced barrier every wave's have
      wait_vm(8 * min(kDwtBufs - 3, nst - 2 - s));
      __builtin_amdgcn_s_barrier();
      if (s + kDwtBufs - 1 < nst) issue(s + kDwtBufs - 1);
    }
    // the next stage's reads go between the two halves of this stage's
    // products: the wait for x (read a step earlier) comes before the first
    // half, and nothing waits for y until the next step (after the last
    // stage a harmless re-read of it, so that y is always written and the
    // two register sets are never both live across a step).  The scheduling
    // barriers keep the compiler from sinking each read to its first use.
    __builtin_amdgcn_sched_barrier(0);
    mma(x.xa0, x.db0);
    __builtin_amdgcn_sched_barrier(0);
    read_stage(min(s + 1, nst - 1), y);
    __builtin_amdgcn_sched_barrier(0);
    mma(x.xa1, x.db1);
    if (do_bias) {
      bias_sums(x.db0);
      bias_sums(x.db1);
    }
  };
  for (int s = 0; s < kDwtBufs - 1 && s < nst; ++s) issue(s);
  Frags fa, fb;
  wait_vm(8 * min(kDwtBufs - 2, nst - 1));
  __builtin_amdgcn_s_barrier();
  read_stage(0, fa);
  int s = 0;
#pragma unroll 1
  for (; s + 1 < nst; s += 2) {
    step(s, fa, fb);
    step(s + 1, fb, fa);
  }
  if (s < nst) step(s, fa, fb);

  if (do_bias) {
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) bsum[nb] += __shfl_xor(bsum[nb], 32, 64);
    if (hi == 0) {
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int n = n0 + 128 * wn + 32 * nb + col;
        if (n < N) glb(P.partb)[(int64_t)split * N + n] = bsum[nb];
      }
    }
  }
  // lane: output n = n0 + 128 wn + 32 nb + col, inputs
  // k = k0 + 128 wk + 32 kb + 8 g + 4 hi + (0 .. 3) in acc[kb][nb][4 g ..]
  // (the plan gives this kernel at least two row chunks: the SGD is the
  // reduction's).  The partials go out through LDS (the stage buffers are
  // free by now): per wavefront and round, its 64 outputs of two blocks nb
  // as rows of 128 inputs (padded by 4 floats: the 16 lanes of a quarter
  // wavefront write distinct banks), read back a row per 32 lanes, so that
  // each store instruction writes two runs of 512 consecutive bytes.
  constexpr int kEpiPitch = kDwtK / 2 + 4;
  static_assert(4 * 64 * kEpiPitch * 4 <= kDwtLds, "epilogue staging exceeds the stage buffers");
  VFL_GLOBAL float* part = glb(P.part) + (int64_t)split * N * P.kp;
  float* E = (float*)(smem + wave * 64 * kEpiPitch * 4);
  __syncthreads();   // every wavefront is done with the stage buffers
#pragma unroll
  for (int r = 0; r < 2; ++r) {
#pragma unroll
    for (int nbi = 0; nbi < 2; ++nbi)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          *(f32x4*)(E + (32 * nbi + col) * kEpiPitch + 32 * kb + 8 * g + 4 * hi) =
              f32x4{acc[kb][2 * r + nbi][4 * g], acc[kb][2 * r + nbi][4 * g + 1], acc[kb][2 * r + nbi][4 * g + 2],
                    acc[kb][2 * r + nbi][4 * g + 3]};
    __syncthreads();
    const int kk = k0 + 128 * wk + 4 * col;
#pragma unroll 4
    for (int it = 0; it < 32; ++it) {
      const int row = 2 * it + hi;
      const f32x4 v = *(const f32x4*)(E + row * kEpiPitch + 4 * col);
      const int n = n0 + 128 * wn + 64 * r + row;
      if (n < N && kk < K) *(VFL_GLOBAL f32x4*)(part + (int64_t)n * P.kp + kk) = v;
    }
    __syncthreads();
  }
}

// The logit layer's block partials {loss, dl, dl * h} (one row of Hd + 2
// floats per chain block): columns 4 lb .. 4 lb + 3, the rows split over 64
// slices and summed slice by slice; then SGD of the logit weights and bias
// and the group's mean loss.
__device__ __forceinline__ void logit_reduce(const DwJob& J, int lb, int R, float scale, float* loss_out) {
  __shared__ float red[64][5];
  const int W = J.Hd + 2;
  const int cl = threadIdx.x & 3, sl = threadIdx.x >> 2;
  const int c = lb * 4 + cl;
  const int rows = (R + J.lrows - 1) / J.lrows;
  const VFL_GLOBAL float* lp = glb(J.lpart);
  float acc = 0.f;
  if (c < W) {
    int b = sl;
    for (; b + 3 * 64 < rows; b += 4 * 64) {
      const float v0 = lp[(int64_t)b * W + c], v1 = lp[(int64_t)(b + 64) * W + c];
      const float v2 = lp[(int64_t)(b + 128) * W + c], v3 = lp[(int64_t)(b + 192) * W + c];
      acc += ((v0 + v1) + v2) + v3;
    }
    for (; b < rows; b += 64) acc += lp[(int64_t)b * W + c];
  }
  red[sl][cl] = acc;
  __syncthreads();
  if (sl == 0 && c < W) {
    float tot = 0.f;
    for (int i = 0; i < 64; ++i) tot += red[i][cl];
    if (c == 0) {
      if (loss_out) *glb(loss_out) = tot / (float)R;
    } else if (c == 1) {
      glb(J.lb)[0] -= scale * tot;
    } else {
      glb(J.lw)[c - 2] -= scale * tot;
    }
  }
}

// Unsplit weight gradient over 32 x 32 output tiles, for groups small
// enough that one block can contract all their rows: the block's four
// wavefronts take interleaved MFMA row steps (wavefront w: steps w, w + 4,
// ...) and accumulate the whole tile each; the four sums meet in LDS and
// are added in wavefront order; the SGD of the tile's master weights (and
// bias, for the tiles of the first 32 inputs) and the operand-copy refresh
// follow in the same block, so no reduction launch is needed.  Blocks past
// the tiles reduce the logit layer's partials.
template <typename T>
__global__ __launch_bounds__(256) void k_dw32(const DwJob* __restrict__ jp, int Rarg, float scale_arg,
                                              float* loss_out, TickRef tr, float* loss_base) {
  constexpr int RR = 16 / (int)sizeof(T);   // rows per chunk
  constexpr int KR = 4 * RR;                // rows per MFMA step
  constexpr int PF = 4;                     // MFMA steps per load group
  const DwJob& J = *jp;
  int R = Rarg;
  float scale = scale_arg;
  if (tr.src) {
    const TickArgs ta = tick_args(tr);
    R = ta.rows;
    scale = ta.scale;
    loss_out = loss_base ? loss_base + ta.loss_idx : nullptr;
  }
  if ((int)blockIdx.x >= J.blocks) {
    logit_reduce(J, (int)blockIdx.x - J.blocks, R, scale, loss_out);
    return;
  }
  int q = 0;
#pragma unroll 1
  while (q + 1 < J.n && (int)blockIdx.x >= J.p[q + 1].first_block) ++q;
  const DwProb& P = J.p[q];
  const int N = P.N, K = P.K;
  const int tiles_k = (K + 31) / 32;
  const int lb = blockIdx.x - P.first_block;
  const int n0 = (lb / tiles_k) * 32, k0 = (lb % tiles_k) * 32;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int kc = lane >> 4, lr = lane & 15;
  const bool do_bias = k0 == 0;

  const VFL_GLOBAL char* dcol[2];
  const VFL_GLOBAL char* xcol[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    dcol[i] = glb((const char*)P.D.p) + (int64_t)min(n0 + 16 * i + lr, N - 1) * 16;
    xcol[i] = glb((const char*)P.X.p) + (int64_t)min(k0 + 16 * i + lr, K - 1) * 16;
  }
  const int64_t dcp = P.D.cp, xcp = P.X.cp;
  // every wavefront takes the same number of row steps, covering all the
  // RC rows (a multiple of 1024; the delta rows past the group are zero):
  // an even number of load groups, no step conditional
  const int nsw = J.rows_pad / KR / 4;                      // steps per wavefront
  const int ngr = nsw / PF;                                 // load groups
  // loads of group g (past the last group they repeat its last step:
  // unconditional, never used)
  auto load = [&](int g, u32x4 (&df)[PF][2], u32x4 (&xf)[PF][2]) {
#pragma unroll
    for (int st = 0; st < PF; ++st) {
      const int sw = min(g * PF + st, nsw - 1);
      const int64_t rg = (int64_t)(wave + 4 * sw) * (KR / RR) + kc;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        df[st][i] = *(const VFL_GLOBAL u32x4*)(dcol[i] + rg * dcp * 16);
        xf[st][i] = *(const VFL_GLOBAL u32x4*)(xcol[i] + rg * xcp * 16);
      }
    }
  };
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jn = 0; jn < 2; ++jn) acc[i][jn] = f32x4{0.f, 0.f, 0.f, 0.f};
  float bsum[2] = {0.f, 0.f};
  auto group = [&](const u32x4 (&df)[PF][2], const u32x4 (&xf)[PF][2]) {
#pragma unroll
    for (int st = 0; st < PF; ++st) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int jn = 0; jn < 2; ++jn) {
          if constexpr (sizeof(T) == 2) {
            acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, xf[st][i]), __builtin_bit_cast(bf16x8, df[st][jn]), acc[i][jn], 0, 0, 0);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                  __uint_as_float(xf[st][i][e]), __uint_as_float(df[st][jn][e]), acc[i][jn], 0, 0, 0);
          }
        }
      }
      if (do_bias) {
#pragma unroll
        for (int jn = 0; jn < 2; ++jn) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if constexpr (sizeof(T) == 2) {
              bsum[jn] += __uint_as_float(df[st][jn][e] << 16) + __uint_as_float(df[st][jn][e] & 0xffff0000u);
            } else {
              bsum[jn] += __uint_as_float(df[st][jn][e]);
            }
          }
        }
      }
    }
  };
  // two groups in flight at the top of every iteration (A: group g, B:
  // group g + 1); each is refilled as soon as its MFMAs have read it
  // (the first iteration is peeled, so that the loop is entered with the
  // loads in flight exactly as at its back edge: the compiler's wait
  // counts stay exact)
  u32x4 dA[PF][2], xA[PF][2], dB[PF][2], xB[PF][2];
  load(0, dA, xA);
  load(1, dB, xB);
  group(dA, xA);
  load(2, dA, xA);
  group(dB, xB);
  load(3, dB, xB);
#pragma unroll 1
  for (int g = 2; g < ngr; g += 2) {
    group(dA, xA);
    load(g + 2, dA, xA);
    group(dB, xB);
    load(g + 3, dB, xB);
  }

  // the SGD operands (their loads overlap the LDS reduction): thread t
  // updates W[n0 + t / 8][k0 + 4 (t % 8) .. +4] and, t < 32, bias[n0 + t]
  const int tn = threadIdx.x >> 3, tk = 4 * (threadIdx.x & 7);
  float w[4];
  sgd_load4<T>(P, n0 + tn, k0 + tk, w);
  const float b0 = glb(P.bias)[min(n0 + (int)(threadIdx.x & 31), N - 1)];
  // the wavefronts' tiles, added in wavefront order (rows padded to 9
  // float4: the 16 lanes of a column group hit distinct banks)
  __shared__ f32x4 red[4][32][9];
  __shared__ float rb[4][32];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jn = 0; jn < 2; ++jn) red[wave][16 * jn + lr][4 * i + kc] = acc[i][jn];
  if (do_bias) {
#pragma unroll
    for (int jn = 0; jn < 2; ++jn) {
      bsum[jn] += __shfl_xor(bsum[jn], 16, 64);
      bsum[jn] += __shfl_xor(bsum[jn], 32, 64);
    }
    if (kc == 0) {
      rb[wave][lr] = bsum[0];
      rb[wave][16 + lr] = bsum[1];
    }
  }
  __syncthreads();
  const f32x4 g = ((red[0][tn][tk / 4] + red[1][tn][tk / 4]) + red[2][tn][tk / 4]) + red[3][tn][tk / 4];
  sgd_store4<T>(P, n0 + tn, k0 + tk, w, g, scale);
  if (do_bias && threadIdx.x < 32) {
    const int n = n0 + threadIdx.x;
    const float gb = ((rb[0][threadIdx.x] + rb[1][threadIdx.x]) + rb[2][threadIdx.x]) + rb[3][threadIdx.x];
    if (n < N) glb(P.bias)[n] = b0 - scale * gb;
  }
}

constexpr int kRedBatch = 16;   // split partials loaded at once per thread

// Sum of the split partials s = 0 .. splits-1 at src + s * stride, in split
// order, the loads of a batch of kRedBatch all in flight before its first
// add (addresses past the last split repeat it; those values are not added).
__device__ __forceinline__ f32x4 split_sum4(const VFL_GLOBAL float* src, int64_t stride, int splits) {
  f32x4 sum = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < splits; s += kRedBatch) {
    f32x4 v[kRedBatch];
#pragma unroll
    for (int u = 0; u < kRedBatch; ++u) v[u] = *(const VFL_GLOBAL f32x4*)(src + (int64_t)min(s + u, splits - 1) * stride);
#pragma unroll
    for (int u = 0; u < kRedBatch; ++u)
      if (s + u < splits) sum += v[u];
  }
  return sum;
}
__device__ __forceinline__ float split_sum1(const VFL_GLOBAL float* src, int64_t stride, int splits) {
  float sum = 0.f;
  for (int s = 0; s < splits; s += kRedBatch) {
    float v[kRedBatch];
#pragma unroll
    for (int u = 0; u < kRedBatch; ++u) v[u] = src[(int64_t)min(s + u, splits - 1) * stride];
#pragma unroll
    for (int u = 0; u < kRedBatch; ++u)
      if (s + u < splits) sum += v[u];
  }
  return sum;
}

// One reduction tile of a split problem: rows n0 .. n0+7 and columns k0 ..
// k0+kRedK-1 of W (thread t: row n0 + t / 32, columns k0 + 4 (t % 32) ..
// +4).  The summed gradient makes the SGD step of the float32 masters; the
// new values (zero past N and K) go through LDS so that both packed operand
// copies are written as whole 16-byte chunks: CE consecutive inputs of one
// output for Wq, CE consecutive outputs of one input for Wtq (pk_index keeps
// such a run contiguous).
template <typename T>
__device__ __forceinline__ void reduce_tile(const DwProb& P, int n0, int k0, float scale) {
  constexpr int CE = 16 / (int)sizeof(T), KS = 4 * CE;
  constexpr int kPitch = kRedK + 16 / (int)sizeof(T);     // elements per LDS row (padded by 16 bytes)
  __shared__ __attribute__((aligned(16))) T tile[8 * kPitch];
  const int N = P.N, K = P.K, kp = P.kp;
  const int nr = threadIdx.x >> 5, kb = k0 + 4 * (threadIdx.x & 31);
  const int n = n0 + nr;
  const bool nok = n < N;
  // lanes past the problem's rows or inputs load nothing (narrow problems
  // leave half of a tile's lanes idle)
  f32x4 g = f32x4{0.f, 0.f, 0.f, 0.f};
  if (nok && kb < kp) g = split_sum4(glb(P.part) + (int64_t)n * kp + kb, (int64_t)N * kp, P.splits);
  VFL_GLOBAL float* W = glb(P.W) + (int64_t)min(n, N - 1) * K;
  const bool vec = (K & 3) == 0 && kb + 4 <= K;          // whole, 16-byte aligned float4 of W
  float w[4];
  if (vec) {
    const f32x4 x = *(const VFL_GLOBAL f32x4*)(W + kb);
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = x[e];
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = W[min(kb + e, K - 1)];
  }
  float v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = (nok && kb + e < K) ? w[e] - scale * g[e] : 0.f;
  if (nok) {
    if (vec) {
      *(VFL_GLOBAL f32x4*)(W + kb) = f32x4{v[0], v[1], v[2], v[3]};
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (kb + e < K) W[kb + e] = v[e];
    }
  }
  if (!P.Wq && !P.Wtq) return;
#pragma unroll
  for (int e = 0; e < 4; ++e) st1<T>(&tile[nr * kPitch + 4 * (threadIdx.x & 31) + e], v[e]);
  __syncthreads();
  if (P.Wq) {
    // chunk i: row i / (kRedK / CE), inputs k0 + CE (i % (kRedK / CE)) ..
    constexpr int per_row = kRedK / CE;
    for (int i = threadIdx.x; i < 8 * per_row; i += 256) {
      const int r = i / per_row, k = k0 + CE * (i % per_row);
      if (k < P.kq * KS)
        *(VFL_GLOBAL u32x4*)(glb((T*)P.Wq) + pk_index<T>(n0 + r, k, P.kq)) =
            *(const u32x4*)&tile[r * kPitch + (k - k0)];
    }
  }
  if (P.Wtq) {
    // chunk i: input k0 + i / (8 / CE), outputs n0 + CE (i % (8 / CE)) ..
    constexpr int per_k = 8 / CE;
    const int krows = (K + 15) / 16 * 16;                 // rows of the transposed copy's tiles
    for (int i = threadIdx.x; i < kRedK * per_k; i += 256) {
      const int kk = i / per_k, h = i % per_k, k = k0 + kk, ns = n0 + CE * h;
      if (k < krows && ns < P.kt * KS) {
        u32x4 c;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          if constexpr (sizeof(T) == 4) {
            c[w] = __float_as_uint(tile[(CE * h + w) * kPitch + kk]);
          } else {
            c[w] = (uint32_t)tile[(2 * w) * kPitch + kk] | ((uint32_t)tile[(2 * w + 1) * kPitch + kk] << 16);
          }
        }
        *(VFL_GLOBAL u32x4*)(glb((T*)P.Wtq) + pk_index<T>(k, ns, P.kt)) = c;
      }
    }
  }
}

// Blocks [0, red_blocks): per split problem, one block per reduction tile
// (8 outputs x kRedK inputs), then one per 256 biases.  Blocks after: 4 logit columns
// each, the partial rows split over 64 slices and summed slice by slice.
template <typename T>
__global__ __launch_bounds__(256) void k_dw_reduce(const DwJob* __restrict__ jp, int Rarg,
                                                   float scale_arg, float* loss_out,
                                                   TickRef tr, float* loss_base) {
  const DwJob& J = *jp;
  int R = Rarg;
  float scale = scale_arg;
  if (tr.src) {
    const TickArgs ta = tick_args(tr);
    R = ta.rows;
    scale = ta.scale;
    loss_out = loss_base ? loss_base + ta.loss_idx : nullptr;
  }
  if ((int)blockIdx.x < J.red_blocks) {
    int b = blockIdx.x;
    for (int q = 0; q < J.n; ++q) {
      const DwProb& P = J.p[q];
      if (P.splits <= 1) continue;
      const int tk = (P.kp + kRedK - 1) / kRedK, tiles = (P.N + 7) / 8 * tk, nbb = (P.N + 255) / 256;
      if (b >= tiles + nbb) { b -= tiles + nbb; continue; }
      if (b < tiles) {
        reduce_tile<T>(P, b / tk * 8, b % tk * kRedK, scale);
      } else {
        const int nb = (b - tiles) * 256 + threadIdx.x;
        if (nb < P.N) {
          VFL_GLOBAL float* bias = glb(P.bias) + nb;
          const float b0 = *bias;
          *bias = b0 - scale * split_sum1(glb(P.partb) + nb, P.N, P.splits);
        }
      }
      return;
    }
    return;
  }
  logit_reduce(J, (int)blockIdx.x - J.red_blocks, R, scale, loss_out);
}

}  // namespace

hipError_t launch_dw(Elt e, const DwJob* job, int blocks, int R, float scale, TickRef tr,
                     hipStream_t st) {
  if (blocks < 1) return hipErrorInvalidValue;
  const int grid = (blocks + 7) / 8 * 8;       // see dw_item
  if (e == BF16) hipLaunchKernelGGL(k_dw<uint16_t>, dim3(grid), dim3(256), 0, st, job, R, scale, tr);
  else hipLaunchKernelGGL(k_dw<float>, dim3(grid), dim3(256), 0, st, job, R, scale, tr);
  return hipGetLastError();
}

hipError_t dwt_init() {
  return hipFuncSetAttribute((const void*)k_dwt, hipFuncAttributeMaxDynamicSharedMemorySize, kDwtLds);
}

hipError_t launch_dwt(const DwJob* job, int blocks, hipStream_t st) {
  if (blocks < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_dwt, dim3((blocks + 7) / 8 * 8), dim3(256), kDwtLds, st, job);   // see dw_item
  return hipGetLastError();
}

hipError_t launch_dw32(Elt e, const DwJob* job, int blocks, int R, float scale, float* loss_out,
                      TickRef tr, float* loss_base, hipStream_t st) {
  if (blocks < 1) return hipErrorInvalidValue;
  if (e == BF16)
    hipLaunchKernelGGL(k_dw32<uint16_t>, dim3(blocks), dim3(256), 0, st, job, R, scale, loss_out, tr, loss_base);
  else
    hipLaunchKernelGGL(k_dw32<float>, dim3(blocks), dim3(256), 0, st, job, R, scale, loss_out, tr, loss_base);
  return hipGetLastError();
}

hipError_t launch_dw_reduce(Elt e, const DwJob* job, int blocks, int R, float scale,
                            float* loss_out, TickRef tr, float* loss_base, hipStream_t st) {
  if (blocks < 1) return hipErrorInvalidValue;
  if (e == BF16)
    hipLaunchKernelGGL(k_dw_reduce<uint16_t>, dim3(blocks), dim3(256), 0, st, job, R, scale, loss_out,
                       tr, loss_base);
  else
    hipLaunchKernelGGL(k_dw_reduce<float>, dim3(blocks), dim3(256), 0, st, job, R, scale, loss_out, tr,
                       loss_base);
  return hipGetLastError();
}

}  // namespace vfl
