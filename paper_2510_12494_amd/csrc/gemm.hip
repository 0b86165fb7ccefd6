// Input-gradient products of wide bottom layers on gfx950 (k_gemm; see
// kernels.h for the job).
//
// out[r][n] = (mask[r][n] > 0) * sum_k A[r][k] W[n][k] for the rows of a
// group, bf16 operands and float32 accumulation: the delta of a layer's
// output (A, row-major) times the layer's stashed weight copy (W, the packed
// transpose the chain kernels read: pk_index, 16 x 32 fragments), masked by
// the ReLU derivative of the layer below (its stashed output, RC layout),
// written in the RC layout the weight gradient reads.  A block of 256
// threads owns a 256-row x 128-column output tile; K goes through LDS in
// stages of 64 (the A rows and the W fragments of the stage, 48 KB,
// double-buffered), one barrier per stage.  Wavefront (wm, wn) of the 2 x 2
// grid computes 128 x 64 of the tile with v_mfma_f32_32x32x16_bf16: A
// fragments (32 rows x 16 k) as the A operand, W fragments (16 k x 32
// outputs) as the B operand, so a lane ends up with one output column n and
// four runs of four consecutive rows.  The tiles are dealt to the XCDs in
// contiguous ranges, so the column tiles that share an A row slab meet in
// one L2.
//
// Epilogue: the runs of lanes l and l + 32 are exchanged so that each lane
// holds two whole 8-row chunks of its column, which meet the RC mask chunk
// at the same place (all mask chunks are loaded together first) and go to
// the RC output.  Rows past the group are written as zeros (the weight
// gradient reads whole row chunks).
#include "device.h"
#include "kernels.h"

namespace vfl {
namespace {
using namespace dev;

constexpr int kTM = 256, kTN = 128;            // block tile (rows x outputs)
constexpr int kSK = 64;                        // K per LDS stage
constexpr int kSC = kSK / 8;                   // 16-byte chunks per row and stage
constexpr int kPitch = kSC + 1;                // LDS chunks per row (+1: banks)
constexpr int kStageChunks = (kTM + kTN) * kPitch;   // one stage buffer, in chunks
constexpr int kWN = kTN / 2, kNB = kWN / 32;   // wavefront outputs, 32-wide blocks of them
constexpr int kGemmLds = 2 * kStageChunks * 16;

typedef __attribute__((ext_vector_type(16))) float f32x16;

// A_arg: the A operand of this launch (the group's rows of a dataset or of a
// caller batch, lda_arg elements per row; with a tick reference, the
// dataset base, offset by the tick's first row), or null: the job's
// workspace operand (rows of the tick).
__global__ __launch_bounds__(256) void k_gemm(const GemmJob* __restrict__ jp, const void* A_arg,
                                              int64_t lda_arg, int rows_arg, TickRef tr) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  u32x4* L = (u32x4*)smem;
  const GemmJob& J = *jp;
  int rows = rows_arg;
  int64_t a_row0 = 0;
  if (tr.src) {
    const TickArgs ta = tick_args(tr);
    rows = ta.rows;
    if (A_arg) a_row0 = ta.row0;
  }
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  // workgroups are dealt to the 8 XCDs round-robin (block b on XCD b mod
  // 8): XCD x takes the contiguous tile range [x * per, (x + 1) * per), so
  // the n-tiles that share an A row slab meet in one L2
  const int ntiles = J.tiles_n * J.tiles_m;
  const int per = (ntiles + 7) / 8;
  const int tile = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (tile >= ntiles) return;
  const int tile_n = tile % J.tiles_n, tile_m = tile / J.tiles_n;
  const int m0 = tile_m * kTM, n0 = tile_n * kTN;
  const int N = J.N, K = J.K;
  const int half = lane >> 5, col = lane & 31;
  const int64_t rg_end = J.rows_pad / 8;       // RC row groups of the outputs

  if (m0 >= rows) {
    // rows past the group: zero RC chunks (up to the padded row count)
    for (int c = t; c < kTM / 8 * kTN; c += 256) {
      const int rg = c / kTN, n = n0 + c % kTN;
      const int64_t g = m0 / 8 + rg;
      if (n >= N || g >= rg_end) continue;
      *(VFL_GLOBAL u32x4*)(glb((char*)J.out_rc.p) + (g * J.out_rc.cp + n) * 16) = u32x4{0u, 0u, 0u, 0u};
    }
    return;
  }

  // this thread's 16-byte chunks of a stage: A row 32 i + t / 8 of the
  // tile (i = 0 .. 7), k chunk t % 8; W fragment lane j = t % 64 of the
  // 16-output tile 2 i + t / 128 of the block (i = 0 .. 3), 32-k step
  // (t / 64) % 2
  const VFL_GLOBAL char* Ag = glb((const char*)(A_arg ? A_arg : J.A));
  const VFL_GLOBAL char* Wg = glb((const char*)J.W);
  const int64_t lda = A_arg ? lda_arg : J.lda;
  const int lda_c = (int)(lda / 8);            // chunks per A row
  const int ntl = (N + 15) / 16;               // 16-output tiles of W
  const int a_kc = t & 7, a_r = t >> 3;
  const int w_j = t & 63, w_st = (t >> 6) & 1, w_nt = t >> 7;
  const int kst = J.kst;
  const int nst = (K + kSK - 1) / kSK;
  constexpr int kWL = kTN * kSC / 256;         // W loads per thread and stage
  u32x4 stg[8 + kWL];
  // A chunks at or past K are zero (a row holds zeros from K up to the next
  // multiple of 8); W steps past the packing are clamped to its last step
  // (they meet those zero A chunks)
  const int kc_end = (K + 7) / 8;
  auto gload = [&](int s) {
    const int kc = s * kSC + a_kc;
    const int kcl = min(kc, lda_c - 1);
    const int st = min(2 * s + w_st, kst - 1);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t row = a_row0 + min(m0 + 32 * i + a_r, rows - 1);
      const u32x4 v = *(const VFL_GLOBAL u32x4*)(Ag + (row * lda_c + kcl) * 16);
      stg[i] = kc < kc_end ? v : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < kWL; ++i) {
      const int nt = min(n0 / 16 + 2 * i + w_nt, ntl - 1);
      stg[8 + i] = *(const VFL_GLOBAL u32x4*)(Wg + (((int64_t)nt * kst + st) * 64 + w_j) * 16);
    }
  };
  auto lstore = [&](int b) {
    u32x4* S = L + b * kStageChunks;
#pragma unroll
    for (int i = 0; i < 8; ++i) S[(32 * i + a_r) * kPitch + a_kc] = stg[i];
    // W: output n = 16 (2 i + w_nt) + j % 16 of the block, k chunk 4 st + j / 16
#pragma unroll
    for (int i = 0; i < kWL; ++i)
      S[kTM * kPitch + (16 * (2 * i + w_nt) + (w_j & 15)) * kPitch + 4 * w_st + (w_j >> 4)] = stg[8 + i];
  };

  f32x16 acc[4][kNB];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[mb][nb][e] = 0.f;

  auto frags = [&](int b, int k16, u32x4 (&af)[4], u32x4 (&bf)[kNB]) {
    const u32x4* S = L + b * kStageChunks;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) af[mb] = S[(wm * 128 + mb * 32 + col) * kPitch + 2 * k16 + half];
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) bf[nb] = S[kTM * kPitch + (wn * kWN + nb * 32 + col) * kPitch + 2 * k16 + half];
  };
  auto mma = [&](const u32x4 (&af)[4], const u32x4 (&bf)[kNB]) {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb)
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8, af[mb]), __builtin_bit_cast(bf16x8, bf[nb]), acc[mb][nb], 0, 0, 0);
  };
  gload(0);
  lstore(0);
  __syncthreads();
#pragma unroll 1
  for (int s = 0; s < nst; ++s) {
    const int b = s & 1;
    gload(min(s + 1, nst - 1));
    u32x4 a0[4], b0[kNB], a1[4], b1[kNB];
    frags(b, 0, a0, b0);
#pragma unroll
    for (int k16 = 0; k16 < kSK / 16; k16 += 2) {
      frags(b, k16 + 1, a1, b1);
      mma(a0, b0);
      if (k16 + 2 < kSK / 16) frags(b, k16 + 2, a0, b0);
      mma(a1, b1);
    }
    lstore(b ^ 1);
    __syncthreads();
  }

  // ------------------------------------------------------------ epilogue
  // lane: column n = n0 + wn * 64 + nb * 32 + col; rows
  // m0 + wm * 128 + mb * 32 + 8 g + 4 half + (0 .. 3) in acc[mb][nb][4 g ..]
  // (the last barrier of the loop follows every stage read, so the LDS
  // now holds each wavefront's private transpose tile)
  // the mask chunks (if any) all in flight before the first is used:
  // chunk (mb, nb, p) = 8-row group 2 p + half of MFMA tile (mb, nb)
  u32x4 mk[4][kNB][2];
  if (J.mask_rc.p) {
    const VFL_GLOBAL char* Mp = glb((const char*)J.mask_rc.p);
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
      const int n = min(n0 + wn * kWN + nb * 32 + col, N - 1);
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const int64_t rg = min((int64_t)(m0 + wm * 128 + mb * 32) / 8 + 2 * p + half, rg_end - 1);
          mk[mb][nb][p] = *(const VFL_GLOBAL u32x4*)(Mp + (rg * J.mask_rc.cp + n) * 16);
        }
    }
  }
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    const int n = n0 + wn * kWN + nb * 32 + col;
    const bool nok = n < N;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
      const int rl = wm * 128 + mb * 32;           // block row of the MFMA tile
      float v[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = m0 + rl + 8 * (e >> 2) + 4 * half + (e & 3);
        v[e] = (r < rows && nok) ? acc[mb][nb][e] : 0.f;
      }
      // 8-row groups g = 0..3 of the MFMA tile: half 0 holds rows 0..3 of
      // each, half 1 rows 4..7.  After one exchange per pair (2p, 2p + 1),
      // half 0 holds group 2p whole and half 1 group 2p + 1, in w[8p ..]
      float w[16];
#pragma unroll
      for (int p = 0; p < 2; ++p) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float send = half ? v[8 * p + i] : v[8 * p + 4 + i];
          const float got = __shfl_xor(send, 32, 64);
          w[8 * p + i] = half ? got : v[8 * p + i];
          w[8 * p + 4 + i] = half ? v[8 * p + 4 + i] : got;
        }
      }
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const int64_t rg = (m0 + rl) / 8 + 2 * p + half;
        if (!nok || rg >= rg_end) continue;
        float o[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = w[8 * p + i];
        if (J.mask_rc.p) {
          const u32x4 m = mk[mb][nb][p];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            o[2 * i] = __uint_as_float(m[i] << 16) > 0.f ? o[2 * i] : 0.f;
            o[2 * i + 1] = __uint_as_float(m[i] & 0xffff0000u) > 0.f ? o[2 * i + 1] : 0.f;
          }
        }
        const u32x4 q = u32x4{pack_bf16(o[0], o[1]), pack_bf16(o[2], o[3]), pack_bf16(o[4], o[5]),
                              pack_bf16(o[6], o[7])};
        *(VFL_GLOBAL u32x4*)(glb((char*)J.out_rc.p) + (rg * J.out_rc.cp + n) * 16) = q;
      }
    }
  }
}

}  // namespace

hipError_t gemm_init() {
  return hipFuncSetAttribute((const void*)k_gemm, hipFuncAttributeMaxDynamicSharedMemorySize, kGemmLds);
}

// blocks of a launch: the tiles rounded up to a multiple of the 8 XCDs
int gemm_tiles(int rows, int N) { return (((rows + kTM - 1) / kTM) * ((N + kTN - 1) / kTN) + 7) / 8 * 8; }

hipError_t launch_gemm(const GemmJob* job, int blocks, const void* A, int64_t lda, int rows, TickRef tr,
                       hipStream_t st) {
  if (blocks < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_gemm, dim3(blocks), dim3(256), kGemmLds, st, job, A, lda, rows, tr);
  return hipGetLastError();
}

}  // namespace vfl
