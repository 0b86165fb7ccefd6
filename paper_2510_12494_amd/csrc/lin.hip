// Products of party B's wide bottom layers on gfx950 (k_lin; see kernels.h
// for the job): the forward product with bias and ReLU, and the input
// gradient masked by the ReLU derivative of the layer below.
//
// A block of 256 threads owns a 256-row x 256-output tile; K goes through
// LDS in stages of 64 (double-buffered, 2 x 64 KB).  Each stage is copied
// from global memory straight into LDS (global_load_lds_dwordx4: no
// registers, no LDS store instructions) in the order the matrix cores read
// it: one 1 KB block per 32 x 16 operand fragment of
// v_mfma_f32_32x32x16_bf16, lane l's 16 bytes at byte 16 l (row or output
// l mod 32, k chunk l / 32).  Every fragment read is then one contiguous
// ds_read_b128 per lane with no bank conflicts.  Waves 0 and 1 copy the
// A fragments (32-row slabs 0-3 and 4-7), waves 2 and 3 the W fragments
// (gathered from the packed weight copy, whose 16 x 32 fragments hold the
// same 16-byte chunks in another order).  Wavefront (wm, wn) of the 2 x 2
// grid computes 128 x 128 of the tile: per 16-deep step 4 A and 4 W
// fragments feed 16 MFMAs.  The tiles are dealt to the XCDs in contiguous
// ranges, so the output tiles that share an A row slab meet in one L2.
//
// Epilogue: a lane holds one output column and four runs of four rows of
// each 32 x 32 MFMA tile.  The forward product adds the bias, applies the
// ReLU and stores the row-major output element by element (the 32 lanes of
// a half-wavefront write 64 contiguous bytes of one row); for the RC
// output the runs of lanes l and l + 32 are exchanged so that each lane
// holds two whole 8-row chunks of its column, masked chunk by chunk by the
// RC mask (input gradient).  Rows past the group are written as zeros in
// the RC output, up to the padded row count.
#include "device.h"
#include "kernels.h"

namespace vfl {
namespace {
using namespace dev;

constexpr int kBM = 256, kBN = 256, kBK = 64;          // block tile, K per stage
constexpr int kFragBytes = 1024;                        // one 32 x 16 bf16 operand fragment
constexpr int kAFrags = kBM / 32 * (kBK / 16);          // A fragments per stage (32)
constexpr int kWFrags = kBN / 32 * (kBK / 16);          // W fragments per stage (32)
constexpr int kStageBytes = (kAFrags + kWFrags) * kFragBytes;
constexpr int kLinLds = 2 * kStageBytes;                // 128 KB

typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((address_space(3))) void lds_t;

// 16 bytes per lane from global memory into LDS at lds + 16 * lane
__device__ __forceinline__ void dma16(const VFL_GLOBAL char* g, char* lds) {
  __builtin_amdgcn_global_load_lds((VFL_GLOBAL void*)g, (lds_t*)lds, 16, 0, 0);
}

// A_arg: the A operand of this launch (the group's rows of a dataset or of a
// caller batch, lda_arg elements per row; with a tick reference the dataset
// base, offset by the tick's first row), or null: the job's workspace
// operand (rows of the tick).
__global__ __launch_bounds__(256) void k_lin(const LinJob* __restrict__ jp, const void* A_arg,
                                             int64_t lda_arg, int rows_arg, TickRef tr) {
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const LinJob& J = *jp;
  int rows = rows_arg;
  int64_t a_row0 = 0;
  if (tr.src) {
    const TickArgs ta = tick_args(tr);
    rows = ta.rows;
    if (A_arg) a_row0 = ta.row0;
  }
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int col = lane & 31, hi = lane >> 5;
  // workgroups are dealt to the 8 XCDs round-robin (block b on XCD b mod
  // 8): XCD x takes the contiguous tile range [x * per, (x + 1) * per)
  const int ntiles = J.tiles_n * J.tiles_m;
  const int per = (ntiles + 7) / 8;
  const int tile = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (tile >= ntiles) return;
  const int tile_n = tile % J.tiles_n, tile_m = tile / J.tiles_n;
  const int m0 = tile_m * kBM, n0 = tile_n * kBN;
  const int N = J.N;
  const int64_t rg_end = J.rows_pad / 8;       // RC row groups of the outputs
  const bool rc_out = J.out_rc.p != nullptr;

  if (m0 >= rows) {
    // rows past the group: zero RC chunks (up to the padded row count)
    if (!rc_out) return;
    for (int c = t; c < kBM / 8 * kBN; c += 256) {
      const int rg = c / kBN, n = n0 + c % kBN;
      const int64_t g = m0 / 8 + rg;
      if (n >= N || g >= rg_end) continue;
      *(VFL_GLOBAL u32x4*)(glb((char*)J.out_rc.p) + (g * J.out_rc.cp + n) * 16) = u32x4{0u, 0u, 0u, 0u};
    }
    return;
  }

  // ------------------------------------------------------------ main loop
  const VFL_GLOBAL char* Ag = glb((const char*)(A_arg ? A_arg : J.A));
  const VFL_GLOBAL char* Wg = glb((const char*)J.W);
  const int64_t lda_c = (A_arg ? lda_arg : J.lda) / 8;   // 16-byte chunks per A row
  const int kst = J.kst;
  const int Kp = 32 * kst;                     // K of the packing (zero from K on)
  const int nst = (Kp + kBK - 1) / kBK;
  const int ntl = (N + 15) / 16;               // 16-output tiles of the packing
  // the lane's source row (A) or output (W) of the four slabs this wave
  // copies: A rows past the group repeat its last row (their outputs are
  // not kept); outputs past the packing repeat its last tile.  The source
  // of 16-deep step k16 of stage s is src[q] + min(step s + sdel[k16], cap)
  // * unit + sofs[k16] bytes: A chunk 8 s + 2 k16 + hi of the row (clamped
  // to the row), W packed step 2 s + k16 / 2 (clamped to the packing), its
  // 8-k chunk 2 (k16 mod 2) + hi
  const bool copies_a = wave < 2;
  const int wq = copies_a ? wave : wave - 2;
  const VFL_GLOBAL char* src[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t row = a_row0 + min(m0 + 32 * (4 * wq + q) + col, rows - 1);
    const int n = n0 + 32 * (4 * wq + q) + col;
    const int tl = min(n / 16, ntl - 1);
    src[q] = copies_a ? Ag + row * lda_c * 16 : Wg + ((int64_t)tl * kst * 64 + (n & 15)) * 16;
  }
  const int step = copies_a ? 8 : 2;
  const int cap = copies_a ? (int)(lda_c - 1) : kst - 1;
  const int64_t unit = copies_a ? 16 : 1024;
  int sdel[4], sofs[4];
#pragma unroll
  for (int k16 = 0; k16 < 4; ++k16) {
    sdel[k16] = copies_a ? 2 * k16 + hi : k16 >> 1;
    sofs[k16] = copies_a ? 0 : 256 * (2 * (k16 & 1) + hi);
  }
  // stage s into buffer b: fragment i of this wave's 16 (slab 4 wq + i / 4,
  // 16-deep step i % 4) goes to fragment 16 wq + i of its operand's region
  auto issue = [&](int s, int b) {
    char* dst = smem + b * kStageBytes + (copies_a ? 0 : kAFrags * kFragBytes) + wq * 16 * kFragBytes;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int q = i >> 2, k16 = i & 3;
      dma16(src[q] + (int64_t)min(step * s + sdel[k16], cap) * unit + sofs[k16], dst + i * kFragBytes);
    }
  };

  const int wm = wave >> 1, wn = wave & 1;
  f32x16 acc[4][4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[mb][nb][e] = 0.f;

  // the fragments of 16-deep step k16 of the buffer at S
  auto frags = [&](const char* S, int k16, u32x4 (&a)[4], u32x4 (&w)[4]) {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
      a[mb] = *(const u32x4*)(S + ((4 * wm + mb) * 4 + k16) * kFragBytes + lane * 16);
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
      w[nb] = *(const u32x4*)(S + (kAFrags + (4 * wn + nb) * 4 + k16) * kFragBytes + lane * 16);
  };
  auto mma = [&](const u32x4 (&a)[4], const u32x4 (&w)[4]) {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8, a[mb]), __builtin_bit_cast(bf16x8, w[nb]), acc[mb][nb], 0, 0, 0);
  };

  // scheduling of one step: its 16 products with the next step's 8
  // fragment reads issued between the first 8, so that the reads are back
  // long before the products that need them
  auto interleave = [] {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
  };

  issue(0, 0);
#pragma unroll 1
  for (int s = 0; s < nst; ++s) {
    const int b = s & 1;
    // this wave's copies of stage s have landed; after the barrier every
    // wave's have, and every wave is done reading buffer b ^ 1
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (s + 1 < nst) issue(s + 1, b ^ 1);
    const char* S = smem + b * kStageBytes;
    // the packing ends at a multiple of 32: the last stage may hold only
    // two 16-deep steps.  Each step's fragments are read while the
    // previous step's products run.
    const bool full = Kp - s * kBK >= kBK;
    u32x4 a0[4], w0[4], a1[4], w1[4];
    frags(S, 0, a0, w0);
    frags(S, 1, a1, w1);
    mma(a0, w0);
    interleave();
    if (full) {
      frags(S, 2, a0, w0);
      mma(a1, w1);
      interleave();
      frags(S, 3, a1, w1);
      mma(a0, w0);
      interleave();
    }
    mma(a1, w1);
  }

  // ------------------------------------------------------------ epilogue
  // lane: column n = n0 + 128 wn + 32 nb + col; rows
  // m0 + 128 wm + 32 mb + 8 g + 4 hi + (0 .. 3) in acc[mb][nb][4 g ..]
  const bool fwd = J.bias != nullptr;
  const bool relu = J.relu != 0;
  const bool masked = J.mask_rc.p != nullptr;
  VFL_GLOBAL uint16_t* orm = glb((uint16_t*)J.out_rm);
  const int64_t ldo = J.ldo;
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) {
    const int n = n0 + 128 * wn + 32 * nb + col;
    const bool nok = n < N;
    const int nc = min(n, N - 1);
    const float bias = fwd ? glb(J.bias)[nc] : 0.f;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
      const int rl = m0 + 128 * wm + 32 * mb;    // first row of the MFMA tile
      // the tile's mask chunks (8-row group 2 p + hi of the column), loaded
      // before they are needed
      u32x4 mk[2];
      if (masked) {
        const VFL_GLOBAL char* Mp = glb((const char*)J.mask_rc.p);
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const int64_t rg = min((int64_t)rl / 8 + 2 * p + hi, rg_end - 1);
          mk[p] = *(const VFL_GLOBAL u32x4*)(Mp + (rg * J.mask_rc.cp + nc) * 16);
        }
      }
      float v[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = rl + 8 * (e >> 2) + 4 * hi + (e & 3);
        float x = acc[mb][nb][e];
        if (fwd) {
          x += bias;
          if (relu) x = fmaxf(x, 0.f);
        }
        v[e] = (r < rows && nok) ? x : 0.f;
      }
      if (orm && nok) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int r = rl + 8 * (e >> 2) + 4 * hi + (e & 3);
          if (r < rows) orm[(int64_t)r * ldo + n] = (uint16_t)pack_bf16(v[e], 0.f);
        }
      }
      if (!rc_out) continue;
      // 8-row groups g = 0..3 of the MFMA tile: half 0 holds rows 0..3 of
      // each, half 1 rows 4..7.  After one exchange per pair (2p, 2p + 1),
      // half 0 holds group 2p whole and half 1 group 2p + 1, in w[8p ..]
      float w[16];
#pragma unroll
      for (int p = 0; p < 2; ++p) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float send = hi ? v[8 * p + i] : v[8 * p + 4 + i];
          const float got = __shfl_xor(send, 32, 64);
          w[8 * p + i] = hi ? got : v[8 * p + i];
          w[8 * p + 4 + i] = hi ? v[8 * p + 4 + i] : got;
        }
      }
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const int64_t rg = rl / 8 + 2 * p + hi;
        if (!nok || rg >= rg_end) continue;
        float o[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = w[8 * p + i];
        if (masked) {
          const u32x4 m = mk[p];
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

// RC copy of a row-major bf16 input [rows x K] (lda elements per row; A as
// for k_lin): one thread per 8-row x 8-column block, transposed in
// registers.  Columns from K and rows from the group's end up to rows_pad
// are written as zeros.
__global__ __launch_bounds__(256) void k_rows_rc(const void* A, int64_t lda, int K, RCMat out, int rows_arg,
                                                 int rows_pad, TickRef tr) {
  int rows = rows_arg;
  int64_t a_row0 = 0;
  if (tr.src) {
    const TickArgs ta = tick_args(tr);
    rows = ta.rows;
    a_row0 = ta.row0;
  }
  const int nkc = out.cp / 8;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t rg = idx / nkc;
  const int kc = (int)(idx - rg * nkc);
  if (rg * 8 >= rows_pad) return;
  const VFL_GLOBAL uint16_t* a = glb((const uint16_t*)A);
  u32x4 in[8], o[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int64_t r = rg * 8 + i;
    in[i] = r < rows ? mask_tail<uint16_t>(*(const VFL_GLOBAL u32x4*)(a + (a_row0 + r) * lda + 8 * kc), K - 8 * kc)
                     : u32x4{0u, 0u, 0u, 0u};
  }
  transpose8x8_u16(in, o);
  VFL_GLOBAL u32x4* dst = (VFL_GLOBAL u32x4*)glb((char*)out.p) + rg * out.cp + 8 * kc;
#pragma unroll
  for (int j = 0; j < 8; ++j) dst[j] = o[j];
}

}  // namespace

hipError_t launch_rows_rc(const void* A, int64_t lda, int K, RCMat out, int rows, int rows_pad, TickRef tr,
                          hipStream_t st) {
  const int64_t threads = (int64_t)(rows_pad + 7) / 8 * (out.cp / 8);
  if (threads < 1 || out.cp % 8 || out.cp < K) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_rows_rc, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, A, lda, K, out, rows,
                     rows_pad, tr);
  return hipGetLastError();
}

hipError_t lin_init() {
  return hipFuncSetAttribute((const void*)k_lin, hipFuncAttributeMaxDynamicSharedMemorySize, kLinLds);
}

// blocks of a launch: the tiles rounded up to a multiple of the 8 XCDs
int lin_blocks(int rows_pad, int N) {
  return (((rows_pad + kBM - 1) / kBM) * ((N + kBN - 1) / kBN) + 7) / 8 * 8;
}

hipError_t launch_lin(const LinJob* job, int blocks, const void* A, int64_t lda, int rows, TickRef tr,
                      hipStream_t st) {
  if (blocks < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_lin, dim3(blocks), dim3(256), kLinLds, st, job, A, lda, rows, tr);
  return hipGetLastError();
}

}  // namespace vfl
