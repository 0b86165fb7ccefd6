// Input gradient of party B's wide first layer on gfx950 (k_lin; see
// kernels.h for the job): the chain's last delta (row-major) times the
// stashed weight copy, masked by the ReLU derivative of the layer below,
// in the RC layout the weight gradient reads.
//
// A block of 256 threads owns a 256-row x 256-output tile; K goes through
// LDS in stages of 32 (five 32 KB buffers, one barrier per stage).  Each stage is copied from global memory straight
// into LDS (global_load_lds_dwordx4: no registers, no LDS store
// instructions) in the order the matrix cores read it: one 1 KB block per
// 32 x 16 operand fragment of v_mfma_f32_32x32x16_bf16, lane l's 16 bytes
// at byte 16 l (row or output l mod 32, k chunk l / 32).  Every fragment
// read is then one contiguous ds_read_b128 per lane with no bank
// conflicts.  Waves 0 and 1 copy the A fragments (32-row slabs 0-3 and
// 4-7), waves 2 and 3 the W fragments (gathered from the packed weight
// copy, whose 16 x 32 fragments hold the same 16-byte chunks in another
// order).  Wavefront (wm, wn) of the 2 x 2 grid computes 128 x 128 of the
// tile: per 16-deep step 4 A and 4 W fragments feed 16 MFMAs, and the next
// stage's fragment reads are issued between the two steps of a stage.  The
// tiles are dealt to
// the XCDs in contiguous ranges, so the output tiles that share an A row
// slab meet in one L2.
//
// Epilogue: a lane holds one output column and four runs of four rows of
// each 32 x 32 MFMA tile.  The tile goes through LDS as bf16, column by
// column (8-byte writes of four rows); each thread then owns one column and
// writes its 8-row chunks, masked by the bit mask of the layer below (a byte
// per chunk): every store is a full 16-byte chunk and a store instruction
// writes 64 consecutive chunks.  Rows
// past the group are written as zeros, up to the padded row count.
#include "device.h"
#include "kernels.h"

namespace vfl {
namespace {
using namespace dev;

constexpr int kBM = 256, kBN = 256, kBK = 32;          // block tile, K per stage
constexpr int kFragBytes = 1024;                        // one 32 x 16 bf16 operand fragment
constexpr int kAFrags = kBM / 32 * (kBK / 16);          // A fragments per stage (16)
constexpr int kWFrags = kBN / 32 * (kBK / 16);          // W fragments per stage (16)
constexpr int kStageBytes = (kAFrags + kWFrags) * kFragBytes;   // 32 KB
constexpr int kStages = 5;                              // buffers: up to 4 stages in flight
// epilogue staging: the tile column by column, kOutPitch bytes per column,
// its 8-row chunks swizzled (see out_slot) so that both the lanes' 8-byte
// writes and the threads' 16-byte reads spread over the LDS banks
constexpr int kOutPitch = kBM * 2 + 32;
// then the tile's mask bytes: kBM / 8 row groups of kBN bytes
constexpr int kBitsOff = kBN * kOutPitch;
constexpr int kEpiLds = kBitsOff + kBM / 8 * kBN;
constexpr int kLinLds = kEpiLds > kStages * kStageBytes ? kEpiLds : kStages * kStageBytes;

// byte offset of rows 8 rg .. 8 rg + 7 of tile column c in the staging
__device__ __forceinline__ int out_slot(int c, int rg) { return c * kOutPitch + 16 * (rg ^ ((c >> 3) & 31)); }

typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((address_space(3))) void lds_t;

// 16 bytes per lane from global memory into LDS at lds + 16 * lane
__device__ __forceinline__ void dma16(const VFL_GLOBAL char* g, char* lds) {
  __builtin_amdgcn_global_load_lds((VFL_GLOBAL void*)g, (lds_t*)lds, 16, 0, 0);
}

// wait until at most n (0, 8, 16 or 24) of this wave's vector-memory operations
// are outstanding (expcnt and lgkmcnt unconstrained)
__device__ __forceinline__ void wait_vm(int n) {
  if (n >= 24) __builtin_amdgcn_s_waitcnt((1 << 14) | (15 << 8) | (7 << 4) | 8);
  else if (n >= 16) __builtin_amdgcn_s_waitcnt((1 << 14) | (15 << 8) | (7 << 4));
  else if (n >= 8) __builtin_amdgcn_s_waitcnt((15 << 8) | (7 << 4) | 8);
  else __builtin_amdgcn_s_waitcnt((15 << 8) | (7 << 4));
}

__global__ __launch_bounds__(256) void k_lin(const LinJob* __restrict__ jp, int rows_arg, TickRef tr) {
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const LinJob& J = *jp;
  const int rows = tr.src ? tick_args(tr).rows : rows_arg;
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
  const VFL_GLOBAL char* Ag = glb((const char*)J.A);
  const VFL_GLOBAL char* Wg = glb((const char*)J.W);
  const int64_t lda_c = J.lda / 8;             // 16-byte chunks per A row
  const int kst = J.kst;
  const int nst = kst;                         // 32-deep stages: one packed step each
  const int ntl = (N + 15) / 16;               // 16-output tiles of the packing
  // the lane's source row (A) or output (W) of the four slabs this wave
  // copies: A rows past the group repeat its last row (their outputs are
  // not kept); outputs past the packing repeat its last tile.  The source
  // of 16-deep step k16 of stage s is src[q] + min(step s + sdel[k16], cap)
  // * unit + sofs[k16] bytes: A chunk 4 s + 2 k16 + hi of the row (clamped
  // to the row), W packed step s, its 8-k chunk 2 k16 + hi
  const bool copies_a = wave < 2;
  const int wq = copies_a ? wave : wave - 2;
  const VFL_GLOBAL char* src[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t row = min(m0 + 32 * (4 * wq + q) + col, rows - 1);
    const int n = n0 + 32 * (4 * wq + q) + col;
    const int tl = min(n / 16, ntl - 1);
    src[q] = copies_a ? Ag + row * lda_c * 16 : Wg + ((int64_t)tl * kst * 64 + (n & 15)) * 16;
  }
  const int step = copies_a ? 4 : 1;
  const int cap = copies_a ? (int)(lda_c - 1) : kst - 1;
  const int64_t unit = copies_a ? 16 : 1024;
  int sdel[2], sofs[2];
#pragma unroll
  for (int k16 = 0; k16 < 2; ++k16) {
    sdel[k16] = copies_a ? 2 * k16 + hi : 0;
    sofs[k16] = copies_a ? 0 : 256 * (2 * k16 + hi);
  }
  // stage s into buffer s mod kStages: fragment i of this wave's 8 (slab
  // 4 wq + i / 2, 16-deep step i % 2) goes to fragment 8 wq + i of its
  // operand's region
  auto issue = [&](int s) {
    char* dst = smem + (s % kStages) * kStageBytes + (copies_a ? 0 : kAFrags * kFragBytes) + wq * 8 * kFragBytes;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int q = i >> 1, k16 = i & 1;
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
      a[mb] = *(const u32x4*)(S + ((4 * wm + mb) * 2 + k16) * kFragBytes + lane * 16);
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
      w[nb] = *(const u32x4*)(S + (kAFrags + (4 * wn + nb) * 2 + k16) * kFragBytes + lane * 16);
  };
  auto mma = [&](const u32x4 (&a)[4], const u32x4 (&w)[4]) {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8, a[mb]), __builtin_bit_cast(bf16x8, w[nb]), acc[mb][nb], 0, 0, 0);
  };

  // Software pipeline: the fragment reads of stage s + 1 are issued between
  // the two halves of stage s's products (two register sets), after the
  // barrier that makes stage s + 1 visible; that barrier also retires the
  // buffer of stage s - 1, which then takes the copies of stage
  // s + kStages - 1.  (Bare barriers: a fenced one would make every wave
  // wait for all of its copies in flight, the later stages' included.)
  struct Frags { u32x4 a0[4], w0[4], a1[4], w1[4]; };
  auto read_stage = [&](int s, Frags& f) {
    const char* S = smem + (s % kStages) * kStageBytes;
    frags(S, 0, f.a0, f.w0);
    frags(S, 1, f.a1, f.w1);
  };
  auto run_stage = [&](int s, const Frags& x, Frags& y) {
    if (s + 1 < nst) {
      // this wave's copies of stage s + 1 have landed (later stages may be
      // in flight); after the barrier every wave's have
      wait_vm(8 * min(kStages - 3, nst - 2 - s));
      __builtin_amdgcn_s_barrier();
      if (s + kStages - 1 < nst) issue(s + kStages - 1);
    }
    // the wait for x (read a step earlier) comes before the first half;
    // nothing waits for y until the next step (after the last stage a
    // harmless re-read of it, so that y is always written and the two
    // register sets are never both live across a step).  The scheduling
    // barriers keep the compiler from sinking each read to its first use.
    __builtin_amdgcn_sched_barrier(0);
    mma(x.a0, x.w0);
    __builtin_amdgcn_sched_barrier(0);
    read_stage(min(s + 1, nst - 1), y);
    __builtin_amdgcn_sched_barrier(0);
    mma(x.a1, x.w1);
  };
  for (int s = 0; s < kStages - 1 && s < nst; ++s) issue(s);
  Frags fa, fb;
  wait_vm(8 * min(kStages - 2, nst - 1));
  __builtin_amdgcn_s_barrier();
  read_stage(0, fa);
  {
    int s = 0;
#pragma unroll 1
    for (; s + 1 < nst; s += 2) {
      run_stage(s, fa, fb);
      run_stage(s + 1, fb, fa);
    }
    if (s < nst) run_stage(s, fa, fb);
  }

  // ------------------------------------------------------------ epilogue
  // 1. each wave puts its 128 x 128 part of the tile into LDS as bf16,
  //    column-major: lane (col, hi) holds column 128 wn + 32 nb + col and
  //    rows 128 wm + 32 mb + 8 g + 4 hi + (0 .. 3) in acc[mb][nb][4 g ..],
  //    four consecutive rows of one column, written as 8 bytes
  __syncthreads();                             // the last stage's reads are done
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) {
    const int cl = 128 * wn + 32 * nb + col;   // tile column
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x16& x = acc[mb][nb];
        const int rg = 16 * wm + 4 * mb + g;   // 8-row group of the tile
        *(u32x2*)(smem + out_slot(cl, rg) + 8 * hi) =
            u32x2{pack_bf16(x[4 * g], x[4 * g + 1]), pack_bf16(x[4 * g + 2], x[4 * g + 3])};
      }
  }
  //    and the tile's mask bytes (the ReLU derivative of the layer below:
  //    row-group-major, so each row group's 256 bytes are one contiguous
  //    run) go to LDS beside it, 16 bytes per thread and load
  if (J.mbits) {
    const VFL_GLOBAL uint8_t* bp = glb(J.mbits);
    for (int u = t; u < kBM / 8 * (kBN / 16); u += 256) {
      const int g = u / (kBN / 16), ch = u % (kBN / 16);
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (m0 / 8 + g < rg_end && n0 + 16 * ch + 16 <= J.ldb)
        v = *(const VFL_GLOBAL u32x4*)(bp + (int64_t)(m0 / 8 + g) * J.ldb + n0 + 16 * ch);
      *(u32x4*)(smem + kBitsOff + g * kBN + 16 * ch) = v;
    }
  }
  __syncthreads();
  // 2. the RC output: thread t owns tile column t and walks its 8-row
  //    chunks, so that each store instruction writes 64 consecutive chunks
  //    of one row group
  if (n0 + t < N) {
    const int n = n0 + t;
    VFL_GLOBAL u32x4* dst = (VFL_GLOBAL u32x4*)glb((char*)J.out_rc.p) + n;
    const int ng = (int)min((int64_t)kBM / 8, rg_end - m0 / 8);   // row groups inside the padded rows
    uint32_t mb[kBM / 32];
#pragma unroll
    for (int i = 0; i < kBM / 32; ++i) mb[i] = ~0u;
    if (J.mbits) {
#pragma unroll
      for (int i = 0; i < kBM / 32; ++i) {
        uint32_t w = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) w |= (uint32_t)*(const uint8_t*)(smem + kBitsOff + (4 * i + b) * kBN + t) << (8 * b);
        mb[i] = w;
      }
    }
    // fully unrolled: the mask words stay in registers (a runtime index
    // would put them in scratch memory)
#pragma unroll
    for (int rg = 0; rg < kBM / 8; ++rg) {
      if (rg >= ng) break;
      const int64_t g = m0 / 8 + rg;
      u32x4 q = mask_tail<uint16_t>(*(const u32x4*)(smem + out_slot(t, rg)), rows - (m0 + 8 * rg));
      const uint32_t byte = mb[rg >> 2] >> (8 * (rg & 3));
#pragma unroll
      for (int w = 0; w < 4; ++w)
        q[w] &= ((byte >> (2 * w)) & 1u ? 0x0000ffffu : 0u) | ((byte >> (2 * w + 1)) & 1u ? 0xffff0000u : 0u);
      __builtin_nontemporal_store(q, dst + g * J.out_rc.cp);   // read back by the next launch from HBM
    }
  }
}

}  // namespace

hipError_t lin_init() {
  return hipFuncSetAttribute((const void*)k_lin, hipFuncAttributeMaxDynamicSharedMemorySize, kLinLds);
}

// blocks of a launch: the tiles rounded up to a multiple of the 8 XCDs
int lin_blocks(int rows_pad, int N) {
  return (((rows_pad + kBM - 1) / kBM) * ((N + kBN - 1) / kBN) + 7) / 8 * 8;
}

hipError_t launch_lin(const LinJob* job, int blocks, int rows, TickRef tr, hipStream_t st) {
  if (blocks < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_lin, dim3(blocks), dim3(256), kLinLds, st, job, rows, tr);
  return hipGetLastError();
}

}  // namespace vfl
