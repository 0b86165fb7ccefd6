// Fused row-block kernels of the split-learning step on gfx950 (k_fwd,
// k_active, k_bwd; see kernels.h for what each computes).
//
// A workgroup of 512 threads (8 wavefronts, two per SIMD) owns BR = 16 * RT
// (RT = 1 .. 4) consecutive rows of the group and runs every layer of its chain on them,
// the activations and deltas staying in LDS.  Each layer is one MFMA product
// out[BR x N] = in[BR x K] W^T: wavefront w takes the 16-column output tiles
// w, w+8, w+16, ... (two at a time), loads the weight fragments of its tiles
// straight from global memory (L2-resident: the workgroups of an XCD fetch
// the kernel's weights into its L2 at the start) two groups of four MFMA
// steps ahead, across layer boundaries, and the activation fragments from
// LDS; biases come from an LDS table filled at the start;
// v_mfma_f32_16x16x32_bf16 for bf16 operands, v_mfma_f32_16x16x4_f32 for
// float32, float32 accumulation.  The weight fragment is the MFMA's A
// operand, so a lane ends up with four consecutive output columns of one row.
//
// LDS rows are padded to 16 bytes past a multiple of 128, so the 16 rows a
// fragment read touches fall in distinct banks.  After a layer, the tensors a
// later kernel needs go to HBM: row-major for messages, the RC layout for
// the operands of the weight gradients (8 x 8 register transposes of bf16
// chunks, 4 x 4 of float32).
//
// Paper correspondence: bottom models f_A, f_B and the top model g of
// Section 3, the BCE loss of Eq. (1) and its gradient, the embedding and
// gradient messages of Section 4.1 with the per-row clip and Gaussian noise
// of the differential-privacy appendix, and the cut-layer backward through
// the clip of B's published embedding.
#include "device.h"
#include "kernels.h"

namespace vfl {
namespace {
using namespace dev;

template <typename T>
struct Ch {
  static constexpr int CE = 16 / (int)sizeof(T);   // elements per chunk = rows per RC chunk
  static constexpr int KS = 4 * CE;                // contraction depth of one MFMA step
};

// values of this launch, from the call or the tick record
struct Call {
  int rows, group, chk;
  int64_t row0;      // sample id of the group's row 0 (noise counter)
  int64_t in_off;    // dataset row offset of the inputs
  int32_t hdr[3];
};

__device__ __forceinline__ Call resolve(const ChainCall& c, const TickRef& tr) {
  Call k;
  if (tr.src) {
    const TickArgs ta = tick_args(tr);
    k.rows = ta.rows; k.group = ta.group; k.chk = ta.chk;
    k.row0 = ta.row0; k.in_off = ta.row0;
    k.hdr[0] = ta.hdr[0]; k.hdr[1] = ta.hdr[1]; k.hdr[2] = ta.hdr[2];
  } else {
    k.rows = c.rows; k.group = c.group; k.chk = c.chk;
    k.row0 = c.row0; k.in_off = 0;
    k.hdr[0] = c.hdr[0]; k.hdr[1] = c.hdr[1]; k.hdr[2] = c.hdr[2];
  }
  return k;
}

__device__ __forceinline__ char* lp(char* s, const LBuf& b, int r, int byte_col) {
  return s + b.off + r * b.pitch + byte_col;
}

// eight consecutive elements of an LDS row (16 bytes of bf16, 32 of float32)
template <typename T>
__device__ __forceinline__ void ld8(const char* p, float (&v)[8]) {
  if constexpr (sizeof(T) == 4) {
    const f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 16);
#pragma unroll
    for (int e = 0; e < 4; ++e) { v[e] = a[e]; v[4 + e] = b[e]; }
  } else {
    const u32x4 x = *(const u32x4*)p;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] = __uint_as_float(x[e] << 16);
      v[2 * e + 1] = __uint_as_float(x[e] & 0xffff0000u);
    }
  }
}
template <typename T>
__device__ __forceinline__ void st8(char* p, const float (&v)[8]) {
  if constexpr (sizeof(T) == 4) {
    *(f32x4*)p = f32x4{v[0], v[1], v[2], v[3]};
    *(f32x4*)(p + 16) = f32x4{v[4], v[5], v[6], v[7]};
  } else {
    *(u32x4*)p = u32x4{pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3]), pack_bf16(v[4], v[5]), pack_bf16(v[6], v[7])};
  }
}

// ------------------------------------------------------------ block product
constexpr int kNW = kChainWaves;    // wavefronts per block (two per SIMD)
constexpr int kNT = 64 * kNW;        // threads per block
constexpr int kNTW = 2;              // 16-column output tiles per wavefront and pass
constexpr int kPFNarrow = kChainPFNarrow;   // MFMA steps per weight load group
constexpr int kPFWide = kChainPFWide;
constexpr int kLogitChunks = kMaxLogitCols / 256;   // 4-column chunks per lane in the logit stage

// Weight-fragment registers of a chain: two load groups of PF MFMA steps
// (ping-pong).  The groups of a chain's products form one stream: when a
// wavefront has issued the loads of a pass's last group, the next two loads
// it issues are groups 0 and 1 of the next pass or of the next product, so
// a product starts with both of its first groups already in flight.  A
// pass has an even number of groups (steps past K are skipped), so every
// pass starts in `wa`.
template <int PF>
struct Pipe {
  u32x4 wa[PF][kNTW], wb[PF][kNTW];
};

// The RC copy of a stage's LDS output (lds_to_rc of b's first cols columns
// into m at block row r0; m.p null: none), left for the next product to
// issue.  On gfx950 stores count in the same in-order counter as loads, so
// a wait for any load issued after a store also waits for the store's
// write to complete; the next product issues the copy after its last
// weight loads, where nothing waits on them until the product after it.
struct RcPend {
  LBuf b;
  int cols = 0;
  RCMat m;
  int r0 = 0;
};

// A pointer or value the compiler must keep in scalar registers (it is
// uniform, but derived through selects the compiler may place in vector
// registers, and a field loaded through a vector-register pointer is a
// vector-memory load whose wait drains every load in flight).
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const void*)(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// A job descriptor read through the constant address space: the jobs are
// written once, before any launch, so their fields may come through the
// scalar cache (scalar loads, counted apart from the vector loads in flight)
// even after the kernel's own stores.
#define VFL_CONST __attribute__((address_space(4)))
template <typename X>
__device__ __forceinline__ const VFL_CONST X& cst(const X& x) {
  return *(const VFL_CONST X*)&x;
}

// 16-column tiles of a product of N output columns (up to the MFMA depth)
template <typename T>
__device__ __forceinline__ int tiles_of(int N) {
  constexpr int KS = Ch<T>::KS;
  return (N + KS - 1) / KS * (KS / 16);
}

// the loads of group g of a pass (tiles tile[]) of an operand W with kst
// K steps and ntl tiles into d: one contiguous 1 KB fragment per tile and
// step of the packed operand.  Loads are unconditional: tiles past the
// operand's last are clamped to it, steps past K to its last step (never
// used; re-reading lines already fetched keeps them off the L2, and a
// conditional load would make the compiler wait for it on the spot).
template <int PF>
__device__ __forceinline__ void wgroup(const void* Wp, int kst, int ntl, const int (&tile)[kNTW], int g,
                                       u32x4 (&d)[PF][kNTW]) {
  const uint32_t lo = (threadIdx.x & 63) * 16;
#pragma unroll
  for (int j = 0; j < kNTW; ++j) {
    const VFL_GLOBAL char* base = glb((const char*)Wp) + (int64_t)min(tile[j], ntl - 1) * kst * 1024 + lo;
#pragma unroll
    for (int q = 0; q < PF; ++q) d[q][j] = *(const VFL_GLOBAL u32x4*)(base + (int64_t)min(g * PF + q, kst - 1) * 1024);
  }
}

// the tiles of a wavefront's pass: wave + kNW * (kNTW * pass + j)
__device__ __forceinline__ void pass_tiles(int pass, int (&tile)[kNTW]) {
  const int wave = uniform((int)(threadIdx.x >> 6));
#pragma unroll
  for (int j = 0; j < kNTW; ++j) tile[j] = wave + kNW * (kNTW * pass + j);
}

// start the loads of groups 0 and 1 of L's first pass
template <typename T, int PF>
__device__ __forceinline__ void prefetch(const ChainLayer* L, Pipe<PF>& p) {
  int tile[kNTW];
  pass_tiles(0, tile);
  const VFL_CONST ChainLayer& C = cst(*(const ChainLayer*)uniform_ptr(L));
  const void* W = uniform_ptr(C.W);
  const int kst = uniform(C.kst), ntl = uniform(tiles_of<T>(C.N));
  wgroup(W, kst, ntl, tile, 0, p.wa);
  wgroup(W, kst, ntl, tile, 1, p.wb);
}

// Copy of a chain kernel's bias table into LDS (see BiasTab).
__device__ __forceinline__ void copy_bias(char* s, const BiasTab& b) {
  const VFL_GLOBAL f32x4* src = glb((const f32x4*)b.src);
  for (int i = threadIdx.x; i < b.n4; i += kNT) *(f32x4*)(s + b.off + 16 * i) = src[i];
}

// One 4-byte load per 128-byte line of this workgroup's slice of the
// kernel's weight ranges (slice = workgroup / 8 mod 32: the workgroups of
// one XCD share its L2), returned so that the caller can consume the values
// where it waits for its inputs anyway.  Up to 2 lines per thread and
// range; addresses are clamped into the range, so the loads are
// unconditional.
__device__ __forceinline__ uint32_t warm_l2(const WarmSet& w, const void* dummy) {
  const int slice = (blockIdx.x >> 3) & 31;
  uint32_t x = 0u;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int lines = w.lines[r];
    const int per = (lines + 31) >> 5;
    const int c0 = slice * per, c1 = min(lines, c0 + per);
    const VFL_GLOBAL uint32_t* base = glb((const uint32_t*)(lines > 0 ? w.p[r] : dummy));
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int c = c0 + (int)threadIdx.x + k * kNT;
      x ^= base[(int64_t)(c < c1 ? c : 0) * 32];
    }
  }
  return x;
}

// out[r][n] = epi(r, n, sum_k in[r][k] W[n][k], bias) for the block's rows:
// epi(r, n, acc, bias) receives block row r, output columns n .. n+3 (n a
// multiple of 4; bias[i] = bias[n + i] from the LDS table, zero without a
// bias or past N), for every row of the block and every column below N
// rounded up to the MFMA depth.  On entry p holds groups 0 and 1 of L's
// first pass; on return, groups 0 and 1 of `next`'s (nullable).  The
// pending RC copy (whose LDS rows this product does not write) is issued
// in the last pass once every weight load of the pass is out.
template <typename T, int BR, bool NT>
__device__ __forceinline__ void lds_to_rc_(const char* s, const LBuf& b, int cols, const RCMat& m, int r0);
template <typename T, int BR>
__device__ __forceinline__ void lds_to_rc_hint(const char* s, const LBuf& b, int cols, const RCMat& m, int r0);

template <typename T, int RT, typename Epi, bool HINT = false, int PF>
__device__ __forceinline__ void block_mm(const char* s, const ChainLayer& L, Pipe<PF>& p,
                                         const ChainLayer* next, const RcPend& pend, Epi&& epi) {
  constexpr int NTW = kNTW;
  const int lane = threadIdx.x & 63;
  const int kc = lane >> 4, lr = lane & 15;
  const VFL_CONST ChainLayer& C = cst(L);
  const void* W = uniform_ptr(C.W);
  const int ntl = uniform(tiles_of<T>(C.N));
  const int nks = uniform(C.kst);
  const int ng = ((nks + PF - 1) / PF + 1) & ~1;
  const int bl = uniform(C.bl);
  LBuf in;
  in.off = C.in.off;
  in.pitch = C.in.pitch;
  const int npass = (ntl + kNW * NTW - 1) / (kNW * NTW);
  // the next product's operand; past the chain's end the loads repeat this
  // product's (never used: every refill issues the same loads, so the
  // compiler's wait counts stay exact)
  next = (const ChainLayer*)uniform_ptr(next);
  const VFL_CONST ChainLayer& CN = cst(next ? *next : L);
  const void* nW = uniform_ptr(CN.W);
  const int nkst = uniform(CN.kst), nntl = uniform(tiles_of<T>(CN.N));
#pragma unroll 1
  for (int pass = 0; pass < npass; ++pass) {
    int tile[NTW], ntile[NTW];
    pass_tiles(pass, tile);
    // where the loads go once this pass's groups are all issued: the next
    // pass, or the next product's first
    const bool more = pass + 1 < npass;
    pass_tiles(more ? pass + 1 : 0, ntile);
    const void* rW = more ? W : nW;
    const int rkst = more ? nks : nkst, rntl = more ? ntl : nntl;
    f32x4 acc[NTW][RT];
#pragma unroll
    for (int j = 0; j < NTW; ++j)
#pragma unroll
      for (int t = 0; t < RT; ++t) acc[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto step = [&](int ks, const u32x4 (&w)[NTW]) {
      if (ks >= nks) return;
      u32x4 xf[RT];
#pragma unroll
      for (int t = 0; t < RT; ++t)
        xf[t] = *(const u32x4*)(s + in.off + (t * 16 + lr) * in.pitch + (ks * 4 + kc) * 16);
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        if (tile[j] >= ntl) continue;
#pragma unroll
        for (int t = 0; t < RT; ++t) {
          if constexpr (sizeof(T) == 2) {
            acc[j][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, w[j]), __builtin_bit_cast(bf16x8, xf[t]), acc[j][t], 0, 0, 0);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              acc[j][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                  __uint_as_float(w[j][e]), __uint_as_float(xf[t][e]), acc[j][t], 0, 0, 0);
          }
        }
      }
    };
    auto group = [&](int g, const u32x4 (&w)[PF][NTW]) {
#pragma unroll
      for (int q = 0; q < PF; ++q) step(g * PF + q, w[q]);
    };
    // group g of this pass into w, or group g - ng of the next pass/product
    auto refill = [&](int g, u32x4 (&w)[PF][NTW]) {
      const bool cur = g < ng;
      int tt[NTW];
#pragma unroll
      for (int j = 0; j < NTW; ++j) tt[j] = cur ? tile[j] : ntile[j];
      wgroup(cur ? W : rW, cur ? nks : rkst, cur ? ntl : rntl, tt, cur ? g : g - ng, w);
    };
#pragma unroll 1
    for (int g = 0; g < ng; g += 2) {
      group(g, p.wa);
      refill(g + 2, p.wa);
      group(g + 1, p.wb);
      refill(g + 3, p.wb);
    }
    if (!more && pend.m.p) {
      if constexpr (HINT) lds_to_rc_hint<T, 16 * RT>(s, pend.b, pend.cols, pend.m, pend.r0);
      else lds_to_rc_<T, 16 * RT, false>(s, pend.b, pend.cols, pend.m, pend.r0);
    }
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
      if (tile[j] >= ntl) continue;
      const int n = tile[j] * 16 + 4 * kc;
      const f32x4 bv = bl >= 0 ? *(const f32x4*)(s + bl + 4 * n) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < RT; ++t) epi(t * 16 + lr, n, acc[j][t], bv);
    }
  }
}

// Forward or input-gradient layer into LDS (see ChainLayer).
// MB: the mask (when there is one) is the byte form of the ReLU bits
template <typename T, int RT, bool HINT = false, int PF, bool MB = false>
__device__ __forceinline__ void run_layer(char* s, const ChainLayer& L, int rv, Pipe<PF>& p,
                                          const ChainLayer* next, const RcPend& pend) {
  const int N = L.N;
  const bool relu = L.relu != 0, msk = L.mask.pitch > 0, nopad = L.nopad != 0;
  const LBuf out = L.out, mk = L.mask;
  // branch-free: every condition is a select (a short-circuit test here
  // compiles to one exec-mask branch per element)
  auto epi = [&](int r, int n, const f32x4& a, const f32x4& b) {
    float m[4] = {1.f, 1.f, 1.f, 1.f}, v[4];
    if constexpr (MB) {
      if (msk) {
        // the 4 columns' bytes of r's row group in one word
        const uint32_t w = *(const uint32_t*)(s + mk.off + (r >> 3) * mk.pitch + n);
#pragma unroll
        for (int i = 0; i < 4; ++i) m[i] = (w >> (8 * i + (r & 7))) & 1u ? 1.f : 0.f;
      }
    } else {
      if (msk) ld4<T>(lp(s, mk, r, n * (int)sizeof(T)), m);
    }
    const bool rok = r < rv;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float x0 = a[i] + b[i];
      const float x = relu ? fmaxf(x0, 0.f) : x0;
      const bool keep = rok & (n + i < N) & (m[i] > 0.f);
      v[i] = keep ? x : 0.f;
    }
    // n is a multiple of 4 and a nopad N of 8: the four columns are all
    // below N or all past it
    if (!nopad || n < N) st4<T>(lp(s, out, r, n * (int)sizeof(T)), v);
  };
  block_mm<T, RT, decltype(epi)&, HINT>(s, L, p, next, pend, epi);
}

// Input gradient of the embedding columns of a bottom input: float32 rows
// of gx (block rows below rv).
template <typename T, int RT, int PF>
__device__ __forceinline__ void run_gx(const char* s, const ChainLayer& L, float* gx, int64_t ldgx,
                                       int r0, int rv, Pipe<PF>& p, const RcPend& pend) {
  const int N = L.N;
  VFL_GLOBAL float* gxg = glb(gx);
  block_mm<T, RT>(s, L, p, nullptr, pend, [&](int r, int n, const f32x4& a, const f32x4&) {
    if (r >= rv) return;
    VFL_GLOBAL float* dst = gxg + (int64_t)(r0 + r) * ldgx + n;
    if (n + 4 <= N) {
      *(VFL_GLOBAL f32x4*)dst = a;
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (n + i < N) dst[i] = a[i];
    }
  });
}

// ------------------------------------------------------------ data movement
// LDS rows -> RC global matrix (block rows at tick rows r0 ..): one lane per
// output chunk (RR rows of one column), built from RR element reads of the
// LDS rows, so every lane of the block works and consecutive lanes store
// consecutive chunks of a row group.  Columns up to the next multiple of RR
// (zero in LDS) are written too.
template <typename T, int BR, bool NT>
__device__ __forceinline__ void lds_to_rc_(const char* s, const LBuf& b, int cols, const RCMat& m, int r0) {
  constexpr int RR = Ch<T>::CE;
  const int cw = (cols + RR - 1) / RR * RR;
  VFL_GLOBAL char* g = glb((char*)m.p);
  const int64_t cp = m.cp;
  const int nrg = m.rows > 0 ? min(BR / RR, (m.rows - r0) / RR) : BR / RR;   // row groups inside m
  for (int u = threadIdx.x; u < nrg * cw; u += kNT) {
    const int rg = u / cw, c = u - rg * cw;
    const char* src = s + b.off + rg * RR * b.pitch + c * (int)sizeof(T);
    u32x4 v;
    if constexpr (RR == 8) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t lo = *(const uint16_t*)(src + (2 * w) * b.pitch);
        const uint32_t hi = *(const uint16_t*)(src + (2 * w + 1) * b.pitch);
        v[w] = lo | (hi << 16);
      }
    } else {
#pragma unroll
      for (int w = 0; w < 4; ++w) v[w] = *(const uint32_t*)(src + w * b.pitch);
    }
    VFL_GLOBAL u32x4* dst = (VFL_GLOBAL u32x4*)(g + ((int64_t)(r0 / RR + rg) * cp + c) * 16);
    if constexpr (NT) __builtin_nontemporal_store(v, dst);
    else *dst = v;
    if constexpr (RR == 8) {
      if (m.bits && c < cols) {
        // the chunk's positive rows, one bit each (ReLU outputs: a row is
        // positive when its sign bit is clear and it is not zero)
        uint32_t byte = 0;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const uint32_t lo = v[w] & 0xffffu, hi = v[w] >> 16;
          byte |= (uint32_t)(lo != 0 && !(lo & 0x8000u)) << (2 * w);
          byte |= (uint32_t)(hi != 0 && !(hi & 0x8000u)) << (2 * w + 1);
        }
        glb(m.bits)[(int64_t)(r0 / RR + rg) * m.ldb + c] = (uint8_t)byte;
      }
    }
  }
}

template <typename T, int BR>
__device__ __forceinline__ void lds_to_rc(const char* s, const LBuf& b, int cols, const RCMat& m, int r0) {
  lds_to_rc_<T, BR, false>(s, b, cols, m, r0);
}

// the same with the streaming hint when m.nt (matrices too large for the
// L2; the two loops are kept apart so that the hint survives), for B's
// forward, whose copies are its largest output
template <typename T, int BR>
__device__ __forceinline__ void lds_to_rc_hint(const char* s, const LBuf& b, int cols, const RCMat& m, int r0) {
  if (m.nt) lds_to_rc_<T, BR, true>(s, b, cols, m, r0);
  else lds_to_rc_<T, BR, false>(s, b, cols, m, r0);
}

// zero rows r0 .. r0+BR-1 of an RC global matrix (columns below cols)
template <typename T, int BR>
__device__ __forceinline__ void zero_rc(const RCMat& m, int cols, int r0) {
  constexpr int RR = Ch<T>::CE;
  if (!m.p) return;
  const int ncc = (cols + RR - 1) / RR;
  VFL_GLOBAL char* g = glb((char*)m.p);
  const int nrg = m.rows > 0 ? min(BR / RR, (m.rows - r0) / RR) : BR / RR;   // row groups inside m
  for (int u = threadIdx.x; u < nrg * ncc * RR; u += kNT) {
    const int rg = u / (ncc * RR), c = u % (ncc * RR);
    *(VFL_GLOBAL u32x4*)(g + ((int64_t)(r0 / RR + rg) * m.cp + c) * 16) = u32x4{0u, 0u, 0u, 0u};
  }
}

// RC global matrix -> LDS rows (columns below cols; zeros up to the MFMA
// depth): one lane per chunk (RR rows of one column), one 16-byte load (or
// a byte of the matrix's ReLU bits when it has them) and RR element writes.
// Past one chunk per lane, the loads of NB units per lane are issued
// before their first use (one round trip to HBM per NB units, not per
// unit), and bits go a lane per 4 chunks (one 4-byte load, an 8-byte write
// per row).  Blocks with at most one chunk per lane keep the one-chunk
// loop (narrow masks: there the batched form was slower beside the other
// party's kernels).
// The ReLU bits of a block's BR rows as they are (a byte per 8 rows and
// column) into b: BR / 8 rows of b.pitch bytes, 16 bytes per lane and load,
// columns up to cols rounded to 16 (within m.ldb).  Row groups past m.rows
// repeat its last (their rows are past the tick's and never kept).
template <int BR>
__device__ __forceinline__ void bits_to_lds(char* s, const LBuf& b, int cols, const RCMat& m, int r0) {
  const int nc = (cols + 15) / 16;
  const int rg_last = m.rows > 0 ? max(m.rows / 8 - 1, 0) : (1 << 30);
  const VFL_GLOBAL uint8_t* bits = glb((const uint8_t*)m.bits);
  for (int u = threadIdx.x; u < (BR / 8) * nc; u += kNT) {
    const int rg = u / nc, c = 16 * (u - rg * nc);
    const u32x4 v = __builtin_nontemporal_load((const VFL_GLOBAL u32x4*)(bits + (int64_t)min(r0 / 8 + rg, rg_last) * m.ldb + c));
    *(u32x4*)(s + b.off + rg * b.pitch + c) = v;
  }
}

template <typename T, int BR>
__device__ __forceinline__ void rc_to_lds(char* s, const LBuf& b, int cols, const RCMat& m, int r0) {
  constexpr int RR = Ch<T>::CE, KS = Ch<T>::KS;
  constexpr int NB = 4;                       // units whose loads are in flight together
  const int cw = (cols + KS - 1) / KS * KS;   // columns up to the MFMA depth
  const VFL_GLOBAL char* g = glb((const char*)m.p);
  const int64_t cp = m.cp;
  const VFL_GLOBAL uint8_t* bits = glb((const uint8_t*)m.bits);
  const int rg_last = m.rows > 0 ? max(m.rows / RR - 1, 0) : (1 << 30);
  const int units = (BR / RR) * cw;
  if constexpr (RR == 8) {
    if (bits && units > kNT) {
      // the ReLU bits: a lane takes 4 columns of a row group (one 4-byte
      // load, byte j = column c + j, bit i = row i), written as bf16 ones
      // (which the mask test reads as positive), 8 bytes per LDS row
      const int nc4 = cw / 4, nu = (BR / RR) * nc4;
      for (int u0 = threadIdx.x; u0 < nu; u0 += NB * kNT) {
        uint32_t wv[NB];
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          const int u = min(u0 + i * kNT, nu - 1);
          const int rg = u / nc4, c = 4 * (u - rg * nc4);
          wv[i] = *(const VFL_GLOBAL uint32_t*)(bits + (int64_t)min(r0 / RR + rg, rg_last) * m.ldb + c);
        }
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          const int u = u0 + i * kNT;
          if (u >= nu) continue;
          const int rg = u / nc4, c = 4 * (u - rg * nc4);
          const bool in_m = m.rows == 0 || r0 + rg * RR < m.rows;
          uint32_t w = in_m ? wv[i] : 0u;
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (c + j >= cols) w &= ~(0xffu << (8 * j));
          char* dst = s + b.off + rg * RR * b.pitch + c * (int)sizeof(T);
#pragma unroll
          for (int r = 0; r < 8; ++r) {
            uint2 q;
            q.x = ((w >> r) & 1u ? 0x3f80u : 0u) | ((w >> (8 + r)) & 1u ? 0x3f800000u : 0u);
            q.y = ((w >> (16 + r)) & 1u ? 0x3f80u : 0u) | ((w >> (24 + r)) & 1u ? 0x3f800000u : 0u);
            *(uint2*)(dst + r * b.pitch) = q;
          }
        }
      }
      return;
    }
  }
  if (units <= kNT) {
    // at most one chunk per lane: a chunk of RC data or of bits each
    const int u = threadIdx.x;
    if (u < units) {
      const int rg = u / cw, c = u - rg * cw;
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (c < cols && (m.rows == 0 || r0 + rg * RR < m.rows)) {
        if constexpr (RR == 8) {
          if (bits) {
            const uint32_t byte = bits[(int64_t)(r0 / RR + rg) * m.ldb + c];
#pragma unroll
            for (int w = 0; w < 4; ++w)
              v[w] = ((byte >> (2 * w)) & 1u ? 0x3f80u : 0u) | ((byte >> (2 * w + 1)) & 1u ? 0x3f800000u : 0u);
          } else {
            v = *(const VFL_GLOBAL u32x4*)(g + ((int64_t)(r0 / RR + rg) * cp + c) * 16);
          }
        } else {
          v = *(const VFL_GLOBAL u32x4*)(g + ((int64_t)(r0 / RR + rg) * cp + c) * 16);
        }
      }
      char* dst = s + b.off + rg * RR * b.pitch + c * (int)sizeof(T);
      if constexpr (RR == 8) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          *(uint16_t*)(dst + (2 * w) * b.pitch) = (uint16_t)(v[w] & 0xffffu);
          *(uint16_t*)(dst + (2 * w + 1) * b.pitch) = (uint16_t)(v[w] >> 16);
        }
      } else {
#pragma unroll
        for (int w = 0; w < 4; ++w) *(uint32_t*)(dst + w * b.pitch) = v[w];
      }
    }
    return;
  }
  // the RC chunks, several per lane: batches of NB 16-byte loads
  const int nu = units;
  for (int u0 = threadIdx.x; u0 < nu; u0 += NB * kNT) {
    u32x4 v[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int u = min(u0 + i * kNT, nu - 1);
      const int rg = u / cw, c = min(u - rg * cw, cols - 1);
      v[i] = *(const VFL_GLOBAL u32x4*)(g + ((int64_t)min(r0 / RR + rg, rg_last) * cp + c) * 16);
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int u = u0 + i * kNT;
      if (u >= nu) continue;
      const int rg = u / cw, c = u - rg * cw;
      const bool ok = c < cols && (m.rows == 0 || r0 + rg * RR < m.rows);
      const u32x4 x = ok ? v[i] : u32x4{0u, 0u, 0u, 0u};
      char* dst = s + b.off + rg * RR * b.pitch + c * (int)sizeof(T);
      if constexpr (RR == 8) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          *(uint16_t*)(dst + (2 * w) * b.pitch) = (uint16_t)(x[w] & 0xffffu);
          *(uint16_t*)(dst + (2 * w + 1) * b.pitch) = (uint16_t)(x[w] >> 16);
        }
      } else {
#pragma unroll
        for (int w = 0; w < 4; ++w) *(uint32_t*)(dst + w * b.pitch) = x[w];
      }
    }
  }
}

// LDS rows -> row-major global rows (16-byte chunks; rows below rv)
template <typename T, int BR>
__device__ __forceinline__ void lds_to_rows(const char* s, const LBuf& b, int cols, void* dst,
                                            int64_t ld, int r0, int rv) {
  constexpr int CE = Ch<T>::CE;
  const int nch = (cols + CE - 1) / CE;
  VFL_GLOBAL char* d = glb((char*)dst);
  for (int u = threadIdx.x; u < rv * nch; u += kNT) {
    const int r = u / nch, ch = u % nch;
    *(VFL_GLOBAL u32x4*)(d + ((int64_t)(r0 + r) * ld + ch * CE) * sizeof(T)) =
        *(const u32x4*)(s + b.off + r * b.pitch + ch * 16);
  }
}

// an embedding id clamped into [0, V)
__device__ __forceinline__ int32_t clamp_id(int32_t id, int32_t V) { return min(max(id, 0), V - 1); }

// Bottom input [embeddings | dense] of the block into LDS (zeros beyond the
// input width up to the MFMA depth and for rows below the group).
template <typename T, int BR>
__device__ __forceinline__ void load_input(char* s, const RowInput& in, const ChainCall& cc,
                                           const Call& k, int r0, int rv) {
  constexpr int CE = Ch<T>::CE, KS = Ch<T>::KS;
  const int ne = in.n_cat * in.E;
  const int din = ne + in.dense_in;
  const int nch = (din + KS - 1) / KS * 4;
  const VFL_GLOBAL T* dense = glb((const T*)cc.dense);
  const VFL_GLOBAL int32_t* ids = glb(cc.ids);
  const VFL_GLOBAL float* tab = glb(in.T);
  if (in.idt) {
    // field-major copy of the block's ids (read contiguously)
    VFL_GLOBAL int32_t* idt = glb(in.idt);
    const VFL_GLOBAL int32_t* src = ids + (k.in_off + r0) * in.n_cat;
    for (int u = threadIdx.x; u < rv * in.n_cat; u += kNT) {
      const int r = u / in.n_cat, f = u - r * in.n_cat;
      int32_t id = src[u];
      if ((uint32_t)id >= (uint32_t)in.V) {
        if (in.bad_ids) atomicAdd(in.bad_ids, 1);
        id = id < 0 ? 0 : in.V - 1;
      }
      idt[(int64_t)f * in.ldi + r0 + r] = id;
    }
  }
  if (ne == 0 && in.dense_vec && BR * nch > kNT) {
    // dense rows only, several chunks per lane: NB chunks per lane in
    // flight before the first LDS write (one round trip to HBM per NB
    // chunks; NB grows with the rows per block, so that narrow blocks keep
    // their register count); chunks past the rows or the width load a valid
    // chunk of the block's first row and store zero.  (With one chunk per
    // lane the loop below issues each lane's only load at once anyway.)
    constexpr int NB = BR / 8 < 8 ? BR / 8 : 8;
    const int nu = BR * nch;
    for (int u0 = threadIdx.x; u0 < nu; u0 += NB * kNT) {
      u32x4 v[NB];
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const int u = u0 + i * kNT, r = u / nch, c0 = (u % nch) * CE;
        const bool ok = u < nu && r < rv && c0 < din;
        const int64_t row = k.in_off + r0 + (ok ? r : 0);
        v[i] = __builtin_nontemporal_load((const VFL_GLOBAL u32x4*)(dense + row * cc.ld + (ok ? c0 : 0)));
      }
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const int u = u0 + i * kNT, r = u / nch, ch = u % nch, c0 = ch * CE;
        if (u >= nu) continue;
        const bool ok = r < rv && c0 < din;
        *(u32x4*)(s + in.buf.off + r * in.buf.pitch + ch * 16) =
            ok ? mask_tail<T>(v[i], din - c0) : u32x4{0u, 0u, 0u, 0u};
      }
    }
    return;
  }
  for (int u = threadIdx.x; u < BR * nch; u += kNT) {
    const int r = u / nch, ch = u % nch, c0 = ch * CE;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (r < rv && c0 < din) {
      const int64_t row = k.in_off + r0 + r;
      if (c0 >= ne && in.dense_vec && (ne % CE) == 0) {
        v = mask_tail<T>(__builtin_nontemporal_load((const VFL_GLOBAL u32x4*)(dense + row * cc.ld + (c0 - ne))),
                         din - c0);
      } else if (c0 + CE <= ne && (in.E % CE) == 0) {
        const int f = c0 / in.E, o = c0 % in.E;
        const VFL_GLOBAL float* src = tab + ((int64_t)f * in.V + clamp_id(ids[row * in.n_cat + f], in.V)) * in.E + o;
        float x[CE];
#pragma unroll
        for (int q = 0; q < CE / 4; ++q) {
          const f32x4 t = *(const VFL_GLOBAL f32x4*)(src + 4 * q);
          x[4 * q] = t[0]; x[4 * q + 1] = t[1]; x[4 * q + 2] = t[2]; x[4 * q + 3] = t[3];
        }
        if constexpr (sizeof(T) == 4) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = __float_as_uint(x[e]);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = pack_bf16(x[2 * e], x[2 * e + 1]);
        }
      } else {
        float x[CE];
#pragma unroll
        for (int e = 0; e < CE; ++e) {
          const int c = c0 + e;
          float val = 0.f;
          if (c < ne) {
            const int f = c / in.E;
            val = tab[((int64_t)f * in.V + clamp_id(ids[row * in.n_cat + f], in.V)) * in.E + (c % in.E)];
          } else if (c < din) {
            val = ld1<T>((const T*)(dense + row * cc.ld + (c - ne)));
          }
          x[e] = val;
        }
        if constexpr (sizeof(T) == 4) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = __float_as_uint(x[e]);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = pack_bf16(x[2 * e], x[2 * e + 1]);
        }
      }
    }
    *(u32x4*)(s + in.buf.off + r * in.buf.pitch + ch * 16) = v;
  }
}

// Per-row clip + noise of an LDS message of D columns (element V) into
// row-major element-T rows; norm/cfac (nullable) receive ||v|| and the clip
// factor.  16 lanes per row (4 rows per wavefront at a time), each lane on
// the 4-column groups cg, cg + 16, ...; the noise is keyed by the row's
// sample id, two groups' Philox blocks at a time (independent instruction
// streams, so one lane keeps the VALU busy).
template <typename V>
__device__ __forceinline__ void msg_ld4(const char* row, int g, int D, float (&x)[4]) {
  ld4<V>(row + 4 * g * (int)sizeof(V), x);
#pragma unroll
  for (int e = 0; e < 4; ++e) x[e] = 4 * g + e < D ? x[e] : 0.f;   // columns past D may hold anything
}
template <typename T>
__device__ __forceinline__ void msg_st4(VFL_GLOBAL T* o, int g, int D, const float (&v)[4]) {
  if (4 * g + 4 <= D) {
    st4<T>((T*)(o + 4 * g), v);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (4 * g + e < D) st1<T>((T*)(o + 4 * g + e), v[e]);
  }
}
template <typename T, typename V, int BR>
__device__ __forceinline__ void msg_rows(const char* s, const LBuf& src, int D, const MsgOp& m,
                                         uint32_t step, int64_t sample0, void* out, int64_t ldo,
                                         float* norm, float* cfac, int r0, int rv) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane >> 4, cg = lane & 15;
  const int ngrp = (D + 3) >> 2;
  for (int rb = 0; rb < BR; rb += 4 * kNW) {
    const int r = rb + wave * 4 + sub;
    if (r >= rv) continue;   // uniform within the row's 16 lanes
    const char* row = s + src.off + r * src.pitch;
    float ss = 0.f;
    for (int g = cg; g < ngrp; g += 16) {
      float x[4];
      msg_ld4<V>(row, g, D, x);
#pragma unroll
      for (int e = 0; e < 4; ++e) ss += x[e] * x[e];
    }
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) ss += __shfl_xor(ss, o, 64);
    const float n = sqrtf(ss);
    const float cf = (m.clip && n > m.C) ? m.C / n : 1.f;
    if (cg == 0) {
      if (norm) glb(norm)[r0 + r] = n;
      if (cfac) glb(cfac)[r0 + r] = cf;
    }
    VFL_GLOBAL T* o = glb((T*)out) + (int64_t)(r0 + r) * ldo;
    const uint32_t grow = (uint32_t)(sample0 + r0 + r);
    for (int g = cg; g < ngrp; g += 32) {
      // groups g and g + 16 (the second past the row: computed, never stored)
      float xa[4] = {0.f, 0.f, 0.f, 0.f}, xb[4] = {0.f, 0.f, 0.f, 0.f};
      if (m.noise) {
        gauss4(m.seed, step, grow, (uint32_t)g, m.tag, xa);
        gauss4(m.seed, step, grow, (uint32_t)(g + 16), m.tag, xb);
      }
      float va[4], vb[4];
      msg_ld4<V>(row, g, D, va);
      msg_ld4<V>(row, min(g + 16, ngrp - 1), D, vb);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        va[e] = 4 * g + e < D ? cf * va[e] + m.stdv * xa[e] : 0.f;
        vb[e] = cf * vb[e] + m.stdv * xb[e];
      }
      msg_st4<T>(o, g, D, va);
      if (g + 16 < ngrp) msg_st4<T>(o, g + 16, D, vb);
    }
  }
}

// ------------------------------------------------------------------ kernels
template <typename T, int RT, int PF>
__global__ __launch_bounds__(kNT) void k_fwd(const FwdJob* __restrict__ jp, ChainCall cc,
                                             TickRef tr) {
  constexpr int BR = 16 * RT;
  extern __shared__ __attribute__((aligned(16))) char s[];
  const FwdJob& j = *jp;
  const int nL = cst(j).L;
  const Call k = resolve(cc, tr);
  if (blockIdx.x == 0 && threadIdx.x == 0 && j.hdr_out) {
    VFL_GLOBAL int32_t* h = glb(j.hdr_out);
    h[0] = k.hdr[0]; h[1] = k.hdr[1]; h[2] = k.hdr[2];
  }
  const int r0 = blockIdx.x * BR;
  if (r0 >= k.rows) return;
  const int rv = min(BR, k.rows - r0);
  Pipe<PF> pp;
  prefetch<T>(&j.l[0], pp);   // overlaps the input rows' loads
  const uint32_t wx = warm_l2(j.warm, jp);
  copy_bias(s, j.bt);
  load_input<T, BR>(s, j.in, cc, k, r0, rv);
  __syncthreads();
  asm volatile("" ::"v"(wx));   // the L2 fetches have landed with the inputs
  // each stage's RC copy goes out during the next product
  RcPend pend{j.in.buf, j.in.n_cat * j.in.E + j.in.dense_in, j.in.rc, r0};
  for (int l = 0; l < nL; ++l) {
    run_layer<T, RT, true>(s, j.l[l], rv, pp, l + 1 < nL ? &j.l[l + 1] : nullptr, pend);
    __syncthreads();
    pend = RcPend{j.l[l].out, j.l[l].N, j.l[l].rc, r0};
  }
  if (pend.m.p) lds_to_rc_hint<T, BR>(s, pend.b, pend.cols, pend.m, r0);
  const ChainLayer& last = j.l[nL - 1];
  lds_to_rows<T, BR>(s, last.out, last.N, j.z, j.ldz, r0, rv);
  if (j.publish)
    msg_rows<T, T, BR>(s, last.out, last.N, j.m, (uint32_t)k.group, k.row0, j.zhat, j.ldzh, j.norm,
                       j.cfac, r0, rv);
}

template <typename T, int RT, int PF>
__global__ __launch_bounds__(kNT) void k_active(const ActiveJob* __restrict__ jp, ChainCall cc,
                                                TickRef tr) {
  constexpr int BR = 16 * RT;
  constexpr int CE = Ch<T>::CE, KS = Ch<T>::KS;
  extern __shared__ __attribute__((aligned(16))) char s[];
  const ActiveJob& j = *jp;
  const int LA = cst(j).LA;
  const int H = cst(j).H;
  const int nda = cst(j).nda;
  const int has_gx = cst(j).has_gx;
  const Call k = resolve(cc, tr);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    if (j.hdr_chk && glb(j.hdr_chk)[0] != k.chk) atomicAdd(j.err, 1);
    if (j.hdr_out) {
      VFL_GLOBAL int32_t* h = glb(j.hdr_out);
      h[0] = k.hdr[0]; h[1] = k.hdr[1]; h[2] = k.hdr[2];
    }
  }
  const int r0 = blockIdx.x * BR;
  if (r0 >= k.rows) {
    // rows past a short group: zero delta rows, so that the weight
    // gradient may read whole row steps
    zero_rc<T, BR>(j.dh_rc, j.ft[H - 1].N, r0);
    for (int q = 0; q + 1 < H; ++q) zero_rc<T, BR>(j.dt[q].rc, j.dt[q].N, r0);
    zero_rc<T, BR>(j.dc.rc, j.dA, r0);
    for (int q = 0; q < nda; ++q) zero_rc<T, BR>(j.da[q].rc, j.da[q].N, r0);
    return;
  }
  const int rv = min(BR, k.rows - r0);
  const int Hd = j.ft[H - 1].N;
  // the labels (to LDS with the inputs) and the logit weights of the lane's
  // columns in the logit stage (columns 256 i + 4 lane .. +4, kept in
  // registers); loads clamped, so all are unconditional
  float* yl = (float*)(s + j.red.off);
  float py;
  float lwr[kLogitChunks][4];
  {
    const VFL_GLOBAL float* lw = glb(j.lw);
    const VFL_GLOBAL float* y = glb(cc.labels) + k.in_off + r0;
#pragma unroll
    for (int i = 0; i < kLogitChunks; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = 256 * i + 4 * lane + e;
        const float v = lw[min(c, Hd - 1)];
        lwr[i][e] = c < Hd ? v : 0.f;
      }
    py = y[min((int)threadIdx.x, rv - 1)];
  }
  const float lbias = glb(j.lb)[0];
  Pipe<PF> pp;
  prefetch<T, PF>(&j.fa[0], pp);
  const uint32_t wx = warm_l2(j.warm, jp);
  copy_bias(s, j.bt);

  // A's bottom input, and B's embedding into cat[:, dA:dA+dB) with zeros up
  // to the MFMA depth (published before this launch; A's last layer fills
  // cat[:, 0:dA) and leaves these columns alone)
  load_input<T, BR>(s, j.in, cc, k, r0, rv);
  if ((int)threadIdx.x < BR) yl[threadIdx.x] = (int)threadIdx.x < rv ? py : 0.f;
  {
    const int dA = j.dA, dB = j.dB;
    const int nch = ((dA + dB + KS - 1) / KS * KS - dA) / CE;
    const VFL_GLOBAL T* zb = glb((const T*)j.zb);
    for (int u = threadIdx.x; u < BR * nch; u += kNT) {
      const int r = u / nch, ch = u % nch, c = ch * CE;
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (r < rv && c < dB) v = mask_tail<T>(*(const VFL_GLOBAL u32x4*)(zb + (int64_t)(r0 + r) * j.ldzb + c), dB - c);
      *(u32x4*)(s + j.cat.off + r * j.cat.pitch + (dA + c) * (int)sizeof(T)) = v;
    }
  }
  __syncthreads();
  asm volatile("" ::"v"(wx));   // the L2 fetches have landed with the inputs
  // each stage's RC copy goes out during the next product (A's last
  // layer writes cat, copied whole)
  RcPend pend{j.in.buf, j.in.n_cat * j.in.E + j.in.dense_in, j.in.rc, r0};
  for (int l = 0; l < LA; ++l) {
    run_layer<T, RT>(s, j.fa[l], rv, pp, l + 1 < LA ? &j.fa[l + 1] : &j.ft[0], pend);
    __syncthreads();
    pend = l + 1 < LA ? RcPend{j.fa[l].out, j.fa[l].N, j.fa[l].rc, r0} : RcPend{j.cat, j.dA + j.dB, j.cat_rc, r0};
  }
  // top hidden layers
  for (int q = 0; q < H; ++q) {
    run_layer<T, RT>(s, j.ft[q], rv, pp, q + 1 < H ? &j.ft[q + 1] : (H > 1 ? &j.dt[0] : &j.dc), pend);
    __syncthreads();
    pend = RcPend{j.ft[q].out, j.ft[q].N, j.ft[q].rc, r0};
  }
  // the logit stage reads the last hidden output, not a product's input
  if (pend.m.p) lds_to_rc<T, BR>(s, pend.b, pend.cols, pend.m, r0);
  // logit + BCE (Eq. 1), dl = sigmoid(l) - y, or for regression the
  // squared error and dl = 2 (l - y): a wavefront per row (its
  // BR / 8 rows one after the other), lane on the columns 256 i + 4 lane
  // .. +4; the last hidden delta dl * w (ReLU-masked) goes to LDS.  The
  // logit layer's weight gradient sum_r dl_r h[r][c], the loss and dl
  // accumulate per wavefront in registers and are then summed over the
  // wavefronts in order.  The loss only reports progress: its exp and log
  // are the hardware's.
  {
    const LBuf Hb = j.ft[H - 1].out, Db = j.dh;
    constexpr int KS = Ch<T>::KS, RW = BR / kNW;
    const int Hw = (Hd + KS - 1) / KS * KS;     // LDS width of h and dh
    const int Hd4 = (Hd + 3) / 4 * 4;
    float* wpart = yl + BR;                     // [kNW][Hd4]
    float* wl = wpart + kNW * Hd4;              // [kNW][2]
    float g[kLogitChunks][4];
#pragma unroll
    for (int i = 0; i < kLogitChunks; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) g[i][e] = 0.f;
    float lsum = 0.f, dsum = 0.f;
    const bool relu_h = j.relu_h != 0;
    auto load_h = [&](int r, float (&h)[kLogitChunks][4]) {
#pragma unroll
      for (int i = 0; i < kLogitChunks; ++i) {
        const int c0 = 256 * i + 4 * lane;
        if (c0 < Hw) ld4<T>(lp(s, Hb, r, c0 * (int)sizeof(T)), h[i]);
        else {
#pragma unroll
          for (int e = 0; e < 4; ++e) h[i][e] = 0.f;
        }
      }
    };
    // the logits of the wavefront's rows: partial dots first, then their
    // wavefront reductions side by side (independent shuffle chains)
    float dots[RW];
#pragma unroll
    for (int rr = 0; rr < RW; ++rr) {
      float h[kLogitChunks][4];
      load_h(wave * RW + rr, h);
      float dot = 0.f;
#pragma unroll
      for (int i = 0; i < kLogitChunks; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) dot += h[i][e] * lwr[i][e];
      dots[rr] = dot;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
#pragma unroll
      for (int rr = 0; rr < RW; ++rr) dots[rr] += __shfl_xor(dots[rr], o, 64);
    // the loss terms and dl of every row first: their exp / reciprocal /
    // log chains are independent, while the stage below alternates LDS
    // reads and writes the compiler must keep in order (they may alias)
    float dls[RW];
    if (cst(j).mse) {
      // regression: squared error (l - y)^2, dl = 2 (l - y)
#pragma unroll
      for (int rr = 0; rr < RW; ++rr) {
        const int r = wave * RW + rr;
        const bool ok = r < rv;
        const float e = dots[rr] + lbias - yl[r];
        const float dl = ok ? 2.f * e : 0.f;
        if (ok) lsum += e * e;
        dsum += dl;
        dls[rr] = dl;
      }
    } else {
#pragma unroll
      for (int rr = 0; rr < RW; ++rr) {
        const int r = wave * RW + rr;
        const bool ok = r < rv;
        const float l = dots[rr] + lbias;
        const float yy = yl[r];
        const float ex = __expf(-fabsf(l));
        const float inv = __frcp_rn(1.f + ex);
        const float sig = l >= 0.f ? inv : ex * inv;
        const float dl = ok ? sig - yy : 0.f;
        if (ok) lsum += fmaxf(l, 0.f) - yy * l + __logf(1.f + ex);
        dsum += dl;
        dls[rr] = dl;
      }
    }
#pragma unroll
    for (int rr = 0; rr < RW; ++rr) {
      const int r = wave * RW + rr;
      const float dl = dls[rr];
      float h[kLogitChunks][4];
      load_h(r, h);
#pragma unroll
      for (int i = 0; i < kLogitChunks; ++i) {
        const int c0 = 256 * i + 4 * lane;
        float d[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          d[e] = dl * lwr[i][e];
          if (relu_h && !(h[i][e] > 0.f)) d[e] = 0.f;
          g[i][e] += dl * h[i][e];
        }
        if (c0 < Hw) st4<T>(lp(s, Db, r, c0 * (int)sizeof(T)), d);
      }
    }
#pragma unroll
    for (int i = 0; i < kLogitChunks; ++i) {
      const int c0 = 256 * i + 4 * lane;
      if (c0 < Hd4) *(f32x4*)(wpart + wave * Hd4 + c0) = f32x4{g[i][0], g[i][1], g[i][2], g[i][3]};
    }
    if (lane == 0) {
      wl[2 * wave] = lsum;
      wl[2 * wave + 1] = dsum;
    }
    __syncthreads();
    VFL_GLOBAL float* part = glb(j.part) + (int64_t)blockIdx.x * (Hd + 2);
    for (int c = threadIdx.x; c < Hd + 2; c += kNT) {
      float t = 0.f;
      if (c < 2) {
#pragma unroll
        for (int w = 0; w < kNW; ++w) t += wl[2 * w + c];
      } else {
#pragma unroll
        for (int w = 0; w < kNW; ++w) t += wpart[w * Hd4 + c - 2];
      }
      part[c] = t;
    }
  }
  pend = RcPend{j.dh, j.ft[H - 1].N, j.dh_rc, r0};
  // top input-gradient chain
  for (int q = 0; q + 1 < H; ++q) {
    run_layer<T, RT>(s, j.dt[q], rv, pp, q + 2 < H ? &j.dt[q + 1] : &j.dc, pend);
    __syncthreads();
    pend = RcPend{j.dt[q].out, j.dt[q].N, j.dt[q].rc, r0};
  }
  // concat product: A's cut delta and the gradient message for B
  {
    const int dA = j.dA, dAB = j.dA + j.dB;
    const int dApad = (dA + KS - 1) / KS * KS;
    const LBuf ob = j.dc.out, cat = j.cat, msg = j.msg;
    const bool maskA = j.dc.mask.pitch > 0, gextra = j.gextra != 0;
    VFL_GLOBAL T* ring = glb((T*)j.ring);
    const int64_t ldr = j.ldring;
    block_mm<T, RT>(s, j.dc, pp, nda > 0 ? &j.da[0] : (has_gx ? &j.gx : nullptr), pend,
                    [&](int r, int n, const f32x4& a, const f32x4&) {
      const bool ok = r < rv;
      if (n + 4 <= dA) {
        float m[4] = {1.f, 1.f, 1.f, 1.f}, v[4];
        if (maskA) ld4<T>(lp(s, cat, r, n * (int)sizeof(T)), m);
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = (ok && m[i] > 0.f) ? a[i] : 0.f;
        st4<T>(lp(s, ob, r, n * (int)sizeof(T)), v);
        return;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = n + i;
        const float x = ok ? a[i] : 0.f;
        if (c < dA) {
          const bool keep = !maskA || ld1<T>((const T*)lp(s, cat, r, 0) + c) > 0.f;
          st1<T>((T*)lp(s, ob, r, 0) + c, keep ? x : 0.f);
        } else if (c < dApad) {
          st1<T>((T*)lp(s, ob, r, 0) + c, 0.f);
        }
        if (c >= dA && c < dAB) {
          if (gextra) ((float*)lp(s, msg, r, 0))[c - dA] = x;
          else if (ok) st1<T>((T*)(ring + (int64_t)(r0 + r) * ldr + (c - dA)), x);
        }
      }
    });
    __syncthreads();
    pend = RcPend{ob, dA, j.dc.rc, r0};
    if (gextra)
      msg_rows<T, float, BR>(s, msg, j.dB, j.m, (uint32_t)k.group, k.row0, j.ring, j.ldring, nullptr,
                             nullptr, r0, rv);
  }
  // A's input-gradient chain
  for (int q = 0; q < nda; ++q) {
    run_layer<T, RT>(s, j.da[q], rv, pp, q + 1 < nda ? &j.da[q + 1] : (has_gx ? &j.gx : nullptr), pend);
    __syncthreads();
    pend = RcPend{j.da[q].out, j.da[q].N, j.da[q].rc, r0};
  }
  if (has_gx) run_gx<T, RT>(s, j.gx, j.gxp, j.ldgx, r0, rv, pp, pend);
  else if (pend.m.p) lds_to_rc<T, BR>(s, pend.b, pend.cols, pend.m, r0);
}

template <typename T, int RT, int PF>
__global__ __launch_bounds__(kNT) void k_bwd(const BwdJob* __restrict__ jp, ChainCall cc,
                                             TickRef tr) {
  constexpr int BR = 16 * RT;
  constexpr int KS = Ch<T>::KS;
  extern __shared__ __attribute__((aligned(16))) char s[];
  const BwdJob& j = *jp;
  const int nd = cst(j).nd;
  const int has_gx = cst(j).has_gx;
  const Call k = resolve(cc, tr);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (blockIdx.x == 0 && threadIdx.x == 0 && j.hdr_chk && glb(j.hdr_chk)[0] != k.chk) atomicAdd(j.err, 1);
  const int r0 = blockIdx.x * BR;
  if (r0 >= k.rows) {
    zero_rc<T, BR>(j.d_rc, j.D, r0);
    for (int q = 0; q < nd; ++q) zero_rc<T, BR>(j.dx[q].rc, j.dx[q].N, r0);
    return;
  }
  const int rv = min(BR, k.rows - r0);
  Pipe<PF> pp;
  if (nd > 0 || has_gx) prefetch<T, PF>(nd > 0 ? &j.dx[0] : &j.gx, pp);
  const uint32_t wx = warm_l2(j.warm, jp);
  // the ReLU masks of every layer of the chain, each in an LDS buffer of
  // its own (bf16: the ReLU bits of this group's forward as bytes; float32:
  // its stashed activations)
  for (int q = 0; q < nd; ++q)
    if (j.dx[q].mask_src.p) {
      if constexpr (sizeof(T) == 2) bits_to_lds<BR>(s, j.dx[q].mask, j.dx[q].N, j.dx[q].mask_src, r0);
      else rc_to_lds<T, BR>(s, j.dx[q].mask, j.dx[q].N, j.dx[q].mask_src, r0);
    }
  // cut-layer backward: through the clip when the row was clipped
  // (d(c v)/dv = c (I - u u^T) with u = v / ||v||), then the ReLU of B's
  // last layer; 16 lanes per row, 4 rows per wavefront at a time
  {
    const int D = j.D;
    const int hq = (D + KS - 1) / KS * KS / 4;
    const int sub = lane >> 4, cg = lane & 15;
    for (int rb = 0; rb < BR; rb += 4 * kNW) {
      const int r = rb + wave * 4 + sub;
      if (r >= BR) continue;   // uniform within the row's 16 lanes
      const bool ok = r < rv;
      const int64_t row = r0 + r;
      const VFL_GLOBAL T* G = glb((const T*)j.g) + row * j.ldg;
      const VFL_GLOBAL T* Z = glb((const T*)j.z) + row * j.ldz;
      const bool clipped = ok && j.clip && glb(j.norm)[row] > j.C;
      float dot = 0.f, inv = 0.f, cf = 1.f;
      if (clipped) {
        inv = 1.f / glb(j.norm)[row];
        cf = glb(j.cfac)[row];
        for (int q = cg; 4 * q < D; q += 16)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (4 * q + e < D) dot += ld1<T>((const T*)(Z + 4 * q + e)) * inv * ld1<T>((const T*)(G + 4 * q + e));
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) dot += __shfl_xor(dot, o, 64);
      }
      for (int q = cg; q < hq; q += 16) {
        float gv[4] = {0.f, 0.f, 0.f, 0.f}, zv[4] = {0.f, 0.f, 0.f, 0.f}, v[4];
        if (ok && 4 * q + 4 <= D) {
          ld4<T>((const T*)(G + 4 * q), gv);
          ld4<T>((const T*)(Z + 4 * q), zv);
        } else if (ok) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (4 * q + e < D) { gv[e] = ld1<T>((const T*)(G + 4 * q + e)); zv[e] = ld1<T>((const T*)(Z + 4 * q + e)); }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float g = gv[e];
          if (clipped) g = cf * (g - zv[e] * inv * dot);
          if (j.relu && !(zv[e] > 0.f)) g = 0.f;
          v[e] = (ok && 4 * q + e < D) ? g : 0.f;
        }
        st4<T>(lp(s, j.d, r, 4 * q * (int)sizeof(T)), v);
      }
    }
  }
  __syncthreads();
  asm volatile("" ::"v"(wx));   // the L2 fetches have landed with the inputs
  // each stage's RC copy goes out during the next product
  RcPend pend{j.d, j.D, j.d_rc, r0};
  for (int q = 0; q < nd; ++q) {
    const ChainLayer& L = j.dx[q];
    run_layer<T, RT, true, PF, sizeof(T) == 2>(s, L, rv, pp, q + 1 < nd ? &j.dx[q + 1] : (has_gx ? &j.gx : nullptr),
                                               pend);
    __syncthreads();
    pend = RcPend{L.out, L.N, L.rc, r0};
  }
  if (has_gx) run_gx<T, RT>(s, j.gx, j.gxp, j.ldgx, r0, rv, pp, pend);
  else if (pend.m.p) lds_to_rc_hint<T, BR>(s, pend.b, pend.cols, pend.m, r0);
  if (j.drm) {
    // the last delta of the chain, row-major, for the layer product below it
    const LBuf last = nd > 0 ? j.dx[nd - 1].out : j.d;
    const int w = nd > 0 ? j.dx[nd - 1].N : j.D;
    lds_to_rows<T, BR>(s, last, w, j.drm, j.lddrm, r0, rv);
  }
}

template <typename K>
hipError_t raise_lds(K kernel) {
  return hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsMax);
}

}  // namespace


#define VFL_PF_RT(K, T, PF, rt, ...)                                                            \
  do {                                                                                       \
    if (rt == 1) hipLaunchKernelGGL((K<T, 1, PF>), __VA_ARGS__);                          \
    else if (rt == 2) hipLaunchKernelGGL((K<T, 2, PF>), __VA_ARGS__);                     \
    else if (rt == 3) hipLaunchKernelGGL((K<T, 3, PF>), __VA_ARGS__);                     \
    else if (rt == 4) hipLaunchKernelGGL((K<T, 4, PF>), __VA_ARGS__);                     \
    else return hipErrorInvalidValue;                                                        \
  } while (0)

hipError_t launch_fwd(Elt e, int rt, int pf, const FwdJob* job, int lds, int blocks, const ChainCall& c,
                      TickRef tr, hipStream_t st) {
  if (lds > kLdsMax || blocks < 1) return hipErrorInvalidValue;
  if (pf == kPFWide && e == BF16) VFL_PF_RT(k_fwd, uint16_t, kPFWide, rt, dim3(blocks), dim3(kNT), lds, st, job, c, tr);
  else if (pf == kPFNarrow && e == BF16) VFL_PF_RT(k_fwd, uint16_t, kPFNarrow, rt, dim3(blocks), dim3(kNT), lds, st, job, c, tr);
  else if (pf == kPFNarrow) VFL_PF_RT(k_fwd, float, kPFNarrow, rt, dim3(blocks), dim3(kNT), lds, st, job, c, tr);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_active(Elt e, int rt, int pf, const ActiveJob* job, int lds, int blocks,
                         const ChainCall& c, TickRef tr, hipStream_t st) {
  if (lds > kLdsMax || blocks < 1) return hipErrorInvalidValue;
  if (pf == kPFWide && e == BF16) VFL_PF_RT(k_active, uint16_t, kPFWide, rt, dim3(blocks), dim3(kNT), lds, st, job, c, tr);
  else if (pf == kPFNarrow && e == BF16) VFL_PF_RT(k_active, uint16_t, kPFNarrow, rt, dim3(blocks), dim3(kNT), lds, st, job, c, tr);
  else if (pf == kPFNarrow) VFL_PF_RT(k_active, float, kPFNarrow, rt, dim3(blocks), dim3(kNT), lds, st, job, c, tr);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_bwd(Elt e, int rt, int pf, const BwdJob* job, int lds, int blocks, const ChainCall& c,
                      TickRef tr, hipStream_t st) {
  if (lds > kLdsMax || blocks < 1) return hipErrorInvalidValue;
  if (pf == kPFWide && e == BF16) VFL_PF_RT(k_bwd, uint16_t, kPFWide, rt, dim3(blocks), dim3(kNT), lds, st, job, c, tr);
  else if (pf == kPFNarrow && e == BF16) VFL_PF_RT(k_bwd, uint16_t, kPFNarrow, rt, dim3(blocks), dim3(kNT), lds, st, job, c, tr);
  else if (pf == kPFNarrow) VFL_PF_RT(k_bwd, float, kPFNarrow, rt, dim3(blocks), dim3(kNT), lds, st, job, c, tr);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t chain_init() {
  const hipError_t r[] = {
      raise_lds(k_fwd<uint16_t, 1, kPFNarrow>), raise_lds(k_fwd<uint16_t, 2, kPFNarrow>),
      raise_lds(k_fwd<uint16_t, 3, kPFNarrow>), raise_lds(k_fwd<uint16_t, 4, kPFNarrow>),
      raise_lds(k_fwd<uint16_t, 1, kPFWide>), raise_lds(k_fwd<uint16_t, 2, kPFWide>),
      raise_lds(k_fwd<uint16_t, 3, kPFWide>), raise_lds(k_fwd<uint16_t, 4, kPFWide>),
      raise_lds(k_fwd<float, 1, kPFNarrow>), raise_lds(k_fwd<float, 2, kPFNarrow>),
      raise_lds(k_fwd<float, 3, kPFNarrow>), raise_lds(k_fwd<float, 4, kPFNarrow>),
      raise_lds(k_active<uint16_t, 1, kPFNarrow>), raise_lds(k_active<uint16_t, 2, kPFNarrow>),
      raise_lds(k_active<uint16_t, 3, kPFNarrow>), raise_lds(k_active<uint16_t, 4, kPFNarrow>),
      raise_lds(k_active<uint16_t, 1, kPFWide>), raise_lds(k_active<uint16_t, 2, kPFWide>),
      raise_lds(k_active<uint16_t, 3, kPFWide>), raise_lds(k_active<uint16_t, 4, kPFWide>),
      raise_lds(k_active<float, 1, kPFNarrow>), raise_lds(k_active<float, 2, kPFNarrow>),
      raise_lds(k_active<float, 3, kPFNarrow>), raise_lds(k_active<float, 4, kPFNarrow>),
      raise_lds(k_bwd<uint16_t, 1, kPFNarrow>), raise_lds(k_bwd<uint16_t, 2, kPFNarrow>),
      raise_lds(k_bwd<uint16_t, 3, kPFNarrow>), raise_lds(k_bwd<uint16_t, 4, kPFNarrow>),
      raise_lds(k_bwd<uint16_t, 1, kPFWide>), raise_lds(k_bwd<uint16_t, 2, kPFWide>),
      raise_lds(k_bwd<uint16_t, 3, kPFWide>), raise_lds(k_bwd<uint16_t, 4, kPFWide>),
      raise_lds(k_bwd<float, 1, kPFNarrow>), raise_lds(k_bwd<float, 2, kPFNarrow>),
      raise_lds(k_bwd<float, 3, kPFNarrow>), raise_lds(k_bwd<float, 4, kPFNarrow>)};
  for (hipError_t x : r)
    if (x != hipSuccess) return x;
  const hipError_t d = dwt_init();
  return d != hipSuccess ? d : lin_init();
}

}  // namespace vfl
