// Internal launch interface of the gfx950 kernels (not part of the C ABI).
//
// One tick of the training step runs as a handful of fused kernels:
//   k_fwd     party B: bottom forward of a row block through every layer,
//             then the published embedding (clip + Philox noise);
//   k_active  party A: bottom forward, concat with B's embedding, the top
//             model, logit + BCE, and the whole input-gradient chain back
//             through the top model and A's bottom, emitting the gradient
//             message for B (clip + noise);
//   k_bwd     party B: cut-layer backward of the message and the
//             input-gradient chain through B's bottom;
//   k_dw      every layer's weight gradient of one party (one launch),
//             rows split into chunks; SGD fused when a layer is unsplit;
//   k_dw_reduce  split chunks and the logit layer's block partials summed
//             in a fixed order, SGD, weight operand copies refreshed.
// The three chain kernels give each workgroup (kChainWaves wavefronts) a
// block of BR = 16 * RT rows and keep the block's activations and deltas in
// LDS from layer to layer:
// only the tensors a later kernel reads go to HBM.  Those that the weight
// gradient contracts over rows are written in the row-chunked layout below.
//
// Row-chunked ("RC") layout of a [rows x cols] matrix: element (r, c) lives
// at ((r / RR) * cp + c) * RR + r % RR, RR = 16 bytes / element size (8 rows
// of bf16, 4 of float32), cp = cols rounded up to 8.  Every 16-byte chunk
// holds RR consecutive rows of one column, which is exactly an MFMA operand
// fragment of a product that contracts over rows.  Rows of a block beyond
// the group's row count are written as zeros, and so are the delta rows of
// blocks past a short group's end.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vfl {

// Element type of activations, messages and weight copies.
enum Elt { F32 = 0, BF16 = 1 };

inline int elt_size(Elt e) { return e == F32 ? 4 : 2; }

constexpr int kMaxChain = 16;         // layers per chain (bottom or top)
constexpr int kMaxDw = 16;            // weight-gradient problems per launch
constexpr int kMaxLogitCols = 512;    // widest last hidden layer of the top model
constexpr int kLdsMax = 160 * 1024;   // LDS of one gfx950 workgroup
constexpr int kChainWaves = 8;        // wavefronts per chain-kernel block
constexpr int kChainPFNarrow = 2;     // MFMA steps per chain weight load group
constexpr int kChainPFWide = 4;       // the same for bf16 chains with large weights

// The values of one tick of the deterministic schedule over a resident
// dataset of n_rows rows (group g covers rows [(g mod E) * R, ...), E =
// ceil(n_rows / R), the last group of an epoch short), as a kernel uses them.
struct TickArgs {
  int32_t rows;        // rows of the batch group
  int32_t group;       // batch-group id (noise step, header sequence)
  int64_t row0;        // dataset row of the group's first row
  int32_t hdr[3];      // channel header to write {group, tick, version}
  int32_t chk;         // group expected in the header of the slot read
  float scale;         // lr / rows
  int64_t loss_idx;    // index of the group's loss in the loss ring
};

// Replayed graphs: a captured launch refers to tick base + off, base being
// the first tick of the current replay (written before the first replay,
// advanced by the graph's last node).  role 0: party B publishes group t;
// role 1: party A consumes group u = t - s; role 2: party B back-propagates
// u.  A null src means the launch's values are given directly.  B's forward
// of group g used version max(0, g - s - vofs): vofs counts the groups
// dropped before the replays (each leaves B's version one step behind).
struct TickSrc {
  int64_t base = 0;
  int64_t n_rows = 0;
  int32_t R = 0, s = 0;
  float lr = 0.f;
  int32_t vofs = 0;
  int64_t loss_len = 1;
};
struct TickRef {
  const TickSrc* src = nullptr;
  int32_t off = 0, role = 0;
};

__device__ __forceinline__ TickArgs tick_args(const TickRef& r) {
  const TickSrc& x = *r.src;
  const int64_t t = x.base + r.off;
  const int64_t g = r.role == 0 ? t : t - x.s;
  const int64_t E = (x.n_rows + x.R - 1) / x.R;
  const int64_t start = (g % E) * x.R;
  TickArgs a;
  a.rows = (int32_t)(x.n_rows - start < x.R ? x.n_rows - start : x.R);
  a.group = (int32_t)g;
  a.row0 = start;
  a.chk = (int32_t)g;
  a.scale = x.lr / (float)a.rows;
  a.loss_idx = g % x.loss_len;
  a.hdr[0] = (int32_t)g;
  a.hdr[1] = (int32_t)t;
  a.hdr[2] = (int32_t)(g - x.s - x.vofs > 0 ? g - x.s - x.vofs : 0);
  return a;
}

// the graph's last node: base += cyc
hipError_t launch_tick_base(TickSrc* src, int cyc, hipStream_t st);
// the record a run of replays starts from (a one-thread kernel: no copy)
hipError_t launch_tick_set(TickSrc* dst, const TickSrc& v, hipStream_t st);

// ------------------------------------------------------------ chain kernels
// LDS region of a row block: byte offset in the kernel's dynamic LDS and row
// pitch in bytes (a pitch of 0 marks an absent buffer).
struct LBuf { int32_t off = 0, pitch = 0; };

// RC-layout global matrix (null p: not written); rows: the rows it holds
// (a chain block's rows past it are not written; 0: unbounded).  bits (bf16
// chain copies only; null: none): a byte per 8-row chunk as well, bit i set
// when row i of the chunk is positive, at bits[(row / 8) * ldb + column] (the
// ReLU derivative of a layer, for B's backward and the wide input-gradient
// product; as a mask source, a set bits pointer is read instead of p).
struct RCMat {
  void* p = nullptr; int32_t cp = 0, rows = 0;
  uint8_t* bits = nullptr; int32_t ldb = 0;
  int32_t nt = 0;      // store with the non-temporal hint (matrices too large for the L2)
};

// One product of a row block with a weight operand W [N x K] (element type,
// packed: see pk_index; kst = K steps of the packing, tiles up to N rounded
// up to the MFMA depth, padding zero):
// out[r][n] = sum_k in[r][k] * W[n][k], n < N, then
//   forward:         + bias[n] (bias set), ReLU when relu;
//   input gradient:  * (mask[r][n] > 0) when mask.pitch > 0.
// Columns of `out` from N up to the next multiple of the MFMA depth are
// written as zeros, as are rows beyond the group.  rc: RC copy of out.
// mask_src (k_bwd): the mask is first loaded into `mask` from this matrix.
// bl: byte offset of the layer's bias row in the kernel's LDS bias table
// (-1: no bias).  nopad: columns from N on are left as they are (another
// tensor shares the LDS rows there).
struct ChainLayer {
  const void* W = nullptr;
  int32_t kst = 0, N = 0, K = 0, relu = 0;
  int32_t bl = -1, nopad = 0;
  // mask_bits: `mask` holds a byte per 8 rows and column (bit r % 8 of byte
  // (r / 8) * pitch + column: the ReLU bits as B's forward records them),
  // else one element per row and column (kept where positive)
  int32_t mask_bits = 0;
  LBuf in, out, mask;
  RCMat rc, mask_src;
};

// The biases a chain kernel adds: one contiguous float32 array in global
// memory (the masters of consecutive layers, each row padded to a multiple
// of 32 floats), copied to LDS at byte offset `off` when the kernel starts.
struct BiasTab {
  const float* src = nullptr;
  int32_t off = 0, n4 = 0;            // n4: float4 count
};

// The packed weight copies a chain kernel reads: up to two ranges of
// 128-byte lines, fetched into L2 when the kernel starts (the workgroups of
// one XCD each fetch a slice).
struct WarmSet {
  const void* p[2] = {nullptr, nullptr};
  int32_t lines[2] = {0, 0};
};

// Bottom-model input of a row block: [embeddings of n_cat fields | dense],
// gathered into LDS (`buf`) and copied to `rc` (for the first layer's
// weight gradient).  T: float32 tables [n_cat * V x E]; idt (with tables):
// field-major copy of the group's ids (clamped into [0, V)),
// idt[f * ldi + tick row], for the sparse table step.
struct RowInput {
  int32_t dense_in = 0, n_cat = 0, V = 0, E = 0;
  int32_t dense_vec = 0;              // dense rows 16-byte aligned: vector loads
  const float* T = nullptr;
  int32_t* idt = nullptr; int32_t ldi = 0;
  // ids outside [0, V) are clamped into it (so no access leaves the
  // field's table) and counted here once per copy into idt
  int32_t* bad_ids = nullptr;
  LBuf buf;
  RCMat rc;
};

// Per-row clip to L2 norm C and Philox Gaussian noise of std stdv keyed by
// (seed, step = group, global row, column / 4, tag).
struct MsgOp {
  int32_t clip = 0, noise = 0;
  float C = 0.f, stdv = 0.f;
  uint64_t seed = 0;
  uint32_t tag = 0;
};

// Values of one chain launch (with a tick reference its tick record replaces
// rows, group, row0 and the headers, and then dense / ids / labels are
// dataset bases).
struct ChainCall {
  const void* dense = nullptr;
  int64_t ld = 0;
  const int32_t* ids = nullptr;
  const float* labels = nullptr;
  int64_t row0 = 0;                   // global sample id of row 0
  int32_t rows = 0, group = 0;
  int32_t hdr[3] = {0, 0, 0};         // header written by block 0
  int32_t chk = 0;                    // group expected in the header read
};

// Party B's forward of a group: input, L layers (ping-pong LDS buffers),
// the last layer's output row-major in z, and the embedding message in
// zhat (zhat == z when neither clip nor noise is on), with norm/cfac per
// row when clipping; block 0 writes the slot header.
struct FwdJob {
  RowInput in;
  BiasTab bt;
  WarmSet warm;
  int32_t L = 0;
  ChainLayer l[kMaxChain];
  void* z = nullptr; int32_t ldz = 0;
  int32_t publish = 0;
  MsgOp m;
  void* zhat = nullptr; int32_t ldzh = 0;
  float* norm = nullptr; float* cfac = nullptr;
  int32_t* hdr_out = nullptr;
};

// Party A's step of a group: forward of A's layers fa (the last writes the
// first dA columns of `cat`), B's embedding zb into columns [dA, dA + dB) of
// cat, the top hidden layers ft, logit + BCE (mse: output + squared error)
// into the last hidden delta dh
// (per-block partials {sum loss, sum dl, sum_r dl * h[r][c]} to
// part[block]; `red`: LDS for the logit weights, labels, dl and loss of the
// block's rows), the top input-gradient chain dt (j = H-1 .. 1), the concat
// product dc (columns < dA: A's cut delta into dc.out, masked by cat when
// A's last layer has a ReLU; columns >= dA: the gradient message, staged as
// float32 in `msg` when clip/noise run, else written to ring directly), and
// A's chain da (l = LA-1 .. 1); with tables, gx = the float32 gradient of
// the embedding columns.
struct ActiveJob {
  RowInput in;
  BiasTab bt;
  WarmSet warm;
  int32_t LA = 0;
  ChainLayer fa[kMaxChain];
  LBuf cat; RCMat cat_rc; int32_t dA = 0, dB = 0;
  const void* zb = nullptr; int32_t ldzb = 0;
  const int32_t* hdr_chk = nullptr; int32_t* err = nullptr;
  int32_t H = 0;
  ChainLayer ft[kMaxChain];
  const float* lw = nullptr; const float* lb = nullptr; int32_t relu_h = 0;
  int32_t mse = 0;                    // squared-error loss on the output (else BCE)
  LBuf dh; RCMat dh_rc;
  float* part = nullptr;
  LBuf red;
  ChainLayer dt[kMaxChain];
  ChainLayer dc;
  int32_t gextra = 0;
  MsgOp m;
  LBuf msg;
  void* ring = nullptr; int32_t ldring = 0;
  int32_t* hdr_out = nullptr;
  int32_t nda = 0;
  ChainLayer da[kMaxChain];
  int32_t has_gx = 0;
  ChainLayer gx;
  float* gxp = nullptr; int32_t ldgx = 0;
};

// Party B's backward of a group: cut-layer backward of the message g
// (row-major) at the stashed output z (clip backward with norm/cfac when
// clip), then the chain dx (l = L-1 .. 1, or down to 2 when layer 1's input
// gradient is a layer product: then the last delta also goes row-major to
// drm), masks loaded from the stashed ReLU bits (bf16) or RC activations;
// with tables, gx as in ActiveJob.
struct BwdJob {
  BiasTab bt;
  WarmSet warm;
  const void* g = nullptr; int32_t ldg = 0;
  const void* z = nullptr; int32_t ldz = 0;
  const float* norm = nullptr; const float* cfac = nullptr;
  int32_t clip = 0, relu = 0, D = 0;
  float C = 0.f;
  LBuf d; RCMat d_rc;
  const int32_t* hdr_chk = nullptr; int32_t* err = nullptr;
  int32_t nd = 0;
  ChainLayer dx[kMaxChain];
  int32_t has_gx = 0;
  ChainLayer gx;
  float* gxp = nullptr; int32_t ldgx = 0;
  void* drm = nullptr; int32_t lddrm = 0;
};

// Jobs live in device memory (written once when the context is created);
// `rt` selects 16 * rt rows per block, `lds` the dynamic LDS bytes.
// pf: MFMA steps per weight load group of the chain kernel,
// kChainPFNarrow, or kChainPFWide for bf16
hipError_t launch_fwd(Elt e, int rt, int pf, const FwdJob* job, int lds, int blocks, const ChainCall& c,
                      TickRef tr, hipStream_t st);
hipError_t launch_active(Elt e, int rt, int pf, const ActiveJob* job, int lds, int blocks,
                         const ChainCall& c, TickRef tr, hipStream_t st);
hipError_t launch_bwd(Elt e, int rt, int pf, const BwdJob* job, int lds, int blocks, const ChainCall& c,
                      TickRef tr, hipStream_t st);
// Raise the dynamic-LDS limit of every chain kernel to kLdsMax.
hipError_t chain_init();

// --------------------------------------------------------- weight gradients
// One layer's weight gradient over the group's rows from RC operands:
// G[n][k] = sum_r D[r][n] X[r][k], g_b[n] = sum_r D[r][n]; W -= scale * G,
// bias -= scale * g_b, then the packed operand copies Wq of W (kq steps)
// and Wtq of W^T (kt steps; both nullable) are rewritten from the new W.
// Rows are cut into
// `splits` chunks of rps rows (a multiple of 128); with more than one chunk
// each block writes float32 partials part[s][n][kp] (kp = K rounded up to
// 4) and partb[s][n], and k_dw_reduce finishes the layer.  Blocks
// [first_block, first_block + tiles * splits) work on this problem.
constexpr int kRedK = 128;   // inputs per reduction tile (k_dw_reduce)
struct DwProb {
  RCMat D, X;
  float* W = nullptr; float* bias = nullptr;
  void* Wq = nullptr; void* Wtq = nullptr;
  int32_t kq = 0, kt = 0;
  float* part = nullptr; float* partb = nullptr;
  int32_t N = 0, K = 0, kp = 0, splits = 1, rps = 0, first_block = 0;
};
struct DwJob {
  int32_t n = 0, blocks = 0;
  DwProb p[kMaxDw];
  // reduction launch: split problems' tiles (8 outputs x kRedK inputs)
  // and bias blocks (256 each), problem by problem, then the logit layer's
  // columns (lblocks partial
  // rows of Hd + 2 floats, of which the first ceil(rows / lrows) are the
  // group's)
  int32_t red_blocks = 0;
  int32_t rows_pad = 0;               // RC rows (k_dw32: its row steps cover them all)
  float* lpart = nullptr; int32_t Hd = 0, lrows = 0;
  float* lw = nullptr; float* lb = nullptr;
};
hipError_t launch_dw(Elt e, const DwJob* job, int blocks, int R, float scale, TickRef tr,
                     hipStream_t st);
// bf16 problems over 256 x 256 tiles (tiles counted with that shape; rps a
// multiple of 32, at least two chunks per problem): float32 partials only,
// which k_dw_reduce sums (with the SGD step).
hipError_t dwt_init();
hipError_t launch_dwt(const DwJob* job, int blocks, hipStream_t st);
// Unsplit problems over 32 x 32 tiles (every problem's splits == 1, tiles
// counted with 32-wide tiles; `blocks` = job->blocks + the logit blocks):
// products, SGD and copy refresh in one launch, the logit reduction in the
// blocks past job->blocks (loss_out / loss_base as for k_dw_reduce).
hipError_t launch_dw32(Elt e, const DwJob* job, int blocks, int R, float scale, float* loss_out,
                       TickRef tr, float* loss_base, hipStream_t st);
// loss_out: the group's mean loss (from the logit partials); with a tick
// reference, loss_base + the tick's loss index instead.
hipError_t launch_dw_reduce(Elt e, const DwJob* job, int blocks, int R, float scale,
                            float* loss_out, TickRef tr, float* loss_base, hipStream_t st);

// ---------------------------------------------------------- layer products
// The input gradient of a wide bottom layer of party B over the rows of a
// group (bf16), in large tiles:
//   out[r][n] = mask(r, n) * sum_k A[r][k] W[n][k]
// for r < rows, into out_rc (rows from the group's end up to rows_pad zero);
// mask(r, n) = bit r mod 8 of mbits[(r / 8) * ldb + n] (mbits null: 1).
// A: row-major bf16, lda elements per row (a multiple of 8; finite values
// from K up to lda); W: packed [N x K] (pk_index, kst 32-k steps, zero past
// K).  Blocks: lin_blocks(rows_pad, N): 256 x 256 output tiles rounded up
// to a multiple of the 8 XCDs.
struct LinJob {
  const void* A = nullptr; int64_t lda = 0;
  const void* W = nullptr; int32_t kst = 0;
  int32_t N = 0, K = 0;
  RCMat out_rc;
  const uint8_t* mbits = nullptr; int32_t ldb = 0;
  int32_t tiles_n = 0, tiles_m = 0, rows_pad = 0;
};
int lin_blocks(int rows_pad, int N);
hipError_t lin_init();
hipError_t launch_lin(const LinJob* job, int blocks, int rows, TickRef tr, hipStream_t st);

// ------------------------------------------------------- replica averaging
// In place over n parameter sets of the same layout (base[i]: a context's
// workspace): every float32 element x of the segments becomes
// sum_i w[ws][i] * x_i (accumulated in the order i = 0 .. n-1; ws = the
// segment's weight set), written back to every set.  Segment s: cnt[s]
// floats at byte offset off[s] (16-byte aligned), weight set wsel[s];
// first[s] = float4 units before segment s (first[nseg] = total).
constexpr int kMaxAvgSets = 16;
constexpr int kMaxAvgSegs = 2 * (2 * kMaxChain + 4);   // both parties' layers, the top, tables
struct AvgJob {
  int32_t n = 0, nseg = 0;
  float w[2][kMaxAvgSets];
  char* base[kMaxAvgSets];
  int64_t off[kMaxAvgSegs], cnt[kMaxAvgSegs], first[kMaxAvgSegs + 1];
  uint8_t wsel[kMaxAvgSegs];
};
hipError_t launch_avg(const AvgJob& j, hipStream_t st);

// ---------------------------------------------------------------- others
// Operand copies of one layer's float32 weight W [out x in], element type
// e, packed (pk_index): Wq of W (kq = K steps over `in`), Wtq of W^T (kt =
// steps over `out`).
struct CastJob {
  const float* W; void* Wq; void* Wtq; int out, in; int kq, kt;
};
hipError_t launch_cast(Elt e, const CastJob* jobs, int n_jobs, hipStream_t st);

// Sparse SGD on the tables: for every row f*V + id touched by field f,
// T[row][c] -= scale * sum over samples r with idt[f][r] == id of G[r][f*E + c]
// (one rounding per touched row and pass of 8192 samples; deterministic).
// idt: the field-major id copy the chain kernel's gather wrote
// (idt[f * ldi + r]).  E <= kMaxEmbDim and a multiple of 4, V <= 2^19.
constexpr int kMaxEmbDim = 16;
struct ScatterJob {
  float* T; const int32_t* idt; int64_t ldi; int n_cat, V, E;
  const float* G; int64_t ldg; int R; float scale;
  TickRef tr;                          // R, scale
};
hipError_t launch_scatter_sgd(const ScatterJob& j, hipStream_t st);

// Raw Philox4x32-10 words: out[(r * groups + q) * 4 + i] = word i of the
// counter (step, row0 + r, q, tag) under key (seed low, seed high).
hipError_t launch_philox_words(uint64_t seed, uint32_t step, uint32_t tag, uint32_t row0,
                               int rows, int groups, uint32_t* out, hipStream_t st);

}  // namespace vfl
