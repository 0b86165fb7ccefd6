// Internal launch interface of the gfx950 kernels (not part of the C ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vfl {

// Element type of activations, messages and weight copies.
enum Elt { F32 = 0, BF16 = 1 };

inline int elt_size(Elt e) { return e == F32 ? 4 : 2; }

// Per-tick values that a replayed graph reads from device memory; k_advance
// writes them at the start of each stream's part of a tick.  A job whose
// `ta` is set takes its row count (and the values listed with each job)
// from *ta instead of its immediate fields; with ta_in set its dataset
// input pointers are bases, offset by ta->row0 rows.
struct TickArgs {
  int32_t rows;        // rows of the batch group
  int32_t group;       // batch-group id (noise step, header sequence)
  int64_t row0;        // dataset row of the group's first row
  int32_t hdr[3];      // channel header to write {group, tick, version}
  int32_t chk;         // group expected in the header of the slot read
  float scale;         // lr / rows
  int32_t pad;
  int64_t loss_idx;    // index of the group's loss in the loss ring
};

// k_advance: one thread reads this stream's tick counter t, writes the
// records of tick t of the deterministic schedule over a resident dataset
// of n_rows rows (group g covers rows [(g mod E) * R, ...), E = ceil(n/R),
// the last group of an epoch short) and increments the counter.
// Party A (kind 0): out[0] = group t - s.  Party B (kind 1): out[0] =
// group t (its forward), out[1] = group t - s (its backward).
struct AdvanceJob {
  int64_t* counter = nullptr;
  TickArgs* out[2] = {nullptr, nullptr};
  int kind = 0;
  int64_t n_rows = 0;
  int R = 0, s = 0;
  float lr = 0.f;
  int64_t loss_len = 1;
};
hipError_t launch_advance(const AdvanceJob& j, hipStream_t st);

// C[m][n] = epilogue( sum_k A[m][k] * B[n][k] ), A = [A1 | A2] split at
// column ksplit (A2 may be null when ksplit >= K).  Epilogue: + bias[n],
// optional ReLU, then columns n < nsplit go to C1 (multiplied by
// (mask[m][n] > 0) when mask is set), columns n >= nsplit to C2 at column
// n - nsplit (float32 when c2_f32).  All matrices row-major with leading
// dimensions in elements; rows must be 16-byte aligned.
struct GemmNT {
  const void* A1 = nullptr; int64_t lda1 = 0;
  const void* A2 = nullptr; int64_t lda2 = 0; int ksplit = 1 << 30;
  const void* B = nullptr; int64_t ldb = 0;
  void* C1 = nullptr; int64_t ldc1 = 0;
  void* C2 = nullptr; int64_t ldc2 = 0; int nsplit = 1 << 30; int c2_f32 = 0;
  const float* bias = nullptr;
  const void* mask = nullptr; int64_t ldm = 0;
  int relu = 0;
  int M = 0, N = 0, K = 0;
  // channel slot header written by block 0 (hdr_out != null) / checked by
  // block 0 against chk_seq (mismatch -> atomic increment of *err)
  int32_t* hdr_out = nullptr; int32_t hdr[3] = {0, 0, 0};
  const int32_t* hdr_chk = nullptr; int32_t chk_seq = 0; int32_t* err = nullptr;
  // tick record: M = ta->rows; ta_in: A1 += ta->row0 rows; header values
  // and the expected sequence from *ta
  const TickArgs* ta = nullptr; int ta_in = 0;
};

// One layer's weight gradient + SGD: G[n][k] = sum over rows r of
// D[r][n] * X[r][k], g_b[n] = sum_r D[r][n]; W -= scale * G, bias -= scale *
// g_b, then the operand copies Wq [N x ldq] and Wtq [K x ldt] (nullable) are
// rewritten from the new W.  X = [X1 | X2] split at column ksplit.  The rows
// are cut into `splits` chunks of rows_per_split (a multiple of the stage
// depth); with more than one chunk each block writes float32 partials
// part[s][n][k] (partb[s][n]) and k_multi_reduce finishes the layer.
struct GemmDW {
  const void* D = nullptr; int64_t ldd = 0;
  const void* X1 = nullptr; int64_t ldx1 = 0;
  const void* X2 = nullptr; int64_t ldx2 = 0; int ksplit = 1 << 30;
  float* W = nullptr; float* bias = nullptr;
  void* Wq = nullptr; int64_t ldq = 0; void* Wtq = nullptr; int64_t ldt = 0;
  float* part = nullptr; float* partb = nullptr;
  int N = 0, K = 0, splits = 1, rows_per_split = 0;
  int x_ta = 0;                        // X1 += ta->row0 rows (dataset input)
};
constexpr int kMaxDw = 8;
// Several layers' weight gradients over the same R rows (one launch).
struct MultiDW {
  GemmDW p[kMaxDw];
  int n = 0, R = 0;
  float scale = 0.f;
  int first_block[kMaxDw + 1] = {0};   // filled by launch_multi_dw
  const TickArgs* ta = nullptr;        // R = ta->rows, scale = ta->scale
};

hipError_t launch_gemm_nt(Elt e, const GemmNT& g, hipStream_t st);
hipError_t launch_multi_dw(Elt e, MultiDW& m, hipStream_t st);
int dw_stage_rows(Elt e);   // rows per pipeline stage of the dW kernel
int dw_tiles(int N, int K); // 64 x 64 output tiles of one layer

// Operand copies of one layer's float32 weight W [out x in]:
// Wq [out x ldq] and Wtq [in x ldt] of element type e (ldq, ldt padded).
struct CastJob {
  const float* W; void* Wq; void* Wtq; int out, in; int64_t ldq, ldt;
};
hipError_t launch_cast(Elt e, const CastJob* jobs, int n_jobs, hipStream_t st);

constexpr int kMaxLogitCols = 512;   // widest last hidden layer of the top model

// Logit layer + BCE on the last hidden activation H [R x ldh] (width Hd):
// l = H w + b, loss_i = BCE(l, y), dl = sigmoid(l) - y; writes
// delta [R x ldd] = dl * w * (H > 0) (element type e).  Each block writes
// partial sums part[blk] = {loss, sum dl, sum_r dl * H[r][0..Hd)} (Hd + 2
// floats); k_multi_reduce reduces them in block order:
// *loss_out = sum loss / R (loss_out may be null), w -= scale * sum dl*H,
// b -= scale * sum dl.
struct LogitJob {
  const void* H; int64_t ldh; int Hd, R;
  float* w; float* b; const float* y;
  void* delta; int64_t ldd; int relu;
  float* part; int blocks; float scale; float* loss_out;
  // tick record: R, scale, y += row0, loss_out = loss_base + loss_idx
  const TickArgs* ta; float* loss_base;
};
hipError_t launch_logit_bce(Elt e, const LogitJob& j, hipStream_t st);
// Second stage of the split layers of m and (lj != null) of the logit
// kernel's partials, in one launch.
hipError_t launch_multi_reduce(Elt e, const MultiDW& m, const LogitJob* lj, hipStream_t st);

// Segments mapping a row of a tick to its global sample id (<= 8 replicas).
struct RowMap {
  int n = 1;
  int32_t start[8] = {0};
  int64_t row0[8] = {0};
};

// Per-row clip + Gaussian noise: out[r] = c_r * v[r] + std * xi(seed, step,
// global row, col, tag), c_r = min(1, C / ||v[r]||) when clip (else 1).
// v is element type e (or float32 when v_f32); out is element type e.
// norm/cfac (nullable) receive ||v[r]|| and c_r.  Block 0 writes the slot
// header.
struct ClipNoiseJob {
  const void* v; int64_t ldv; int v_f32;
  void* out; int64_t ldo;
  float* norm; float* cfac;
  int R, D; int clip; float C; int noise; float stdv;
  uint64_t seed; uint32_t step; uint32_t tag; RowMap rows;
  int32_t* hdr_out; int32_t hdr[3];
  // tick record: R, step = group, global rows from row0, header values
  const TickArgs* ta;
};
hipError_t launch_clip_noise(Elt e, const ClipNoiseJob& j, hipStream_t st);

// Cut-layer backward of party B: g = message row; if clipped (n_r > C):
// g = c_r (g - u (u . g)), u = z_r / n_r; delta = g * (z > 0 when relu).
// Block 0 checks the slot header.
struct CutBwdJob {
  const void* g; int64_t ldg; const void* z; int64_t ldz;
  const float* norm; const float* cfac; int clip; float C; int relu;
  void* delta; int64_t ldd; int R, D;
  const int32_t* hdr_chk; int32_t chk_seq; int32_t* err;
  const TickArgs* ta;                  // R and the expected sequence
};
hipError_t launch_cut_backward(Elt e, const CutBwdJob& j, hipStream_t st);

// Embedding gather + concat: X[r] = [T[f*V + ids[r][f]] for f | dense[r]]
// (float32 tables; X and dense of element type e).
struct GatherJob {
  const float* T; const int32_t* ids; int n_cat, V, E;
  const void* dense; int64_t ldx_in; int dense_in;
  void* X; int64_t ldx; int R;
  const TickArgs* ta;                  // R; ids and dense offset by row0 rows
};
hipError_t launch_gather(Elt e, const GatherJob& j, hipStream_t st);

// Sparse SGD on the tables: for every row f*V + id touched by field f,
// T[row][c] -= scale * sum over samples r with ids[r][f] == id of G[r][f*E + c]
// (one rounding per touched row; deterministic).  E <= kMaxEmbDim,
// V <= 2^19.
constexpr int kMaxEmbDim = 16;
struct ScatterJob {
  float* T; const int32_t* ids; int n_cat, V, E;
  const float* G; int64_t ldg; int R; float scale;
  const TickArgs* ta;                  // R, scale; ids offset by row0 rows
};
hipError_t launch_scatter_sgd(const ScatterJob& j, hipStream_t st);

// Raw Philox4x32-10 words: out[(r * groups + q) * 4 + i] = word i of the
// counter (step, row0 + r, q, tag) under key (seed low, seed high).
hipError_t launch_philox_words(uint64_t seed, uint32_t step, uint32_t tag, uint32_t row0,
                               int rows, int groups, uint32_t* out, hipStream_t st);

}  // namespace vfl
