// C ABI of the publisher/subscriber split-learning step (include/vfl.h).
//
// Host side only: it validates shapes, lays the caller's workspace out,
// plans the LDS layout of the fused chain kernels, writes their job
// descriptors into the workspace once, keeps the channel state machine
// (which group each slot holds, B's parameter version, how many groups are
// in flight) and enqueues the kernels of kernels.h on the two party streams.
// Party A's work goes to stream_a, party B's to stream_b; the only
// cross-stream edges are the per-slot "embedding published" and "gradient
// published" events.
//
// Slot reuse needs no further edges: B rewrites embedding slot g mod (s+1)
// with group g + s + 1 only after its backward of group g, which waited for
// g's gradient event, recorded by A after A read embedding g; A rewrites
// gradient slot u mod (s+1) with group u + s + 1 only after waiting for that
// group's embedding event, recorded by B after its backward of group u.
//
// Per tick and party: B runs k_fwd (forward + publish) for group t, and for
// group u = t - s k_bwd, k_dw and k_dw_reduce; A runs k_active, k_dw and
// k_dw_reduce for group u (plus the sparse table step with embedding
// tables).  The weight update refreshes the operand copies of party B in the
// slot of the group just back-propagated, which is the slot B's next
// forward uses; a forward casts the master weights only when its slot's
// copies hold another version.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/vfl.h"
#include "kernels.h"

using namespace vfl;

namespace {

constexpr int kMaxSlots = VFL_MAX_STALENESS + 1;
constexpr int kGemmMinWidth = 512;    // B's first-layer width from which its input gradient is a layer product
constexpr int kMinBlocks = 256;       // row blocks a chain launch aims at (one per CU)
constexpr int kDwBlocks = 256;        // weight-gradient blocks a launch aims at
constexpr double kRcStreamBytes = 32e6;  // RC copies above this size use streaming stores
constexpr int kDwRows = 256;          // rows of two k_dw load groups (4 MFMA steps each) in bf16;
                                      // float32 chunks hold half the rows: 128
constexpr int kTimedEvery = 4;        // ticks of a captured cycle between timed ticks

int64_t ld_of(int w) { return ((int64_t)w + 7) / 8 * 8; }  // 16-byte rows for both types

struct Layout {
  size_t off = 0;
  size_t take(size_t bytes) {
    off = (off + 255) / 256 * 256;
    size_t o = off;
    off += bytes;
    return o;
  }
};

struct Party {
  vfl_bottom_spec spec{};
  int L = 0, din = 0, nslots = 1;
  int in[VFL_MAX_LAYERS]{}, out[VFL_MAX_LAYERS]{};
  bool relu[VFL_MAX_LAYERS]{};
  int kq[VFL_MAX_LAYERS]{}, kt[VFL_MAX_LAYERS]{};   // K steps of the packed copies of W, W^T
  size_t W[VFL_MAX_LAYERS]{}, b[VFL_MAX_LAYERS]{}, T = 0;
  size_t Wq[kMaxSlots][VFL_MAX_LAYERS]{}, Wtq[kMaxSlots][VFL_MAX_LAYERS]{};
  size_t x0rc[kMaxSlots]{};                     // RC copy of the bottom input
  size_t arc[kMaxSlots][VFL_MAX_LAYERS]{};      // RC outputs of layers 0 .. L-2
  size_t drc[VFL_MAX_LAYERS]{};                 // RC deltas of every layer
  size_t z[kMaxSlots]{}, zhat[kMaxSlots]{};     // party B: last layer, published message
  size_t norm[kMaxSlots]{}, cfac[kMaxSlots]{};
  size_t gx = 0;
  int64_t ldgx = 0;
  size_t idt[kMaxSlots]{};                      // field-major id copies (tables)
  size_t part[VFL_MAX_LAYERS]{}, partb[VFL_MAX_LAYERS]{};
  int bo[VFL_MAX_LAYERS]{};                     // bias offsets (floats) in the party's bias table
  size_t wq_end[kMaxSlots]{}, wtq_end[kMaxSlots]{};   // ends of the packed ranges
};

struct Top {
  vfl_top_spec spec{};
  int H = 0;                          // hidden layers (n_layers - 1)
  int in[VFL_MAX_LAYERS]{}, out[VFL_MAX_LAYERS]{};
  bool relu[VFL_MAX_LAYERS]{};
  int kq[VFL_MAX_LAYERS]{}, kt[VFL_MAX_LAYERS]{};
  size_t W[VFL_MAX_LAYERS]{}, b[VFL_MAX_LAYERS]{};
  size_t Wq[VFL_MAX_LAYERS]{}, Wtq[VFL_MAX_LAYERS]{};
  size_t arc[VFL_MAX_LAYERS]{}, drc[VFL_MAX_LAYERS]{};
  size_t part[VFL_MAX_LAYERS]{}, partb[VFL_MAX_LAYERS]{};
  size_t logit_part = 0;
  int bo[VFL_MAX_LAYERS]{};           // hidden-layer bias offsets (floats) in A's bias table
  size_t packed_end = 0;
};

// LDS layout of one chain kernel at BR rows per block
struct Lds {
  int KS = 32, BR = 16, off = 0;
  LBuf take(int width, int elt_bytes) {
    const int cols = (width + KS - 1) / KS * KS;
    LBuf b;
    b.off = off;
    b.pitch = (cols * elt_bytes + 127) / 128 * 128 + 16;
    off += b.pitch * BR;
    off = (off + 15) / 16 * 16;
    return b;
  }
  LBuf raw(int bytes) {
    LBuf b;
    b.off = off;
    b.pitch = 1;
    off += (bytes + 15) / 16 * 16;
    return b;
  }
  // two buffers that are never live at the same time: one region as large
  // as the larger, each with its own pitch
  void take_shared(LBuf& a, int wa, int ea, LBuf& b, int wb, int eb) {
    const int o = off;
    a = take(wa, ea);
    const int ea_end = off;
    off = o;
    b = take(wb, eb);
    off = std::max(off, ea_end);
  }
};

struct FwdLds { LBuf buf[2], bias; int bytes = 0; };
struct ActLds {
  LBuf in, fa[VFL_MAX_LAYERS], cat, ft[VFL_MAX_LAYERS], P[2], msg, red, bias;
  int bytes = 0;
};
struct BwdLds { LBuf P[2], mask[VFL_MAX_LAYERS]; int bytes = 0; };

struct KMeta { int rt = 1, blocks = 1, lds = 0, pf = kChainPFNarrow; };
constexpr size_t kPFWideElts = 256 * 1024;   // chain weights taking the deeper load groups

// Weight-gradient launch shape of a party: tile 32 (one unsplit launch,
// k_dw32) or 64 (row chunks, k_dw + k_dw_reduce).
struct DwMeta { int tile = 64, splits = 1, rps = 0, blocks = 0, red_blocks = 0, logit_blocks = 0; };

struct Plan {
  Elt e = F32;
  int s = 0, k = 1, B = 1, R = 1, Ra = 64, dA = 0, dB = 0;
  bool dw32 = false;                  // unsplit 32 x 32 weight gradients
  Party A, P;                         // P: party B (passive)
  Top T;
  size_t cat_rc = 0;
  // bias tables: A's layers then the top model's hidden layers; B's layers
  // (each row padded to 32 floats)
  size_t bias_a = 0, bias_b = 0;
  int nbias_a = 0, nbias_b = 0;       // floats
  size_t ring_g[kMaxSlots]{};
  size_t hdr = 0;                     // int32 [2][kMaxSlots][4] + error counter
  size_t tsrc = 0;                    // TickSrc of the replayed graphs
  size_t job_fwd = 0, job_act = 0, job_bwd = 0, job_dwa = 0, job_dwb = 0;
  // party B's layer-1 input gradient as a large-tile layer product (wide
  // first layer): the backward chain stops at layer 2 and writes its last
  // delta row-major to d1rm; LinJob per slot
  bool bgemm = false;
  size_t d1rm = 0, job_lin = 0;
  int lin_blocks_dx = 0;
  size_t mbits[kMaxSlots][VFL_MAX_LAYERS]{};   // B's ReLU bits per slot and layer [Ra / 8 x ldb[l]] (0: none)
  int ldb[VFL_MAX_LAYERS]{};                  // their row pitch (bytes: the layer width rounded up to 64)
  KMeta kf, ka, kb;
  FwdLds lf;
  ActLds la;
  BwdLds lb;
  DwMeta da, db;
  size_t total = 0;
};

struct SlotState {
  int64_t group = -1;
  int64_t version = -1;
  bool published = false;
  int rows = 0;
  int64_t row0 = 0;                   // sample id of row 0
  const void* dense = nullptr;
  int64_t ld = 0;
  const int32_t* ids = nullptr;
  const float* labels = nullptr;
};

// Event pairs bracketing the launches of the selected kernel classes.
struct Timing {
  static constexpr int kPool = 4096;
  uint32_t mask = 0;
  bool created = false;
  hipEvent_t ev0[kPool]{}, ev1[kPool]{};
  int cls[kPool]{};
  double work[kPool]{};
  bool used[kPool]{};
  int next = 0;
  double ms[VFL_K_COUNT]{}, wk[VFL_K_COUNT]{};
  int64_t n[VFL_K_COUNT]{};
};

}  // namespace

struct vfl_ctx {
  Plan p;
  Timing tm;
  vfl_opts o{};
  char* ws = nullptr;
  int static_dev = -1;  // device whose static workspace this context holds (-1: caller's)
  hipStream_t sa = nullptr, sb = nullptr;
  hipEvent_t ev_emb[kMaxSlots]{}, ev_grad[kMaxSlots]{};
  // B
  int64_t b_next_fwd = 0, b_next_bwd = 0, b_version = 0, b_pub_next = 0;
  SlotState bslot[kMaxSlots];
  int64_t b_copy_version[kMaxSlots];  // version held by each slot's operand copies (-1: none)
  int64_t grad_group[kMaxSlots];
  int grad_rows[kMaxSlots]{};
  // A (and the top model)
  int64_t a_next = 0, a_version = 0, a_copy_version = -1;
  int a_phase = 0;                    // 0 forward, 1 top step, 2 backward
  SlotState aslot;
  float* a_loss = nullptr;
  // rows each party has applied since its last replica average (the
  // average's weights)
  int64_t a_rows_avg = 0, b_rows_avg = 0;
  hipEvent_t ev_avg = nullptr;
  // discarded groups (Section 4.1 "System Design": the buffer and waiting-deadline
  // mechanisms), each until B's backward of it releases its slot without
  // an update; grad: A had consumed the group (B must wait for A's
  // gradient event before reusing the slot)
  struct Drop { int64_t group; bool grad; };
  std::vector<Drop> drops;
  std::vector<int64_t> trace;
  std::string err;
  // resident dataset + captured graphs (one per phase t mod (s+1))
  bool bound = false;
  vfl_dataset ds_a{}, ds_b{};
  int64_t n_rows = 0;
  // graph i < kMaxSlots: VFL_GRAPH_CYCLES * (s+1) ticks from phase i;
  // graph kMaxSlots + i: a shorter remainder from phase i
  static constexpr int kGraphs = 2 * kMaxSlots;
  hipGraph_t graph[kGraphs]{};
  hipGraphExec_t gexec[kGraphs]{};
  float* graph_loss[kGraphs]{};
  int64_t graph_loss_len[kGraphs]{};
  uint32_t graph_mask[kGraphs]{};
  int graph_len[kGraphs]{};
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  int capture_phase = -1;             // >= 0 while capturing that graph (its index)
  int capture_tick = -1;              // tick of the cycle being captured
  struct GPair { hipEvent_t e0, e1; int cls; double work; };
  std::vector<GPair> gpairs[kGraphs];     // created before capture
  int gused[kGraphs]{};                   // pairs used by the captured graph
  hipError_t tm_err = hipSuccess;         // first failed event record in a capture
  std::string tm_err_what;
  int last_phase = -1;                // the graph replayed last
};

namespace {

template <typename T>
T* at(vfl_ctx* c, size_t off) { return (T*)(c->ws + off); }

// Failures of calls that have no context yet (vfl_workspace_size, vfl_create)
// keep their text per host thread; vfl_last_error(NULL) returns it.
thread_local std::string t_create_err;

vfl_status fail(vfl_ctx* c, vfl_status st, const std::string& msg) {
  if (c) c->err = msg;
  return st;
}

vfl_status fail_create(vfl_status st, const std::string& msg) {
  t_create_err = msg;
  return st;
}

#define HIPCHK(expr)                                                                     \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess)                                                                \
      return fail(c, VFL_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_));     \
  } while (0)

#define HIPCHK0(ctx, expr)                                                               \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess)                                                                \
      return fail((ctx), VFL_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_));  \
  } while (0)

bool check_bottom(const vfl_bottom_spec* s, std::string& why) {
  if (!s) { why = "null bottom spec"; return false; }
  if (s->n_layers < 1 || s->n_layers > VFL_MAX_LAYERS) { why = "bottom n_layers out of range"; return false; }
  if (s->dense_in < 0 || s->n_cat < 0) { why = "negative bottom input width"; return false; }
  if (s->n_cat > 0 && (s->vocab < 1 || s->vocab > (1 << 19) || s->emb_dim < 4 || s->emb_dim % 4 ||
                       s->emb_dim > kMaxEmbDim)) {
    why = "embedding dims: vocab in [1, 2^19], emb_dim a multiple of 4 in [4, 16]"; return false;
  }
  if (s->n_cat * (int64_t)std::max(s->emb_dim, 0) + s->dense_in < 1) { why = "empty bottom input"; return false; }
  if (s->n_cat * (int64_t)std::max(s->emb_dim, 0) + s->dense_in > 65536) { why = "bottom input too wide"; return false; }
  for (int l = 0; l < s->n_layers; ++l)
    if (s->widths[l] < 1 || s->widths[l] > 65536) { why = "bad bottom width"; return false; }
  return true;
}

// output tiles of a weight gradient [N x K]: square tiles of 32, 64 or 256
// (tile == 256: the large-tile kernel)
int dw_tiles(int N, int K, int tile = 64) {
  return ((N + tile - 1) / tile) * ((K + tile - 1) / tile);
}

// Parties whose weight gradient per tick reaches this many FLOPs (bf16)
// take the large-tile kernel (one 96 KB-LDS block per CU, so at most one
// block per CU is planned).
constexpr double kDwtMinFlops = 4e9;

// Groups whose RC operand columns hold at most this many bytes (rows times
// element size) contract all their rows in one block per 32 x 32 tile.
constexpr int kDwUnsplitBytes = 2048;

// Chunks of at least this many rows may be cut at any 32-row stage.
constexpr int kDwtFineRows = 1024;

// Row chunks of a weight-gradient launch over `tiles` output tiles: at
// most kDwBlocks blocks (one round on the CUs: a few blocks past it would
// double the launch), chunks a multiple of two load groups (kDwRows rows
// in bf16, half that in float32).
void dw_split(int R, int tiles, bool bf16, DwMeta& m) {
  auto split = [&](int gran) {
    const int max_splits = std::max(1, (R + gran - 1) / gran);
    const int s = std::min(max_splits, std::max(1, kDwBlocks / tiles));
    m.rps = ((R + s - 1) / s + gran - 1) / gran * gran;
    m.splits = (R + m.rps - 1) / m.rps;
  };
  split(bf16 ? kDwRows : kDwRows / 2);
  if (m.tile == 256 && m.rps >= kDwtFineRows) {
    // long chunks of the large-tile kernel need only whole 32-row stages:
    // the finer granularity lets them fill the CUs (hetero's B: 14 chunks of
    // 2368 rows, 252 blocks, instead of 13 of 2560, 234 blocks); short ones
    // keep the coarser chunks, whose fewer partials shorten the reduction
    split(32);
  }
  if (m.tile == 256 && m.splits < 2) {
    // the large-tile kernel writes partials only: two chunks of a multiple
    // of its 32-row stage
    m.rps = ((R + 1) / 2 + 31) / 32 * 32;
    m.splits = 2;
  }
}

// LDS layouts at BR rows per block (bytes in .bytes)
void plan_fwd_lds(const Plan& p, int BR, FwdLds& f) {
  Lds l;
  l.KS = p.e == BF16 ? 32 : 16;
  l.BR = BR;
  // layer l reads buf[l % 2] and writes buf[(l + 1) % 2]; the input is in
  // buf[0]: each buffer is as wide as the widest tensor it holds
  int w[2] = {p.P.din, 1};
  for (int i = 0; i < p.P.L; ++i) w[(i + 1) % 2] = std::max(w[(i + 1) % 2], p.P.out[i]);
  const int es = elt_size(p.e);
  f.buf[0] = l.take(w[0], es);
  f.buf[1] = l.take(w[1], es);
  f.bias = l.raw(4 * p.nbias_b);
  f.bytes = l.off;
}

void plan_act_lds(const Plan& p, int BR, bool gextra, ActLds& a) {
  Lds l;
  l.KS = p.e == BF16 ? 32 : 16;
  l.BR = BR;
  const int es = elt_size(p.e);
  for (int i = 0; i + 1 < p.A.L; ++i) a.fa[i] = l.take(p.A.out[i], es);
  a.cat = l.take(p.dA + p.dB, es);
  for (int j = 0; j + 1 < p.T.H; ++j) a.ft[j] = l.take(p.T.out[j], es);
  int w = 1;
  for (int j = 0; j < p.T.H; ++j) w = std::max(w, p.T.out[j]);
  for (int i = 0; i < p.A.L; ++i) w = std::max(w, p.A.out[i]);
  a.P[0] = l.take(w, es);
  // buffers never live at the same time share LDS: the input (read by A's
  // first layer only) with P[1] (first written after the logit stage), and
  // the last top hidden output (dead once the logit stage has formed dh)
  // with the float32 gradient-message staging (written by the concat
  // product)
  l.take_shared(a.in, p.A.din, es, a.P[1], w, es);
  if (gextra) l.take_shared(a.ft[p.T.H - 1], p.T.out[p.T.H - 1], es, a.msg, p.dB, 4);
  else a.ft[p.T.H - 1] = l.take(p.T.out[p.T.H - 1], es);
  // logit weights [Hd], the block's labels, dl and loss [BR each]
  // the block's labels, per-wavefront partials of the logit layer's
  // weight gradient [kChainWaves][Hd rounded to 4] and of {loss, dl}
  a.red = l.raw(4 * (BR + kChainWaves * ((p.T.out[p.T.H - 1] + 3) / 4 * 4) + 2 * kChainWaves));
  a.bias = l.raw(4 * p.nbias_a);
  a.bytes = l.off;
}

void plan_bwd_lds(const Plan& p, int BR, BwdLds& b) {
  Lds l;
  l.KS = p.e == BF16 ? 32 : 16;
  l.BR = BR;
  const int es = elt_size(p.e);
  // the chain's deltas: every layer's output, or (layer product below)
  // those of layers 1 .. L-1
  const int lo = p.bgemm ? 1 : 0;
  // the cut delta (layer L-1's output) is in P[0], the delta of layer i's
  // output in P[(L-1-i) % 2]; the table input gradient reads layer 0's
  int w[2] = {1, 1};
  for (int i = lo; i < p.P.L; ++i) w[(p.P.L - 1 - i) % 2] = std::max(w[(p.P.L - 1 - i) % 2], p.P.out[i]);
  b.P[0] = l.take(w[0], es);
  b.P[1] = l.take(w[1], es);
  // one mask buffer per ReLU layer the chain crosses: all are loaded up
  // front; bf16 keeps the bits B's forward recorded (a byte per 8 rows and
  // column), float32 the stashed activations
  for (int i = lo; i + 1 < p.P.L; ++i) {
    if (!p.P.relu[i]) continue;
    if (p.e == BF16) {
      const int pitch = p.ldb[i] + 16;
      b.mask[i] = l.raw(BR / 8 * pitch);
      b.mask[i].pitch = pitch;
    } else {
      b.mask[i] = l.take(p.P.out[i], es);
    }
  }
  b.bytes = l.off;
}

// Rows per block: the largest of 64, 48, 32, 16 whose layout fits the LDS
// and that still gives kMinBlocks blocks (16 when nothing gives that many).
template <typename F>
bool pick_rt(int R, KMeta& m, F&& bytes_at) {
  for (int rt : {4, 3, 2, 1}) {
    const int BR = 16 * rt;
    const int blocks = (R + BR - 1) / BR;
    const int lds = bytes_at(BR);
    if (lds > kLdsMax) continue;
    if (rt > 1 && blocks < kMinBlocks) continue;
    m.rt = rt;
    m.blocks = blocks;
    m.lds = lds;
    return true;
  }
  return false;
}

std::string build_plan(const vfl_bottom_spec* a, const vfl_bottom_spec* b, const vfl_top_spec* t,
                       const vfl_opts* o, Plan& p) {
  std::string why;
  if (!o) return "null opts";
  // the caller's dtype as the integer it is (a C caller may pass any value;
  // loading it as the enum type would not be defined for other values)
  int32_t dtype = 0;
  static_assert(sizeof(o->dtype) == sizeof(dtype), "vfl_dtype is an int");
  std::memcpy(&dtype, &o->dtype, sizeof(dtype));
  if (dtype != VFL_F32 && dtype != VFL_BF16) return "dtype must be VFL_F32 or VFL_BF16";
  if (o->batch < 1) return "batch must be >= 1";
  if (o->staleness < 0 || o->staleness > VFL_MAX_STALENESS) return "staleness out of [0, 4]";
  if (o->replicas < 1 || o->replicas > VFL_MAX_REPLICAS) return "replicas out of [1, 8]";
  if (!std::isfinite(o->lr)) return "lr not finite";
  if ((o->flags & (VFL_CLIP_EMB | VFL_CLIP_GRAD)) && !(o->clip_c > 0.f)) return "clip needs clip_c > 0";
  if ((o->flags & (VFL_NOISE_EMB | VFL_NOISE_GRAD)) && !(o->sigma >= 0.f)) return "sigma must be >= 0";
  if (!check_bottom(a, why) || !check_bottom(b, why)) return why;
  if (!t || t->n_layers < 2 || t->n_layers > VFL_MAX_LAYERS)
    return "top needs 2.." + std::to_string(VFL_MAX_LAYERS) + " layers (>= 1 hidden + output)";
  if (t->widths[t->n_layers - 1] != 1) return "last top layer must have width 1";
  for (int j = 0; j + 1 < t->n_layers; ++j)
    if (t->widths[j] < 1 || t->widths[j] > 65536) return "bad top width";
  if (t->widths[t->n_layers - 2] > kMaxLogitCols) return "last hidden top width must be <= 512";
  if (a->widths[a->n_layers - 1] % 8) return "party A's embedding width must be a multiple of 8";
  if (a->n_layers + t->n_layers - 1 > kMaxDw)
    return "party A's + the top's hidden layers must be <= " + std::to_string(kMaxDw);
  if ((int64_t)o->batch * o->replicas > (1 << 28)) return "rows per tick too large";

  p.e = dtype == VFL_BF16 ? BF16 : F32;
  p.s = o->staleness;
  p.k = o->replicas;
  p.B = o->batch;
  p.R = o->batch * o->replicas;
  // weight-gradient launch shapes (they fix the RC row count Ra): small
  // groups take the unsplit 32 x 32 weight gradient, whose four wavefronts
  // run two groups of four row steps per iteration over rows rounded up to
  // 1024; larger ones row chunks of rps rows (a multiple of two load
  // groups) over 64 x 64 tiles.  Every block contracts whole chunks: the
  // rows past the group are zero deltas.
  {
    auto bottom_tiles = [&](const vfl_bottom_spec* sp, int tile) {
      int in = sp->n_cat * sp->emb_dim + sp->dense_in, n = 0;
      for (int l = 0; l < sp->n_layers; ++l) { n += dw_tiles(sp->widths[l], in, tile); in = sp->widths[l]; }
      return n;
    };
    auto top_tiles = [&](int tile) {
      int in = a->widths[a->n_layers - 1] + b->widths[b->n_layers - 1], n = 0;
      for (int j = 0; j + 1 < t->n_layers; ++j) { n += dw_tiles(t->widths[j], in, tile); in = t->widths[j]; }
      return n;
    };
    const int Ra128 = (p.R + 127) / 128 * 128;
    p.dw32 = (int64_t)Ra128 * elt_size(p.e) <= kDwUnsplitBytes;
    if (p.dw32) {
      p.Ra = (p.R + 1023) / 1024 * 1024;
      p.da.blocks = bottom_tiles(a, 32) + top_tiles(32);
      p.db.blocks = bottom_tiles(b, 32);
      for (DwMeta* m : {&p.da, &p.db}) { m->tile = 32; m->splits = 1; m->rps = p.Ra; }
    } else {
      // MACs per row of each party's weight gradients
      auto bottom_macs = [&](const vfl_bottom_spec* sp) {
        double in = sp->n_cat * sp->emb_dim + sp->dense_in, n = 0;
        for (int l = 0; l < sp->n_layers; ++l) { n += in * sp->widths[l]; in = sp->widths[l]; }
        return n;
      };
      double top_macs = 0;
      {
        double in = a->widths[a->n_layers - 1] + b->widths[b->n_layers - 1];
        for (int j = 0; j + 1 < t->n_layers; ++j) { top_macs += in * t->widths[j]; in = t->widths[j]; }
      }
      const bool bf = dtype == VFL_BF16;
      p.da.tile = bf && 2.0 * p.R * (bottom_macs(a) + top_macs) >= kDwtMinFlops ? 256 : 64;
      p.db.tile = bf && 2.0 * p.R * bottom_macs(b) >= kDwtMinFlops ? 256 : 64;
      const int ta = bottom_tiles(a, p.da.tile) + top_tiles(p.da.tile), tb = bottom_tiles(b, p.db.tile);
      dw_split(p.R, ta, bf, p.da);
      dw_split(p.R, tb, bf, p.db);
      p.da.blocks = ta * p.da.splits;
      p.db.blocks = tb * p.db.splits;
      p.Ra = std::max(p.da.splits * p.da.rps, p.db.splits * p.db.rps);
    }
  }
  const int es = elt_size(p.e);
  const int64_t R = p.R, Ra = p.Ra;
  const bool eextra = o->flags & (VFL_CLIP_EMB | VFL_NOISE_EMB);
  const bool gextra = o->flags & (VFL_CLIP_GRAD | VFL_NOISE_GRAD);
  Layout ly;
  auto rc_bytes = [&](int cols) { return (size_t)es * Ra * ld_of(cols); };
  // packed MFMA operands: tiles of 16 rows up to the MFMA depth, K steps of
  // one fragment (1 KB) each
  const int KS = p.e == BF16 ? 32 : 16;
  auto ksteps = [&](int K) { return (K + KS - 1) / KS; };
  // (+ slack for the loads of a chain pass's last group, which may run up
  // to 2 * 4 - 1 MFMA steps past the last tile)
  auto packed_bytes = [&](int N, int K) { return (size_t)((N + KS - 1) / KS * KS) * ksteps(K) * 64 + 8192; };

  auto party = [&](Party& P, const vfl_bottom_spec* s, int nslots, bool passive) {
    P.spec = *s;
    P.L = s->n_layers;
    P.din = s->n_cat * s->emb_dim + s->dense_in;
    P.nslots = nslots;
    int in = P.din;
    for (int l = 0; l < P.L; ++l) {
      P.in[l] = in;
      P.out[l] = s->widths[l];
      P.relu[l] = (s->relu_mask >> l) & 1u;
      P.kq[l] = ksteps(in);
      P.kt[l] = ksteps(P.out[l]);
      P.W[l] = ly.take(sizeof(float) * (size_t)P.out[l] * in);
      P.drc[l] = ly.take(rc_bytes(P.out[l]));
      in = P.out[l];
    }
    if (s->n_cat) P.T = ly.take(sizeof(float) * (size_t)s->n_cat * s->vocab * s->emb_dim);
    for (int q = 0; q < nslots; ++q) {
      // the forward's packed copies, then the backward's: two ranges
      for (int l = 0; l < P.L; ++l) P.Wq[q][l] = ly.take(packed_bytes(P.out[l], P.in[l]));
      P.wq_end[q] = ly.off;
      for (int l = 0; l < P.L; ++l) P.Wtq[q][l] = ly.take(packed_bytes(P.in[l], P.out[l]));
      P.wtq_end[q] = ly.off;
      for (int l = 0; l + 1 < P.L; ++l) P.arc[q][l] = ly.take(rc_bytes(P.out[l]));
      P.x0rc[q] = ly.take(rc_bytes(P.din));
      if (passive) {
        P.z[q] = ly.take((size_t)es * R * ld_of(P.out[P.L - 1]));
        P.zhat[q] = eextra ? ly.take((size_t)es * R * ld_of(P.out[P.L - 1])) : P.z[q];
        if (o->flags & VFL_CLIP_EMB) {
          P.norm[q] = ly.take(sizeof(float) * R);
          P.cfac[q] = ly.take(sizeof(float) * R);
        }
      }
    }
    if (s->n_cat) {
      P.ldgx = ld_of(s->n_cat * s->emb_dim);
      P.gx = ly.take(sizeof(float) * R * P.ldgx);
      for (int q = 0; q < nslots; ++q) P.idt[q] = ly.take(sizeof(int32_t) * R * s->n_cat);
    }
  };

  party(p.A, a, 1, false);
  party(p.P, b, p.s + 1, true);
  p.dA = p.A.out[p.A.L - 1];
  p.dB = p.P.out[p.P.L - 1];
  // B's first layer at least kGemmMinWidth wide (its deltas would crowd the
  // chain's LDS), no tables, bf16: layer 1's input gradient is a layer
  // product over the whole group
  p.bgemm = p.e == BF16 && p.P.L >= 2 && p.P.spec.n_cat == 0 && p.P.out[0] >= kGemmMinWidth;
  if (p.bgemm) p.d1rm = ly.take((size_t)es * R * ld_of(p.P.out[1]));
  // bf16: B's forward records one bit per activation of every ReLU layer
  // below the cut layer, which B's delayed backward (and the wide layer's
  // input-gradient product) read as the ReLU derivative instead of the
  // stashed activations
  if (p.e == BF16) {
    for (int l = 0; l + 1 < p.P.L; ++l) p.ldb[l] = (p.P.out[l] + 63) / 64 * 64;
    for (int q = 0; q <= p.s; ++q)
      for (int l = 0; l + 1 < p.P.L; ++l)
        if (p.P.relu[l]) p.mbits[q][l] = ly.take((size_t)(Ra / 8) * p.ldb[l]);
  }

  Top& T = p.T;
  T.spec = *t;
  T.H = t->n_layers - 1;
  int in = p.dA + p.dB;
  for (int j = 0; j < t->n_layers; ++j) {
    T.in[j] = in;
    T.out[j] = t->widths[j];
    T.relu[j] = j < T.H && ((t->relu_mask >> j) & 1u);
    T.kq[j] = ksteps(in);
    T.kt[j] = ksteps(T.out[j]);
    T.W[j] = ly.take(sizeof(float) * (size_t)T.out[j] * in);
    if (j < T.H) {
      if (j + 1 < T.H) T.arc[j] = ly.take(rc_bytes(T.out[j]));
      T.drc[j] = ly.take(rc_bytes(T.out[j]));
    }
    in = T.out[j];
  }
  // the top model's packed copies, contiguous
  for (int j = 0; j < T.H; ++j) T.Wq[j] = ly.take(packed_bytes(T.out[j], T.in[j]));
  for (int j = 0; j < T.H; ++j) T.Wtq[j] = ly.take(packed_bytes(T.in[j], T.out[j]));
  T.packed_end = ly.off;
  // bias tables (rows padded to 32 floats; the padding stays zero)
  auto pad32 = [](int n) { return (n + 31) / 32 * 32; };
  p.nbias_a = 0;
  for (int l = 0; l < p.A.L; ++l) { p.A.bo[l] = p.nbias_a; p.nbias_a += pad32(p.A.out[l]); }
  for (int j = 0; j < T.H; ++j) { T.bo[j] = p.nbias_a; p.nbias_a += pad32(T.out[j]); }
  p.bias_a = ly.take(sizeof(float) * (size_t)p.nbias_a);
  for (int l = 0; l < p.A.L; ++l) p.A.b[l] = p.bias_a + sizeof(float) * p.A.bo[l];
  for (int j = 0; j < T.H; ++j) T.b[j] = p.bias_a + sizeof(float) * T.bo[j];
  T.b[T.H] = ly.take(sizeof(float));  // the logit's bias
  p.nbias_b = 0;
  for (int l = 0; l < p.P.L; ++l) { p.P.bo[l] = p.nbias_b; p.nbias_b += pad32(p.P.out[l]); }
  p.bias_b = ly.take(sizeof(float) * (size_t)p.nbias_b);
  for (int l = 0; l < p.P.L; ++l) p.P.b[l] = p.bias_b + sizeof(float) * p.P.bo[l];
  p.cat_rc = ly.take(rc_bytes(p.dA + p.dB));

  // chain kernels: rows per block and LDS layouts
  if (!pick_rt(p.R, p.kf, [&](int BR) { FwdLds f; plan_fwd_lds(p, BR, f); return f.bytes; }))
    return "party B's widths exceed the LDS of one workgroup";
  if (!pick_rt(p.R, p.ka, [&](int BR) { ActLds x; plan_act_lds(p, BR, gextra, x); return x.bytes; }))
    return "party A's and the top model's widths exceed the LDS of one workgroup";
  if (!pick_rt(p.R, p.kb, [&](int BR) { BwdLds x; plan_bwd_lds(p, BR, x); return x.bytes; }))
    return "party B's widths exceed the LDS of one workgroup";
  {
    // B's backward starts every block with its loads (ReLU masks, gradient
    // message, stashed output): 32-row blocks when two of them fit one CU's
    // LDS and the larger pick would not, so that one block's loads overlap
    // the other's products.  Only where B's stream carries most of the
    // tick's work (its bottom has over twice the per-row MACs of A's bottom
    // and the top model): two backward blocks per CU leave no room beside
    // them for A's kernels, which would otherwise be the longer stream.
    auto macs = [](const Party& q) {
      double m = 0;
      for (int l = 0; l < q.L; ++l) m += (double)q.in[l] * q.out[l];
      return m;
    };
    double macs_a = macs(p.A);
    for (int j = 0; j < T.H; ++j) macs_a += (double)T.in[j] * T.out[j];
    BwdLds two, cur;
    plan_bwd_lds(p, 32, two);
    plan_bwd_lds(p, 16 * p.kb.rt, cur);
    if (p.kb.rt > 2 && 2 * two.bytes <= kLdsMax && 2 * cur.bytes > kLdsMax && macs(p.P) > 2 * macs_a) {
      p.kb.rt = 2;
      p.kb.blocks = (p.R + 31) / 32;
      p.kb.lds = two.bytes;
    }
  }
  {
    // deeper weight load groups for bf16 chains whose weights are large
    // (hetero's B, ten 256-wide layers): there they keep the L2 stream busy,
    // while small chains run faster with the shallower groups (the forward
    // of 64 -> 256 -> 128 at 16384 rows: 36 -> 26 us).  B's backward takes
    // the deeper groups only through more than three such layers: hetero's
    // three-layer backward runs faster with the shallow ones (42 -> 40 us),
    // the ten-layer one of 256-wide layers slower (tick 265 -> 278 us).
    auto welts = [](const Party& P) {
      size_t n = 0;
      for (int l = 0; l < P.L; ++l) n += (size_t)P.in[l] * P.out[l];
      return n;
    };
    size_t wa = welts(p.A);
    for (int j = 0; j < p.T.H; ++j) wa += (size_t)p.T.in[j] * p.T.out[j];
    if (p.e == BF16 && welts(p.P) >= kPFWideElts) p.kf.pf = kChainPFWide;
    if (p.e == BF16 && wa >= kPFWideElts) p.ka.pf = kChainPFWide;
    if (p.e == BF16 && welts(p.P) >= kPFWideElts && p.P.L > 3) p.kb.pf = kChainPFWide;
  }
  plan_fwd_lds(p, 16 * p.kf.rt, p.lf);
  plan_act_lds(p, 16 * p.ka.rt, gextra, p.la);
  plan_bwd_lds(p, 16 * p.kb.rt, p.lb);
  T.logit_part = ly.take(sizeof(float) * (size_t)p.ka.blocks * (T.out[T.H - 1] + 2));

  // messages and control
  for (int q = 0; q <= p.s; ++q) p.ring_g[q] = ly.take((size_t)es * R * ld_of(p.dB));
  p.hdr = ly.take(sizeof(int32_t) * (2 * kMaxSlots * 4 + 4));
  p.tsrc = ly.take(sizeof(TickSrc));

  // weight gradients: partials of the split problems
  auto parts = [&](DwMeta& m, int N, int K, size_t& pw, size_t& pb) {
    if (m.splits <= 1) return;
    const int kp = (K + 3) / 4 * 4;
    pw = ly.take(sizeof(float) * (size_t)m.splits * N * kp);
    pb = ly.take(sizeof(float) * (size_t)m.splits * N);
    m.red_blocks += (N + 7) / 8 * ((kp + kRedK - 1) / kRedK) + (N + 255) / 256;   // k_dw_reduce's tiles, biases
  };
  p.da.red_blocks = p.db.red_blocks = 0;
  for (int l = 0; l < p.A.L; ++l) parts(p.da, p.A.out[l], p.A.in[l], p.A.part[l], p.A.partb[l]);
  for (int j = 0; j < T.H; ++j) parts(p.da, T.out[j], T.in[j], T.part[j], T.partb[j]);
  for (int l = 0; l < p.P.L; ++l) parts(p.db, p.P.out[l], p.P.in[l], p.P.part[l], p.P.partb[l]);
  p.da.logit_blocks = (T.out[T.H - 1] + 2 + 3) / 4;

  // device job descriptors
  p.job_fwd = ly.take(sizeof(FwdJob) * (p.s + 1));
  p.job_act = ly.take(sizeof(ActiveJob) * (p.s + 1));
  p.job_bwd = ly.take(sizeof(BwdJob) * (p.s + 1));
  p.job_dwa = ly.take(sizeof(DwJob));
  p.job_dwb = ly.take(sizeof(DwJob) * (p.s + 1));
  if (p.bgemm) {
    p.job_lin = ly.take(sizeof(LinJob) * (p.s + 1));
    // row tiles up to the tick's rows only: the padded rows past them are
    // zero from the workspace's creation and no launch writes them, and a
    // 256-row tile more per XCD (Ra = 34048 at hetero) cost a third round
    // of blocks on the CUs
    p.lin_blocks_dx = lin_blocks(p.R, p.P.out[0]);
  }
  p.total = (ly.off + 255) / 256 * 256;
  return "";
}

int32_t* hdr_ptr(vfl_ctx* c, int which, int slot) { return at<int32_t>(c, c->p.hdr) + (which * kMaxSlots + slot) * 4; }
int32_t* err_ptr(vfl_ctx* c) { return at<int32_t>(c, c->p.hdr) + 2 * kMaxSlots * 4; }

ChainLayer layer(const void* W, int kst, int bl, int N, int K, bool relu, LBuf in, LBuf out) {
  ChainLayer L;
  L.W = W; L.kst = kst; L.bl = bl;
  L.N = N; L.K = K; L.relu = relu ? 1 : 0;
  L.in = in; L.out = out;
  return L;
}

MsgOp msg_op(const vfl_opts& o, bool clip, bool noise, uint32_t tag) {
  MsgOp m;
  m.clip = clip; m.noise = noise; m.C = o.clip_c;
  m.stdv = o.sigma * ((o.flags & (VFL_CLIP_EMB | VFL_CLIP_GRAD)) ? o.clip_c : 1.f);
  m.seed = o.seed; m.tag = tag;
  return m;
}

// Host check of what a chain kernel touches in LDS and in a weight operand:
// the input buffer holds K columns rounded up to the MFMA depth, the output
// and mask buffers N columns, all inside the block's LDS, and the packed
// operand has the K steps of the product; the RC copy holds
// rc_cols columns (N unless given).
// rc_cols / out_cols: the columns the RC copy / the LDS output hold when
// fewer than N (the concat product keeps only A's columns of both).
bool layer_fits(const Plan& p, const ChainLayer& L, int BR, int lds, bool lds_out, int rc_cols = -1,
                int out_cols = -1) {
  const int es = elt_size(p.e), KS = p.e == BF16 ? 32 : 16;
  auto inside = [&](const LBuf& b, int cols) {
    const int need = (cols + KS - 1) / KS * KS * es;
    return b.pitch >= need && b.off >= 0 && b.off + b.pitch * BR <= lds && b.off % 16 == 0 && b.pitch % 16 == 0;
  };
  if (!L.W || L.N < 1 || L.K < 1 || L.kst != (L.K + KS - 1) / KS) return false;
  if (L.bl >= 0 && (L.bl % 16 || L.bl + 4 * ((L.N + 31) / 32 * 32) > lds)) return false;
  if (!inside(L.in, L.K)) return false;
  if (lds_out && !inside(L.out, out_cols < 0 ? L.N : out_cols)) return false;
  if (L.mask.pitch && L.mask_bits) {
    // a byte per 8 rows and column, copied 16 columns at a time
    const int nb = (L.N + 15) / 16 * 16;
    if (BR % 8 || L.mask.off < 0 || L.mask.off % 16 || L.mask.pitch % 16 || L.mask.pitch < nb ||
        L.mask.off + L.mask.pitch * (BR / 8) > lds || !L.mask_src.bits || L.mask_src.ldb < nb ||
        L.mask_src.ldb % 16)
      return false;
  } else if (L.mask.pitch && !inside(L.mask, L.N)) {
    return false;
  }
  if (L.rc.p && L.rc.cp < ((rc_cols < 0 ? L.N : rc_cols) + 7) / 8 * 8) return false;
  return true;
}

struct Jobs {
  std::vector<FwdJob> fj;
  std::vector<ActiveJob> aj;
  std::vector<BwdJob> bj;
  std::vector<DwJob> dwb;
  DwJob dwa;
  std::vector<LinJob> lin;            // party B's layer-1 input gradient per slot (bgemm)
};

// The job descriptors of every slot for a workspace at `ws` (host only;
// empty string when every layer's layout checks out).
std::string build_jobs(const Plan& p, const vfl_opts& o, char* ws, Jobs& J) {
  struct Base { char* ws; } cb{ws};
  const Base* c = &cb;
  const Party& A = p.A;
  const Party& P = p.P;
  const Top& T = p.T;
  const int S1 = p.s + 1;
  const bool eextra = o.flags & (VFL_CLIP_EMB | VFL_NOISE_EMB);
  const bool gextra = o.flags & (VFL_CLIP_GRAD | VFL_NOISE_GRAD);
  J.fj.assign(S1, FwdJob());
  J.aj.assign(S1, ActiveJob());
  J.bj.assign(S1, BwdJob());
  J.dwb.assign(S1, DwJob());
  J.dwa = DwJob();
  J.lin.assign(p.bgemm ? S1 : 0, LinJob());
  std::vector<FwdJob>& fj = J.fj;
  std::vector<ActiveJob>& aj = J.aj;
  std::vector<BwdJob>& bj = J.bj;
  std::vector<DwJob>& dwb = J.dwb;
  DwJob& dwa = J.dwa;
  auto at_f = [&](size_t off) { return (float*)(ws + off); };
  auto hdrp = [&](int which, int slot) { return (int32_t*)(ws + p.hdr) + (which * kMaxSlots + slot) * 4; };
  auto rcm = [&](const Base*, size_t off, int cols) {
    RCMat m;
    m.p = ws + off;
    m.cp = (int32_t)ld_of(cols);
    m.rows = p.Ra;
    // a copy larger than the L2s is written with the streaming hint: its
    // reader (the weight gradient, several launches later) finds it in HBM
    // either way
    m.nt = (double)p.Ra * m.cp * (p.e == BF16 ? 2 : 4) > kRcStreamBytes;
    return m;
  };
  for (int q = 0; q < S1; ++q) {
    // party B forward + publish
    FwdJob& f = fj[q];
    f.in.dense_in = P.spec.dense_in; f.in.n_cat = P.spec.n_cat; f.in.V = P.spec.vocab; f.in.E = P.spec.emb_dim;
    f.in.dense_vec = P.spec.n_cat == 0;
    f.in.T = P.spec.n_cat ? at_f(P.T) : nullptr;
    f.in.idt = P.spec.n_cat ? (int32_t*)(ws + P.idt[q]) : nullptr; f.in.ldi = p.R;
    f.in.bad_ids = (int32_t*)(ws + p.hdr) + 2 * kMaxSlots * 4 + 1;
    f.in.buf = p.lf.buf[0];
    f.in.rc = rcm(c, P.x0rc[q], P.din);
    f.bt.src = at_f(p.bias_b); f.bt.off = p.lf.bias.off; f.bt.n4 = p.nbias_b / 4;
    f.warm.p[0] = c->ws + P.Wq[q][0];
    f.warm.lines[0] = (int32_t)((P.wq_end[q] - P.Wq[q][0]) / 128);
    f.L = P.L;
    for (int l = 0; l < P.L; ++l) {
      f.l[l] = layer(c->ws + P.Wq[q][l], P.kq[l], p.lf.bias.off + 4 * P.bo[l], P.out[l], P.in[l], P.relu[l],
                     p.lf.buf[l % 2], p.lf.buf[(l + 1) % 2]);
      if (l + 1 < P.L) f.l[l].rc = rcm(c, P.arc[q][l], P.out[l]);
    }
    for (int l = 0; l + 1 < P.L; ++l)
      if (p.mbits[q][l]) {
        f.l[l].rc.bits = (uint8_t*)(ws + p.mbits[q][l]);
        f.l[l].rc.ldb = p.ldb[l];
      }
    f.z = c->ws + P.z[q]; f.ldz = (int32_t)ld_of(p.dB);
    f.publish = eextra;
    f.m = msg_op(o, o.flags & VFL_CLIP_EMB, o.flags & VFL_NOISE_EMB, 0);
    f.zhat = c->ws + P.zhat[q]; f.ldzh = (int32_t)ld_of(p.dB);
    f.norm = P.norm[q] ? at_f(P.norm[q]) : nullptr;
    f.cfac = P.cfac[q] ? at_f(P.cfac[q]) : nullptr;
    f.hdr_out = hdrp(0, q);

    // party A's step against embedding slot q
    ActiveJob& a = aj[q];
    const ActLds& la = p.la;
    a.in.dense_in = A.spec.dense_in; a.in.n_cat = A.spec.n_cat; a.in.V = A.spec.vocab; a.in.E = A.spec.emb_dim;
    a.in.dense_vec = A.spec.n_cat == 0;
    a.in.T = A.spec.n_cat ? at_f(A.T) : nullptr;
    a.in.idt = A.spec.n_cat ? (int32_t*)(ws + A.idt[0]) : nullptr; a.in.ldi = p.R;
    a.in.bad_ids = (int32_t*)(ws + p.hdr) + 2 * kMaxSlots * 4 + 1;
    a.in.buf = la.in;
    a.in.rc = rcm(c, A.x0rc[0], A.din);
    a.bt.src = at_f(p.bias_a); a.bt.off = la.bias.off; a.bt.n4 = p.nbias_a / 4;
    a.warm.p[0] = c->ws + A.Wq[0][0];
    a.warm.lines[0] = (int32_t)((A.wtq_end[0] - A.Wq[0][0]) / 128);
    a.warm.p[1] = c->ws + T.Wq[0];
    a.warm.lines[1] = (int32_t)((T.packed_end - T.Wq[0]) / 128);
    a.LA = A.L;
    for (int l = 0; l < A.L; ++l) {
      const LBuf src = l == 0 ? la.in : la.fa[l - 1];
      const LBuf dst = l + 1 < A.L ? la.fa[l] : la.cat;
      a.fa[l] = layer(c->ws + A.Wq[0][l], A.kq[l], la.bias.off + 4 * A.bo[l], A.out[l], A.in[l], A.relu[l],
                      src, dst);
      if (l + 1 < A.L) a.fa[l].rc = rcm(c, A.arc[0][l], A.out[l]);
      else a.fa[l].nopad = 1;   // B's embedding is already in cat past dA
    }
    a.cat = la.cat; a.cat_rc = rcm(c, p.cat_rc, p.dA + p.dB); a.dA = p.dA; a.dB = p.dB;
    a.zb = c->ws + P.zhat[q]; a.ldzb = (int32_t)ld_of(p.dB);
    a.hdr_chk = hdrp(0, q); a.err = (int32_t*)(ws + p.hdr) + 2 * kMaxSlots * 4;
    a.H = T.H;
    for (int j = 0; j < T.H; ++j) {
      a.ft[j] = layer(c->ws + T.Wq[j], T.kq[j], la.bias.off + 4 * T.bo[j], T.out[j], T.in[j], T.relu[j],
                      j == 0 ? la.cat : la.ft[j - 1], la.ft[j]);
      if (j + 1 < T.H) a.ft[j].rc = rcm(c, T.arc[j], T.out[j]);
    }
    a.lw = at_f(T.W[T.H]); a.lb = at_f(T.b[T.H]); a.relu_h = T.relu[T.H - 1];
    a.mse = (o.flags & VFL_LOSS_MSE) != 0;
    a.dh = la.P[0]; a.dh_rc = rcm(c, T.drc[T.H - 1], T.out[T.H - 1]);
    a.part = at_f(T.logit_part);
    a.red = la.red;
    for (int qq = 0; qq + 1 < T.H; ++qq) {
      const int j = T.H - 1 - qq;           // delta of top layer j -> layer j-1
      ChainLayer& L = a.dt[qq];
      L = layer(c->ws + T.Wtq[j], T.kt[j], -1, T.in[j], T.out[j], false, la.P[qq % 2], la.P[(qq + 1) % 2]);
      if (T.relu[j - 1]) L.mask = la.ft[j - 1];
      L.rc = rcm(c, T.drc[j - 1], T.out[j - 1]);
    }
    {
      const int h = T.H - 1;
      ChainLayer& L = a.dc;
      L = layer(c->ws + T.Wtq[0], T.kt[0], -1, p.dA + p.dB, T.out[0], false, la.P[h % 2], la.P[(h + 1) % 2]);
      if (A.relu[A.L - 1]) L.mask = la.cat;
      L.rc = rcm(c, A.drc[A.L - 1], p.dA);
    }
    a.gextra = gextra;
    a.m = msg_op(o, o.flags & VFL_CLIP_GRAD, o.flags & VFL_NOISE_GRAD, 1);
    a.msg = la.msg;
    a.ring = c->ws + p.ring_g[q]; a.ldring = (int32_t)ld_of(p.dB);
    a.hdr_out = hdrp(1, q);
    a.nda = A.L - 1;
    for (int qq = 0; qq + 1 < A.L; ++qq) {
      const int l = A.L - 1 - qq;           // delta of A's layer l -> layer l-1
      const int h = T.H + qq;
      ChainLayer& L = a.da[qq];
      L = layer(c->ws + A.Wtq[0][l], A.kt[l], -1, A.in[l], A.out[l], false, la.P[h % 2], la.P[(h + 1) % 2]);
      if (A.relu[l - 1]) L.mask = la.fa[l - 1];
      L.rc = rcm(c, A.drc[l - 1], A.out[l - 1]);
    }
    a.has_gx = A.spec.n_cat > 0;
    if (a.has_gx) {
      const int h = T.H + A.L - 1;
      a.gx = layer(c->ws + A.Wtq[0][0], A.kt[0], -1, A.spec.n_cat * A.spec.emb_dim, A.out[0], false,
                   la.P[h % 2], LBuf());
      a.gxp = at_f(A.gx); a.ldgx = (int32_t)A.ldgx;
    }

    // party B's backward of the group stashed in slot q
    BwdJob& b = bj[q];
    const BwdLds& lb = p.lb;
    b.g = c->ws + p.ring_g[q]; b.ldg = (int32_t)ld_of(p.dB);
    b.z = c->ws + P.z[q]; b.ldz = (int32_t)ld_of(p.dB);
    b.clip = (o.flags & VFL_CLIP_EMB) != 0;
    b.norm = b.clip ? at_f(P.norm[q]) : nullptr;
    b.cfac = b.clip ? at_f(P.cfac[q]) : nullptr;
    b.C = o.clip_c; b.relu = P.relu[P.L - 1]; b.D = p.dB;
    b.d = lb.P[0]; b.d_rc = rcm(c, P.drc[P.L - 1], p.dB);
    b.hdr_chk = hdrp(1, q); b.err = (int32_t*)(ws + p.hdr) + 2 * kMaxSlots * 4;
    b.warm.p[0] = c->ws + P.Wtq[q][0];
    b.warm.lines[0] = (int32_t)((P.wtq_end[q] - P.Wtq[q][0]) / 128);
    b.nd = P.L - 1 - (p.bgemm ? 1 : 0);
    for (int qq = 0; qq < b.nd; ++qq) {
      const int l = P.L - 1 - qq;
      ChainLayer& L = b.dx[qq];
      L = layer(c->ws + P.Wtq[q][l], P.kt[l], -1, P.in[l], P.out[l], false, lb.P[qq % 2], lb.P[(qq + 1) % 2]);
      if (P.relu[l - 1]) {
        L.mask = lb.mask[l - 1];
        L.mask_src = rcm(c, P.arc[q][l - 1], P.out[l - 1]);
        if (p.mbits[q][l - 1]) {
          L.mask_src.bits = (uint8_t*)(ws + p.mbits[q][l - 1]);
          L.mask_src.ldb = p.ldb[l - 1];
          L.mask_bits = 1;
        }
        // bf16 backward kernels read masks only in the byte form
        if ((p.e == BF16) != (L.mask_bits != 0)) return "party B's backward: bf16 masks without ReLU bits";
      }
      L.rc = rcm(c, P.drc[l - 1], P.out[l - 1]);
    }
    b.has_gx = P.spec.n_cat > 0;
    if (b.has_gx) {
      b.gx = layer(c->ws + P.Wtq[q][0], P.kt[0], -1, P.spec.n_cat * P.spec.emb_dim, P.out[0], false,
                   lb.P[(P.L - 1) % 2], LBuf());
      b.gxp = at_f(P.gx); b.ldgx = (int32_t)P.ldgx;
    }
    if (p.bgemm) {
      // layer 1's input gradient over the group: the chain's last delta
      // (row-major) times the stashed W1, masked by the stashed layer-0 output
      b.drm = ws + p.d1rm; b.lddrm = (int32_t)ld_of(P.out[1]);
      LinJob& g = J.lin[q];
      g.A = ws + p.d1rm; g.lda = ld_of(P.out[1]);
      g.W = c->ws + P.Wtq[q][1]; g.kst = P.kt[1];
      g.N = P.out[0]; g.K = P.out[1];
      if (P.relu[0]) { g.mbits = (const uint8_t*)(ws + p.mbits[q][0]); g.ldb = p.ldb[0]; }
      g.out_rc = rcm(c, P.drc[0], P.out[0]);
      g.tiles_n = (g.N + 255) / 256; g.tiles_m = (p.R + 255) / 256;
      g.rows_pad = p.Ra;
    }
  }

  // weight gradients
  auto add = [&](DwJob& J, const DwMeta& m, size_t D, size_t X, int N, int K, size_t W, size_t bias,
                 size_t Wq, int kq, size_t Wtq, int kt, size_t part, size_t partb) {
    DwProb& d = J.p[J.n++];
    d.D = rcm(c, D, N);
    d.X = rcm(c, X, K);
    d.W = at_f(W); d.bias = at_f(bias);
    d.Wq = c->ws + Wq; d.Wtq = c->ws + Wtq; d.kq = kq; d.kt = kt;
    d.part = part ? at_f(part) : nullptr;
    d.partb = partb ? at_f(partb) : nullptr;
    d.N = N; d.K = K; d.kp = (K + 3) / 4 * 4;
    d.splits = m.splits; d.rps = m.rps;
    d.first_block = J.blocks;
    J.blocks += dw_tiles(N, K, m.tile) * m.splits;
  };
  for (int j = 0; j < T.H; ++j)
    add(dwa, p.da, T.drc[j], j == 0 ? p.cat_rc : T.arc[j - 1], T.out[j], T.in[j], T.W[j], T.b[j], T.Wq[j],
        T.kq[j], T.Wtq[j], T.kt[j], T.part[j], T.partb[j]);
  for (int l = 0; l < A.L; ++l)
    add(dwa, p.da, A.drc[l], l == 0 ? A.x0rc[0] : A.arc[0][l - 1], A.out[l], A.in[l], A.W[l], A.b[l],
        A.Wq[0][l], A.kq[l], A.Wtq[0][l], A.kt[l], A.part[l], A.partb[l]);
  dwa.rows_pad = p.Ra;
  dwa.red_blocks = p.da.red_blocks;
  dwa.lpart = at_f(T.logit_part);
  dwa.Hd = T.out[T.H - 1];
  dwa.lrows = 16 * p.ka.rt;
  dwa.lw = at_f(T.W[T.H]);
  dwa.lb = at_f(T.b[T.H]);
  for (int q = 0; q < S1; ++q) {
    DwJob& J = dwb[q];
    for (int l = 0; l < P.L; ++l)
      add(J, p.db, P.drc[l], l == 0 ? P.x0rc[q] : P.arc[q][l - 1], P.out[l], P.in[l], P.W[l], P.b[l],
          P.Wq[q][l], P.kq[l], P.Wtq[q][l], P.kt[l], P.part[l], P.partb[l]);
    J.rows_pad = p.Ra;
    J.red_blocks = p.db.red_blocks;
  }
  if (dwa.blocks != p.da.blocks || dwb[0].blocks != p.db.blocks)
    return "internal: weight-gradient block count mismatch";
  for (int q = 0; q < S1; ++q) {
    bool ok = true;
    const int bf = 16 * p.kf.rt, ba = 16 * p.ka.rt, bb = 16 * p.kb.rt;
    for (int l = 0; l < fj[q].L; ++l) ok = ok && layer_fits(p, fj[q].l[l], bf, p.kf.lds, true);
    for (int l = 0; l < aj[q].LA; ++l) ok = ok && layer_fits(p, aj[q].fa[l], ba, p.ka.lds, true);
    for (int j = 0; j < aj[q].H; ++j) ok = ok && layer_fits(p, aj[q].ft[j], ba, p.ka.lds, true);
    for (int j = 0; j + 1 < aj[q].H; ++j) ok = ok && layer_fits(p, aj[q].dt[j], ba, p.ka.lds, true);
    ok = ok && layer_fits(p, aj[q].dc, ba, p.ka.lds, true, p.dA, p.dA);   // A's columns only
    for (int l = 0; l < aj[q].nda; ++l) ok = ok && layer_fits(p, aj[q].da[l], ba, p.ka.lds, true);
    if (aj[q].has_gx) ok = ok && layer_fits(p, aj[q].gx, ba, p.ka.lds, false);
    for (int l = 0; l < bj[q].nd; ++l) ok = ok && layer_fits(p, bj[q].dx[l], bb, p.kb.lds, true);
    if (bj[q].has_gx) ok = ok && layer_fits(p, bj[q].gx, bb, p.kb.lds, false);
    ok = ok && p.la.red.off + 4 * (ba + kChainWaves * ((p.T.out[p.T.H - 1] + 3) / 4 * 4) + 2 * kChainWaves) <=
                   p.ka.lds;
    if (!ok) return "internal: chain layout does not cover a layer";
  }
  return "";
}

// Write the job descriptors into the workspace (once, at creation).
vfl_status write_jobs(vfl_ctx* c) {
  const Plan& p = c->p;
  const int S1 = p.s + 1;
  Jobs J;
  const std::string why = build_jobs(p, c->o, c->ws, J);
  if (!why.empty()) return fail(c, VFL_E_INVALID, why);
  const std::vector<FwdJob>& fj = J.fj;
  const std::vector<ActiveJob>& aj = J.aj;
  const std::vector<BwdJob>& bj = J.bj;
  const std::vector<DwJob>& dwb = J.dwb;
  const DwJob& dwa = J.dwa;

  HIPCHK(hipMemcpy(c->ws + p.job_fwd, fj.data(), sizeof(FwdJob) * S1, hipMemcpyHostToDevice));
  HIPCHK(hipMemcpy(c->ws + p.job_act, aj.data(), sizeof(ActiveJob) * S1, hipMemcpyHostToDevice));
  HIPCHK(hipMemcpy(c->ws + p.job_bwd, bj.data(), sizeof(BwdJob) * S1, hipMemcpyHostToDevice));
  HIPCHK(hipMemcpy(c->ws + p.job_dwa, &dwa, sizeof(DwJob), hipMemcpyHostToDevice));
  HIPCHK(hipMemcpy(c->ws + p.job_dwb, dwb.data(), sizeof(DwJob) * S1, hipMemcpyHostToDevice));
  if (p.bgemm) HIPCHK(hipMemcpy(c->ws + p.job_lin, J.lin.data(), sizeof(LinJob) * J.lin.size(), hipMemcpyHostToDevice));
  return VFL_OK;
}

// Validate k back-to-back replica batches; fills the slot description.
vfl_status take_batches(vfl_ctx* c, const Party& P, const vfl_batch* br, int n, bool need_labels,
                        SlotState& st) {
  const Plan& p = c->p;
  if (!br || n < 1 || n > p.k) return fail(c, VFL_E_INVALID, "need 1..k replica batches");
  const int es = elt_size(p.e);
  const int64_t ld = br[0].ld ? br[0].ld : P.spec.dense_in;
  if (P.spec.dense_in) {
    if (!br[0].dense) return fail(c, VFL_E_INVALID, "dense input missing");
    if (ld < P.spec.dense_in || (!P.spec.n_cat && ((ld * es) % 16 || ((uintptr_t)br[0].dense) % 16)))
      return fail(c, VFL_E_INVALID, "dense rows must be 16-byte aligned (ld * element size % 16 == 0)");
  }
  if (P.spec.n_cat && !br[0].ids) return fail(c, VFL_E_INVALID, "ids missing");
  if (need_labels && !br[0].labels) return fail(c, VFL_E_INVALID, "labels missing");
  int64_t off = 0;
  for (int r = 0; r < n; ++r) {
    const vfl_batch& x = br[r];
    if (x.rows < 1 || x.rows > p.B || (r + 1 < n && x.rows != p.B))
      return fail(c, VFL_E_INVALID, "each replica holds `batch` rows (the last may hold fewer)");
    if ((x.ld ? x.ld : P.spec.dense_in) != ld) return fail(c, VFL_E_INVALID, "replicas differ in ld");
    if (r > 0) {
      bool ok = x.row0 == br[0].row0 + off;
      if (P.spec.dense_in) ok = ok && (const char*)x.dense == (const char*)br[0].dense + off * ld * es;
      if (P.spec.n_cat) ok = ok && x.ids == br[0].ids + off * P.spec.n_cat;
      if (need_labels) ok = ok && x.labels == br[0].labels + off;
      if (!ok) return fail(c, VFL_E_INVALID, "replica batches must lie back to back");
    }
    off += x.rows;
  }
  st.rows = (int)off;
  st.row0 = br[0].row0;
  st.dense = br[0].dense;
  st.ld = ld;
  st.ids = br[0].ids;
  st.labels = br[0].labels;
  return VFL_OK;
}

// ------------------------------------------------------------- timing hook
void harvest(vfl_ctx* c, int i) {
  Timing& T = c->tm;
  if (!T.used[i]) return;
  float ms = 0.f;
  if (hipEventSynchronize(T.ev1[i]) == hipSuccess && hipEventElapsedTime(&ms, T.ev0[i], T.ev1[i]) == hipSuccess) {
    T.ms[T.cls[i]] += ms;
    T.wk[T.cls[i]] += T.work[i];
    T.n[T.cls[i]] += 1;
  }
  T.used[i] = false;
}

// An event-record node appended to the stream's captured work: it depends on
// the stream's current capture dependencies and becomes the only one, so the
// next captured launch on the stream starts after it.
bool capture_record(vfl_ctx* c, hipEvent_t ev, hipStream_t st, int cls, int end) {
  hipStreamCaptureStatus cs;
  unsigned long long id = 0;
  hipGraph_t g = nullptr;
  const hipGraphNode_t* deps = nullptr;
  size_t nd = 0;
  hipGraphNode_t node;
  const char* what = "hipStreamGetCaptureInfo_v2";
  hipError_t he = hipStreamGetCaptureInfo_v2(st, &cs, &id, &g, &deps, &nd);
  if (he == hipSuccess) { what = "hipGraphAddEventRecordNode"; he = hipGraphAddEventRecordNode(&node, g, deps, nd, ev); }
  if (he == hipSuccess) {
    what = "hipStreamUpdateCaptureDependencies";
    he = hipStreamUpdateCaptureDependencies(st, &node, 1, hipStreamSetCaptureDependencies);
  }
  if (he == hipSuccess) return true;
  (void)hipGetLastError();   // do not leave it to the next launch's check
  if (c->tm_err == hipSuccess) {
    c->tm_err = he;
    c->tm_err_what = std::string(what) + (end ? " (end" : " (begin") + ", class " + std::to_string(cls) +
                     ", stream " + (st == c->sa ? "A" : st == c->sb ? "B" : "?") + ", deps " +
                     std::to_string(nd) + ", pair " + std::to_string(c->gused[c->capture_phase]) + ")";
  }
  return false;
}

int tbegin(vfl_ctx* c, int cls, double work, hipStream_t st) {
  Timing& T = c->tm;
  if (!((T.mask >> cls) & 1u)) return -1;
  if (c->capture_phase >= 0) {
    // inside a captured graph: an event pair of its own (created before the
    // capture), recorded as graph nodes, read after the graph's last replay;
    // only every kTimedEvery-th tick of the cycle is timed (each pair adds
    // two nodes that the host launches with every replay)
    if (c->capture_tick % kTimedEvery != 0) return -1;
    const int ph = c->capture_phase;
    if (c->gused[ph] >= (int)c->gpairs[ph].size()) return -1;
    vfl_ctx::GPair& gp = c->gpairs[ph][c->gused[ph]];
    gp.cls = cls;
    gp.work = work;
    if (!capture_record(c, gp.e0, st, cls, 0)) return -1;
    return c->gused[ph]++ + (1 << 20);
  }
  const int i = T.next;
  T.next = (T.next + 1) % Timing::kPool;
  harvest(c, i);
  T.cls[i] = cls;
  T.work[i] = work;
  if (hipEventRecord(T.ev0[i], st) != hipSuccess) return -1;
  return i;
}

void tend(vfl_ctx* c, int i, hipStream_t st) {
  if (i < 0) return;
  if (i >= (1 << 20)) {
    (void)capture_record(c, c->gpairs[c->capture_phase][i - (1 << 20)].e1, st, -1, 1);
    return;
  }
  if (hipEventRecord(c->tm.ev1[i], st) == hipSuccess) c->tm.used[i] = true;
}

#define TIMED(cls, work, st, call)                      \
  do {                                                  \
    const int ts_ = tbegin(c, (cls), (work), (st));     \
    HIPCHK(call);                                       \
    tend(c, ts_, (st));                                 \
  } while (0)

double mm_flops(int R, int N, int K) { return 2.0 * R * (double)N * K; }

// ------------------------------------------------------------ enqueue steps
// Every enqueue function below takes a tick reference `tr`: null (src) when
// the call's values are known on the host (the per-call API), the tick of a
// captured launch when the work is captured into a replayed graph.
vfl_status enqueue_cast(vfl_ctx* c, const Party& P, int slot, const Top* T, hipStream_t st) {
  CastJob jobs[2 * VFL_MAX_LAYERS + 2];
  int n = 0;
  for (int l = 0; l < P.L; ++l)
    jobs[n++] = CastJob{at<float>(c, P.W[l]), c->ws + P.Wq[slot][l], c->ws + P.Wtq[slot][l],
                        P.out[l], P.in[l], P.kq[l], P.kt[l]};
  if (T)
    for (int j = 0; j < T->H; ++j)
      jobs[n++] = CastJob{at<float>(c, T->W[j]), c->ws + T->Wq[j], c->ws + T->Wtq[j],
                          T->out[j], T->in[j], T->kq[j], T->kt[j]};
  double bytes = 0;
  for (int i = 0; i < n; ++i) bytes += (double)jobs[i].out * jobs[i].in * (4 + 2 * elt_size(c->p.e));
  TIMED(VFL_K_CAST, bytes, st, launch_cast(c->p.e, jobs, n, st));
  return VFL_OK;
}

ChainCall call_of(const SlotState& st, int64_t group, const int32_t hdr[3], int64_t chk) {
  ChainCall k;
  k.dense = st.dense; k.ld = st.ld; k.ids = st.ids; k.labels = st.labels;
  k.row0 = st.row0; k.rows = st.rows; k.group = (int32_t)group;
  if (hdr) { k.hdr[0] = hdr[0]; k.hdr[1] = hdr[1]; k.hdr[2] = hdr[2]; }
  k.chk = (int32_t)chk;
  return k;
}

double party_fwd_flops(const Party& P, int R) {
  double f = 0;
  for (int l = 0; l < P.L; ++l) f += mm_flops(R, P.out[l], P.in[l]);
  return f;
}

double party_dx_flops(const Party& P, int R) {
  double f = 0;
  for (int l = 1; l < P.L; ++l) f += mm_flops(R, P.in[l], P.out[l]);
  if (P.spec.n_cat) f += mm_flops(R, P.spec.n_cat * P.spec.emb_dim, P.out[0]);
  return f;
}

// sparse SGD of a party's tables from its float32 input gradient gx
vfl_status enqueue_table_sgd(vfl_ctx* c, const Party& P, int slot, int R, float scale, hipStream_t st,
                             TickRef tr) {
  if (!P.spec.n_cat) return VFL_OK;
  ScatterJob sj{at<float>(c, P.T), at<int32_t>(c, P.idt[slot]), c->p.R, P.spec.n_cat, P.spec.vocab,
                P.spec.emb_dim, at<float>(c, P.gx), P.ldgx, R, scale, tr};
  TIMED(VFL_K_EMB_SGD, (double)R * P.spec.n_cat * 4.0 * (1 + P.spec.emb_dim), st,
        launch_scatter_sgd(sj, st));
  return VFL_OK;
}

// one party's weight gradients + SGD (+ the logit layer and loss for A)
vfl_status enqueue_dw(vfl_ctx* c, bool party_a, int slot, int R, float* loss, TickRef tr,
                      hipStream_t st) {
  const Plan& p = c->p;
  const DwMeta& m = party_a ? p.da : p.db;
  const DwJob* job = party_a ? (const DwJob*)(c->ws + p.job_dwa) : (const DwJob*)(c->ws + p.job_dwb) + slot;
  const float scale = c->o.lr / (float)R;
  double flops = 0;
  if (party_a) {
    for (int j = 0; j < p.T.H; ++j) flops += mm_flops(R, p.T.out[j], p.T.in[j]);
    flops += party_fwd_flops(p.A, R);
  } else {
    flops += party_fwd_flops(p.P, R);
  }
  if (m.tile == 32) {
    // one launch: products, SGD, copy refresh and (A) the logit reduction
    TIMED(VFL_K_DW, flops, st,
          launch_dw32(p.e, job, m.blocks + (party_a ? m.logit_blocks : 0), R, scale, tr.src ? nullptr : loss, tr,
                      tr.src ? loss : nullptr, st));
    return VFL_OK;
  }
  if (m.tile == 256) TIMED(VFL_K_DWT, flops, st, launch_dwt(job, m.blocks, st));
  else TIMED(VFL_K_DW, flops, st, launch_dw(p.e, job, m.blocks, R, scale, tr, st));
  const int blocks = m.red_blocks + (party_a ? m.logit_blocks : 0);
  if (blocks > 0) {
    double bytes = 0;
    const Party& P = party_a ? p.A : p.P;
    auto add = [&](int N, int K) { bytes += 4.0 * ((double)N * K + N) * (m.splits + 2); };
    if (m.splits > 1) {
      for (int l = 0; l < P.L; ++l) add(P.out[l], P.in[l]);
      if (party_a)
        for (int j = 0; j < p.T.H; ++j) add(p.T.out[j], p.T.in[j]);
    }
    if (party_a) bytes += 4.0 * p.ka.blocks * (p.T.out[p.T.H - 1] + 2);
    TIMED(VFL_K_REDUCE, bytes, st,
          launch_dw_reduce(p.e, job, blocks, R, scale, tr.src ? nullptr : loss, tr, tr.src ? loss : nullptr, st));
  }
  return VFL_OK;
}

// ---- the phases of a tick (enqueue only; the callers keep the host state)

// B's forward + publish of `st` (group st.group) into `slot`.
vfl_status b_forward(vfl_ctx* c, int slot, const SlotState& st, TickRef tr) {
  const Plan& p = c->p;
  const int32_t hdr[3] = {(int32_t)st.group, (int32_t)st.group, (int32_t)st.version};
  const ChainCall k = call_of(st, st.group, hdr, 0);
  TIMED(VFL_K_FWD, party_fwd_flops(p.P, p.R), c->sb,
        launch_fwd(p.e, p.kf.rt, p.kf.pf, (const FwdJob*)(c->ws + p.job_fwd) + slot, p.kf.lds, p.kf.blocks, k,
                   tr, c->sb));
  return VFL_OK;
}

vfl_status b_publish(vfl_ctx* c, int slot) {
  HIPCHK(hipEventRecord(c->ev_emb[slot], c->sb));
  return VFL_OK;
}

// A's forward, top model, loss and input-gradient chains of group `group`
// (A's batch in `st`) against embedding slot `slot`; gradient message +
// event.
vfl_status a_top(vfl_ctx* c, int64_t group, int slot, const SlotState& st, int32_t b_version,
                 TickRef tr, bool wait_emb = true) {
  const Plan& p = c->p;
  if (wait_emb) HIPCHK(hipStreamWaitEvent(c->sa, c->ev_emb[slot], 0));
  const int32_t hdr[3] = {(int32_t)group, (int32_t)(group + p.s), b_version};
  const ChainCall k = call_of(st, group, hdr, group);
  const int R = p.R;
  double f = party_fwd_flops(p.A, R) + party_dx_flops(p.A, R) + mm_flops(R, p.dA + p.dB, p.T.out[0]);
  for (int j = 0; j < p.T.H; ++j) f += mm_flops(R, p.T.out[j], p.T.in[j]);
  for (int j = 1; j < p.T.H; ++j) f += mm_flops(R, p.T.in[j], p.T.out[j]);
  TIMED(VFL_K_ACTIVE, f, c->sa,
        launch_active(p.e, p.ka.rt, p.ka.pf, (const ActiveJob*)(c->ws + p.job_act) + slot, p.ka.lds, p.ka.blocks, k,
                      tr, c->sa));
  HIPCHK(hipEventRecord(c->ev_grad[slot], c->sa));
  return VFL_OK;
}

// A's and the top model's SGD for A's group (rows R).
vfl_status a_backward(vfl_ctx* c, const SlotState& st, float* loss, TickRef tr) {
  const Plan& p = c->p;
  vfl_status r = enqueue_dw(c, true, 0, st.rows, loss, tr, c->sa);
  if (r) return r;
  return enqueue_table_sgd(c, p.A, 0, st.rows, c->o.lr / (float)st.rows, c->sa, tr);
}

// B's delayed backward of the group stashed in `slot` + SGD on B's current
// weights; the refreshed operand copies go to this slot, which B's next
// forward uses.
vfl_status b_backward(vfl_ctx* c, int slot, const SlotState& st, int64_t group, TickRef tr) {
  const Plan& p = c->p;
  HIPCHK(hipStreamWaitEvent(c->sb, c->ev_grad[slot], 0));
  const ChainCall k = call_of(st, group, nullptr, group);
  const double gf = p.bgemm ? mm_flops(p.R, p.P.out[0], p.P.out[1]) : 0.0;
  TIMED(VFL_K_BWD, party_dx_flops(p.P, p.R) - gf, c->sb,
        launch_bwd(p.e, p.kb.rt, p.kb.pf, (const BwdJob*)(c->ws + p.job_bwd) + slot, p.kb.lds, p.kb.blocks, k, tr, c->sb));
  if (p.bgemm)
    TIMED(VFL_K_GEMM, gf, c->sb,
          launch_lin((const LinJob*)(c->ws + p.job_lin) + slot, p.lin_blocks_dx, st.rows, tr, c->sb));
  vfl_status r = enqueue_dw(c, false, slot, st.rows, nullptr, tr, c->sb);
  if (r) return r;
  return enqueue_table_sgd(c, p.P, slot, st.rows, c->o.lr / (float)st.rows, c->sb, tr);
}

// Discard of group g (A will not, or no longer, use it): noted until B's
// backward of g releases the slot.
void note_drop(vfl_ctx* c, int64_t g, bool grad) { c->drops.push_back(vfl_ctx::Drop{g, grad}); }

// B's backward of a discarded group: the slot is released, nothing is
// updated (B's version stays); returns false when g was not discarded.
bool release_drop(vfl_ctx* c, int64_t g, vfl_status& r) {
  for (size_t i = 0; i < c->drops.size(); ++i) {
    if (c->drops[i].group != g) continue;
    const bool grad = c->drops[i].grad;
    c->drops.erase(c->drops.begin() + (long)i);
    r = VFL_OK;
    if (grad) {
      // A read the embedding slot: B's next forward into it follows A's
      // gradient event, as after an ordinary backward
      const hipError_t e = hipStreamWaitEvent(c->sb, c->ev_grad[g % (c->p.s + 1)], 0);
      if (e != hipSuccess) r = fail(c, VFL_E_HIP, std::string("hipStreamWaitEvent: ") + hipGetErrorString(e));
    }
    c->b_next_bwd = g + 1;
    return true;
  }
  return false;
}

bool dropped(const vfl_ctx* c, int64_t g) {
  for (const auto& d : c->drops)
    if (d.group == g) return true;
  return false;
}

// ---- checkpoint / resume: host channel state + the whole workspace

// Fixed header of a state image, followed by the workspace bytes and the
// schedule trace (int64).  Slot inputs are not kept: a slot's batch
// pointers are read only by the forward that filled it.
struct StateHead {
  char magic[8];
  uint32_t format, n_slots;
  uint64_t layout, ws_bytes, trace_len;
  int64_t b_next_fwd, b_next_bwd, b_version, b_pub_next, a_next, a_version, a_copy_version;
  int64_t a_rows_avg, b_rows_avg;
  int64_t b_copy_version[kMaxSlots], grad_group[kMaxSlots], grad_rows[kMaxSlots];
  int64_t slot_group[kMaxSlots], slot_version[kMaxSlots], slot_row0[kMaxSlots], slot_rows[kMaxSlots],
      slot_published[kMaxSlots];
};
constexpr char kStateMagic[8] = {'V', 'F', 'L', 'S', 'T', 'A', 'T', 'E'};
constexpr uint32_t kStateFormat = 2;

// FNV-1a over everything that fixes the workspace layout: element type,
// batch, staleness, replicas and both bottom specs and the top spec.
uint64_t layout_signature(const vfl_ctx* c) {
  uint64_t h = 1469598103934665603ull;
  auto mix = [&](int64_t v) {
    for (int i = 0; i < 8; ++i) {
      h ^= (uint64_t)((v >> (8 * i)) & 0xff);
      h *= 1099511628211ull;
    }
  };
  const Plan& p = c->p;
  mix(p.e); mix(p.B); mix(p.s); mix(p.k); mix((int64_t)p.total);
  for (const vfl_bottom_spec* b : {&p.A.spec, &p.P.spec}) {
    mix(b->dense_in); mix(b->n_cat); mix(b->vocab); mix(b->emb_dim); mix(b->n_layers); mix(b->relu_mask);
    for (int l = 0; l < b->n_layers; ++l) mix(b->widths[l]);
  }
  mix(p.T.spec.n_layers); mix(p.T.spec.relu_mask);
  for (int j = 0; j < p.T.spec.n_layers; ++j) mix(p.T.spec.widths[j]);
  return h;
}

size_t state_bytes(const vfl_ctx* c) {
  return sizeof(StateHead) + c->p.total + sizeof(int64_t) * c->trace.size();
}

vfl_status param_loc(vfl_ctx* c, vfl_party party, int layer, int kind, size_t& off, size_t& bytes) {
  const Plan& p = c->p;
  if (party == VFL_PARTY_A || party == VFL_PARTY_B) {
    const Party& P = party == VFL_PARTY_A ? p.A : p.P;
    if (kind == VFL_PARAM_TABLE) {
      if (!P.spec.n_cat) return fail(c, VFL_E_INVALID, "party has no embedding table");
      off = P.T; bytes = sizeof(float) * (size_t)P.spec.n_cat * P.spec.vocab * P.spec.emb_dim;
      return VFL_OK;
    }
    if (layer < 0 || layer >= P.L) return fail(c, VFL_E_INVALID, "layer out of range");
    if (kind == VFL_PARAM_W) { off = P.W[layer]; bytes = sizeof(float) * (size_t)P.out[layer] * P.in[layer]; }
    else if (kind == VFL_PARAM_B) { off = P.b[layer]; bytes = sizeof(float) * P.out[layer]; }
    else return fail(c, VFL_E_INVALID, "bad parameter kind");
    return VFL_OK;
  }
  if (party == VFL_TOP) {
    const Top& T = p.T;
    if (layer < 0 || layer > T.H) return fail(c, VFL_E_INVALID, "layer out of range");
    if (kind == VFL_PARAM_W) { off = T.W[layer]; bytes = sizeof(float) * (size_t)T.out[layer] * T.in[layer]; }
    else if (kind == VFL_PARAM_B) { off = T.b[layer]; bytes = sizeof(float) * T.out[layer]; }
    else return fail(c, VFL_E_INVALID, "bad parameter kind");
    return VFL_OK;
  }
  return fail(c, VFL_E_INVALID, "bad party");
}

// The slot description of group g of the bound dataset for one party.
SlotState dataset_slot(vfl_ctx* c, int party, int64_t g) {
  const Plan& p = c->p;
  const int64_t E = (c->n_rows + p.R - 1) / p.R;
  const int64_t start = (g % E) * p.R;
  const vfl_dataset& d = party == 0 ? c->ds_a : c->ds_b;
  const Party& P = party == 0 ? p.A : p.P;
  const int es = elt_size(p.e);
  SlotState st;
  st.rows = (int)std::min<int64_t>(p.R, c->n_rows - start);
  st.row0 = start;
  st.ld = d.ld ? d.ld : P.spec.dense_in;
  st.dense = d.dense ? (const char*)d.dense + start * st.ld * es : nullptr;
  st.ids = d.ids ? d.ids + start * P.spec.n_cat : nullptr;
  st.labels = d.labels ? d.labels + start : nullptr;
  st.group = g;
  return st;
}

// the same group as replica batches (what a caller of vfl_step would pass)
int dataset_batches(vfl_ctx* c, int party, int64_t g, vfl_batch* out) {
  const Plan& p = c->p;
  const SlotState st = dataset_slot(c, party, g);
  const int es = elt_size(p.e);
  const Party& P = party == 0 ? p.A : p.P;
  int n = 0;
  for (int64_t o = 0; o < st.rows; o += p.B, ++n) {
    vfl_batch& b = out[n];
    b = vfl_batch{};
    if (st.dense) { b.dense = (const char*)st.dense + o * st.ld * es; b.ld = st.ld; }
    if (st.ids) b.ids = st.ids + o * P.spec.n_cat;
    if (st.labels) b.labels = st.labels + o;
    b.rows = (int32_t)std::min<int64_t>(p.B, st.rows - o);
    b.row0 = st.row0 + o;
  }
  return n;
}

// Graph gi of `len` ticks whose first tick has phase `phase` (t mod (s+1)),
// captured once for a loss ring and timing mask; launches refer to tick
// base + i of the replay, so the graph is independent of the absolute tick,
// and its last node advances the base by len.
vfl_status ensure_graph(vfl_ctx* c, int gi, int phase, int len, float* loss_ring, int64_t loss_len) {
  const Plan& p = c->p;
  const int s = p.s, S1 = s + 1;
  const uint32_t mask = c->tm.mask;
  const bool stale = c->gexec[gi] &&
      (c->graph_loss[gi] != loss_ring || c->graph_loss_len[gi] != loss_len || c->graph_mask[gi] != mask ||
       c->graph_len[gi] != len);
  if (stale) {
    // an earlier replay of it may still run
    HIPCHK(hipStreamSynchronize(c->sa));
    (void)hipGraphExecDestroy(c->gexec[gi]);
    (void)hipGraphDestroy(c->graph[gi]);
    c->gexec[gi] = nullptr;
    c->graph[gi] = nullptr;
  }
  if (c->gexec[gi]) return VFL_OK;
  c->gused[gi] = 0;
  if (mask && c->gpairs[gi].empty()) {
    constexpr int kGraphPairs = 1024;
    c->gpairs[gi].resize(kGraphPairs);
    for (auto& gp : c->gpairs[gi]) {
      HIPCHK(hipEventCreate(&gp.e0));
      HIPCHK(hipEventCreate(&gp.e1));
    }
  }
  TickSrc* tsrc = at<TickSrc>(c, p.tsrc);
  // dataset bases: the tick records supply rows, row0 and the headers
  SlotState sa_in, sb_in;
  sa_in.rows = p.R; sa_in.dense = c->ds_a.dense; sa_in.ld = c->ds_a.ld; sa_in.ids = c->ds_a.ids;
  sa_in.labels = c->ds_a.labels;
  sb_in.rows = p.R; sb_in.dense = c->ds_b.dense; sb_in.ld = c->ds_b.ld; sb_in.ids = c->ds_b.ids;
  c->tm_err = hipSuccess;
  HIPCHK(hipStreamBeginCapture(c->sa, hipStreamCaptureModeThreadLocal));
  c->capture_phase = gi;
  vfl_status r = VFL_OK;
  hipError_t he = hipEventRecord(c->ev_fork, c->sa);
  if (he == hipSuccess) he = hipStreamWaitEvent(c->sb, c->ev_fork, 0);
  for (int i = 0; i < len && he == hipSuccess && r == VFL_OK; ++i) {
    const int fs = (phase + i) % S1;                   // slot of group t
    const int us = ((phase + i - s) % S1 + S1) % S1;   // slot of group t - s
    const TickRef tb{tsrc, i, 0}, ta{tsrc, i, 1}, tu{tsrc, i, 2};
    c->capture_tick = i;
    if ((r = b_forward(c, fs, sb_in, tb))) break;
    if ((r = b_publish(c, fs))) break;
    // the first s ticks consume groups published before this graph;
    // replays on one stream never overlap, so the publish of those groups
    // is already complete
    if ((r = a_top(c, 0, us, sa_in, 0, ta, i >= s))) break;
    if ((r = a_backward(c, sa_in, loss_ring, ta))) break;
    if ((r = b_backward(c, us, sb_in, 0, tu))) break;
  }
  c->capture_tick = -1;
  if (he == hipSuccess && r == VFL_OK) he = hipEventRecord(c->ev_join, c->sb);
  if (he == hipSuccess && r == VFL_OK) he = hipStreamWaitEvent(c->sa, c->ev_join, 0);
  if (he == hipSuccess && r == VFL_OK) he = launch_tick_base(tsrc, len, c->sa);
  hipGraph_t g = nullptr;
  const hipError_t he2 = hipStreamEndCapture(c->sa, &g);
  c->capture_phase = -1;
  if (r) { if (g) (void)hipGraphDestroy(g); return r; }
  if (he != hipSuccess || he2 != hipSuccess) {
    if (g) (void)hipGraphDestroy(g);
    return fail(c, VFL_E_HIP, std::string("graph capture: ") + hipGetErrorString(he != hipSuccess ? he : he2));
  }
  if (c->tm_err != hipSuccess) {
    const hipError_t te = c->tm_err;
    c->tm_err = hipSuccess;
    (void)hipGraphDestroy(g);
    return fail(c, VFL_E_HIP, std::string("timing event record in graph capture: ") + c->tm_err_what +
                           ": " + hipGetErrorString(te));
  }
  c->graph[gi] = g;
  HIPCHK(hipGraphInstantiate(&c->gexec[gi], g, nullptr, nullptr, 0));
  c->graph_loss[gi] = loss_ring;
  c->graph_loss_len[gi] = loss_len;
  c->graph_mask[gi] = mask;
  c->graph_len[gi] = len;
  return VFL_OK;
}

}  // namespace

extern "C" vfl_status vfl_destroy(vfl_ctx* c);

namespace {

// The workspace of vfl_create_static: one array per device, in the code
// object's zero-initialised data, held from the library's load on a device
// until the process ends.  Host code reaches it only through the address
// hipGetSymbolAddress returns for the current device (the array's name is a
// host-side stand-in); at most one context holds a device's array at a time.
static __device__ __align__(256) unsigned char scratch[VFL_STATIC_WORKSPACE_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_static_mu;
void* g_static_ptr[kMaxDevices] = {};
bool g_static_held[kMaxDevices] = {};

// Take the current device's static workspace: its address (looked up once
// per device, with that device current) or an error.
vfl_status static_ws_acquire(int& dev, void*& ptr, std::string& why) {
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    why = std::string("hipGetDevice: ") + hipGetErrorString(e);
    return VFL_E_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    why = "device index beyond the static workspace table";
    return VFL_E_INVALID;
  }
  std::lock_guard<std::mutex> lock(g_static_mu);
  if (g_static_held[dev]) {
    why = "the static workspace of device " + std::to_string(dev) +
          " is held by another context (destroy that one first)";
    return VFL_E_STATE;
  }
  if (!g_static_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p || ((uintptr_t)p) % 256) {
      why = std::string("hipGetSymbolAddress of the static workspace: ") + hipGetErrorString(e);
      return VFL_E_HIP;
    }
    g_static_ptr[dev] = p;
  }
  g_static_held[dev] = true;
  ptr = g_static_ptr[dev];
  return VFL_OK;
}

void static_ws_release(int dev) {
  std::lock_guard<std::mutex> lock(g_static_mu);
  g_static_held[dev] = false;
}

// The part of context creation shared by vfl_create and vfl_create_static:
// plan checked, workspace chosen.  On failure the context is destroyed (which
// also releases a static workspace).
vfl_status finish_create(vfl_ctx* c, const vfl_opts* o, void* workspace, void* stream_a,
                         void* stream_b, vfl_ctx** out) {
  c->o = *o;
  c->ws = (char*)workspace;
  c->sa = (hipStream_t)stream_a;
  c->sb = (hipStream_t)stream_b;
  for (int q = 0; q < kMaxSlots; ++q) {
    c->grad_group[q] = -1;
    c->b_copy_version[q] = -1;
  }
  hipError_t e = chain_init();
  for (int q = 0; q <= c->p.s && e == hipSuccess; ++q) {
    e = hipEventCreateWithFlags(&c->ev_emb[q], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_grad[q], hipEventDisableTiming);
  }
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_fork, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_join, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_avg, hipEventDisableTiming);
  // parameters, headers and the error counter start at zero
  if (e == hipSuccess) e = hipMemsetAsync(c->ws, 0, c->p.total, c->sa);
  if (e == hipSuccess) e = hipStreamSynchronize(c->sa);
  if (e != hipSuccess) {
    vfl_destroy(c);
    return fail_create(VFL_E_HIP, std::string("context set-up: ") + hipGetErrorString(e));
  }
  const vfl_status js = write_jobs(c);
  if (js != VFL_OK) {
    const std::string msg = c->err;
    vfl_destroy(c);
    return fail_create(js, msg);
  }
  t_create_err.clear();
  *out = c;
  return VFL_OK;
}

}  // namespace

extern "C" {

vfl_status vfl_workspace_size(const vfl_bottom_spec* a, const vfl_bottom_spec* b,
                              const vfl_top_spec* top, const vfl_opts* o, size_t* bytes) {
  if (!bytes) return fail_create(VFL_E_INVALID, "null bytes");
  Plan p;
  std::string why = build_plan(a, b, top, o, p);
  if (!why.empty()) return fail_create(VFL_E_INVALID, why);
  // the kernels' layouts are checked here already (against a nominal base)
  Jobs J;
  why = build_jobs(p, *o, (char*)(uintptr_t)4096, J);
  if (!why.empty()) return fail_create(VFL_E_INVALID, why);
  t_create_err.clear();
  *bytes = p.total;
  return VFL_OK;
}

vfl_status vfl_create(const vfl_bottom_spec* a, const vfl_bottom_spec* b, const vfl_top_spec* top,
                      const vfl_opts* o, void* workspace, size_t bytes, void* stream_a,
                      void* stream_b, vfl_ctx** out) {
  if (!out) return fail_create(VFL_E_INVALID, "null out");
  *out = nullptr;
  vfl_ctx* c = new vfl_ctx();
  std::string why = build_plan(a, b, top, o, c->p);
  if (!why.empty()) { delete c; return fail_create(VFL_E_INVALID, why); }
  if (!workspace || ((uintptr_t)workspace) % 256) {
    delete c;
    return fail_create(VFL_E_INVALID, "workspace null or not 256-byte aligned");
  }
  if (bytes < c->p.total) { delete c; return fail_create(VFL_E_NOMEM, "workspace too small"); }
  return finish_create(c, o, workspace, stream_a, stream_b, out);
}

vfl_status vfl_create_static(const vfl_bottom_spec* a, const vfl_bottom_spec* b,
                             const vfl_top_spec* top, const vfl_opts* o, void* stream_a,
                             void* stream_b, vfl_ctx** out) {
  if (!out) return fail_create(VFL_E_INVALID, "null out");
  *out = nullptr;
  vfl_ctx* c = new vfl_ctx();
  std::string why = build_plan(a, b, top, o, c->p);
  if (!why.empty()) { delete c; return fail_create(VFL_E_INVALID, why); }
  if (c->p.total > (size_t)VFL_STATIC_WORKSPACE_BYTES) {
    const std::string msg = "configuration needs " + std::to_string(c->p.total) +
                            " bytes of workspace; the static workspace holds " +
                            std::to_string((size_t)VFL_STATIC_WORKSPACE_BYTES);
    delete c;
    return fail_create(VFL_E_NOMEM, msg);
  }
  int dev = -1;
  void* ws = nullptr;
  const vfl_status st = static_ws_acquire(dev, ws, why);
  if (st != VFL_OK) { delete c; return fail_create(st, why); }
  c->static_dev = dev;
  return finish_create(c, o, ws, stream_a, stream_b, out);
}

vfl_status vfl_set_param(vfl_ctx* c, vfl_party party, int32_t layer, int32_t kind, const void* src,
                         size_t bytes, int32_t src_on_device) {
  if (!c || !src) return VFL_E_INVALID;
  size_t off = 0, nb = 0;
  vfl_status st = param_loc(c, party, layer, kind, off, nb);
  if (st) return st;
  if (bytes != nb) return fail(c, VFL_E_INVALID, "parameter size mismatch");
  HIPCHK(hipStreamSynchronize(c->sa));
  HIPCHK(hipStreamSynchronize(c->sb));
  HIPCHK(hipMemcpy(c->ws + off, src, nb, src_on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice));
  // operand copies of the changed party no longer hold its weights
  if (party == VFL_PARTY_B)
    for (int q = 0; q < kMaxSlots; ++q) c->b_copy_version[q] = -1;
  else
    c->a_copy_version = -1;
  return VFL_OK;
}

vfl_status vfl_get_param(vfl_ctx* c, vfl_party party, int32_t layer, int32_t kind, void* dst,
                         size_t bytes, int32_t dst_on_device) {
  if (!c || !dst) return VFL_E_INVALID;
  size_t off = 0, nb = 0;
  vfl_status st = param_loc(c, party, layer, kind, off, nb);
  if (st) return st;
  if (bytes != nb) return fail(c, VFL_E_INVALID, "parameter size mismatch");
  HIPCHK(hipStreamSynchronize(c->sa));
  HIPCHK(hipStreamSynchronize(c->sb));
  HIPCHK(hipMemcpy(dst, c->ws + off, nb, dst_on_device ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost));
  return VFL_OK;
}

vfl_status vfl_bottom_forward(vfl_ctx* c, vfl_party party, int64_t group, const vfl_batch* br,
                              int32_t n) {
  if (!c) return VFL_E_INVALID;
  Plan& p = c->p;
  if (party == VFL_PARTY_B) {
    if (group != c->b_next_fwd || c->b_pub_next != group)
      return fail(c, VFL_E_STATE, "B's forward must take the next group after publishing the last");
    // a full channel: with FIFO discard the oldest group in flight goes
    // (its embedding if A has not taken it, else its gradient), once the
    // call is known to be valid
    const int64_t g0 = c->b_next_bwd;
    const bool full = group - g0 > p.s;
    if (full) {
      if (!(c->o.flags & VFL_FIFO_DISCARD) || group - g0 != p.s + 1 || c->bslot[g0 % (p.s + 1)].group != g0)
        return fail(c, VFL_E_STALE, "more than s+1 groups in flight");
      if (!dropped(c, g0) && c->a_next == g0 && c->a_phase != 0)
        return fail(c, VFL_E_STALE, "the oldest group is inside A's step");
    }
    const int slot = (int)(group % (p.s + 1));
    SlotState st;
    vfl_status r = take_batches(c, p.P, br, n, false, st);
    if (r) return r;
    if (full) {
      if (!dropped(c, g0)) {
        const bool consumed = c->a_next > g0;
        if (!consumed) c->a_next = g0 + 1;
        note_drop(c, g0, consumed);
      }
      (void)release_drop(c, g0, r);
      if (r) return r;
    }
    st.group = group;
    st.version = c->b_version;
    st.published = false;
    if (c->b_copy_version[slot] != c->b_version) {
      if ((r = enqueue_cast(c, p.P, slot, nullptr, c->sb))) return r;
      c->b_copy_version[slot] = c->b_version;
    }
    if ((r = b_forward(c, slot, st, TickRef()))) return r;
    c->bslot[slot] = st;
    c->b_next_fwd = group + 1;
    return VFL_OK;
  }
  if (party == VFL_PARTY_A) {
    // A's forward runs fused with its top step; this call takes the batch
    if (group != c->a_next || c->a_phase != 0)
      return fail(c, VFL_E_STATE, "A's forward must take the next group A consumes");
    SlotState st;
    vfl_status r = take_batches(c, p.A, br, n, true, st);
    if (r) return r;
    st.group = group;
    c->aslot = st;
    c->a_phase = 1;
    return VFL_OK;
  }
  return fail(c, VFL_E_INVALID, "bad party");
}

vfl_status vfl_publish(vfl_ctx* c, int64_t group) {
  if (!c) return VFL_E_INVALID;
  Plan& p = c->p;
  const int slot = (int)(group % (p.s + 1));
  if (group != c->b_pub_next || c->b_next_fwd != group + 1 || c->bslot[slot].group != group)
    return fail(c, VFL_E_STATE, "publish must follow B's forward of the same group");
  vfl_status r = b_publish(c, slot);
  if (r) return r;
  c->bslot[slot].published = true;
  c->b_pub_next = group + 1;
  return VFL_OK;
}

vfl_status vfl_top_step(vfl_ctx* c, int64_t group, float* loss_dev) {
  if (!c) return VFL_E_INVALID;
  Plan& p = c->p;
  if (group != c->a_next || c->a_phase != 1)
    return fail(c, VFL_E_STATE, "top step must follow A's forward of the same group");
  const int slot = (int)(group % (p.s + 1));
  SlotState& bs = c->bslot[slot];
  if (bs.group != group || !bs.published)
    return fail(c, VFL_E_NOT_READY, "embedding of this group not published");
  if (bs.rows != c->aslot.rows) return fail(c, VFL_E_INVALID, "A and B batches differ in rows");
  vfl_status r;
  if (c->a_copy_version != c->a_version) {
    if ((r = enqueue_cast(c, p.A, 0, &p.T, c->sa))) return r;
    c->a_copy_version = c->a_version;
  }
  if ((r = a_top(c, group, slot, c->aslot, (int32_t)bs.version, TickRef()))) return r;
  c->grad_group[slot] = group;
  c->grad_rows[slot] = c->aslot.rows;
  c->a_loss = loss_dev;
  c->a_phase = 2;
  return VFL_OK;
}

vfl_status vfl_bottom_backward(vfl_ctx* c, vfl_party party, int64_t group) {
  if (!c) return VFL_E_INVALID;
  Plan& p = c->p;
  if (party == VFL_PARTY_A) {
    if (group != c->a_next || c->a_phase != 2)
      return fail(c, VFL_E_STATE, "A's backward must follow its top step");
    vfl_status r = a_backward(c, c->aslot, c->a_loss, TickRef());
    if (r) return r;
    c->a_version += 1;
    c->a_rows_avg += c->aslot.rows;
    c->a_copy_version = c->a_version;
    c->a_next = group + 1;
    c->a_phase = 0;
    return VFL_OK;
  }
  if (party == VFL_PARTY_B) {
    if (group != c->b_next_bwd) return fail(c, VFL_E_STATE, "B back-propagates groups in order");
    const int slot = (int)(group % (p.s + 1));
    if (c->bslot[slot].group == group) {
      vfl_status rr = VFL_OK;
      if (release_drop(c, group, rr)) return rr;
    }
    if (c->grad_group[slot] != group || c->bslot[slot].group != group)
      return fail(c, VFL_E_NOT_READY, "gradient of this group not published");
    vfl_status r = b_backward(c, slot, c->bslot[slot], group, TickRef());
    if (r) return r;
    c->b_next_bwd = group + 1;
    c->b_version += 1;
    c->b_rows_avg += c->bslot[slot].rows;
    c->b_copy_version[slot] = c->b_version;
    return VFL_OK;
  }
  return fail(c, VFL_E_INVALID, "bad party");
}

vfl_status vfl_discard(vfl_ctx* c, int64_t group) {
  if (!c) return VFL_E_INVALID;
  if (group != c->a_next || c->a_phase != 0)
    return fail(c, VFL_E_STATE, "A discards the next group it would consume, before its forward");
  if (group < c->b_next_bwd || dropped(c, group)) return fail(c, VFL_E_STATE, "group already released");
  note_drop(c, group, false);
  c->a_next = group + 1;
  return VFL_OK;
}

vfl_status vfl_step(vfl_ctx* c, int64_t t, const vfl_batch* a, int32_t n_a, const vfl_batch* b,
                    int32_t n_b, float* loss_dev) {
  if (!c) return VFL_E_INVALID;
  const int s = c->p.s;
  int64_t row[7] = {t, -1, -1, -1, -1, -1, -1};
  vfl_status r;
  if (n_b > 0) {
    row[1] = t; row[2] = t % (s + 1); row[3] = c->b_version;
    if ((r = vfl_bottom_forward(c, VFL_PARTY_B, t, b, n_b))) return r;
    if ((r = vfl_publish(c, t))) return r;
  }
  if (n_a > 0) {
    const int64_t u = t - s;
    if (u < 0) return fail(c, VFL_E_STATE, "no group to consume before tick s");
    // a group discarded by vfl_discard: no A step, B releases its slot
    if (!(dropped(c, u) && c->a_next > u)) {
      if ((r = vfl_bottom_forward(c, VFL_PARTY_A, u, a, n_a))) return r;
      if ((r = vfl_top_step(c, u, loss_dev))) return r;
      if ((r = vfl_bottom_backward(c, VFL_PARTY_A, u))) return r;
    }
    if ((r = vfl_bottom_backward(c, VFL_PARTY_B, u))) return r;
    row[4] = u; row[5] = u % (s + 1); row[6] = c->b_version;
  }
  c->trace.insert(c->trace.end(), row, row + 7);
  return VFL_OK;
}

vfl_status vfl_bind_dataset(vfl_ctx* c, const vfl_dataset* a, const vfl_dataset* b, int64_t n_rows) {
  if (!c || !a || !b || n_rows < 1) return VFL_E_INVALID;
  const Plan& p = c->p;
  const int es = elt_size(p.e);
  const vfl_dataset* ds[2] = {a, b};
  const Party* P[2] = {&p.A, &p.P};
  for (int i = 0; i < 2; ++i) {
    const int64_t ld = ds[i]->ld ? ds[i]->ld : P[i]->spec.dense_in;
    if (P[i]->spec.dense_in) {
      if (!ds[i]->dense || ld < P[i]->spec.dense_in)
        return fail(c, VFL_E_INVALID, "dataset dense input missing or ld too small");
      if (!P[i]->spec.n_cat && ((ld * es) % 16 || ((uintptr_t)ds[i]->dense) % 16))
        return fail(c, VFL_E_INVALID, "dataset dense rows must be 16-byte aligned");
    }
    if (P[i]->spec.n_cat && !ds[i]->ids) return fail(c, VFL_E_INVALID, "dataset ids missing");
  }
  if (!a->labels) return fail(c, VFL_E_INVALID, "dataset labels missing");
  // captured graphs point at the previous binding
  for (int q = 0; q < vfl_ctx::kGraphs; ++q) {
    if (c->gexec[q]) (void)hipGraphExecDestroy(c->gexec[q]);
    if (c->graph[q]) (void)hipGraphDestroy(c->graph[q]);
    c->gexec[q] = nullptr;
    c->graph[q] = nullptr;
  }
  c->ds_a = *a;
  c->ds_b = *b;
  if (!c->ds_a.ld) c->ds_a.ld = p.A.spec.dense_in;
  if (!c->ds_b.ld) c->ds_b.ld = p.P.spec.dense_in;
  c->n_rows = n_rows;
  c->bound = true;
  return VFL_OK;
}

vfl_status vfl_run(vfl_ctx* c, int64_t t0, int64_t n, float* loss_ring, int64_t loss_len) {
  if (!c || n < 0) return VFL_E_INVALID;
  if (!c->bound) return fail(c, VFL_E_STATE, "no dataset bound");
  Plan& p = c->p;
  const int s = p.s, S1 = s + 1;
  if (loss_ring && loss_len < 1) return fail(c, VFL_E_INVALID, "loss_len must be >= 1");
  if (t0 < S1 || c->b_next_fwd != t0 || c->b_pub_next != t0 || c->b_next_bwd != t0 - s ||
      c->a_next != t0 - s || c->a_phase != 0)
    return fail(c, VFL_E_STATE, "vfl_run continues a run of ticks 0 .. t0-1 with t0 >= s+1");
  if (!c->drops.empty()) return fail(c, VFL_E_STATE, "discarded groups in flight: run those ticks with vfl_step");
  // the replays derive B's version for group g as max(0, g - s - vofs); the
  // groups in flight must already follow that (s + 1 ticks after a drop)
  const int64_t vofs = (t0 - s) - c->b_version;
  for (int64_t g = t0 - s; g < t0; ++g)
    if (c->bslot[g % S1].group != g || c->bslot[g % S1].version != std::max<int64_t>(0, g - s - vofs))
      return fail(c, VFL_E_STATE, "groups in flight predate a discard: run s+1 ticks with vfl_step first");
  if (c->b_copy_version[t0 % S1] != c->b_version || c->a_copy_version != c->a_version)
    return fail(c, VFL_E_STATE, "operand copies not current; run vfl_step first");
  const int cyc = VFL_GRAPH_CYCLES * S1;
  const int64_t reps = n / cyc;
  const int rem = (int)(n % cyc);
  if (n == 0) return VFL_OK;
  const int phase = (int)(t0 % S1);   // every graph starts at a multiple of s+1 ticks from t0
  if (reps > 0) {
    vfl_status r = ensure_graph(c, phase, phase, cyc, loss_ring, loss_len);
    if (r) return r;
  }
  if (rem > 0) {
    vfl_status r = ensure_graph(c, kMaxSlots + phase, phase, rem, loss_ring, loss_len);
    if (r) return r;
  }
  // the replays start at tick t0 (the dataset and schedule constants with it)
  TickSrc src;
  src.base = t0; src.n_rows = c->n_rows; src.R = p.R; src.s = s; src.lr = c->o.lr;
  src.vofs = (int32_t)vofs;
  src.loss_len = loss_ring ? loss_len : 1;
  HIPCHK(launch_tick_set(at<TickSrc>(c, p.tsrc), src, c->sa));
  // the graphs run both parties' work from stream A: they must follow the
  // work already enqueued on stream B
  HIPCHK(hipEventRecord(c->ev_fork, c->sb));
  HIPCHK(hipStreamWaitEvent(c->sa, c->ev_fork, 0));
  for (int64_t k = 0; k < reps; ++k) HIPCHK(hipGraphLaunch(c->gexec[phase], c->sa));
  if (rem > 0) HIPCHK(hipGraphLaunch(c->gexec[kMaxSlots + phase], c->sa));
  // later work on stream B must follow the graphs
  HIPCHK(hipEventRecord(c->ev_join, c->sa));
  HIPCHK(hipStreamWaitEvent(c->sb, c->ev_join, 0));
  c->last_phase = rem > 0 ? kMaxSlots + phase : phase;
  // host state as if the ticks had been enqueued one by one
  for (int64_t t = t0; t < t0 + n; ++t) {
    const int64_t u = t - s;
    const int fs = (int)(t % S1), us = (int)(u % S1);
    int64_t row[7] = {t, t, fs, c->b_version, u, us, -1};
    SlotState st = dataset_slot(c, 1, t);
    st.version = c->b_version;
    st.published = true;
    c->bslot[fs] = st;
    c->grad_group[us] = u;
    c->grad_rows[us] = c->bslot[us].rows;
    c->a_version += 1;
    c->b_version += 1;
    c->a_rows_avg += c->grad_rows[us];
    c->b_rows_avg += c->grad_rows[us];
    c->b_copy_version[us] = c->b_version;
    row[6] = c->b_version;
    c->trace.insert(c->trace.end(), row, row + 7);
  }
  c->a_copy_version = c->a_version;
  c->b_next_fwd = c->b_pub_next = t0 + n;
  c->b_next_bwd = c->a_next = t0 + n - s;
  return VFL_OK;
}

vfl_status vfl_replica_average(vfl_ctx* const* ctxs, int32_t n, uint32_t parties) {
  if (!ctxs || n < 1 || n > kMaxAvgSets || !parties || (parties & ~3u)) return VFL_E_INVALID;
  vfl_ctx* c0 = ctxs[0];
  if (!c0) return VFL_E_INVALID;
  int dev = -1;
  HIPCHK0(c0, hipGetDevice(&dev));
  for (int i = 0; i < n; ++i) {
    vfl_ctx* c = ctxs[i];
    if (!c) return fail(c0, VFL_E_INVALID, "null context");
    for (int j = 0; j < i; ++j)
      if (ctxs[j] == c) return fail(c0, VFL_E_INVALID, "a context appears twice");
    if (layout_signature(c) != layout_signature(c0))
      return fail(c0, VFL_E_INVALID, "contexts of different configurations");
    if (c->capture_phase >= 0) return fail(c0, VFL_E_STATE, "graph capture in progress");
    if ((parties & 1u) && c->a_phase != 0)
      return fail(c0, VFL_E_STATE, "party A of a context is inside a group's step");
    hipPointerAttribute_t pa;
    HIPCHK0(c0, hipPointerGetAttributes(&pa, c->ws));
    if (pa.device != dev) return fail(c0, VFL_E_INVALID, "contexts must live on the current device");
  }
  const Plan& p = c0->p;
  // one launch for the selected parties; weights per party: the rows each
  // context applied since that party's last average
  AvgJob j;
  j.n = n;
  j.first[0] = 0;
  for (int i = 0; i < n; ++i) j.base[i] = ctxs[i]->ws;
  for (int party = 0; party < 2; ++party) {
    if (!(parties & (1u << party))) continue;
    int64_t tot = 0;
    for (int i = 0; i < n; ++i) tot += party == 0 ? ctxs[i]->a_rows_avg : ctxs[i]->b_rows_avg;
    if (tot <= 0) return fail(c0, VFL_E_STATE, "no rows applied since the last average");
    for (int i = 0; i < n; ++i) {
      const int64_t r = party == 0 ? ctxs[i]->a_rows_avg : ctxs[i]->b_rows_avg;
      j.w[party][i] = (float)((double)r / (double)tot);
    }
    // the party's float32 masters: bottom layers, table, and for A the top
    const Party& P = party == 0 ? p.A : p.P;
    auto seg = [&](size_t off, int64_t cnt) {
      j.off[j.nseg] = (int64_t)off;
      j.cnt[j.nseg] = cnt;
      j.wsel[j.nseg] = (uint8_t)party;
      j.first[j.nseg + 1] = j.first[j.nseg] + (cnt + 3) / 4;
      ++j.nseg;
    };
    for (int l = 0; l < P.L; ++l) {
      seg(P.W[l], (int64_t)P.out[l] * P.in[l]);
      seg(P.b[l], P.out[l]);
    }
    if (P.spec.n_cat) seg(P.T, (int64_t)P.spec.n_cat * P.spec.vocab * P.spec.emb_dim);
    if (party == 0)
      for (int l = 0; l <= p.T.H; ++l) {
        seg(p.T.W[l], (int64_t)p.T.out[l] * p.T.in[l]);
        seg(p.T.b[l], p.T.out[l]);
      }
  }
  // ordered after every context's pending work on the selected parties'
  // streams, and their later work after the average
  const bool pa = parties & 1u, pb = parties & 2u;
  hipStream_t st0 = pa ? c0->sa : c0->sb;
  auto streams = [&](vfl_ctx* c, hipStream_t out[2]) {
    int m = 0;
    if (pa) out[m++] = c->sa;
    if (pb && !(pa && c->sb == c->sa)) out[m++] = c->sb;
    return m;
  };
  for (int i = 0; i < n; ++i) {
    hipStream_t q[2];
    const int m = streams(ctxs[i], q);
    for (int k = 0; k < m; ++k) {
      if (q[k] == st0) continue;
      HIPCHK0(c0, hipEventRecord(ctxs[i]->ev_avg, q[k]));
      HIPCHK0(c0, hipStreamWaitEvent(st0, ctxs[i]->ev_avg, 0));
    }
  }
  {
    vfl_ctx* c = c0;
    double bytes = 0;
    for (int q = 0; q < j.nseg; ++q) bytes += 8.0 * n * (double)j.cnt[q];
    TIMED(VFL_K_AVG, bytes, st0, launch_avg(j, st0));
  }
  HIPCHK0(c0, hipEventRecord(c0->ev_avg, st0));
  for (int i = 0; i < n; ++i) {
    vfl_ctx* c = ctxs[i];
    hipStream_t q[2];
    const int m = streams(c, q);
    for (int k = 0; k < m; ++k)
      if (q[k] != st0) HIPCHK0(c0, hipStreamWaitEvent(q[k], c0->ev_avg, 0));
    // operand copies of the averaged weights: A's current copies; B's
    // copies in the slot of its next forward when that slot is free (the
    // slots of groups in flight keep the weights their forward used)
    vfl_status r;
    if (pa) {
      if ((r = enqueue_cast(c, p.A, 0, &p.T, c->sa))) return r;
      c->a_copy_version = c->a_version;
      c->a_rows_avg = 0;
    }
    if (pb) {
      const int S1 = p.s + 1;
      for (int qs = 0; qs < S1; ++qs) {
        bool busy = false;
        for (int64_t g = c->b_next_bwd; g < c->b_next_fwd; ++g) busy |= (int)(g % S1) == qs;
        if (busy) continue;
        if (qs == (int)(c->b_next_fwd % S1)) {
          if ((r = enqueue_cast(c, p.P, qs, nullptr, c->sb))) return r;
          c->b_copy_version[qs] = c->b_version;
        } else {
          c->b_copy_version[qs] = -1;
        }
      }
      c->b_rows_avg = 0;
    }
  }
  return VFL_OK;
}

vfl_status vfl_get_message(vfl_ctx* c, int32_t which, int64_t group, void* dst, size_t bytes,
                           int32_t header[3]) {
  if (!c || !dst) return VFL_E_INVALID;
  Plan& p = c->p;
  const int slot = (int)(group % (p.s + 1));
  int rows = 0;
  size_t off = 0;
  if (which == 0) {
    if (c->bslot[slot].group != group || !c->bslot[slot].published)
      return fail(c, VFL_E_STATE, "embedding slot does not hold this group");
    rows = c->bslot[slot].rows;
    off = p.P.zhat[slot];
  } else if (which == 1) {
    if (c->grad_group[slot] != group) return fail(c, VFL_E_STATE, "gradient slot does not hold this group");
    rows = c->grad_rows[slot];
    off = p.ring_g[slot];
  } else {
    return fail(c, VFL_E_INVALID, "which must be 0 or 1");
  }
  const int es = elt_size(p.e);
  if (bytes != (size_t)rows * p.dB * es) return fail(c, VFL_E_INVALID, "message size mismatch");
  HIPCHK(hipStreamSynchronize(c->sa));
  HIPCHK(hipStreamSynchronize(c->sb));
  HIPCHK(hipMemcpy2D(dst, (size_t)p.dB * es, c->ws + off, (size_t)ld_of(p.dB) * es, (size_t)p.dB * es,
                     rows, hipMemcpyDeviceToHost));
  if (header) HIPCHK(hipMemcpy(header, hdr_ptr(c, which, slot), 3 * sizeof(int32_t), hipMemcpyDeviceToHost));
  return VFL_OK;
}

vfl_status vfl_get_trace(vfl_ctx* c, int64_t* buf, size_t cap_rows, size_t* rows) {
  if (!c) return VFL_E_INVALID;
  const size_t n = c->trace.size() / 7;
  if (rows) *rows = n;
  if (buf) std::memcpy(buf, c->trace.data(), sizeof(int64_t) * 7 * std::min(n, cap_rows));
  return VFL_OK;
}

vfl_status vfl_check(vfl_ctx* c, uint32_t* mismatches, uint32_t* bad_ids) {
  if (!c || !mismatches) return VFL_E_INVALID;
  HIPCHK(hipStreamSynchronize(c->sa));
  HIPCHK(hipStreamSynchronize(c->sb));
  int32_t v[2] = {0, 0};
  HIPCHK(hipMemcpy(v, err_ptr(c), sizeof(v), hipMemcpyDeviceToHost));
  *mismatches = (uint32_t)v[0];
  if (bad_ids) *bad_ids = (uint32_t)v[1];
  return VFL_OK;
}

vfl_status vfl_philox(uint64_t seed, uint32_t step, uint32_t tag, uint32_t row0, int32_t rows,
                      int32_t groups, uint32_t* out_dev, void* stream) {
  if (!out_dev || rows < 0 || groups < 0) return VFL_E_INVALID;
  if (hipSuccess != launch_philox_words(seed, step, tag, row0, rows, groups, out_dev, (hipStream_t)stream))
    return VFL_E_HIP;
  return VFL_OK;
}

vfl_status vfl_timing_enable(vfl_ctx* c, uint32_t mask) {
  if (!c) return VFL_E_INVALID;
  Timing& T = c->tm;
  if (mask && !T.created) {
    for (int i = 0; i < Timing::kPool; ++i) {
      HIPCHK(hipEventCreate(&T.ev0[i]));
      HIPCHK(hipEventCreate(&T.ev1[i]));
    }
    T.created = true;
  }
  T.mask = mask;
  return VFL_OK;
}

vfl_status vfl_timing_read(vfl_ctx* c, int32_t cls, double* ms, int64_t* launches, double* work) {
  if (!c || cls < 0 || cls >= VFL_K_COUNT) return VFL_E_INVALID;
  Timing& T = c->tm;
  HIPCHK(hipStreamSynchronize(c->sa));
  HIPCHK(hipStreamSynchronize(c->sb));
  if (T.created)
    for (int i = 0; i < Timing::kPool; ++i) harvest(c, i);
  // event pairs inside the last replayed graph: its last replay's launches
  if (c->last_phase >= 0)
    for (int i = 0; i < c->gused[c->last_phase]; ++i) {
      const vfl_ctx::GPair& gp = c->gpairs[c->last_phase][i];
      float ms_ = 0.f;
      if (gp.cls == cls && hipEventElapsedTime(&ms_, gp.e0, gp.e1) == hipSuccess) {
        T.ms[cls] += ms_;
        T.wk[cls] += gp.work;
        T.n[cls] += 1;
      }
    }
  if (ms) *ms = T.ms[cls];
  if (launches) *launches = T.n[cls];
  if (work) *work = T.wk[cls];
  T.ms[cls] = 0.0;
  T.wk[cls] = 0.0;
  T.n[cls] = 0;
  return VFL_OK;
}

vfl_status vfl_state_size(const vfl_ctx* c, size_t* bytes) {
  if (!c || !bytes) return VFL_E_INVALID;
  *bytes = state_bytes(c);
  return VFL_OK;
}

vfl_status vfl_get_state(vfl_ctx* c, void* host_buf, size_t bytes) {
  if (!c || !host_buf) return VFL_E_INVALID;
  if (c->a_phase != 0) return fail(c, VFL_E_STATE, "A is inside a group's step (forward or top step pending)");
  if (c->capture_phase >= 0) return fail(c, VFL_E_STATE, "graph capture in progress");
  if (!c->drops.empty()) return fail(c, VFL_E_STATE, "discarded groups not yet released by B");
  if (bytes < state_bytes(c)) return fail(c, VFL_E_INVALID, "buffer smaller than vfl_state_size()");
  const Plan& p = c->p;
  StateHead h;
  std::memset(&h, 0, sizeof(h));
  std::memcpy(h.magic, kStateMagic, sizeof(h.magic));
  h.format = kStateFormat;
  h.n_slots = (uint32_t)(p.s + 1);
  h.layout = layout_signature(c);
  h.ws_bytes = p.total;
  h.trace_len = c->trace.size();
  h.b_next_fwd = c->b_next_fwd; h.b_next_bwd = c->b_next_bwd; h.b_version = c->b_version;
  h.b_pub_next = c->b_pub_next; h.a_next = c->a_next; h.a_version = c->a_version;
  h.a_copy_version = c->a_copy_version;
  h.a_rows_avg = c->a_rows_avg; h.b_rows_avg = c->b_rows_avg;
  for (int q = 0; q < kMaxSlots; ++q) {
    h.b_copy_version[q] = c->b_copy_version[q];
    h.grad_group[q] = c->grad_group[q];
    h.grad_rows[q] = c->grad_rows[q];
    const SlotState& st = c->bslot[q];
    h.slot_group[q] = st.group; h.slot_version[q] = st.version; h.slot_row0[q] = st.row0;
    h.slot_rows[q] = st.rows; h.slot_published[q] = st.published;
  }
  char* out = (char*)host_buf;
  HIPCHK(hipStreamSynchronize(c->sa));
  HIPCHK(hipStreamSynchronize(c->sb));
  std::memcpy(out, &h, sizeof(h));
  HIPCHK(hipMemcpy(out + sizeof(h), c->ws, p.total, hipMemcpyDeviceToHost));
  if (!c->trace.empty())
    std::memcpy(out + sizeof(h) + p.total, c->trace.data(), sizeof(int64_t) * c->trace.size());
  return VFL_OK;
}

vfl_status vfl_set_state(vfl_ctx* c, const void* host_buf, size_t bytes) {
  if (!c || !host_buf) return VFL_E_INVALID;
  if (c->capture_phase >= 0) return fail(c, VFL_E_STATE, "graph capture in progress");
  const Plan& p = c->p;
  StateHead h;
  if (bytes < sizeof(h)) return fail(c, VFL_E_INVALID, "state image too short");
  std::memcpy(&h, host_buf, sizeof(h));
  if (std::memcmp(h.magic, kStateMagic, sizeof(h.magic)) || h.format != kStateFormat)
    return fail(c, VFL_E_INVALID, "not a state image of this library");
  if (h.layout != layout_signature(c) || h.ws_bytes != p.total || h.n_slots != (uint32_t)(p.s + 1))
    return fail(c, VFL_E_INVALID, "state image of another configuration");
  if (h.trace_len % 7 || bytes < sizeof(h) + h.ws_bytes + sizeof(int64_t) * h.trace_len)
    return fail(c, VFL_E_INVALID, "state image truncated");
  const char* in = (const char*)host_buf;
  HIPCHK(hipStreamSynchronize(c->sa));
  HIPCHK(hipStreamSynchronize(c->sb));
  HIPCHK(hipMemcpy(c->ws, in + sizeof(h), p.total, hipMemcpyHostToDevice));
  // the image's job descriptors point into the workspace it was taken from
  const vfl_status js = write_jobs(c);
  if (js != VFL_OK) return js;
  c->b_next_fwd = h.b_next_fwd; c->b_next_bwd = h.b_next_bwd; c->b_version = h.b_version;
  c->b_pub_next = h.b_pub_next; c->a_next = h.a_next; c->a_version = h.a_version;
  c->a_copy_version = h.a_copy_version;
  c->a_rows_avg = h.a_rows_avg; c->b_rows_avg = h.b_rows_avg;
  c->a_phase = 0;
  c->aslot = SlotState();
  c->a_loss = nullptr;
  c->drops.clear();
  for (int q = 0; q < kMaxSlots; ++q) {
    c->b_copy_version[q] = h.b_copy_version[q];
    c->grad_group[q] = h.grad_group[q];
    c->grad_rows[q] = (int)h.grad_rows[q];
    SlotState st;
    st.group = h.slot_group[q]; st.version = h.slot_version[q]; st.row0 = h.slot_row0[q];
    st.rows = (int)h.slot_rows[q]; st.published = h.slot_published[q] != 0;
    c->bslot[q] = st;
  }
  c->trace.assign((const int64_t*)(in + sizeof(h) + h.ws_bytes),
                  (const int64_t*)(in + sizeof(h) + h.ws_bytes) + h.trace_len);
  // the channel events: everything they guarded is in place
  for (int q = 0; q <= p.s; ++q) {
    HIPCHK(hipEventRecord(c->ev_emb[q], c->sb));
    HIPCHK(hipEventRecord(c->ev_grad[q], c->sa));
  }
  return VFL_OK;
}

const char* vfl_last_error(const vfl_ctx* c) { return c ? c->err.c_str() : t_create_err.c_str(); }

vfl_status vfl_destroy(vfl_ctx* c) {
  if (!c) return VFL_E_INVALID;
  vfl_status r = VFL_OK;
  if (c->ws) {
    if (hipStreamSynchronize(c->sa) != hipSuccess) r = VFL_E_HIP;
    if (hipStreamSynchronize(c->sb) != hipSuccess) r = VFL_E_HIP;
  }
  if (c->tm.created)
    for (int i = 0; i < Timing::kPool; ++i) {
      (void)hipEventDestroy(c->tm.ev0[i]);
      (void)hipEventDestroy(c->tm.ev1[i]);
    }
  for (int q = 0; q < kMaxSlots; ++q) {
    if (c->ev_emb[q]) (void)hipEventDestroy(c->ev_emb[q]);
    if (c->ev_grad[q]) (void)hipEventDestroy(c->ev_grad[q]);
  }
  for (int q = 0; q < vfl_ctx::kGraphs; ++q) {
    if (c->gexec[q]) (void)hipGraphExecDestroy(c->gexec[q]);
    if (c->graph[q]) (void)hipGraphDestroy(c->graph[q]);
    for (auto& gp : c->gpairs[q]) {
      (void)hipEventDestroy(gp.e0);
      (void)hipEventDestroy(gp.e1);
    }
  }
  if (c->ev_fork) (void)hipEventDestroy(c->ev_fork);
  if (c->ev_join) (void)hipEventDestroy(c->ev_join);
  if (c->ev_avg) (void)hipEventDestroy(c->ev_avg);
  if (c->static_dev >= 0) static_ws_release(c->static_dev);
  delete c;
  return r;
}

}  // extern "C"
