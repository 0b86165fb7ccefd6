// C ABI of the publisher/subscriber split-learning step (include/vfl.h).
//
// Host side only: it validates shapes, lays the caller's workspace out,
// keeps the channel state machine (which group each slot holds, B's
// parameter version, how many groups are in flight) and enqueues the
// kernels of kernels.h on the two party streams.  Party A's work goes to
// stream_a, party B's to stream_b; the only cross-stream edges are the
// per-slot "embedding published" and "gradient published" events.
//
// Slot reuse needs no further edges: B rewrites embedding slot g mod (s+1)
// with group g + s + 1 only after its backward of group g, which waited for
// g's gradient event, recorded by A after A read embedding g; A rewrites
// gradient slot u mod (s+1) with group u + s + 1 only after waiting for that
// group's embedding event, recorded by B after its backward of group u.
//
// Backward order per party: the input-gradient chain first (every layer's
// delta kept in its own buffer), then one launch for all layers' weight
// gradients (SGD fused, operand copies of the new weights refreshed) and one
// reduction launch for the layers whose rows were split across blocks.  The
// refreshed copies of party B land in the slot of the group just
// back-propagated, which is the slot B's next forward uses; a forward casts
// the master weights only when its slot's copies hold another version.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/vfl.h"
#include "kernels.h"

using namespace vfl;

namespace {

constexpr int kMaxSlots = VFL_MAX_STALENESS + 1;
constexpr int kLogitBlocks = 512;

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
  int64_t ldq[VFL_MAX_LAYERS]{}, ldt[VFL_MAX_LAYERS]{};
  size_t W[VFL_MAX_LAYERS]{}, b[VFL_MAX_LAYERS]{}, T = 0;
  size_t Wq[kMaxSlots][VFL_MAX_LAYERS]{}, Wtq[kMaxSlots][VFL_MAX_LAYERS]{};
  size_t x0[kMaxSlots]{};
  int64_t ldx0 = 0;
  size_t act[kMaxSlots][VFL_MAX_LAYERS]{};
  size_t zhat[kMaxSlots]{};          // published embedding (party B)
  size_t norm[kMaxSlots]{}, cfac[kMaxSlots]{};
  size_t dlt[VFL_MAX_LAYERS]{};      // gradient w.r.t. each layer's pre-activation
  size_t gx = 0;
  int64_t ldgx = 0;
  size_t part[VFL_MAX_LAYERS]{}, partb[VFL_MAX_LAYERS]{};
};

struct Top {
  vfl_top_spec spec{};
  int H = 0;                          // hidden layers (n_layers - 1)
  int in[VFL_MAX_LAYERS]{}, out[VFL_MAX_LAYERS]{};
  bool relu[VFL_MAX_LAYERS]{};
  int64_t ldq[VFL_MAX_LAYERS]{}, ldt[VFL_MAX_LAYERS]{};
  size_t W[VFL_MAX_LAYERS]{}, b[VFL_MAX_LAYERS]{};
  size_t Wq[VFL_MAX_LAYERS]{}, Wtq[VFL_MAX_LAYERS]{};
  size_t act[VFL_MAX_LAYERS]{};
  size_t dlt[VFL_MAX_LAYERS]{};
  size_t part[VFL_MAX_LAYERS]{}, partb[VFL_MAX_LAYERS]{};
  size_t logit_part = 0;
};

struct Plan {
  Elt e = F32;
  int s = 0, k = 1, B = 1, R = 1, dA = 0, dB = 0;
  Party A, P;                         // P: party B (passive)
  Top T;
  int splits_a = 1, rps_a = 0, splits_b = 1, rps_b = 0;   // weight-gradient row chunks
  size_t ring_g[kMaxSlots]{};
  size_t gpre = 0;                    // float32 gradient message before clip/noise
  size_t hdr = 0;                     // int32 [2][kMaxSlots][4] + error counter
  size_t ta_a = 0, ta_bf = 0, ta_bb = 0;   // tick records (graph replay)
  size_t ctr = 0;                     // int64 tick counters of streams A and B
  size_t total = 0;
};

struct SlotState {
  int64_t group = -1;
  int64_t version = -1;
  bool published = false;
  int rows = 0;
  const void* dense = nullptr;
  int64_t ld = 0;
  const int32_t* ids = nullptr;
  RowMap rmap;
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
  const float* a_labels = nullptr;
  float* a_loss = nullptr;
  std::vector<int64_t> trace;
  std::string err;
  // resident dataset + captured graphs (one per phase t mod (s+1))
  bool bound = false;
  vfl_dataset ds_a{}, ds_b{};
  int64_t n_rows = 0;
  hipGraph_t graph[kMaxSlots]{};
  hipGraphExec_t gexec[kMaxSlots]{};
  float* graph_loss[kMaxSlots]{};
  int64_t graph_loss_len[kMaxSlots]{};
  uint32_t graph_mask[kMaxSlots]{};
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  int capture_phase = -1;             // >= 0 while capturing that phase's graph
  struct GPair { hipEvent_t e0, e1; int cls; double work; };
  std::vector<GPair> gpairs[kMaxSlots];   // created before capture
  int gused[kMaxSlots]{};                 // pairs used by the captured graph
  hipError_t tm_err = hipSuccess;         // first failed event record in a capture
  std::string tm_err_what;
  int last_phase = -1;                // phase of the graph replayed last
};

namespace {

template <typename T>
T* at(vfl_ctx* c, size_t off) { return (T*)(c->ws + off); }

vfl_status fail(vfl_ctx* c, vfl_status st, const std::string& msg) {
  if (c) c->err = msg;
  return st;
}

#define HIPCHK(expr)                                                                     \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess)                                                                \
      return fail(c, VFL_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_));     \
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
  for (int l = 0; l < s->n_layers; ++l)
    if (s->widths[l] < 1 || s->widths[l] > 65536) { why = "bad bottom width"; return false; }
  return true;
}

// rows per weight-gradient chunk for a launch over `tiles` output tiles:
// aim at >= 256 blocks, chunks a multiple of the kernel's stage depth
void dw_chunks(Elt e, int R, int tiles, int& splits, int& rps) {
  const int RE = dw_stage_rows(e);
  const int max_splits = std::max(1, (R + RE - 1) / RE);
  int s = std::min(max_splits, std::max(1, (256 + tiles - 1) / tiles));
  rps = (R + s - 1) / s;
  rps = (rps + RE - 1) / RE * RE;
  splits = (R + rps - 1) / rps;
}

std::string build_plan(const vfl_bottom_spec* a, const vfl_bottom_spec* b, const vfl_top_spec* t,
                       const vfl_opts* o, Plan& p) {
  std::string why;
  if (!o) return "null opts";
  if (o->dtype != VFL_F32 && o->dtype != VFL_BF16) return "dtype must be VFL_F32 or VFL_BF16";
  if (o->batch < 1) return "batch must be >= 1";
  if (o->staleness < 0 || o->staleness > VFL_MAX_STALENESS) return "staleness out of [0, 4]";
  if (o->replicas < 1 || o->replicas > VFL_MAX_REPLICAS) return "replicas out of [1, 8]";
  if (!std::isfinite(o->lr)) return "lr not finite";
  if ((o->flags & (VFL_CLIP_EMB | VFL_CLIP_GRAD)) && !(o->clip_c > 0.f)) return "clip needs clip_c > 0";
  if ((o->flags & (VFL_NOISE_EMB | VFL_NOISE_GRAD)) && !(o->sigma >= 0.f)) return "sigma must be >= 0";
  if (!check_bottom(a, why) || !check_bottom(b, why)) return why;
  if (!t || t->n_layers < 2 || t->n_layers > VFL_MAX_LAYERS) return "top needs 2..8 layers (>= 1 hidden + logit)";
  if (t->widths[t->n_layers - 1] != 1) return "last top layer must have width 1";
  for (int j = 0; j + 1 < t->n_layers; ++j)
    if (t->widths[j] < 1 || t->widths[j] > 65536) return "bad top width";
  if (t->widths[t->n_layers - 2] > kMaxLogitCols) return "last hidden top width must be <= 512";
  if (a->widths[a->n_layers - 1] % 8) return "party A's embedding width must be a multiple of 8";
  if (a->n_layers + t->n_layers - 1 > kMaxDw) return "party A + top hidden layers must be <= 8";
  if ((int64_t)o->batch * o->replicas > (1 << 28)) return "rows per tick too large";

  p.e = o->dtype == VFL_BF16 ? BF16 : F32;
  p.s = o->staleness;
  p.k = o->replicas;
  p.B = o->batch;
  p.R = o->batch * o->replicas;
  const int es = elt_size(p.e);
  const int64_t R = p.R;
  Layout ly;

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
      P.ldq[l] = ld_of(in);
      P.ldt[l] = ld_of(P.out[l]);
      P.W[l] = ly.take(sizeof(float) * (size_t)P.out[l] * in);
      P.b[l] = ly.take(sizeof(float) * (size_t)P.out[l]);
      P.dlt[l] = ly.take((size_t)es * R * ld_of(P.out[l]));
      in = P.out[l];
    }
    if (s->n_cat) P.T = ly.take(sizeof(float) * (size_t)s->n_cat * s->vocab * s->emb_dim);
    P.ldx0 = ld_of(P.din);
    for (int q = 0; q < nslots; ++q) {
      for (int l = 0; l < P.L; ++l) {
        P.Wq[q][l] = ly.take((size_t)es * P.out[l] * P.ldq[l]);
        P.Wtq[q][l] = ly.take((size_t)es * P.in[l] * P.ldt[l]);
        P.act[q][l] = ly.take((size_t)es * R * ld_of(P.out[l]));
      }
      if (s->n_cat) P.x0[q] = ly.take((size_t)es * R * P.ldx0);
      if (passive) {
        const bool extra = o->flags & (VFL_CLIP_EMB | VFL_NOISE_EMB);
        P.zhat[q] = extra ? ly.take((size_t)es * R * ld_of(P.out[P.L - 1])) : P.act[q][P.L - 1];
        if (o->flags & VFL_CLIP_EMB) {
          P.norm[q] = ly.take(sizeof(float) * R);
          P.cfac[q] = ly.take(sizeof(float) * R);
        }
      }
    }
    if (s->n_cat) {
      P.ldgx = ld_of(s->n_cat * s->emb_dim);
      P.gx = ly.take(sizeof(float) * R * P.ldgx);
    }
  };

  party(p.A, a, 1, false);
  party(p.P, b, p.s + 1, true);
  p.dA = p.A.out[p.A.L - 1];
  p.dB = p.P.out[p.P.L - 1];

  Top& T = p.T;
  T.spec = *t;
  T.H = t->n_layers - 1;
  int in = p.dA + p.dB;
  for (int j = 0; j < t->n_layers; ++j) {
    T.in[j] = in;
    T.out[j] = t->widths[j];
    T.relu[j] = j < T.H && ((t->relu_mask >> j) & 1u);
    T.ldq[j] = ld_of(in);
    T.ldt[j] = ld_of(T.out[j]);
    T.W[j] = ly.take(sizeof(float) * (size_t)T.out[j] * in);
    T.b[j] = ly.take(sizeof(float) * (size_t)T.out[j]);
    if (j < T.H) {
      T.Wq[j] = ly.take((size_t)es * T.out[j] * T.ldq[j]);
      T.Wtq[j] = ly.take((size_t)es * T.in[j] * T.ldt[j]);
      T.act[j] = ly.take((size_t)es * R * ld_of(T.out[j]));
      T.dlt[j] = ly.take((size_t)es * R * ld_of(T.out[j]));
    }
    in = T.out[j];
  }
  T.logit_part = ly.take(sizeof(float) * kLogitBlocks * (T.out[T.H - 1] + 2));

  // messages
  for (int q = 0; q <= p.s; ++q) p.ring_g[q] = ly.take((size_t)es * R * ld_of(p.dB));
  if (o->flags & (VFL_CLIP_GRAD | VFL_NOISE_GRAD)) p.gpre = ly.take(sizeof(float) * R * ld_of(p.dB));
  p.hdr = ly.take(sizeof(int32_t) * (2 * kMaxSlots * 4 + 4));
  p.ta_a = ly.take(sizeof(TickArgs));
  p.ta_bf = ly.take(sizeof(TickArgs));
  p.ta_bb = ly.take(sizeof(TickArgs));
  p.ctr = ly.take(2 * sizeof(int64_t));

  // weight-gradient row chunks and partials (one region per layer: all
  // layers of a party are in flight in the same launch)
  int tiles_a = 0, tiles_b = 0;
  for (int l = 0; l < p.A.L; ++l) tiles_a += dw_tiles(p.A.out[l], p.A.in[l]);
  for (int j = 0; j < T.H; ++j) tiles_a += dw_tiles(T.out[j], T.in[j]);
  for (int l = 0; l < p.P.L; ++l) tiles_b += dw_tiles(p.P.out[l], p.P.in[l]);
  dw_chunks(p.e, p.R, tiles_a, p.splits_a, p.rps_a);
  dw_chunks(p.e, p.R, tiles_b, p.splits_b, p.rps_b);
  auto parts = [&](int splits, int N, int K, size_t& pw, size_t& pb) {
    if (splits <= 1) return;
    pw = ly.take(sizeof(float) * (size_t)splits * N * K);
    pb = ly.take(sizeof(float) * (size_t)splits * N);
  };
  for (int l = 0; l < p.A.L; ++l) parts(p.splits_a, p.A.out[l], p.A.in[l], p.A.part[l], p.A.partb[l]);
  for (int j = 0; j < T.H; ++j) parts(p.splits_a, T.out[j], T.in[j], T.part[j], T.partb[j]);
  for (int l = 0; l < p.P.L; ++l) parts(p.splits_b, p.P.out[l], p.P.in[l], p.P.part[l], p.P.partb[l]);
  p.total = (ly.off + 255) / 256 * 256;
  return "";
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
  st.rmap = RowMap();
  st.rmap.n = n;
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
    st.rmap.start[r] = (int32_t)off;
    st.rmap.row0[r] = x.row0;
    off += x.rows;
  }
  st.rows = (int)off;
  st.dense = br[0].dense;
  st.ld = ld;
  st.ids = br[0].ids;
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
    // capture), recorded as graph nodes, read after the graph's last replay
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

double gemm_flops(int M, int N, int K) { return 2.0 * M * (double)N * K; }

int32_t* hdr_ptr(vfl_ctx* c, int which, int slot) { return at<int32_t>(c, c->p.hdr) + (which * kMaxSlots + slot) * 4; }
int32_t* err_ptr(vfl_ctx* c) { return at<int32_t>(c, c->p.hdr) + 2 * kMaxSlots * 4; }

// ------------------------------------------------------------ enqueue steps
// Every enqueue function below takes an optional tick record `ta`: null when
// the call's values are known on the host (the per-call API), the device
// record of the stream when the work is captured into a replayed graph.
vfl_status enqueue_cast(vfl_ctx* c, const Party& P, int slot, const Top* T, hipStream_t st) {
  CastJob jobs[2 * VFL_MAX_LAYERS + 2];
  int n = 0;
  for (int l = 0; l < P.L; ++l)
    jobs[n++] = CastJob{at<float>(c, P.W[l]), c->ws + P.Wq[slot][l], c->ws + P.Wtq[slot][l],
                        P.out[l], P.in[l], P.ldq[l], P.ldt[l]};
  if (T)
    for (int j = 0; j < T->H; ++j)
      jobs[n++] = CastJob{at<float>(c, T->W[j]), c->ws + T->Wq[j], c->ws + T->Wtq[j],
                          T->out[j], T->in[j], T->ldq[j], T->ldt[j]};
  double bytes = 0;
  for (int i = 0; i < n; ++i) bytes += (double)jobs[i].out * jobs[i].in * (4 + 2 * elt_size(c->p.e));
  TIMED(VFL_K_CAST, bytes, st, launch_cast(c->p.e, jobs, n, st));
  return VFL_OK;
}

// Party bottom forward (gather + layers) into slot `slot`.  With a tick
// record the input pointers in `in` are dataset bases.
vfl_status enqueue_bottom_forward(vfl_ctx* c, const Party& P, int slot, const SlotState& in,
                                  hipStream_t st, int32_t* hdr_out, const int32_t hdr[3],
                                  const TickArgs* ta) {
  const Plan& p = c->p;
  const int R = in.rows;
  const void* x = in.dense;
  int64_t ldx = in.ld;
  if (P.spec.n_cat) {
    GatherJob gj{at<float>(c, P.T), in.ids, P.spec.n_cat, P.spec.vocab, P.spec.emb_dim,
                 in.dense, in.ld, P.spec.dense_in, c->ws + P.x0[slot], P.ldx0, R, ta};
    const double gb = (double)R * P.spec.n_cat * (4 + P.spec.emb_dim * (4.0 + elt_size(p.e))) +
                      2.0 * R * P.spec.dense_in * elt_size(p.e);
    TIMED(VFL_K_GATHER, gb, st, launch_gather(p.e, gj, st));
    x = c->ws + P.x0[slot];
    ldx = P.ldx0;
  }
  for (int l = 0; l < P.L; ++l) {
    GemmNT g;
    g.A1 = l == 0 ? x : c->ws + P.act[slot][l - 1];
    g.lda1 = l == 0 ? ldx : ld_of(P.out[l - 1]);
    g.B = c->ws + P.Wq[slot][l];
    g.ldb = P.ldq[l];
    g.C1 = c->ws + P.act[slot][l];
    g.ldc1 = ld_of(P.out[l]);
    g.bias = at<float>(c, P.b[l]);
    g.relu = P.relu[l];
    g.M = R; g.N = P.out[l]; g.K = P.in[l];
    g.ta = ta;
    g.ta_in = (ta && l == 0 && !P.spec.n_cat) ? 1 : 0;
    if (l == P.L - 1 && hdr_out) {
      g.hdr_out = hdr_out;
      if (hdr) { g.hdr[0] = hdr[0]; g.hdr[1] = hdr[1]; g.hdr[2] = hdr[2]; }
    }
    TIMED(VFL_K_GEMM_FWD, gemm_flops(g.M, g.N, g.K), st, launch_gemm_nt(p.e, g, st));
  }
  return VFL_OK;
}

// Input-gradient chain of a bottom model: from dlt[L-1] down to dlt[0], and
// for tables the float32 gradient of the gathered input columns.
vfl_status enqueue_dx_chain(vfl_ctx* c, const Party& P, int slot, int R, hipStream_t st,
                            const TickArgs* ta) {
  const Plan& p = c->p;
  for (int l = P.L - 1; l >= 1; --l) {
    GemmNT g;
    g.A1 = c->ws + P.dlt[l]; g.lda1 = ld_of(P.out[l]);
    g.B = c->ws + P.Wtq[slot][l]; g.ldb = P.ldt[l];
    g.C1 = c->ws + P.dlt[l - 1]; g.ldc1 = ld_of(P.out[l - 1]);
    if (P.relu[l - 1]) { g.mask = c->ws + P.act[slot][l - 1]; g.ldm = ld_of(P.out[l - 1]); }
    g.M = R; g.N = P.in[l]; g.K = P.out[l];
    g.ta = ta;
    TIMED(VFL_K_GEMM_DX, gemm_flops(g.M, g.N, g.K), st, launch_gemm_nt(p.e, g, st));
  }
  if (P.spec.n_cat) {
    GemmNT g;
    g.A1 = c->ws + P.dlt[0]; g.lda1 = ld_of(P.out[0]);
    g.B = c->ws + P.Wtq[slot][0]; g.ldb = P.ldt[0];
    g.C2 = c->ws + P.gx; g.ldc2 = P.ldgx; g.nsplit = 0; g.c2_f32 = 1;
    g.M = R; g.N = P.spec.n_cat * P.spec.emb_dim; g.K = P.out[0];
    g.ta = ta;
    TIMED(VFL_K_GEMM_DX, gemm_flops(g.M, g.N, g.K), st, launch_gemm_nt(p.e, g, st));
  }
  return VFL_OK;
}

void add_dw(MultiDW& m, const void* D, int N, const void* X1, int64_t ldx1, const void* X2,
            int64_t ldx2, int ksplit, int K, float* W, float* bias, void* Wq, int64_t ldq,
            void* Wtq, int64_t ldt, float* part, float* partb, int splits, int rps) {
  GemmDW& d = m.p[m.n++];
  d.D = D; d.ldd = ld_of(N);
  d.X1 = X1; d.ldx1 = ldx1; d.X2 = X2; d.ldx2 = ldx2; d.ksplit = ksplit;
  d.W = W; d.bias = bias; d.Wq = Wq; d.ldq = ldq; d.Wtq = Wtq; d.ldt = ldt;
  d.part = part; d.partb = partb;
  d.N = N; d.K = K;
  d.splits = splits; d.rows_per_split = rps;
}

// Bottom layers' weight gradients of one party appended to m.  With a tick
// record the dense input in `in` is a dataset base.
void add_party_dw(vfl_ctx* c, MultiDW& m, const Party& P, int slot, const SlotState& in,
                  int splits, int rps, bool dataset_in) {
  const void* x = P.spec.n_cat ? (const void*)(c->ws + P.x0[slot]) : in.dense;
  const int64_t ldx = P.spec.n_cat ? P.ldx0 : in.ld;
  for (int l = 0; l < P.L; ++l) {
    add_dw(m, c->ws + P.dlt[l], P.out[l], l == 0 ? x : c->ws + P.act[slot][l - 1],
           l == 0 ? ldx : ld_of(P.out[l - 1]), nullptr, 0, 1 << 30, P.in[l], at<float>(c, P.W[l]),
           at<float>(c, P.b[l]), c->ws + P.Wq[slot][l], P.ldq[l], c->ws + P.Wtq[slot][l], P.ldt[l],
           P.part[l] ? at<float>(c, P.part[l]) : nullptr, P.partb[l] ? at<float>(c, P.partb[l]) : nullptr,
           splits, rps);
    if (l == 0 && dataset_in && !P.spec.n_cat) m.p[m.n - 1].x_ta = 1;
  }
}

vfl_status enqueue_weight_update(vfl_ctx* c, MultiDW& m, const LogitJob* lj, hipStream_t st) {
  const Plan& p = c->p;
  double flops = 0, rbytes = 0;
  bool split = false;
  for (int q = 0; q < m.n; ++q) {
    flops += gemm_flops(m.R, m.p[q].N, m.p[q].K);
    if (m.p[q].splits > 1) {
      split = true;
      rbytes += 4.0 * ((double)m.p[q].N * m.p[q].K + m.p[q].N) * (m.p[q].splits + 2);
    }
  }
  TIMED(VFL_K_GEMM_DW, flops, st, launch_multi_dw(p.e, m, st));
  if (split || lj) {
    if (lj) rbytes += 4.0 * lj->blocks * (lj->Hd + 2) + 8.0 * lj->Hd;
    TIMED(VFL_K_REDUCE, rbytes, st, launch_multi_reduce(p.e, m, lj, st));
  }
  return VFL_OK;
}

vfl_status enqueue_table_sgd(vfl_ctx* c, const Party& P, const SlotState& in, float scale,
                             hipStream_t st, const TickArgs* ta) {
  if (!P.spec.n_cat) return VFL_OK;
  ScatterJob sj{at<float>(c, P.T), in.ids, P.spec.n_cat, P.spec.vocab, P.spec.emb_dim,
                at<float>(c, P.gx), P.ldgx, in.rows, scale, ta};
  TIMED(VFL_K_EMB_SGD, (double)in.rows * P.spec.n_cat * 4.0 * (1 + P.spec.emb_dim), st,
        launch_scatter_sgd(sj, st));
  return VFL_OK;
}

LogitJob logit_job(vfl_ctx* c, int R, const float* labels, float* loss_dev, const TickArgs* ta) {
  const Plan& p = c->p;
  const Top& T = p.T;
  LogitJob lj{};
  lj.H = c->ws + T.act[T.H - 1]; lj.ldh = ld_of(T.out[T.H - 1]); lj.Hd = T.out[T.H - 1]; lj.R = R;
  lj.w = at<float>(c, T.W[T.H]); lj.b = at<float>(c, T.b[T.H]); lj.y = labels;
  lj.delta = c->ws + T.dlt[T.H - 1]; lj.ldd = ld_of(T.out[T.H - 1]); lj.relu = T.relu[T.H - 1];
  lj.part = at<float>(c, T.logit_part);
  // blocking from the configured rows per tick, so that a short group is
  // cut the same way whether its row count is known on the host or read
  // from a tick record
  lj.blocks = std::max(1, std::min(kLogitBlocks, (p.R + 15) / 16));
  lj.scale = c->o.lr / (float)R;
  lj.loss_out = ta ? nullptr : loss_dev;
  lj.ta = ta;
  lj.loss_base = ta ? loss_dev : nullptr;
  return lj;
}

// ---- the phases of a tick (enqueue only; the callers keep the host state)

// B's forward of group `group` into `slot`; the embedding slot header is
// written by the last layer unless clip/noise publish it.
vfl_status b_forward(vfl_ctx* c, int slot, const SlotState& st, const TickArgs* ta) {
  const Plan& p = c->p;
  const bool extra = c->o.flags & (VFL_CLIP_EMB | VFL_NOISE_EMB);
  const int32_t hdr[3] = {(int32_t)st.group, (int32_t)st.group, (int32_t)st.version};
  return enqueue_bottom_forward(c, p.P, slot, st, c->sb, extra ? nullptr : hdr_ptr(c, 0, slot),
                                ta ? nullptr : hdr, ta);
}

vfl_status b_publish(vfl_ctx* c, int slot, const SlotState& st, const TickArgs* ta) {
  const Plan& p = c->p;
  if (c->o.flags & (VFL_CLIP_EMB | VFL_NOISE_EMB)) {
    ClipNoiseJob j{};
    j.v = c->ws + p.P.act[slot][p.P.L - 1]; j.ldv = ld_of(p.dB); j.v_f32 = p.e == F32;
    j.out = c->ws + p.P.zhat[slot]; j.ldo = ld_of(p.dB);
    j.norm = p.P.norm[slot] ? at<float>(c, p.P.norm[slot]) : nullptr;
    j.cfac = p.P.cfac[slot] ? at<float>(c, p.P.cfac[slot]) : nullptr;
    j.R = st.rows; j.D = p.dB;
    j.clip = (c->o.flags & VFL_CLIP_EMB) != 0; j.C = c->o.clip_c;
    j.noise = (c->o.flags & VFL_NOISE_EMB) != 0;
    j.stdv = c->o.sigma * ((c->o.flags & (VFL_CLIP_EMB | VFL_CLIP_GRAD)) ? c->o.clip_c : 1.f);
    j.seed = c->o.seed; j.step = (uint32_t)st.group; j.tag = 0; j.rows = st.rmap;
    j.hdr_out = hdr_ptr(c, 0, slot);
    j.hdr[0] = (int32_t)st.group; j.hdr[1] = (int32_t)st.group; j.hdr[2] = (int32_t)st.version;
    j.ta = ta;
    TIMED(VFL_K_CLIP_NOISE, (double)st.rows * p.dB * (elt_size(p.e) * 2.0) + 8.0 * st.rows, c->sb,
          launch_clip_noise(p.e, j, c->sb));
  }
  HIPCHK(hipEventRecord(c->ev_emb[slot], c->sb));
  return VFL_OK;
}

vfl_status a_forward(vfl_ctx* c, const SlotState& st, const TickArgs* ta) {
  return enqueue_bottom_forward(c, c->p.A, 0, st, c->sa, nullptr, nullptr, ta);
}

// Top model step of A's group (rows R) against embedding slot `slot`:
// forward, logit + BCE, input-gradient chain, gradient message + event.
vfl_status a_top(vfl_ctx* c, int64_t group, int slot, int R, const float* labels,
                 int32_t b_version, float* loss_dev, const TickArgs* ta, bool wait_emb = true) {
  const Plan& p = c->p;
  hipStream_t st = c->sa;
  if (wait_emb) HIPCHK(hipStreamWaitEvent(st, c->ev_emb[slot], 0));
  const Top& T = p.T;
  const void* zA = c->ws + p.A.act[0][p.A.L - 1];
  const void* zB = c->ws + p.P.zhat[slot];
  for (int j = 0; j < T.H; ++j) {
    GemmNT g;
    if (j == 0) {
      g.A1 = zA; g.lda1 = ld_of(p.dA);
      g.A2 = zB; g.lda2 = ld_of(p.dB); g.ksplit = p.dA;
      g.hdr_chk = hdr_ptr(c, 0, slot); g.chk_seq = (int32_t)group; g.err = err_ptr(c);
    } else {
      g.A1 = c->ws + T.act[j - 1]; g.lda1 = ld_of(T.out[j - 1]);
    }
    g.B = c->ws + T.Wq[j]; g.ldb = T.ldq[j];
    g.C1 = c->ws + T.act[j]; g.ldc1 = ld_of(T.out[j]);
    g.bias = at<float>(c, T.b[j]); g.relu = T.relu[j];
    g.M = R; g.N = T.out[j]; g.K = T.in[j];
    g.ta = ta;
    TIMED(VFL_K_GEMM_FWD, gemm_flops(g.M, g.N, g.K), st, launch_gemm_nt(p.e, g, st));
  }
  // logit + BCE; its reduction and SGD run with the weight update
  LogitJob lj = logit_job(c, R, labels, loss_dev, ta);
  TIMED(VFL_K_LOGIT, (double)R * lj.Hd * 2.0 * elt_size(p.e) + 4.0 * R, st, launch_logit_bce(p.e, lj, st));
  // input-gradient chain of the top model; the last product splits into A's
  // cut-layer delta and the per-row gradient message for B
  const bool gextra = c->o.flags & (VFL_CLIP_GRAD | VFL_NOISE_GRAD);
  for (int j = T.H - 1; j >= 0; --j) {
    GemmNT g;
    g.A1 = c->ws + T.dlt[j]; g.lda1 = ld_of(T.out[j]);
    g.B = c->ws + T.Wtq[j]; g.ldb = T.ldt[j];
    g.M = R; g.N = T.in[j]; g.K = T.out[j];
    g.ta = ta;
    if (j > 0) {
      g.C1 = c->ws + T.dlt[j - 1]; g.ldc1 = ld_of(T.out[j - 1]);
      if (T.relu[j - 1]) { g.mask = c->ws + T.act[j - 1]; g.ldm = ld_of(T.out[j - 1]); }
    } else {
      g.C1 = c->ws + p.A.dlt[p.A.L - 1]; g.ldc1 = ld_of(p.dA);
      if (p.A.relu[p.A.L - 1]) { g.mask = zA; g.ldm = ld_of(p.dA); }
      g.nsplit = p.dA;
      if (gextra) { g.C2 = c->ws + p.gpre; g.ldc2 = ld_of(p.dB); g.c2_f32 = 1; }
      else {
        g.C2 = c->ws + p.ring_g[slot]; g.ldc2 = ld_of(p.dB);
        g.hdr_out = hdr_ptr(c, 1, slot);
        g.hdr[0] = (int32_t)group; g.hdr[1] = (int32_t)(group + p.s); g.hdr[2] = b_version;
      }
    }
    TIMED(VFL_K_GEMM_DX, gemm_flops(g.M, g.N, g.K), st, launch_gemm_nt(p.e, g, st));
  }
  if (gextra) {
    ClipNoiseJob j{};
    j.v = c->ws + p.gpre; j.ldv = ld_of(p.dB); j.v_f32 = 1;
    j.out = c->ws + p.ring_g[slot]; j.ldo = ld_of(p.dB);
    j.R = R; j.D = p.dB;
    j.clip = (c->o.flags & VFL_CLIP_GRAD) != 0; j.C = c->o.clip_c;
    j.noise = (c->o.flags & VFL_NOISE_GRAD) != 0;
    j.stdv = c->o.sigma * ((c->o.flags & (VFL_CLIP_EMB | VFL_CLIP_GRAD)) ? c->o.clip_c : 1.f);
    j.seed = c->o.seed; j.step = (uint32_t)group; j.tag = 1; j.rows = c->aslot.rmap;
    j.hdr_out = hdr_ptr(c, 1, slot);
    j.hdr[0] = (int32_t)group; j.hdr[1] = (int32_t)(group + p.s); j.hdr[2] = b_version;
    j.ta = ta;
    TIMED(VFL_K_CLIP_NOISE, (double)R * p.dB * (4.0 + elt_size(p.e)), st, launch_clip_noise(p.e, j, st));
  }
  HIPCHK(hipEventRecord(c->ev_grad[slot], st));
  return VFL_OK;
}

// A's and the top model's backward + SGD for A's group in `st` (rows R);
// `slot` is the embedding slot the top model read.
vfl_status a_backward(vfl_ctx* c, int slot, const SlotState& st, const float* labels,
                      float* loss_dev, const TickArgs* ta) {
  const Plan& p = c->p;
  const int R = st.rows;
  vfl_status r = enqueue_dx_chain(c, p.A, 0, R, c->sa, ta);
  if (r) return r;
  // one weight update for the top model's hidden layers and A's layers,
  // with the logit layer's reduction, SGD and loss in the same reduction
  MultiDW m;
  m.R = R;
  m.scale = c->o.lr / (float)R;
  m.ta = ta;
  const Top& T = p.T;
  const void* zA = c->ws + p.A.act[0][p.A.L - 1];
  const void* zB = c->ws + p.P.zhat[slot];
  for (int j = 0; j < T.H; ++j)
    add_dw(m, c->ws + T.dlt[j], T.out[j], j == 0 ? zA : c->ws + T.act[j - 1],
           j == 0 ? ld_of(p.dA) : ld_of(T.out[j - 1]), j == 0 ? zB : nullptr,
           j == 0 ? ld_of(p.dB) : 0, j == 0 ? p.dA : 1 << 30, T.in[j], at<float>(c, T.W[j]),
           at<float>(c, T.b[j]), c->ws + T.Wq[j], T.ldq[j], c->ws + T.Wtq[j], T.ldt[j],
           T.part[j] ? at<float>(c, T.part[j]) : nullptr, T.partb[j] ? at<float>(c, T.partb[j]) : nullptr,
           p.splits_a, p.rps_a);
  add_party_dw(c, m, p.A, 0, st, p.splits_a, p.rps_a, ta != nullptr);
  LogitJob lj = logit_job(c, R, labels, loss_dev, ta);
  if ((r = enqueue_weight_update(c, m, &lj, c->sa))) return r;
  return enqueue_table_sgd(c, p.A, st, c->o.lr / (float)R, c->sa, ta);
}

// B's delayed backward of the group stashed in `slot` + SGD on B's current
// weights; the refreshed operand copies go to this slot, which B's next
// forward uses.
vfl_status b_backward(vfl_ctx* c, int slot, const SlotState& st, int64_t group, const TickArgs* ta) {
  const Plan& p = c->p;
  HIPCHK(hipStreamWaitEvent(c->sb, c->ev_grad[slot], 0));
  CutBwdJob cj{};
  cj.g = c->ws + p.ring_g[slot]; cj.ldg = ld_of(p.dB);
  cj.z = c->ws + p.P.act[slot][p.P.L - 1]; cj.ldz = ld_of(p.dB);
  cj.clip = (c->o.flags & VFL_CLIP_EMB) != 0;
  cj.norm = cj.clip ? at<float>(c, p.P.norm[slot]) : nullptr;
  cj.cfac = cj.clip ? at<float>(c, p.P.cfac[slot]) : nullptr;
  cj.C = c->o.clip_c; cj.relu = p.P.relu[p.P.L - 1];
  cj.delta = c->ws + p.P.dlt[p.P.L - 1]; cj.ldd = ld_of(p.dB);
  cj.R = st.rows; cj.D = p.dB;
  cj.hdr_chk = hdr_ptr(c, 1, slot); cj.chk_seq = (int32_t)group; cj.err = err_ptr(c);
  cj.ta = ta;
  TIMED(VFL_K_CUT_BWD, (double)st.rows * p.dB * 3.0 * elt_size(p.e) + (cj.clip ? 8.0 * st.rows : 0.0),
        c->sb, launch_cut_backward(p.e, cj, c->sb));
  vfl_status r = enqueue_dx_chain(c, p.P, slot, st.rows, c->sb, ta);
  if (r) return r;
  MultiDW m;
  m.R = st.rows;
  m.scale = c->o.lr / (float)st.rows;
  m.ta = ta;
  add_party_dw(c, m, p.P, slot, st, p.splits_b, p.rps_b, ta != nullptr);
  if ((r = enqueue_weight_update(c, m, nullptr, c->sb))) return r;
  return enqueue_table_sgd(c, p.P, st, c->o.lr / (float)st.rows, c->sb, ta);
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

// Replica batches of group g of the bound dataset (consecutive chunks of at
// most `batch` rows of the group's rows).
int dataset_batches(vfl_ctx* c, int party, int64_t g, vfl_batch* out) {
  const Plan& p = c->p;
  const int64_t E = (c->n_rows + p.R - 1) / p.R;
  const int64_t start = (g % E) * p.R;
  const int64_t rows = std::min<int64_t>(p.R, c->n_rows - start);
  const vfl_dataset& d = party == 0 ? c->ds_a : c->ds_b;
  const Party& P = party == 0 ? p.A : p.P;
  const int es = elt_size(p.e);
  const int64_t ld = d.ld ? d.ld : P.spec.dense_in;
  int n = 0;
  for (int64_t o = 0; o < rows; o += p.B, ++n) {
    vfl_batch& b = out[n];
    b = vfl_batch{};
    const int64_t r0 = start + o;
    if (d.dense) { b.dense = (const char*)d.dense + r0 * ld * es; b.ld = ld; }
    if (d.ids) b.ids = d.ids + r0 * P.spec.n_cat;
    if (d.labels) b.labels = d.labels + r0;
    b.rows = (int32_t)std::min<int64_t>(p.B, rows - o);
    b.row0 = r0;
  }
  return n;
}

}  // namespace

extern "C" {

vfl_status vfl_workspace_size(const vfl_bottom_spec* a, const vfl_bottom_spec* b,
                              const vfl_top_spec* top, const vfl_opts* o, size_t* bytes) {
  if (!bytes) return VFL_E_INVALID;
  Plan p;
  if (!build_plan(a, b, top, o, p).empty()) return VFL_E_INVALID;
  *bytes = p.total;
  return VFL_OK;
}

vfl_status vfl_create(const vfl_bottom_spec* a, const vfl_bottom_spec* b, const vfl_top_spec* top,
                      const vfl_opts* o, void* workspace, size_t bytes, void* stream_a,
                      void* stream_b, vfl_ctx** out) {
  if (!out) return VFL_E_INVALID;
  *out = nullptr;
  vfl_ctx* c = new vfl_ctx();
  std::string why = build_plan(a, b, top, o, c->p);
  if (!why.empty()) { delete c; return VFL_E_INVALID; }
  if (!workspace || ((uintptr_t)workspace) % 256) { delete c; return VFL_E_INVALID; }
  if (bytes < c->p.total) { delete c; return VFL_E_NOMEM; }
  c->o = *o;
  c->ws = (char*)workspace;
  c->sa = (hipStream_t)stream_a;
  c->sb = (hipStream_t)stream_b;
  for (int q = 0; q < kMaxSlots; ++q) {
    c->grad_group[q] = -1;
    c->b_copy_version[q] = -1;
  }
  hipError_t e = hipSuccess;
  for (int q = 0; q <= c->p.s && e == hipSuccess; ++q) {
    e = hipEventCreateWithFlags(&c->ev_emb[q], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_grad[q], hipEventDisableTiming);
  }
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_fork, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_join, hipEventDisableTiming);
  // parameters, headers and the error counter start at zero
  if (e == hipSuccess) e = hipMemsetAsync(c->ws, 0, c->p.total, c->sa);
  if (e == hipSuccess) e = hipStreamSynchronize(c->sa);
  if (e != hipSuccess) {
    vfl_destroy(c);
    return VFL_E_HIP;
  }
  *out = c;
  return VFL_OK;
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
    if (group - c->b_next_bwd > p.s)
      return fail(c, VFL_E_STALE, "more than s+1 groups in flight");
    const int slot = (int)(group % (p.s + 1));
    SlotState st;
    vfl_status r = take_batches(c, p.P, br, n, false, st);
    if (r) return r;
    st.group = group;
    st.version = c->b_version;
    st.published = false;
    if (c->b_copy_version[slot] != c->b_version) {
      if ((r = enqueue_cast(c, p.P, slot, nullptr, c->sb))) return r;
      c->b_copy_version[slot] = c->b_version;
    }
    if ((r = b_forward(c, slot, st, nullptr))) return r;
    c->bslot[slot] = st;
    c->b_next_fwd = group + 1;
    return VFL_OK;
  }
  if (party == VFL_PARTY_A) {
    if (group != c->a_next || c->a_phase != 0)
      return fail(c, VFL_E_STATE, "A's forward must take the next group A consumes");
    SlotState st;
    vfl_status r = take_batches(c, p.A, br, n, true, st);
    if (r) return r;
    st.group = group;
    if (c->a_copy_version != c->a_version) {
      if ((r = enqueue_cast(c, p.A, 0, &p.T, c->sa))) return r;
      c->a_copy_version = c->a_version;
    }
    if ((r = a_forward(c, st, nullptr))) return r;
    c->aslot = st;
    c->a_labels = br[0].labels;
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
  vfl_status r = b_publish(c, slot, c->bslot[slot], nullptr);
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
  vfl_status r = a_top(c, group, slot, c->aslot.rows, c->a_labels, (int32_t)bs.version, loss_dev, nullptr);
  if (r) return r;
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
    vfl_status r = a_backward(c, (int)(group % (p.s + 1)), c->aslot, c->a_labels, c->a_loss, nullptr);
    if (r) return r;
    c->a_version += 1;
    c->a_copy_version = c->a_version;
    c->a_next = group + 1;
    c->a_phase = 0;
    return VFL_OK;
  }
  if (party == VFL_PARTY_B) {
    if (group != c->b_next_bwd) return fail(c, VFL_E_STATE, "B back-propagates groups in order");
    const int slot = (int)(group % (p.s + 1));
    if (c->grad_group[slot] != group || c->bslot[slot].group != group)
      return fail(c, VFL_E_NOT_READY, "gradient of this group not published");
    vfl_status r = b_backward(c, slot, c->bslot[slot], group, nullptr);
    if (r) return r;
    c->b_next_bwd = group + 1;
    c->b_version += 1;
    c->b_copy_version[slot] = c->b_version;
    return VFL_OK;
  }
  return fail(c, VFL_E_INVALID, "bad party");
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
    if ((r = vfl_bottom_forward(c, VFL_PARTY_A, u, a, n_a))) return r;
    if ((r = vfl_top_step(c, u, loss_dev))) return r;
    if ((r = vfl_bottom_backward(c, VFL_PARTY_A, u))) return r;
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
  for (int q = 0; q < kMaxSlots; ++q) {
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
  if (c->b_copy_version[t0 % S1] != c->b_version || c->a_copy_version != c->a_version)
    return fail(c, VFL_E_STATE, "operand copies not current; run vfl_step first");
  const int cyc = VFL_GRAPH_CYCLES * S1;
  const int64_t reps = n / cyc;
  if (reps > 0) {
    const int phase = (int)(t0 % S1);
    const uint32_t mask = c->tm.mask;
    const bool stale = c->gexec[phase] &&
        (c->graph_loss[phase] != loss_ring || c->graph_loss_len[phase] != loss_len ||
         c->graph_mask[phase] != mask);
    if (stale) {
      (void)hipGraphExecDestroy(c->gexec[phase]);
      (void)hipGraphDestroy(c->graph[phase]);
      c->gexec[phase] = nullptr;
      c->graph[phase] = nullptr;
    }
    if (!c->gexec[phase]) {
      c->gused[phase] = 0;
      if (mask && c->gpairs[phase].empty()) {
        constexpr int kGraphPairs = 1024;
        c->gpairs[phase].resize(kGraphPairs);
        for (auto& gp : c->gpairs[phase]) {
          HIPCHK(hipEventCreate(&gp.e0));
          HIPCHK(hipEventCreate(&gp.e1));
        }
      }
      // capture cyc ticks starting at this phase; the tick records and
      // counters make the graph independent of the absolute tick
      TickArgs* ta_a = at<TickArgs>(c, p.ta_a);
      TickArgs* ta_bf = at<TickArgs>(c, p.ta_bf);
      TickArgs* ta_bb = at<TickArgs>(c, p.ta_bb);
      int64_t* ctr = at<int64_t>(c, p.ctr);
      AdvanceJob adv_a, adv_b;
      adv_a.counter = ctr; adv_a.out[0] = ta_a; adv_a.kind = 0;
      adv_b.counter = ctr + 1; adv_b.out[0] = ta_bf; adv_b.out[1] = ta_bb; adv_b.kind = 1;
      for (AdvanceJob* aj : {&adv_a, &adv_b}) {
        aj->n_rows = c->n_rows; aj->R = p.R; aj->s = s; aj->lr = c->o.lr;
        aj->loss_len = loss_ring ? loss_len : 1;
      }
      SlotState sa_in, sb_in;
      sa_in.rows = p.R; sa_in.dense = c->ds_a.dense; sa_in.ld = c->ds_a.ld; sa_in.ids = c->ds_a.ids;
      sb_in.rows = p.R; sb_in.dense = c->ds_b.dense; sb_in.ld = c->ds_b.ld; sb_in.ids = c->ds_b.ids;
      c->tm_err = hipSuccess;
      HIPCHK(hipStreamBeginCapture(c->sa, hipStreamCaptureModeThreadLocal));
      c->capture_phase = phase;
      vfl_status r = VFL_OK;
      hipError_t he = hipEventRecord(c->ev_fork, c->sa);
      if (he == hipSuccess) he = hipStreamWaitEvent(c->sb, c->ev_fork, 0);
      for (int i = 0; i < cyc && he == hipSuccess && r == VFL_OK; ++i) {
        const int fs = (phase + i) % S1;             // slot of group t
        const int us = ((phase + i - s) % S1 + S1) % S1;   // slot of group t - s
        he = launch_advance(adv_b, c->sb);
        if (he == hipSuccess) he = launch_advance(adv_a, c->sa);
        if (he != hipSuccess) break;
        if ((r = b_forward(c, fs, sb_in, ta_bf))) break;
        if ((r = b_publish(c, fs, sb_in, ta_bf))) break;
        if ((r = a_forward(c, sa_in, ta_a))) break;
        // the first s ticks consume groups published before this graph;
        // replays of a graph on one stream never overlap, so the publish
        // of those groups is already complete
        if ((r = a_top(c, 0, us, p.R, c->ds_a.labels, 0, loss_ring, ta_a, i >= s))) break;
        if ((r = a_backward(c, us, sa_in, c->ds_a.labels, loss_ring, ta_a))) break;
        if ((r = b_backward(c, us, sb_in, 0, ta_bb))) break;
      }
      if (he == hipSuccess && r == VFL_OK) he = hipEventRecord(c->ev_join, c->sb);
      if (he == hipSuccess && r == VFL_OK) he = hipStreamWaitEvent(c->sa, c->ev_join, 0);
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
      c->graph[phase] = g;
      HIPCHK(hipGraphInstantiate(&c->gexec[phase], g, nullptr, nullptr, 0));
      c->graph_loss[phase] = loss_ring;
      c->graph_loss_len[phase] = loss_len;
      c->graph_mask[phase] = mask;
    }
    // both counters start at t0; the graph's advance kernels read them
    const int64_t ctr_h[2] = {t0, t0};
    HIPCHK(hipMemcpyAsync(at<int64_t>(c, p.ctr), ctr_h, sizeof(ctr_h), hipMemcpyHostToDevice, c->sa));
    // the graph runs both parties' work from stream A: it must follow the
    // work already enqueued on stream B
    HIPCHK(hipEventRecord(c->ev_fork, c->sb));
    HIPCHK(hipStreamWaitEvent(c->sa, c->ev_fork, 0));
    for (int64_t k = 0; k < reps; ++k) HIPCHK(hipGraphLaunch(c->gexec[phase], c->sa));
    // later work on stream B must follow the graph
    HIPCHK(hipEventRecord(c->ev_join, c->sa));
    HIPCHK(hipStreamWaitEvent(c->sb, c->ev_join, 0));
    c->last_phase = phase;
    // host state as if the ticks had been enqueued one by one
    for (int64_t t = t0; t < t0 + reps * cyc; ++t) {
      const int64_t u = t - s;
      const int fs = (int)(t % S1), us = (int)(u % S1);
      int64_t row[7] = {t, t, fs, c->b_version, u, us, -1};
      SlotState st;
      vfl_batch bb[VFL_MAX_REPLICAS];
      const int nb = dataset_batches(c, 1, t, bb);
      st.rows = 0;
      st.rmap = RowMap();
      st.rmap.n = nb;
      for (int i = 0; i < nb; ++i) {
        st.rmap.start[i] = st.rows;
        st.rmap.row0[i] = bb[i].row0;
        st.rows += bb[i].rows;
      }
      st.dense = bb[0].dense; st.ld = bb[0].ld; st.ids = bb[0].ids;
      st.group = t; st.version = c->b_version; st.published = true;
      c->bslot[fs] = st;
      c->grad_group[us] = u;
      c->grad_rows[us] = c->bslot[us].rows;
      c->a_version += 1;
      c->b_version += 1;
      c->b_copy_version[us] = c->b_version;
      row[6] = c->b_version;
      c->trace.insert(c->trace.end(), row, row + 7);
    }
    c->a_copy_version = c->a_version;
    c->b_next_fwd = c->b_pub_next = t0 + reps * cyc;
    c->b_next_bwd = c->a_next = t0 + reps * cyc - s;
  }
  // the remainder tick by tick
  for (int64_t t = t0 + reps * cyc; t < t0 + n; ++t) {
    vfl_batch ab[VFL_MAX_REPLICAS], bb[VFL_MAX_REPLICAS];
    const int na = dataset_batches(c, 0, t - s, ab);
    const int nb = dataset_batches(c, 1, t, bb);
    float* lp = loss_ring ? loss_ring + ((t - s) % loss_len) : nullptr;
    vfl_status r = vfl_step(c, t, ab, na, bb, nb, lp);
    if (r) return r;
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

vfl_status vfl_check(vfl_ctx* c, uint32_t* mismatches) {
  if (!c || !mismatches) return VFL_E_INVALID;
  HIPCHK(hipStreamSynchronize(c->sa));
  HIPCHK(hipStreamSynchronize(c->sb));
  int32_t v = 0;
  HIPCHK(hipMemcpy(&v, err_ptr(c), sizeof(v), hipMemcpyDeviceToHost));
  *mismatches = (uint32_t)v;
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

const char* vfl_last_error(const vfl_ctx* c) { return c ? c->err.c_str() : "null context"; }

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
    if (c->gexec[q]) (void)hipGraphExecDestroy(c->gexec[q]);
    if (c->graph[q]) (void)hipGraphDestroy(c->graph[q]);
    for (auto& gp : c->gpairs[q]) {
      (void)hipEventDestroy(gp.e0);
      (void)hipEventDestroy(gp.e1);
    }
  }
  if (c->ev_fork) (void)hipEventDestroy(c->ev_fork);
  if (c->ev_join) (void)hipEventDestroy(c->ev_join);
  delete c;
  return r;
}

}  // extern "C"
