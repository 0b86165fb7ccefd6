// Test infrastructure: drives the library's host-only logic under the host
// address and undefined-behaviour sanitizers (built by
// tests/test_host_sanitizers.py with the kernel launches stubbed out).  It
// never creates a context, so no call reaches a GPU: configuration plans
// and job layouts for random and malformed specs (vfl_workspace_size), the
// tick schedule, the planner, the delay fit, the interval of Eq. 5, and the
// argument checks of every entry point on null or invalid input.  Exits 0
// after printing "host checks passed"; a sanitizer report aborts it.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <random>

#include "../../include/vfl.h"

namespace {

std::mt19937_64 rng(20260);

int uni(int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); }
double unif(double lo, double hi) { return std::uniform_real_distribution<double>(lo, hi)(rng); }

void random_bottom(vfl_bottom_spec& s, bool wild) {
  std::memset(&s, 0, sizeof(s));
  s.n_cat = uni(0, 1) ? uni(0, 4) : 0;
  s.vocab = s.n_cat ? uni(1, 5000) : 0;
  s.emb_dim = s.n_cat ? 4 * uni(1, 4) : 0;
  s.dense_in = uni(s.n_cat ? 0 : 1, 600);
  s.n_layers = uni(1, wild ? VFL_MAX_LAYERS + 2 : 6);
  for (int l = 0; l < VFL_MAX_LAYERS; ++l) s.widths[l] = uni(1, l == 0 ? 1100 : 520);
  // the cut layer (the published embedding) is a multiple of 8 wide unless wild
  if (s.n_layers >= 1 && s.n_layers <= VFL_MAX_LAYERS && !(wild && uni(0, 3) == 0))
    s.widths[s.n_layers - 1] = 8 * uni(1, 32);
  s.relu_mask = (uint32_t)rng();
  if (wild) {
    switch (uni(0, 6)) {
      case 0: s.dense_in = -uni(1, 5); break;
      case 1: s.widths[uni(0, VFL_MAX_LAYERS - 1)] = uni(-3, 0); break;
      case 2: s.vocab = uni(-2, 0); break;
      case 3: s.emb_dim = uni(17, 70); break;
      case 4: s.n_layers = uni(-1, 0); break;
      default: break;
    }
  }
}

void random_top(vfl_top_spec& t, bool wild) {
  std::memset(&t, 0, sizeof(t));
  t.n_layers = uni(2, wild ? VFL_MAX_LAYERS + 2 : 5);
  for (int j = 0; j < VFL_MAX_LAYERS; ++j) t.widths[j] = uni(1, 520);
  if (t.n_layers >= 1 && t.n_layers <= VFL_MAX_LAYERS) t.widths[t.n_layers - 1] = wild && uni(0, 3) == 0 ? 2 : 1;
  t.relu_mask = (uint32_t)rng();
}

void random_opts(vfl_opts& o, bool wild) {
  std::memset(&o, 0, sizeof(o));
  o.dtype = uni(0, 1) ? VFL_BF16 : VFL_F32;
  o.batch = uni(1, 20000);
  o.staleness = uni(0, VFL_MAX_STALENESS);
  o.replicas = uni(1, VFL_MAX_REPLICAS);
  o.lr = (float)unif(1e-4, 1.0);
  o.clip_c = uni(0, 1) ? (float)unif(0.1, 3.0) : 0.f;
  o.sigma = uni(0, 1) ? (float)unif(0.0, 1.0) : 0.f;
  o.seed = rng();
  o.flags = (uint32_t)uni(0, 63);
  if (o.clip_c <= 0.f && !(wild && uni(0, 3) == 0)) o.flags &= ~(uint32_t)(VFL_CLIP_EMB | VFL_CLIP_GRAD);
  if (wild) {
    switch (uni(0, 5)) {
      case 0: o.batch = uni(-5, 0); break;
      case 1: o.staleness = uni(VFL_MAX_STALENESS + 1, 40); break;
      case 2: o.replicas = uni(VFL_MAX_REPLICAS + 1, 64); break;
      case 3: o.dtype = (vfl_dtype)uni(2, 9); break;
      case 4: o.flags |= 1u << uni(6, 31); break;
      default: break;
    }
  }
}

int fails = 0;
void expect(bool ok, const char* what) {
  if (!ok) {
    std::printf("FAILED: %s\n", what);
    ++fails;
  }
}

}  // namespace

int main() {
  // 1. plans and job layouts
  int ok = 0, refused = 0;
  for (int it = 0; it < 4000; ++it) {
    const bool wild = it % 3 == 0;
    vfl_bottom_spec a, b;
    vfl_top_spec t;
    vfl_opts o;
    random_bottom(a, wild);
    random_bottom(b, wild && uni(0, 1));
    random_top(t, wild && uni(0, 1));
    random_opts(o, wild && uni(0, 1));
    size_t bytes = 0;
    const vfl_status st = vfl_workspace_size(&a, &b, &t, &o, &bytes);
    if (st == VFL_OK) {
      ++ok;
      expect(bytes > 0 && bytes % 256 == 0, "workspace size positive and 256-byte granular");
    } else {
      ++refused;
      const char* why = vfl_last_error(nullptr);
      expect(why && std::strlen(why) > 0, "a refused plan names its reason");
    }
  }
  std::printf("accepted %d refused %d\n", ok, refused);
  expect(ok > 500 && refused > 200, "both accepted and refused configurations were exercised");

  // 2. null and invalid arguments (no context is ever created)
  {
    vfl_bottom_spec a, b;
    vfl_top_spec t;
    vfl_opts o;
    random_bottom(a, false);
    random_bottom(b, false);
    random_top(t, false);
    random_opts(o, false);
    size_t bytes = 0;
    expect(vfl_workspace_size(nullptr, &b, &t, &o, &bytes) != VFL_OK, "null spec refused");
    expect(vfl_workspace_size(&a, &b, &t, &o, nullptr) != VFL_OK, "null size refused");
    vfl_ctx* c = nullptr;
    expect(vfl_create(&a, &b, &t, &o, nullptr, 1 << 20, nullptr, nullptr, &c) != VFL_OK && !c,
           "null workspace refused");
    alignas(256) static char fake[512];
    expect(vfl_create(&a, &b, &t, &o, fake + 16, sizeof(fake), nullptr, nullptr, &c) != VFL_OK && !c,
           "misaligned workspace refused");
    expect(vfl_create(&a, &b, &t, &o, fake, 1, nullptr, nullptr, &c) != VFL_OK && !c,
           "short workspace refused");
    expect(vfl_create(&a, &b, &t, &o, fake, sizeof(fake), nullptr, nullptr, nullptr) != VFL_OK,
           "null out refused");
    expect(vfl_create_static(nullptr, &b, &t, &o, nullptr, nullptr, &c) != VFL_OK && !c,
           "static create with a null spec refused");
    expect(vfl_destroy(nullptr) == VFL_E_INVALID, "destroy(null)");
    expect(vfl_step(nullptr, 0, nullptr, 0, nullptr, 0, nullptr) == VFL_E_INVALID, "step(null)");
    expect(vfl_run(nullptr, 1, 1, nullptr, 0) == VFL_E_INVALID, "run(null)");
    expect(vfl_publish(nullptr, 0) == VFL_E_INVALID, "publish(null)");
    expect(vfl_top_step(nullptr, 0, nullptr) == VFL_E_INVALID, "top_step(null)");
    expect(vfl_bottom_forward(nullptr, VFL_PARTY_B, 0, nullptr, 0) == VFL_E_INVALID, "forward(null)");
    expect(vfl_bottom_backward(nullptr, VFL_PARTY_B, 0) == VFL_E_INVALID, "backward(null)");
    expect(vfl_discard(nullptr, 0) == VFL_E_INVALID, "discard(null)");
    size_t n = 0;
    expect(vfl_state_size(nullptr, &n) == VFL_E_INVALID, "state_size(null)");
    expect(vfl_get_state(nullptr, fake, sizeof(fake)) == VFL_E_INVALID, "get_state(null)");
    expect(vfl_set_state(nullptr, fake, sizeof(fake)) == VFL_E_INVALID, "set_state(null)");
    expect(vfl_replica_average(nullptr, 2, 3) == VFL_E_INVALID, "replica_average(null)");
    vfl_ctx* none[2] = {nullptr, nullptr};
    expect(vfl_replica_average(none, 2, 3) == VFL_E_INVALID, "replica_average(null contexts)");
    expect(vfl_replica_average(none, 0, 3) == VFL_E_INVALID, "replica_average(n = 0)");
    expect(vfl_last_error(nullptr) != nullptr, "last_error(null) is a string");
  }

  // 3. the tick schedule against its closed form
  for (int s = 0; s <= VFL_MAX_STALENESS; ++s)
    for (int64_t ng = 0; ng < 40; ng += 7)
      for (int64_t t = 0; t < 60; ++t) {
        int64_t row[7];
        expect(vfl_schedule_tick(t, s, ng, row) == VFL_OK, "schedule tick");
        const int64_t u = t - s;
        expect(row[1] == (t < ng ? t : -1), "published group");
        expect(row[4] == (u >= 0 && u < ng ? u : -1), "consumed group");
        if (row[1] >= 0) expect(row[3] == (t - s > 0 ? t - s : 0), "forward version");
      }
  int64_t row[7];
  expect(vfl_schedule_tick(-1, 0, 1, row) != VFL_OK, "negative tick refused");
  expect(vfl_schedule_tick(0, VFL_MAX_STALENESS + 1, 1, row) != VFL_OK, "staleness bound");
  expect(vfl_schedule_tick(0, 0, 1, nullptr) != VFL_OK, "null row refused");

  // 4. the planner and the delay fit
  for (int it = 0; it < 300; ++it) {
    vfl_plan_party a, p;
    std::memset(&a, 0, sizeof(a));
    std::memset(&p, 0, sizeof(p));
    for (vfl_plan_party* q : {&a, &p}) {
      q->lambda = unif(1e-5, 1e-2);
      q->gamma = unif(-1.0, 1.2);
      q->phi = unif(1e-5, 1e-2);
      q->beta = unif(-1.0, 1.2);
      q->cores = unif(1.0, 64.0);
      q->w_min = uni(1, 4);
      q->w_max = q->w_min + uni(0, 6);
      q->mem_base = unif(0.0, 1e9);
      q->mem_coef = uni(0, 1) ? unif(1e3, 1e6) : 0.0;
      q->mem_cap = unif(1e9, 1e11);
    }
    a.lambda_top = unif(0.0, 1e-3);
    a.gamma_top = unif(0.0, 1.0);
    vfl_plan_link link{unif(0.0, 1e3), unif(0.0, 1e3), unif(1e8, 1e11), unif(0.5, 1.5)};
    int32_t batches[9];
    const int nb = uni(1, 9);
    for (int i = 0; i < nb; ++i) batches[i] = 16 << uni(0, 10);
    int32_t out[3];
    double cost = 0;
    const vfl_status st = vfl_plan(&a, &p, &link, batches, nb, out, &cost);
    if (st == VFL_OK) expect(std::isfinite(cost) && out[2] > 0, "plan feasible and finite");
  }
  {
    int32_t out[3];
    vfl_plan_link link{1, 1, 1, 1};
    expect(vfl_plan(nullptr, nullptr, &link, nullptr, 0, out, nullptr) != VFL_OK, "plan(null)");
    double xb[5] = {256, 512, 1024, 2048, 4096}, yt[5], coef = 0, ex = 0;
    for (int i = 0; i < 5; ++i) yt[i] = 3e-4 * std::pow(xb[i], -0.7);
    expect(vfl_fit_delay(xb, yt, 5, &coef, &ex) == VFL_OK && std::fabs(ex + 0.7) < 1e-9,
           "fit recovers a power law");
    expect(vfl_fit_delay(xb, yt, 1, &coef, &ex) != VFL_OK, "fit needs two points");
    yt[2] = -1.0;
    expect(vfl_fit_delay(xb, yt, 5, &coef, &ex) != VFL_OK, "fit refuses non-positive delays");
  }

  // 5. the interval of Eq. 5
  for (int dt0 = 1; dt0 <= 64; ++dt0)
    for (int64_t t = 0; t < 400; ++t) {
      int32_t dt = 0;
      expect(vfl_sync_interval(dt0, t, &dt) == VFL_OK && dt >= 1 && dt <= dt0, "interval in [1, dt0]");
    }
  int32_t dt;
  expect(vfl_sync_interval(0, 1, &dt) != VFL_OK, "dt0 = 0 refused");
  expect(vfl_sync_interval(5, -1, &dt) != VFL_OK, "negative unit refused");
  expect(vfl_sync_interval(5, 1, nullptr) != VFL_OK, "null output refused");

  if (fails) {
    std::printf("%d host checks failed\n", fails);
    return 1;
  }
  std::printf("host checks passed (%d plans accepted, %d refused)\n", ok, refused);
  return 0;
}
