// Deterministic tick schedule of the publisher/subscriber loop (pure host
// code).  Tick t: B publishes group t while t < n_groups; A consumes group
// u = t - s and B back-propagates it.  Channel slot of group g: g mod (s+1);
// B's forward of group g runs at version max(0, g - s); the update made
// with group u is applied at tick u + s (delay min(u, s)).  Batch groups
// are keyed by id as the paper's channels are (Section 4.1), and s + 1 <= 5
// slots matches its buffer capacity p = q = 5.
#include <cmath>

#include "../../include/vfl.h"

extern "C" vfl_status vfl_schedule_tick(int64_t t, int32_t s, int64_t n_groups, int64_t out[7]) {
  if (!out || t < 0 || s < 0 || s > VFL_MAX_STALENESS || n_groups < 0) return VFL_E_INVALID;
  const int64_t fwd = t < n_groups ? t : -1;
  const int64_t u = t - s;
  const int64_t bwd = (u >= 0 && u < n_groups) ? u : -1;
  out[0] = t;
  out[1] = fwd;
  out[2] = fwd >= 0 ? fwd % (s + 1) : -1;
  out[3] = fwd >= 0 ? (fwd - s > 0 ? fwd - s : 0) : -1;
  out[4] = bwd;
  out[5] = bwd >= 0 ? bwd % (s + 1) : -1;
  out[6] = bwd >= 0 ? bwd + 1 : -1;
  return VFL_OK;
}

// Synchronisation interval of the intra-party semi-asynchronous mechanism
// (Section 4.1, Eq. 5) for unit t (an epoch in Algorithm 1): the ceiling of
// dt0/2 * tanh(2t/dt0 - 2) + dt0/2, which lies in [1, dt0].
extern "C" vfl_status vfl_sync_interval(int32_t dt0, int64_t t, int32_t* dt) {
  if (!dt || dt0 < 1 || t < 0) return VFL_E_INVALID;
  const double h = 0.5 * dt0;
  const double v = h * std::tanh(2.0 * (double)t / dt0 - 2.0) + h;
  int64_t c = (int64_t)std::ceil(v);
  if (c < 1) c = 1;
  if (c > dt0) c = dt0;
  *dt = (int32_t)c;
  return VFL_OK;
}
