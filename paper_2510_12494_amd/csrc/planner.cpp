// Configuration planner of the system-planning phase (Section 4.3 "System Planning Phase",
// Algorithm 2): host code only.
//
// Per candidate (workers w_a of party A, workers w_p of party B, batch size
// B) the per-iteration delay is
//   max(T_A, T_P) + (E + G) / B_b,
//   T_A = (lambda_a B^gamma_a + phi_a B^beta_a + lambda'_a B^gamma'_a
//          + phi'_a B^beta'_a) w_a / C_a        (Eqs. 7-9),
//   T_P = (lambda_p B^gamma_p + phi_p B^beta_p) w_p / C_p,
// with the exchanged embedding and gradient E, G proportional to B (per-row
// messages); candidates with B above B_max (the memory model
// M(B) = M0 + rho B^chi per worker against each party's cap) are not
// feasible.  Algorithm 2 fills its table over every feasible (w_a, w_p, B),
// so the search below is that enumeration: batch sizes in the caller's
// order, then w_a, then w_p, keeping the first strict minimum.
//
// The delay constants are fitted from measured times over a batch-size
// sweep (the Appendix's Table 7 lists the paper's): vfl_fit_delay fits one
// power law coef * B^exp by least squares in log space.
#include <cmath>
#include <limits>

#include "../../include/vfl.h"

namespace {

double party_delay(const vfl_plan_party& q, double B, int w) {
  const double t = q.lambda * std::pow(B, q.gamma) + q.phi * std::pow(B, q.beta) +
                   q.lambda_top * std::pow(B, q.gamma_top) + q.phi_top * std::pow(B, q.beta_top);
  return t * w / q.cores;
}

// largest batch the party's memory model allows (infinite without a cap)
double batch_cap(const vfl_plan_party& q, double chi) {
  if (!(q.mem_coef > 0.0)) return std::numeric_limits<double>::infinity();
  const double room = q.mem_cap - q.mem_base;
  if (room <= 0.0) return 0.0;
  return std::pow(room / q.mem_coef, 1.0 / chi);
}

bool valid(const vfl_plan_party* q) {
  return q && q->cores > 0.0 && q->w_min >= 1 && q->w_max >= q->w_min;
}

}  // namespace

extern "C" {

vfl_status vfl_plan(const vfl_plan_party* a, const vfl_plan_party* p, const vfl_plan_link* link,
                    const int32_t* batches, int32_t n_batches, int32_t out[3], double* cost) {
  if (!valid(a) || !valid(p) || !link || !batches || n_batches < 1 || !out || !(link->bandwidth > 0.0) ||
      !(link->chi > 0.0))
    return VFL_E_INVALID;
  const double bmax = std::fmin(batch_cap(*a, link->chi), batch_cap(*p, link->chi));
  double best = std::numeric_limits<double>::infinity();
  int32_t arg[3] = {0, 0, 0};
  for (int32_t r = 0; r < n_batches; ++r) {
    const double B = batches[r];
    if (batches[r] < 1 || B > bmax) continue;
    const double comm = B * (link->emb_bytes_per_row + link->grad_bytes_per_row) / link->bandwidth;
    for (int32_t wa = a->w_min; wa <= a->w_max; ++wa) {
      const double ta = party_delay(*a, B, wa);
      for (int32_t wp = p->w_min; wp <= p->w_max; ++wp) {
        const double o = std::fmax(ta, party_delay(*p, B, wp)) + comm;
        if (o < best) {
          best = o;
          arg[0] = wa; arg[1] = wp; arg[2] = batches[r];
        }
      }
    }
  }
  if (!(best < std::numeric_limits<double>::infinity())) return VFL_E_INVALID;   // nothing feasible
  out[0] = arg[0]; out[1] = arg[1]; out[2] = arg[2];
  if (cost) *cost = best;
  return VFL_OK;
}

vfl_status vfl_fit_delay(const double* batch, const double* seconds, int32_t n, double* coef,
                         double* expo) {
  if (!batch || !seconds || !coef || !expo || n < 2) return VFL_E_INVALID;
  // ordinary least squares of log T on log B (centred sums)
  double mx = 0.0, my = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    if (!(batch[i] > 0.0) || !(seconds[i] > 0.0) || !std::isfinite(batch[i]) || !std::isfinite(seconds[i]))
      return VFL_E_INVALID;
    mx += std::log(batch[i]);
    my += std::log(seconds[i]);
  }
  mx /= n;
  my /= n;
  double sxx = 0.0, sxy = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    const double dx = std::log(batch[i]) - mx;
    sxx += dx * dx;
    sxy += dx * (std::log(seconds[i]) - my);
  }
  if (!(sxx > 0.0)) return VFL_E_INVALID;   // a single distinct batch size
  *expo = sxy / sxx;
  *coef = std::exp(my - *expo * mx);
  return VFL_OK;
}

}  // extern "C"
