// Straggler-aware group-size control (SAGC, Algorithm 1): the host-side
// controller and the launcher of the per-group length statistics.  See
// include/sagc.h for the exact update rule and random stream.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <string>

#include "../../include/rollout.h"
#include "../../include/sagc.h"
#include "rg_kernels.h"

// Plain double arithmetic in the written order: no contraction into FMAs, so
// the controller's choices are reproducible bit for bit.
#pragma STDC FP_CONTRACT OFF
#pragma clang fp contract(off)

int rg_set_error(int code, const char* msg);

namespace {

constexpr uint64_t kTagSagc = 2;

struct Words { uint64_t w[4]; };

// Philox4x64-10 (Salmon et al., SC'11) on the host.
Words philox(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3, uint64_t k0, uint64_t k1) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
  for (int r = 0; r < 10; ++r) {
    if (r > 0) { k0 += W0; k1 += W1; }
    const unsigned __int128 p0 = (unsigned __int128)M0 * c0, p1 = (unsigned __int128)M1 * c2;
    const uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
    const uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    const uint64_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  return Words{{c0, c1, c2, c3}};
}

double u53(uint64_t w) { return ((double)(w >> 11) + 0.5) * 0x1p-53; }

// Gamma(a, 1), Marsaglia-Tsang, on stream (step, stream).
double gamma_draw(uint64_t seed, uint64_t step, uint64_t stream, double a) {
  const bool boost = a < 1.0;
  const double shape = boost ? a + 1.0 : a;
  const double d = shape - 1.0 / 3.0;
  const double c = 1.0 / std::sqrt(9.0 * d);
  double g = 0.0, boost_u = 0.0;
  for (uint64_t attempt = 0;; ++attempt) {
    const Words w = philox(step, stream, attempt, 0, seed, kTagSagc);
    if (attempt == 0) boost_u = u53(w.w[3]);
    const double x = std::sqrt(-2.0 * std::log(u53(w.w[0]))) * std::cos(2.0 * M_PI * u53(w.w[1]));
    const double t = 1.0 + c * x;
    if (t <= 0.0) continue;
    const double v = t * t * t;
    if (std::log(u53(w.w[2])) < 0.5 * x * x + d - d * v + d * std::log(v)) {
      g = d * v;
      break;
    }
  }
  if (boost) g = g * std::pow(boost_u, 1.0 / a);
  return g;
}

double beta_draw(uint64_t seed, uint64_t step, int arm, double a, double b) {
  const double x = gamma_draw(seed, step, 2 * (uint64_t)arm, a);
  const double y = gamma_draw(seed, step, 2 * (uint64_t)arm + 1, b);
  return x / (x + y);
}

int check_config(const sagc_config* c) {
  if (!c) return rg_set_error(RG_EINVAL, "sagc: NULL config");
  if (c->n_sizes < 1 || c->n_sizes > SAGC_MAX_SIZES) return rg_set_error(RG_EINVAL, "sagc: n_sizes out of [1, 8]");
  for (int i = 0; i < c->n_sizes; ++i)
    if (c->sizes[i] < 2 || (i > 0 && c->sizes[i] <= c->sizes[i - 1]))
      return rg_set_error(RG_EINVAL, "sagc: sizes must be >= 2 and strictly increasing");
  if (!(c->tau > 1.0) || !(c->delta > 0.0 && c->delta < 1.0) || !(c->eta > 0.0) ||
      !(c->gamma > 0.0 && c->gamma <= 1.0) || !std::isfinite(c->tau) || !std::isfinite(c->eta))
    return rg_set_error(RG_EINVAL, "sagc: need tau > 1, 0 < delta < 1, eta > 0, 0 < gamma <= 1");
  return RG_OK;
}

}  // namespace

extern "C" {

int sagc_init(const sagc_config* cfg, sagc_state* st) {
  int rc = check_config(cfg);
  if (rc) return rc;
  if (!st) return rg_set_error(RG_EINVAL, "sagc_init: NULL state");
  std::memset(st, 0, sizeof(*st));
  for (int i = 0; i < SAGC_MAX_SIZES; ++i) st->alpha[i] = st->beta[i] = 1.0;
  const Words w = philox(1ull << 63, 0, 0, 0, cfg->seed, kTagSagc);
  const int g0 = (int)(u53(w.w[0]) * (double)cfg->n_sizes);
  st->g_index = g0 < cfg->n_sizes ? g0 : cfg->n_sizes - 1;
  return RG_OK;
}

int sagc_step(const sagc_config* cfg, sagc_state* st, const float* stats, int32_t n_groups, int32_t* g_next) {
  int rc = check_config(cfg);
  if (rc) return rc;
  if (!st || !stats || !g_next || n_groups < 1) return rg_set_error(RG_EINVAL, "sagc_step: bad argument");
  if (st->g_index < 0 || st->g_index >= cfg->n_sizes || !(st->lambda >= 0.0))
    return rg_set_error(RG_EINVAL, "sagc_step: state does not match the config");
  const int k = cfg->n_sizes;
  double s_sum = 0.0;
  for (int i = 0; i < n_groups; ++i) {
    const double s = stats[4 * i + 3];
    if (!std::isfinite(s)) return rg_set_error(RG_EINVAL, "sagc_step: non-finite straggler event");
    s_sum += s;
  }
  const double s_bar = s_sum / (double)n_groups;
  // projected dual ascent, then the discounted posterior of the size just used
  const double lam = st->lambda + cfg->eta * (s_bar - cfg->delta);
  st->lambda = lam > 0.0 ? lam : 0.0;
  const int cur = st->g_index;
  st->alpha[cur] = cfg->gamma * st->alpha[cur] + s_bar;
  st->beta[cur] = cfg->gamma * st->beta[cur] + (1.0 - s_bar);
  // Thompson sample and score every size, move within the neighbourhood
  for (int a = 0; a < k; ++a) {
    st->last_sample[a] = beta_draw(cfg->seed, (uint64_t)st->step, a, st->alpha[a], st->beta[a]);
    st->last_score[a] = std::log2((double)cfg->sizes[a]) - st->lambda * st->last_sample[a];
  }
  int best = -1;
  for (int i = cur - 1; i <= cur + 1; ++i)   // ascending size: a strict > keeps the smaller on ties
    if (i >= 0 && i < k && (best < 0 || st->last_score[i] > st->last_score[best])) best = i;
  st->g_index = best;
  st->step += 1;
  st->last_rate = s_bar;
  *g_next = cfg->sizes[best];
  return RG_OK;
}

int sagc_beta_draw(uint64_t seed, int64_t step, int32_t arm, double a, double b, double* out) {
  if (!out || step < 0 || arm < 0 || !(a > 0.0) || !(b > 0.0) || !std::isfinite(a) || !std::isfinite(b))
    return rg_set_error(RG_EINVAL, "sagc_beta_draw: bad argument");
  *out = beta_draw(seed, (uint64_t)step, arm, a, b);
  return RG_OK;
}

int sagc_group_stats(const int32_t* lengths, const int32_t* G, int32_t P, int32_t N, double tau, float* stats,
                     void* stream) {
  if (!lengths || !G || !stats || P < 1 || N < 1 || !(tau > 0.0))
    return rg_set_error(RG_EINVAL, "sagc_group_stats: bad argument");
  const hipError_t e = launch_group_stats(lengths, G, P, N, tau, stats, (hipStream_t)stream);
  if (e != hipSuccess) return rg_set_error(RG_EHIP, (std::string("sagc_group_stats: ") + hipGetErrorString(e)).c_str());
  return RG_OK;
}

}  // extern "C"
