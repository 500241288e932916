/*
 * sagc.h -- C ABI of the straggler-aware group-size controller in
 * librollout.so (paper Sec. 4, Algorithm 1 "SAGC").
 *
 * The controller picks the group size G of the next rollout from the sizes a
 * caller admits.  After each rollout the GPU reduces every group's completion
 * lengths to (l_max, l_median, R = l_max / l_median, S = [R > tau])
 * (Sec. 3.1, Eq. ratio and Eq. event; Sec. 4.4: only these summaries leave
 * the GPU).  The host step then
 *   - averages S over the completed groups (S_bar),
 *   - takes a projected dual-ascent step on lambda (Sec. 4.2, Eq. lambda_update),
 *   - discounts and updates the Beta posterior of the size just used
 *     (Sec. 4.3; every size starts at Beta(1, 1)),
 *   - draws one straggler probability per size from its posterior (Thompson
 *     sampling) and scores log2(G) - lambda * p (Eq. lagrangian_score),
 *   - moves to the best-scoring size among the current one and its two
 *     neighbours in the admitted list, ties going to the smaller size.
 * G_0 is drawn at random from the admitted sizes.
 *
 * Randomness: every draw comes from Philox4x64-10 with key (seed, 2) and
 * counter (step, stream, attempt, 0); a 64-bit word w is the double
 * ((w >> 11) + 0.5) * 2^-53.  Gamma variates follow Marsaglia and Tsang
 * (2000) with Box-Muller normals (attempt words 0 and 1) and the acceptance
 * uniform in word 2; shapes below one are boosted, Gamma(a + 1) * U^(1/a),
 * with U from word 3 of attempt 0.  Beta(a, b) = X / (X + Y), X on stream 2k
 * and Y on stream 2k + 1 for size index k.  G_0 takes word 0 of counter
 * (2^63, 0, 0, 0).  The paper fixes no generator; this one makes every run
 * reproducible from the seed.
 *
 * Status codes and rg_last_error() are those of rollout.h.  Host pointers are
 * read before the call returns; device pointers are HIP device memory.
 */
#ifndef PAPER_2606_02218_SAGC_H
#define PAPER_2606_02218_SAGC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SAGC_MAX_SIZES 8

typedef struct sagc_config {
  int32_t n_sizes;                /* admitted group sizes: 1 .. SAGC_MAX_SIZES              */
  int32_t sizes[SAGC_MAX_SIZES];  /* strictly increasing, each >= 2                         */
  double tau;                     /* straggler threshold on R, > 1 (Eq. event)              */
  double delta;                   /* target straggler rate, in (0, 1)                       */
  double eta;                     /* dual step size, > 0 (Eq. lambda_update)               */
  double gamma;                   /* posterior forgetting factor, in (0, 1]                 */
  uint64_t seed;                  /* Thompson-sampling and G_0 stream                       */
} sagc_config;

/* Controller state: plain data, caller-owned (it can be copied, saved and
 * restored to resume a run). */
typedef struct sagc_state {
  double lambda;                        /* dual variable, >= 0                              */
  double alpha[SAGC_MAX_SIZES];         /* Beta posterior per size                          */
  double beta[SAGC_MAX_SIZES];
  int32_t g_index;                      /* index of the current G in sizes[]                */
  int32_t reserved;
  int64_t step;                         /* controller steps taken                           */
  double last_rate;                     /* S_bar of the last step                           */
  double last_sample[SAGC_MAX_SIZES];   /* p~ drawn in the last step                        */
  double last_score[SAGC_MAX_SIZES];    /* log2(G) - lambda * p~ of the last step           */
} sagc_state;

/* Validate cfg and initialise st: lambda = 0, alpha = beta = 1, G_0 from the
 * seed.  RG_EINVAL on an invalid config. */
int sagc_init(const sagc_config* cfg, sagc_state* st);

/* Per-group length summaries of one rollout.  lengths: device int32 [N],
 * prompt-major (group p holds entries sum(G[0..p-1]) ..); G: device int32
 * [P], 1 <= G[p] <= 1024 and sum(G) <= N.  stats: device float [P][4] =
 * (l_max, l_median, R, S) with the median of an even group the mean of its
 * two middle lengths, R = l_max / l_median and S = 1 if R > tau (R compared
 * in double precision) else 0.  A group that breaks the bounds above, or has
 * a zero median, gets NaN in all four.  Asynchronous on `stream`. */
int sagc_group_stats(const int32_t* lengths, const int32_t* G, int32_t P, int32_t N, double tau,
                     float* stats, void* stream);

/* One controller step after a rollout run with G = sizes[st->g_index]:
 * stats is HOST float [n_groups][4] as written by sagc_group_stats (only S,
 * column 3, is used), n_groups >= 1.  Updates st and writes the next group
 * size to *g_next.  RG_EINVAL on a bad argument or a non-finite S. */
int sagc_step(const sagc_config* cfg, sagc_state* st, const float* stats, int32_t n_groups,
              int32_t* g_next);

/* Test hook: the Beta(a, b) variate drawn for size index `arm` at controller
 * step `step` of a run seeded with `seed` (a, b > 0). */
int sagc_beta_draw(uint64_t seed, int64_t step, int32_t arm, double a, double b, double* out);

#ifdef __cplusplus
}
#endif
#endif /* PAPER_2606_02218_SAGC_H */
