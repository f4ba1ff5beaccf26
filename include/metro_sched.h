/* metro_sched.h -- out-of-order agent scheduler (host C ABI of libmetro.so).
 *
 * The controller of an agent simulation run out of order (AI Metropolis,
 * §3.1-§3.4, Algorithm 3): agents on a 2-D world advance in steps; an agent
 * may run ahead of others as long as the spatio-temporal dependency rules of
 * §3.3 allow, coupled agents proceed together as a cluster (§3.4), and ready
 * clusters are handed out lowest step first (§3.5).  The library keeps the
 * dependency state; the caller runs the clusters (the "workers": the agents'
 * LLM calls through metro.h) and reports their completion with the agents'
 * new positions.
 *
 * Rules (§3.3; the appendix derives them from the validity condition that
 * any two agents at different steps s_A != s_B keep
 * dist(A, B) > radius_p + (|s_A - s_B| - 1) * max_vel):
 *   coupled(A, B):  s_A == s_B and dist(A, B) <= radius_p + max_vel
 *   blocked(A by B): s_B < s_A and dist(A, B) <= (s_A - s_B + 1) * max_vel + radius_p
 * A cluster is a connected component of the coupled relation among the
 * agents waiting at one step; it is ready when none of its members is
 * blocked.  An agent's step counts the steps it has completed.
 *
 * Thread safety: a scheduler is used by one thread at a time.  Errors return
 * a negative metro_status (metro.h); metro_last_error() describes the last.
 */
#ifndef METRO_SCHED_H
#define METRO_SCHED_H

#include <stdint.h>

#include "metro.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct metro_sched metro_sched;

typedef enum {
  METRO_DIST_CHEBYSHEV = 0, /* max(|dx|, |dy|): the square perception area of a grid world */
  METRO_DIST_EUCLIDEAN = 1  /* sqrt(dx^2 + dy^2) */
} metro_dist_metric;

typedef struct {
  int32_t n_agents;     /* > 0 */
  float radius_p;       /* perception radius, >= 0 (4 grid units in the paper's world, §3.3) */
  float max_vel;        /* largest move per step, >= 0 (1 grid unit) */
  int32_t metric;       /* metro_dist_metric */
  int32_t target_step;  /* agents stop after completing this many steps, > 0 */
  int32_t sync;         /* 0: out of order (Algorithm 3); 1: parallel-sync baseline (Algorithm 1): all
                           agents form one cluster per step, released once every agent has finished the
                           step before */
} metro_sched_config;

/* Create a scheduler for cfg->n_agents agents at step 0 at positions
 * xy[2*i], xy[2*i+1] (host array, copied).  Errors: METRO_E_INVAL for a bad
 * config or NULL argument, METRO_E_NOMEM. */
metro_status metro_sched_create(const metro_sched_config* cfg, const int32_t* xy, metro_sched** out);

void metro_sched_destroy(metro_sched* s);

/* Hand out the next ready cluster, lowest step first, then lowest agent id
 * (§3.5: the ready queue is a priority queue on the step).  Its members (in
 * increasing id) go to agents[0 .. *n_out), at most cap of them; *step is the
 * step they are about to run, *cluster an id for metro_sched_ack.  With no
 * ready cluster *n_out = 0 and *cluster = -1.  The members are running until
 * their cluster is acknowledged.  Errors: METRO_E_INVAL (NULL argument),
 * METRO_E_CAPACITY when the cluster has more than cap members (nothing is
 * handed out). */
metro_status metro_sched_next(metro_sched* s, int32_t* cluster, int32_t* step, int32_t* agents, int32_t cap,
                              int32_t* n_out);

/* Completion of a handed-out cluster: every member has finished its step and
 * moved to xy[2*j], xy[2*j+1] (j in the order metro_sched_next returned
 * them).  Errors: METRO_E_INVAL for an unknown or finished cluster, or for a
 * move longer than max_vel (the rules hold only for bounded moves). */
metro_status metro_sched_ack(metro_sched* s, int32_t cluster, const int32_t* xy);

/* Snapshot: steps[i] (completed steps), xy[2i..2i+1], state[i] (0 waiting,
 * 1 running, 2 done at target_step); any pointer may be NULL.  *running =
 * running clusters; *done = 1 once every agent has reached target_step. */
metro_status metro_sched_state(const metro_sched* s, int32_t* steps, int32_t* xy, int32_t* state,
                               int32_t* running, int32_t* done);

#ifdef __cplusplus
}
#endif

#endif /* METRO_SCHED_H */
