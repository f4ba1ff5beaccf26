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

/* ---------------------------------------------------------------------------
 * Mixed continuous batching of the agents' LLM requests: the serving loop
 * between the scheduler above and the model of metro.h.
 *
 * Each request carries the step of the agent that issued it (§3.5: every
 * request includes a step count, and smaller counts run first).  One
 * metro_engine_step runs one forward pass holding
 *   1. the next token of every running request (prompt done, outputs left):
 *      a one-token item each, lowest step first when more than max_items run
 *      (a request is never preempted mid-generation, §3.5);
 *   2. in the token budget left (max_tokens minus those tokens), prompt chunks
 *      of at most `chunk` tokens of waiting requests, admitted lowest step
 *      first, ties by submission order (priority = 1), or in submission order
 *      alone (priority = 0), until max_items items or the budget is used; a
 *      request's last chunk yields its first output token.
 * So prompt prefill and decode share each pass over the weights (chunked
 * prefill mixed with decode, the prior art cited in §5).  A forward with no
 * prompt chunk runs metro_decode_step, otherwise metro_prefill_chunk.  After
 * the forward the engine waits for the greedy tokens on `stream`, appends
 * them to their requests and retires those that have all n_out tokens (their
 * sequences are closed).
 *
 * With model == NULL the engine only plans: metro_engine_step forms the items
 * as above and appends stand-in tokens without device work (for checking the
 * admission rules on a host without a GPU).
 * When the KV pool cannot hold the pages of a forward (the model's call
 * returns METRO_E_NOPAGES and changes nothing), the step is planned again with
 * half the prompt tokens, down to a decode-only forward; only when no forward
 * fits does metro_engine_step return METRO_E_NOPAGES (no request's state
 * changes; retry once requests have retired or others are closed).
 * Errors: METRO_E_INVAL (NULL, bad sizes, a live request id), METRO_E_SEQ
 * (unknown request), METRO_E_NOMEM, METRO_E_NOPAGES as above, and whatever
 * else the model calls return. */
typedef struct metro_engine metro_engine;

typedef struct {
  int32_t max_tokens; /* tokens of one forward (decode tokens + prompt chunks), <= the model's max_tokens */
  int32_t chunk;      /* prompt tokens of one request per forward */
  int32_t max_items;  /* requests in one forward, <= the model's max_batch */
  int32_t priority;   /* 1: lowest step first (§3.5); 0: submission order */
} metro_engine_config;

typedef struct {
  int64_t forwards;      /* forward passes run */
  int64_t items;         /* items over all forwards */
  int64_t prompt_tokens; /* prompt tokens prefilled */
  int64_t decode_tokens; /* one-token decode items */
  int32_t live;          /* requests not yet finished */
  int32_t waiting;       /* of which not yet through their prompt */
  int64_t page_retries;  /* forwards planned again with fewer prompt tokens for lack of KV pages */
} metro_engine_stats;

/* Create an engine on a model (or NULL: planning only); the model must
 * outlive it.  Errors: METRO_E_INVAL, METRO_E_NOMEM. */
metro_status metro_engine_create(metro_model* model, const metro_engine_config* cfg, metro_engine** out);

/* Close the sequences of unfinished requests and free the engine. */
void metro_engine_destroy(metro_engine* engine);

/* Queue a request: generate n_out tokens greedily after prompt[0 .. n_prompt)
 * (host int32, copied).  Opens its sequence through the model's prefix
 * cache (metro_seq_open_cached; with the cache off every prompt token is
 * prefilled).  request must not name a live request. */
metro_status metro_engine_submit(metro_engine* engine, int64_t request, int32_t step, const int32_t* prompt,
                                 int32_t n_prompt, int32_t n_out);

/* One forward (see above); *n_items = its items (0: nothing to run).
 * Returns after the forward's tokens are on the host. */
metro_status metro_engine_step(metro_engine* engine, void* stream, int32_t* n_items);

/* The items of the last metro_engine_step, in forward order: request ids,
 * tokens of each item, and 1 for a decode token, 0 for a prompt chunk.
 * Writes min(cap, n) entries and n to *n. */
metro_status metro_engine_last_plan(const metro_engine* engine, int64_t* requests, int32_t* tokens, int32_t* decode,
                                    int32_t cap, int32_t* n);

/* Requests retired since the last call, in retirement order (at most cap;
 * the rest stay queued). */
metro_status metro_engine_finished(metro_engine* engine, int64_t* requests, int32_t cap, int32_t* n);

/* Output tokens of a request so far (min(cap, n) written, n to *n).  A
 * finished request whose tokens all fit is released: its id may be reused. */
metro_status metro_engine_result(metro_engine* engine, int64_t request, int32_t* tokens, int32_t cap, int32_t* n);

metro_status metro_engine_get_stats(const metro_engine* engine, metro_engine_stats* stats);

#ifdef __cplusplus
}
#endif

#endif /* METRO_SCHED_H */
