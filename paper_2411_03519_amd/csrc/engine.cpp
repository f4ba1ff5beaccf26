// Mixed continuous batching of agents' LLM requests (include/metro_sched.h):
// the serving loop between the out-of-order scheduler and the model.
//
// Every forward carries the next token of each running request (a one-token
// item: no request is preempted mid-generation, §3.5) and, in the token budget
// left, prompt chunks of waiting requests -- chunked prefill mixed with decode
// in one pass over the weights, the prior art the paper cites (§5).  Waiting
// requests are admitted lowest step first (every request carries its agent's
// step; smaller steps run first, §3.5 and the priority ablation of §4.4), ties
// by arrival; with priority off, by arrival alone.  A forward with no prompt
// chunk goes through the decode path (metro_decode_step), which reads each
// row's context with the decode attention kernel.
//
// The engine keeps every request's tokens on the host: after each forward it
// waits for the greedy tokens, appends them, and retires requests that have
// produced their n_out tokens (their sequences are closed).  That wait is also
// where the caller learns which agents may proceed.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <new>
#include <unordered_map>
#include <vector>

#include "../../include/metro.h"
#include "../../include/metro_sched.h"
#include "errors.h"

namespace {

constexpr int32_t kWaiting = 0, kRunning = 1, kFinished = 2;

struct Request {
  int64_t id = 0;
  int32_t step = 0;
  int64_t arrival = 0;
  int64_t seq = -1;
  std::vector<int32_t> prompt;
  int32_t off = 0;    // prompt tokens in the sequence
  int32_t n_out = 0;  // tokens to generate
  std::vector<int32_t> out;
  int32_t state = kWaiting;
};

}  // namespace

struct metro_engine {
  metro_model* model = nullptr;  // NULL: planning only (no device work)
  metro_engine_config cfg{};
  std::unordered_map<int64_t, Request> reqs;
  int64_t arrivals = 0;
  std::vector<int64_t> finished;  // retired, not yet reported by metro_engine_finished
  // the last forward's items, in order
  std::vector<int64_t> plan_id;
  std::vector<int32_t> plan_tokens;
  std::vector<int32_t> plan_decode;
  // device and pinned host buffers for the greedy tokens
  int32_t* next_dev = nullptr;
  int32_t* tok_dev = nullptr;
  int32_t* pinned = nullptr;  // [2 * max_items]: tokens in, tokens out
  metro_engine_stats stats{};

  ~metro_engine() {
    if (next_dev) (void)hipFree(next_dev);
    if (tok_dev) (void)hipFree(tok_dev);
    if (pinned) (void)hipHostFree(pinned);
  }

  // order of admission: lowest step first, then arrival (priority), or arrival
  bool before(const Request* a, const Request* b) const {
    if (cfg.priority && a->step != b->step) return a->step < b->step;
    return a->arrival < b->arrival;
  }

  // The items of the next forward: (request, tokens, is a decode token), with
  // at most prompt_cap prompt tokens.
  void plan(int32_t prompt_cap) {
    plan_id.clear();
    plan_tokens.clear();
    plan_decode.clear();
    std::vector<Request*> run, wait;
    for (auto& kv : reqs) {
      Request& r = kv.second;
      if (r.state == kRunning) run.push_back(&r);
      else if (r.state == kWaiting) wait.push_back(&r);
    }
    auto order = [this](const Request* a, const Request* b) { return before(a, b); };
    std::sort(run.begin(), run.end(), order);
    std::sort(wait.begin(), wait.end(), order);
    for (Request* r : run) {
      if (static_cast<int32_t>(plan_id.size()) >= cfg.max_items) break;
      plan_id.push_back(r->id);
      plan_tokens.push_back(1);
      plan_decode.push_back(1);
    }
    int32_t budget = std::min(cfg.max_tokens - static_cast<int32_t>(plan_id.size()), prompt_cap);
    for (Request* r : wait) {
      if (static_cast<int32_t>(plan_id.size()) >= cfg.max_items || budget <= 0) break;
      const int32_t take = std::min({cfg.chunk, static_cast<int32_t>(r->prompt.size()) - r->off, budget});
      plan_id.push_back(r->id);
      plan_tokens.push_back(take);
      plan_decode.push_back(0);
      budget -= take;
    }
  }

  // Run the planned forward and leave each item's greedy token in next
  // (planning only: a stand-in token per item).  Returns the model's status;
  // on failure no request's state has changed.
  metro_status forward(void* stream, std::vector<int32_t>& next) {
    const int32_t n = static_cast<int32_t>(plan_id.size());
    if (!model) {
      for (int32_t i = 0; i < n; ++i) next[i] = static_cast<int32_t>((plan_id[i] * 31 + stats.forwards) % 1000);
      return METRO_OK;
    }
    bool any_prompt = false;
    for (int32_t d : plan_decode) any_prompt |= d == 0;
    hipStream_t s = static_cast<hipStream_t>(stream);
    std::vector<int64_t> seqs(n);
    for (int32_t i = 0; i < n; ++i) seqs[i] = reqs[plan_id[i]].seq;
    metro_status st;
    if (any_prompt) {
      std::vector<int32_t> cu(n + 1, 0), toks;
      for (int32_t i = 0; i < n; ++i) {
        const Request& r = reqs[plan_id[i]];
        if (plan_decode[i]) toks.push_back(r.out.back());
        else toks.insert(toks.end(), r.prompt.begin() + r.off, r.prompt.begin() + r.off + plan_tokens[i]);
        cu[i + 1] = static_cast<int32_t>(toks.size());
      }
      st = metro_prefill_chunk(model, n, seqs.data(), cu.data(), toks.data(), nullptr, next_dev, stream);
    } else {
      for (int32_t i = 0; i < n; ++i) pinned[i] = reqs[plan_id[i]].out.back();
      if (hipMemcpyAsync(tok_dev, pinned, n * 4, hipMemcpyHostToDevice, s) != hipSuccess)
        return metro::report(METRO_E_HIP, "engine: token upload failed");
      st = metro_decode_step(model, n, seqs.data(), tok_dev, nullptr, next_dev, stream);
    }
    if (st != METRO_OK) return st;
    int32_t* back = pinned + cfg.max_items;
    if (hipMemcpyAsync(back, next_dev, n * 4, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      return metro::report(METRO_E_HIP, "engine: token download failed");
    std::memcpy(next.data(), back, n * 4);
    return METRO_OK;
  }
};

namespace {

using metro::report;

metro_status check_engine(const metro_engine* e) {
  if (!e) return report(METRO_E_INVAL, "engine is NULL");
  return METRO_OK;
}

}  // namespace

extern "C" {

metro_status metro_engine_create(metro_model* model, const metro_engine_config* cfg, metro_engine** out) {
  metro::clear_error();
  if (!cfg || !out) return report(METRO_E_INVAL, "engine: NULL argument");
  *out = nullptr;
  if (cfg->max_tokens <= 0 || cfg->chunk <= 0 || cfg->max_items <= 0 || (cfg->priority != 0 && cfg->priority != 1))
    return report(METRO_E_INVAL, "engine: max_tokens, chunk and max_items must be positive, priority 0 or 1");
  auto* e = new (std::nothrow) metro_engine();
  if (!e) return report(METRO_E_NOMEM, "engine: out of host memory");
  e->model = model;
  e->cfg = *cfg;
  if (model) {
    const int64_t n = cfg->max_items;
    if (hipMalloc(&e->next_dev, n * 4) != hipSuccess || hipMalloc(&e->tok_dev, n * 4) != hipSuccess ||
        hipHostMalloc(reinterpret_cast<void**>(&e->pinned), 2 * n * 4, hipHostMallocDefault) != hipSuccess) {
      delete e;
      return report(METRO_E_NOMEM, "engine: device or pinned buffers of %lld items", (long long)n);
    }
  }
  *out = e;
  return METRO_OK;
}

void metro_engine_destroy(metro_engine* e) {
  if (!e) return;
  if (e->model)
    for (auto& kv : e->reqs)
      if (kv.second.seq >= 0) (void)metro_seq_close(e->model, kv.second.seq);
  delete e;
}

metro_status metro_engine_submit(metro_engine* e, int64_t request, int32_t step, const int32_t* prompt,
                                 int32_t n_prompt, int32_t n_out) {
  metro::clear_error();
  metro_status st = check_engine(e);
  if (st != METRO_OK) return st;
  if (!prompt || n_prompt <= 0 || n_out <= 0 || step < 0)
    return report(METRO_E_INVAL, "engine submit: prompt of %d tokens, %d outputs, step %d", n_prompt, n_out, step);
  if (e->reqs.count(request)) return report(METRO_E_INVAL, "engine submit: request %lld is live", (long long)request);
  Request r;
  r.id = request;
  r.step = step;
  r.arrival = e->arrivals;
  r.prompt.assign(prompt, prompt + n_prompt);
  r.n_out = n_out;
  if (e->model) {
    int32_t cached = 0;
    st = metro_seq_open_cached(e->model, prompt, n_prompt, &r.seq, &cached);
    if (st != METRO_OK) return st;
    r.off = cached;
  }
  e->arrivals += 1;
  try {
    e->reqs.emplace(request, std::move(r));
  } catch (const std::bad_alloc&) {
    if (e->model && r.seq >= 0) (void)metro_seq_close(e->model, r.seq);  // (the id survives the failed move)
    return report(METRO_E_NOMEM, "engine submit: out of host memory");
  }
  return METRO_OK;
}

metro_status metro_engine_step(metro_engine* e, void* stream, int32_t* n_items) {
  metro::clear_error();
  metro_status st = check_engine(e);
  if (st != METRO_OK) return st;
  // When the model runs short of KV pages for the forward, the same step is
  // planned again with half the prompt tokens (the model's calls change no
  // state when they fail that way), down to a decode-only forward.
  int32_t prompt_cap = e->cfg.max_tokens;
  int32_t n = 0;
  std::vector<int32_t> next;
  for (;;) {
    e->plan(prompt_cap);
    n = static_cast<int32_t>(e->plan_id.size());
    if (n_items) *n_items = n;
    int32_t prompt_tokens = 0;
    for (int32_t i = 0; i < n; ++i)
      if (!e->plan_decode[i]) prompt_tokens += e->plan_tokens[i];
    if (n == 0) {
      if (prompt_cap < e->cfg.max_tokens)
        return report(METRO_E_NOPAGES, "engine: too few free KV pages for any forward (%d requests live)",
                      static_cast<int>(e->reqs.size()));
      return METRO_OK;
    }
    next.assign(n, 0);
    st = e->forward(stream, next);
    if (st == METRO_E_NOPAGES && prompt_tokens > 0) {
      prompt_cap = prompt_tokens / 2;
      e->stats.page_retries += 1;
      continue;
    }
    if (st != METRO_OK) return st;
    break;
  }
  e->stats.forwards += 1;
  e->stats.items += n;
  for (int32_t i = 0; i < n; ++i) {
    Request& r = e->reqs[e->plan_id[i]];
    if (e->plan_decode[i]) {
      e->stats.decode_tokens += 1;
    } else {
      e->stats.prompt_tokens += e->plan_tokens[i];
      r.off += e->plan_tokens[i];
      if (r.off < static_cast<int32_t>(r.prompt.size())) continue;  // more chunks to come
      r.state = kRunning;
    }
    r.out.push_back(next[i]);
    if (static_cast<int32_t>(r.out.size()) >= r.n_out) {
      r.state = kFinished;
      if (e->model && r.seq >= 0) (void)metro_seq_close(e->model, r.seq);
      r.seq = -1;
      e->finished.push_back(r.id);
    }
  }
  return METRO_OK;
}

metro_status metro_engine_last_plan(const metro_engine* e, int64_t* requests, int32_t* tokens, int32_t* decode,
                                    int32_t cap, int32_t* n) {
  metro::clear_error();
  metro_status st = check_engine(e);
  if (st != METRO_OK) return st;
  if (!n || (cap > 0 && (!requests || !tokens || !decode))) return report(METRO_E_INVAL, "engine plan: NULL");
  const int32_t m = static_cast<int32_t>(e->plan_id.size());
  for (int32_t i = 0; i < std::min(m, cap); ++i) {
    requests[i] = e->plan_id[i];
    tokens[i] = e->plan_tokens[i];
    decode[i] = e->plan_decode[i];
  }
  *n = m;
  return METRO_OK;
}

metro_status metro_engine_finished(metro_engine* e, int64_t* requests, int32_t cap, int32_t* n) {
  metro::clear_error();
  metro_status st = check_engine(e);
  if (st != METRO_OK) return st;
  if (!n || (cap > 0 && !requests)) return report(METRO_E_INVAL, "engine finished: NULL");
  const int32_t m = std::min(cap, static_cast<int32_t>(e->finished.size()));
  std::copy(e->finished.begin(), e->finished.begin() + m, requests);
  e->finished.erase(e->finished.begin(), e->finished.begin() + m);
  *n = m;
  return METRO_OK;
}

metro_status metro_engine_result(metro_engine* e, int64_t request, int32_t* tokens, int32_t cap, int32_t* n) {
  metro::clear_error();
  metro_status st = check_engine(e);
  if (st != METRO_OK) return st;
  if (!n || (cap > 0 && !tokens)) return report(METRO_E_INVAL, "engine result: NULL");
  auto it = e->reqs.find(request);
  if (it == e->reqs.end()) return report(METRO_E_SEQ, "engine result: unknown request %lld", (long long)request);
  const Request& r = it->second;
  const int32_t m = static_cast<int32_t>(r.out.size());
  std::copy(r.out.begin(), r.out.begin() + std::min(m, cap), tokens);
  *n = m;
  if (r.state == kFinished && cap >= m) e->reqs.erase(it);
  return METRO_OK;
}

metro_status metro_engine_get_stats(const metro_engine* e, metro_engine_stats* out) {
  metro::clear_error();
  metro_status st = check_engine(e);
  if (st != METRO_OK) return st;
  if (!out) return report(METRO_E_INVAL, "engine stats: NULL");
  *out = e->stats;
  out->live = 0;
  out->waiting = 0;
  for (const auto& kv : e->reqs) {
    if (kv.second.state != kFinished) out->live += 1;
    if (kv.second.state == kWaiting) out->waiting += 1;
  }
  return METRO_OK;
}

}  // extern "C"
