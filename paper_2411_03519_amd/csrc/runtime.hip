// Host runtime of libmetro.so: model creation and weight packing, the KV page
// pool, per-call descriptors, the launch sequence of the forward pass, and the
// extern "C" entry points declared in include/metro.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/metro.h"
#include "../../include/metro_ops.h"
#include "errors.h"
#include "kernels/kernels.h"
#include "kv_pool.h"

namespace {

thread_local std::string g_err;

metro_status fail(metro_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

uint64_t splitmix64_host(uint64_t z) {
  z += 0x9e3779b97f4a7c15ull;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

constexpr int kRing = 4;              // pinned descriptor buffers in flight

int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }

struct Layer {
  uint16_t* attn_norm;
  uint16_t* ffn_norm;
  uint16_t* wqkv;   // [(nq + 2 nkv) hd, d]: rows of wq, then wk, then wv
  uint16_t* wo;     // [d, nq hd]
  uint16_t* wgu;    // [2F, d]: blocks of 16 rows = 8 gate rows, then the 8 up rows of the same features
  uint16_t* wdown;  // [d, Fp] (K padded with zeros to a multiple of 128)
};

}  // namespace

namespace metro {

metro_status report(metro_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

void clear_error() { g_err.clear(); }

}  // namespace metro

struct metro_model {
  metro_config cfg{};
  int device = 0;
  int q_dim = 0, kv_dim = 0, qkv_n = 0, group = 0, Fp = 0;
  // weights
  void* wbase = nullptr;
  size_t weight_bytes = 0;
  uint16_t *embed = nullptr, *lm_head = nullptr, *final_norm = nullptr;
  std::vector<Layer> layers;
  float2* rope = nullptr;
  // KV pool
  uint16_t* kv = nullptr;
  int64_t page_elems = 0;   // per layer
  int64_t layer_stride = 0; // elements
  int32_t n_pages = 0;
  size_t kv_bytes = 0;
  // scratch
  void* sbase = nullptr;
  size_t scratch_bytes = 0;
  float* x = nullptr;
  uint16_t* h = nullptr;
  float* qkv = nullptr;
  uint16_t* q = nullptr;
  uint16_t* o = nullptr;
  uint16_t* a = nullptr;
  float* xr = nullptr;
  float* logits_ws = nullptr;
  int32_t* next_ws = nullptr;
  float* parts = nullptr;    // k-slice sums of decode GEMMs, [8][min(kSplitMaxRows, rows)][max(qkv_n, d)]
  int64_t parts_cap = 0;     // floats in parts
  float* attn_part = nullptr;  // decode attention split states
  int32_t* desc_dev = nullptr;
  int64_t desc_cap = 0;  // int32 elements
  // host
  std::unique_ptr<metro::SequenceTable> seqs;
  int32_t* desc_host[kRing] = {};
  hipEvent_t desc_ev[kRing] = {};
  int ring = 0;
  bool poisoned = false;
  bool sync_check = false;  // METRO_SYNC_CHECK: wait for and check every launch
  // launch timing (metro_profile_*)
  int prof_cls = -1;
  int prof_phase = 0;
  int cur_phase = 0;  // 1 prefill, 2 decode
  std::vector<hipEvent_t> prof_ev;  // pairs
  std::vector<char> prof_used;
  int prof_next = 0;
  double prof_ms = 0.0;
  int64_t prof_count = 0;
};

namespace {

metro_status hip_fail(metro_model* m, hipError_t e, const char* what) {
  if (m) m->poisoned = true;
  return fail(METRO_E_HIP, "HIP error %d (%s) in %s", static_cast<int>(e), hipGetErrorString(e), what);
}

#define HIP_TRY(m, expr)                                  \
  do {                                                    \
    hipError_t e_ = (expr);                               \
    if (e_ != hipSuccess) return hip_fail((m), e_, #expr); \
  } while (0)

constexpr int kProfPairs = 4096;

metro_status prof_harvest(metro_model* m, int i) {
  if (!m->prof_used[i]) return METRO_OK;
  HIP_TRY(m, hipEventSynchronize(m->prof_ev[2 * i + 1]));
  float ms = 0.f;
  HIP_TRY(m, hipEventElapsedTime(&ms, m->prof_ev[2 * i], m->prof_ev[2 * i + 1]));
  m->prof_ms += ms;
  m->prof_count += 1;
  m->prof_used[i] = 0;
  return METRO_OK;
}

// Launch through `fn` (returning hipError_t); when this kernel class and call
// phase are being profiled, the kernel records a pair of events on its own
// dispatch (see metro::launch_events).
template <class Fn>
metro_status launch(metro_model* m, int cls, hipStream_t s, const char* what, Fn&& fn) {
  const bool timed = cls == m->prof_cls && (m->prof_phase == 0 || m->prof_phase == m->cur_phase);
  int i = 0;
  if (timed) {
    i = m->prof_next;
    m->prof_next = (i + 1) % kProfPairs;
    metro_status st = prof_harvest(m, i);
    if (st != METRO_OK) return st;
    metro::launch_events = {m->prof_ev[2 * i], m->prof_ev[2 * i + 1]};
  }
  hipError_t e = fn();
  metro::launch_events = {};
  if (e == hipSuccess && m->sync_check) {  // debugging: a failing kernel is named by its own launch
    e = hipStreamSynchronize(s);
    if (e == hipSuccess) e = hipGetLastError();
  }
  if (e != hipSuccess) return hip_fail(m, e, what);
  if (timed) m->prof_used[i] = 1;
  return METRO_OK;
}

#define LAUNCH(m, cls, s, expr)                                                   \
  do {                                                                            \
    metro_status st_ = launch((m), (cls), (s), #expr, [&]() { return (expr); }); \
    if (st_ != METRO_OK) return st_;                                              \
  } while (0)

metro_status check_config(const metro_config* c) {
  if (!c) return fail(METRO_E_INVAL, "config is NULL");
  if (c->n_layers <= 0 || c->d_model <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 || c->ffn_dim <= 0 ||
      c->vocab <= 0 || c->max_batch <= 0 || c->max_tokens <= 0 || c->max_context <= 0 || c->max_seqs <= 0)
    return fail(METRO_E_INVAL, "config: every count must be positive");
  if (c->d_model % 128) return fail(METRO_E_INVAL, "config: d_model %% 128 != 0");
  if (c->d_model > metro::kRmsNormMaxDim) return fail(METRO_E_INVAL, "config: d_model > %d", metro::kRmsNormMaxDim);
  if (c->head_dim != 64 && c->head_dim != 128) return fail(METRO_E_INVAL, "config: head_dim must be 64 or 128");
  if (c->n_heads % c->n_kv_heads) return fail(METRO_E_INVAL, "config: n_heads %% n_kv_heads != 0");
  const int g = c->n_heads / c->n_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8) return fail(METRO_E_INVAL, "config: group size must be 1, 2, 4 or 8");
  if ((c->n_heads * c->head_dim) % 128) return fail(METRO_E_INVAL, "config: n_heads*head_dim %% 128 != 0");
  if (c->ffn_dim % 16) return fail(METRO_E_INVAL, "config: ffn_dim %% 16 != 0");
  if (c->vocab % 32) return fail(METRO_E_INVAL, "config: vocab %% 32 != 0");
  if (c->page_size != 16) return fail(METRO_E_INVAL, "config: page_size must be 16");
  if (!(c->rope_base > 1.0f) || !(c->rms_eps >= 0.0f)) return fail(METRO_E_INVAL, "config: rope_base/rms_eps");
  if (c->kv_pool_bytes < 0) return fail(METRO_E_INVAL, "config: kv_pool_bytes < 0");
  if (c->max_context > (1 << 22)) return fail(METRO_E_INVAL, "config: max_context too large");
  return METRO_OK;
}

struct Carve {
  char* base;
  size_t off = 0;
  template <class T>
  T* take(size_t n) {
    off = static_cast<size_t>(round_up(static_cast<int64_t>(off), 256));
    T* p = reinterpret_cast<T*>(base + off);
    off += n * sizeof(T);
    return p;
  }
};

int64_t decode_work_capacity(const metro_config& c) {
  const int64_t P = (c.max_context + 15) / 16;
  return int64_t(c.max_batch) * ((P + metro::kDecodePagesPerSplit - 1) / metro::kDecodePagesPerSplit);
}

int64_t desc_capacity(const metro_config& c) {
  const int64_t T = c.max_tokens, B = c.max_batch;
  const int64_t P = (c.max_context + 15) / 16;
  // tokens, positions, slots, last rows, item block tables, query blocks, block tables
  const int64_t prefill = 3 * T + 2 * B + 3 * (T + B) + B * P;
  // positions, slots, 5 per-row arrays, work items, block tables
  const int64_t decode = 7 * B + 2 * decode_work_capacity(c) + B * P;
  // + per-array rounding to 16 elements (at most 16 arrays per call)
  return std::max(prefill, decode) + 16 * 16 + 64;
}

void free_model(metro_model* m) {
  if (!m) return;
  for (int i = 0; i < kRing; ++i) {
    if (m->desc_ev[i]) (void)hipEventDestroy(m->desc_ev[i]);
    if (m->desc_host[i]) (void)hipHostFree(m->desc_host[i]);
  }
  for (hipEvent_t e : m->prof_ev) (void)hipEventDestroy(e);
  if (m->kv) (void)hipFree(m->kv);
  if (m->sbase) (void)hipFree(m->sbase);
  if (m->wbase) (void)hipFree(m->wbase);
  delete m;
}

// Descriptor block of one call, built on the host and copied in one piece.
struct Desc {
  std::vector<int64_t> off;  // offsets (int32 elements) of each array
  int32_t* host;
  int64_t n = 0;
  int64_t cap;
  int32_t* put(int64_t count) {
    int32_t* p = host + n;
    off.push_back(n);
    n += (count + 15) / 16 * 16;  // keep each array 64-byte aligned
    if (n > cap) {  // the capacity formula bounds every call; this cannot trigger
      std::fprintf(stderr, "metro: descriptor buffer overflow (%lld > %lld)\n", (long long)n, (long long)cap);
      std::abort();
    }
    return p;
  }
};

// The launch sequence of the decoder blocks over T rows; attention is the
// decode kernel (dec) or the prefill kernel (pre).  Decode-sized GEMMs may
// leave k-slice sums in m->parts; the kernel that next reads their result
// (RMSNorm for the residual stream, RoPE for q/k/v) adds them.  On return
// *x_parts says how many slices the residual stream still has to take.
metro_status launch_layers(metro_model* m, int T, const int32_t* tok_dev, const int32_t* pos, const int32_t* slot,
                           const metro::AttnArgs* dec, const metro::PrefillAttnArgs* pre, int* x_parts,
                           hipStream_t s) {
  const metro_config& c = m->cfg;
  const int d = c.d_model;
  int xp = 0, qp = 0;
  LAUNCH(m, METRO_K_EMBED, s, metro::launch_embed(tok_dev, m->embed, c.vocab, d, m->x, T, s));
  for (int l = 0; l < c.n_layers; ++l) {
    const Layer& L = m->layers[l];
    uint16_t* kv_l = m->kv + static_cast<size_t>(l) * m->layer_stride;
    LAUNCH(m, METRO_K_RMSNORM, s,
           metro::launch_rmsnorm(m->x, d, L.attn_norm, c.rms_eps, m->h, d, T, d, m->parts, xp, s));
    if (metro::gemm_rope_kv_fused(T, m->qkv_n, d)) {
      const metro::RopeKV rk{pos, slot, m->rope, m->q, kv_l, c.n_heads, c.n_kv_heads, c.head_dim};
      LAUNCH(m, METRO_K_GEMM_QKV, s, metro::launch_gemm_rope_kv(m->h, d, L.wqkv, d, T, m->qkv_n, rk, s));
    } else {
      LAUNCH(m, METRO_K_GEMM_QKV, s,
             metro::launch_gemm(m->h, d, L.wqkv, d, T, m->qkv_n, metro::kEpiStoreF32, m->qkv, nullptr, m->qkv_n,
                                m->parts, m->parts_cap, &qp, s));
      LAUNCH(m, METRO_K_ROPE_KV, s,
             metro::launch_rope_kv(qp ? m->parts : m->qkv, qp, T, c.n_heads, c.n_kv_heads, c.head_dim, pos, slot,
                                   m->rope, m->q, kv_l, s));
    }
    if (dec) {
      metro::AttnArgs a = *dec;
      a.kv = kv_l;
      LAUNCH(m, METRO_K_ATTENTION, s, metro::launch_attn_decode(a, s));
      if (a.n_work > a.rows) LAUNCH(m, METRO_K_ATTENTION, s, metro::launch_attn_combine(a, s));
    } else {
      metro::PrefillAttnArgs a = *pre;
      a.kv = kv_l;
      LAUNCH(m, METRO_K_ATTENTION, s, metro::launch_attn_prefill(a, s));
    }
    LAUNCH(m, METRO_K_GEMM_O, s,
           metro::launch_gemm(m->o, m->q_dim, L.wo, m->q_dim, T, d, metro::kEpiAddF32, m->x, nullptr, d, m->parts,
                              m->parts_cap, &xp, s));
    LAUNCH(m, METRO_K_RMSNORM, s,
           metro::launch_rmsnorm(m->x, d, L.ffn_norm, c.rms_eps, m->h, d, T, d, m->parts, xp, s));
    int gp = 0;
    LAUNCH(m, METRO_K_GEMM_GATE_UP, s,
           metro::launch_gemm(m->h, d, L.wgu, d, T, 2 * c.ffn_dim, metro::kEpiSwiGLU, nullptr, m->a, m->Fp, m->parts,
                              m->parts_cap, &gp, s));
    LAUNCH(m, METRO_K_GEMM_DOWN, s,
           metro::launch_gemm(m->a, m->Fp, L.wdown, m->Fp, T, d, metro::kEpiAddF32, m->x, nullptr, d, m->parts,
                              m->parts_cap, &xp, s));
  }
  *x_parts = xp;
  return METRO_OK;
}

// Final RMSNorm (adding x_parts pending slices of the residual), LM head,
// greedy argmax over R rows.
metro_status launch_head(metro_model* m, float* xrows, int R, int x_parts, float* logits, int32_t* next_tok,
                         hipStream_t s) {
  const metro_config& c = m->cfg;
  float* lg = logits ? logits : m->logits_ws;
  int32_t* nt = next_tok ? next_tok : m->next_ws;
  int lp = 0;
  LAUNCH(m, METRO_K_RMSNORM, s,
         metro::launch_rmsnorm(xrows, c.d_model, m->final_norm, c.rms_eps, m->h, c.d_model, R, c.d_model, m->parts,
                               x_parts, s));
  LAUNCH(m, METRO_K_LM_HEAD, s,
         metro::launch_gemm(m->h, c.d_model, m->lm_head, c.d_model, R, c.vocab, metro::kEpiStoreF32, lg, nullptr,
                            c.vocab, nullptr, 0, &lp, s));
  if (next_tok || !logits) LAUNCH(m, METRO_K_ARGMAX, s, metro::launch_argmax(lg, c.vocab, R, nt, s));
  return METRO_OK;
}

// Take the next pinned descriptor buffer (waiting until its last copy is done).
metro_status take_ring(metro_model* m, Desc* d) {
  const int i = m->ring;
  HIP_TRY(m, hipEventSynchronize(m->desc_ev[i]));
  d->host = m->desc_host[i];
  d->cap = m->desc_cap;
  d->n = 0;
  return METRO_OK;
}

metro_status upload_ring(metro_model* m, const Desc& d, hipStream_t s) {
  const int i = m->ring;
  HIP_TRY(m, hipMemcpyAsync(m->desc_dev, d.host, d.n * sizeof(int32_t), hipMemcpyHostToDevice, s));
  HIP_TRY(m, hipEventRecord(m->desc_ev[i], s));
  m->ring = (i + 1) % kRing;
  return METRO_OK;
}

// Work items of decode attention for a row that sees ctx keys: runs of up to
// kDecodePagesPerSplit pages (depends on the row's own context only).
int32_t decode_splits(int32_t ctx) {
  return ((ctx + 15) / 16 + metro::kDecodePagesPerSplit - 1) / metro::kDecodePagesPerSplit;
}

// Query blocks of prefill attention for items of add[i] rows starting at row
// cu[i]: (item, first row, rows) triples of at most tpb rows each.
int64_t prefill_blocks(int n_items, const int32_t* cu, int tpb, int32_t* blocks) {
  int64_t nb = 0;
  for (int i = 0; i < n_items; ++i)
    for (int r0 = cu[i]; r0 < cu[i + 1]; r0 += tpb) {
      if (blocks) {
        blocks[3 * nb] = i;
        blocks[3 * nb + 1] = r0;
        blocks[3 * nb + 2] = std::min(tpb, cu[i + 1] - r0);
      }
      ++nb;
    }
  return nb;
}

metro_status check_live(const metro_model* m) {
  if (!m) return fail(METRO_E_INVAL, "model is NULL");
  if (m->poisoned) return fail(METRO_E_HIP, "model is poisoned by an earlier HIP error");
  return METRO_OK;
}

}  // namespace

namespace {

// ---------------------------------------------------------------------------
// Decode attention without allocation: descriptors and split states live in a
// fixed device array (one copy per GPU) instead of a per-call buffer.
// ---------------------------------------------------------------------------

constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

// Per device: the address of `scratch` on that GPU (hipGetSymbolAddress; the
// host-side name is only a stand-in and must never reach a kernel).
constexpr int kMaxDevices = 64;
static void* g_scratch_ptr[kMaxDevices] = {};
static std::mutex g_scratch_mu;

metro_status scratch_on_current_device(void** out) {
  int dev = 0;
  HIP_TRY(nullptr, hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(METRO_E_INVAL, "device %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY(nullptr, hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(METRO_E_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return METRO_OK;
}

// Descriptor arrays of decode attention built on the device from the rows'
// context lengths, in the order and with the values the host builds them for
// metro_op_attn_decode (row i's pages at the running page offset, its work
// items at the running work offset, splits of decode_splits()).  One thread:
// a few hundred cycles per row.
__global__ void describe_decode_kernel(const int32_t* ctx, int rows, int32_t* row_q, int32_t* row_bt,
                                       int32_t* row_work, int32_t* row_nsplit, int32_t* work) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  int32_t bo = 0, w = 0;
  for (int i = 0; i < rows; ++i) {
    const int32_t np = (ctx[i] + 15) / 16;
    const int32_t ns = (np + metro::kDecodePagesPerSplit - 1) / metro::kDecodePagesPerSplit;
    row_q[i] = i;
    row_bt[i] = bo;
    row_work[i] = w;
    row_nsplit[i] = ns;
    for (int sp = 0; sp < ns; ++sp, ++w) {
      work[2 * w] = i;
      work[2 * w + 1] = sp;
    }
    bo += np;
  }
}

}  // namespace

// ===========================================================================
// extern "C" API
// ===========================================================================

extern "C" {

int32_t metro_abi_version(void) { return METRO_ABI_VERSION; }

const char* metro_last_error(void) { return g_err.c_str(); }

const char* metro_status_name(int32_t st) {
  switch (st) {
    case METRO_OK: return "METRO_OK";
    case METRO_E_INVAL: return "METRO_E_INVAL";
    case METRO_E_NOMEM: return "METRO_E_NOMEM";
    case METRO_E_NOPAGES: return "METRO_E_NOPAGES";
    case METRO_E_SEQ: return "METRO_E_SEQ";
    case METRO_E_CAPACITY: return "METRO_E_CAPACITY";
    case METRO_E_HIP: return "METRO_E_HIP";
    default: return "METRO_E_UNKNOWN";
  }
}

metro_status metro_create_model(const metro_config* cfg, uint64_t init_seed, metro_model** out) {
  g_err.clear();
  if (!out) return fail(METRO_E_INVAL, "out is NULL");
  *out = nullptr;
  metro_status st = check_config(cfg);
  if (st != METRO_OK) return st;
  auto* m = new metro_model();
  m->cfg = *cfg;
  const metro_config& c = m->cfg;
  const int d = c.d_model, hd = c.head_dim, nq = c.n_heads, nkv = c.n_kv_heads, F = c.ffn_dim, V = c.vocab;
  m->q_dim = nq * hd;
  m->kv_dim = nkv * hd;
  m->qkv_n = m->q_dim + 2 * m->kv_dim;
  m->group = nq / nkv;
  m->Fp = static_cast<int>(round_up(F, 128));

  auto bail = [&](metro_status s2) {
    free_model(m);
    return s2;
  };
  if (const char* sc = std::getenv("METRO_SYNC_CHECK")) m->sync_check = std::atoi(sc) != 0;
  hipError_t e = hipGetDevice(&m->device);
  if (e != hipSuccess) return bail(hip_fail(nullptr, e, "hipGetDevice"));

  // ---- weights: one allocation, carved per tensor
  const size_t per_layer = 2 * static_cast<size_t>(d) + static_cast<size_t>(m->qkv_n) * d +
                           static_cast<size_t>(d) * m->q_dim + 2 * static_cast<size_t>(F) * d +
                           static_cast<size_t>(d) * m->Fp;
  const size_t welems = 2 * static_cast<size_t>(V) * d + d + per_layer * c.n_layers;
  m->weight_bytes = welems * 2 + 256 * (6 * c.n_layers + 8);
  const size_t rope_bytes = static_cast<size_t>(c.max_context) * (hd / 2) * sizeof(float2);
  e = hipMalloc(&m->wbase, m->weight_bytes + rope_bytes + 256);
  if (e != hipSuccess) return bail(fail(METRO_E_NOMEM, "hipMalloc of %zu weight bytes failed", m->weight_bytes));
  {
    Carve cv{static_cast<char*>(m->wbase)};
    m->embed = cv.take<uint16_t>(static_cast<size_t>(V) * d);
    m->lm_head = cv.take<uint16_t>(static_cast<size_t>(V) * d);
    m->final_norm = cv.take<uint16_t>(d);
    m->layers.resize(c.n_layers);
    for (auto& L : m->layers) {
      L.attn_norm = cv.take<uint16_t>(d);
      L.ffn_norm = cv.take<uint16_t>(d);
      L.wqkv = cv.take<uint16_t>(static_cast<size_t>(m->qkv_n) * d);
      L.wo = cv.take<uint16_t>(static_cast<size_t>(d) * m->q_dim);
      L.wgu = cv.take<uint16_t>(2 * static_cast<size_t>(F) * d);
      L.wdown = cv.take<uint16_t>(static_cast<size_t>(d) * m->Fp);
    }
    m->rope = cv.take<float2>(static_cast<size_t>(c.max_context) * (hd / 2));
  }

  // ---- scratch
  const int64_t Tm = std::max(c.max_tokens, c.max_batch);
  m->desc_cap = desc_capacity(c);
  {
    const size_t bytes = Tm * d * 4 + Tm * d * 2 + Tm * m->qkv_n * 4 + 2 * Tm * m->q_dim * 2 + Tm * m->Fp * 2 +
                         int64_t(c.max_batch) * d * 4 + int64_t(c.max_batch) * V * 4 + int64_t(c.max_batch) * 4 +
                         8LL * std::min<int64_t>(metro::kSplitMaxRows, Tm) * std::max(m->qkv_n, d) * 4 +
                         decode_work_capacity(c) * nkv * m->group * (hd + 2) * 4 + m->desc_cap * 4 + 256 * 16;
    m->scratch_bytes = bytes;
    e = hipMalloc(&m->sbase, bytes);
    if (e != hipSuccess) return bail(fail(METRO_E_NOMEM, "hipMalloc of %zu scratch bytes failed", bytes));
    Carve cv{static_cast<char*>(m->sbase)};
    m->x = cv.take<float>(Tm * d);
    m->h = cv.take<uint16_t>(Tm * d);
    m->qkv = cv.take<float>(Tm * m->qkv_n);
    m->q = cv.take<uint16_t>(Tm * m->q_dim);
    m->o = cv.take<uint16_t>(Tm * m->q_dim);
    m->a = cv.take<uint16_t>(Tm * m->Fp);
    m->xr = cv.take<float>(int64_t(c.max_batch) * d);
    m->logits_ws = cv.take<float>(int64_t(c.max_batch) * V);
    m->next_ws = cv.take<int32_t>(c.max_batch);
    m->parts_cap = 8LL * std::min<int64_t>(metro::kSplitMaxRows, Tm) * std::max(m->qkv_n, d);
    m->parts = cv.take<float>(m->parts_cap);
    m->attn_part = cv.take<float>(decode_work_capacity(c) * nkv * m->group * (hd + 2));
    m->desc_dev = cv.take<int32_t>(m->desc_cap);
    // the SwiGLU output's padding columns must read as zero
    e = hipMemset(m->a, 0, Tm * m->Fp * 2);
    if (e != hipSuccess) return bail(hip_fail(nullptr, e, "hipMemset(scratch)"));
  }

  // ---- KV pool
  m->page_elems = 2LL * nkv * 16 * hd;
  const int64_t page_bytes_all = m->page_elems * 2 * c.n_layers;
  int64_t pool_bytes = c.kv_pool_bytes;
  if (pool_bytes == 0) {
    size_t fr = 0, tot = 0;
    e = hipMemGetInfo(&fr, &tot);
    if (e != hipSuccess) return bail(hip_fail(nullptr, e, "hipMemGetInfo"));
    const int64_t reserve = 2LL << 30;
    pool_bytes = static_cast<int64_t>(fr) > reserve ? static_cast<int64_t>(fr) - reserve : 0;
  }
  int64_t n_pages = pool_bytes / page_bytes_all;
  n_pages = std::min<int64_t>(n_pages, 1 << 26);
  if (n_pages < 1) return bail(fail(METRO_E_NOMEM, "KV pool of %lld bytes holds no page", (long long)pool_bytes));
  m->n_pages = static_cast<int32_t>(n_pages);
  m->layer_stride = m->page_elems * n_pages;
  m->kv_bytes = static_cast<size_t>(page_bytes_all) * n_pages;
  e = hipMalloc(reinterpret_cast<void**>(&m->kv), m->kv_bytes);
  if (e != hipSuccess) return bail(fail(METRO_E_NOMEM, "hipMalloc of %zu KV-pool bytes failed", m->kv_bytes));
  m->seqs = std::make_unique<metro::SequenceTable>(m->n_pages, 16, c.max_seqs, c.max_context);

  // ---- descriptor ring
  for (int i = 0; i < kRing; ++i) {
    e = hipHostMalloc(reinterpret_cast<void**>(&m->desc_host[i]), m->desc_cap * sizeof(int32_t), hipHostMallocDefault);
    if (e != hipSuccess) return bail(fail(METRO_E_NOMEM, "hipHostMalloc of descriptor ring failed"));
    e = hipEventCreateWithFlags(&m->desc_ev[i], hipEventDisableTiming);
    if (e != hipSuccess) return bail(hip_fail(nullptr, e, "hipEventCreate"));
  }

  // ---- RoPE table: cos/sin of p * base^(-2i/hd), computed in double
  {
    std::vector<float2> tab(static_cast<size_t>(c.max_context) * (hd / 2));
    for (int p = 0; p < c.max_context; ++p)
      for (int i = 0; i < hd / 2; ++i) {
        const double th = std::pow(static_cast<double>(c.rope_base), -2.0 * i / hd);
        const double ph = p * th;
        tab[static_cast<size_t>(p) * (hd / 2) + i] = make_float2(static_cast<float>(std::cos(ph)),
                                                                 static_cast<float>(std::sin(ph)));
      }
    e = hipMemcpy(m->rope, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice);
    if (e != hipSuccess) return bail(hip_fail(nullptr, e, "hipMemcpy(rope)"));
  }

  // ---- random initialisation on the device
  {
    auto key = [&](int id, int layer) {
      return splitmix64_host(init_seed ^ splitmix64_host((static_cast<uint64_t>(id) << 32) |
                                                         static_cast<uint32_t>(layer + 1)));
    };
    const uint16_t one = 0x3f80;
    hipError_t r = hipSuccess;
    auto chk = [&](hipError_t x) {
      if (r == hipSuccess) r = x;
    };
    const metro::RowMap in_order = metro::kRowsInOrder;
    const int half = hd / 2;  // QKV rows: rotate-half interleave per head
    chk(metro::launch_init_normal(m->embed, d, V, d, in_order, key(METRO_W_EMBED, -1), false, 0));
    chk(metro::launch_init_normal(m->lm_head, d, V, d, in_order, key(METRO_W_LM_HEAD, -1), true, 0));
    chk(metro::launch_fill_bf16(m->final_norm, d, one, 0));
    for (int l = 0; l < c.n_layers; ++l) {
      Layer& L = m->layers[l];
      chk(metro::launch_fill_bf16(L.attn_norm, d, one, 0));
      chk(metro::launch_fill_bf16(L.ffn_norm, d, one, 0));
      chk(metro::launch_init_normal(L.wqkv, d, m->q_dim, d, {16, 16, 0, half}, key(METRO_W_WQ, l), true, 0));
      chk(metro::launch_init_normal(L.wqkv, d, m->kv_dim, d, {16, 16, m->q_dim, half}, key(METRO_W_WK, l), true, 0));
      chk(metro::launch_init_normal(L.wqkv, d, m->kv_dim, d, {16, 16, m->q_dim + m->kv_dim, half},
                                    key(METRO_W_WV, l), true, 0));
      chk(metro::launch_init_normal(L.wo, m->q_dim, d, m->q_dim, in_order, key(METRO_W_WO, l), true, 0));
      chk(metro::launch_init_normal(L.wgu, d, F, d, {8, 16, 0, 0}, key(METRO_W_WGATE, l), true, 0));
      chk(metro::launch_init_normal(L.wgu, d, F, d, {8, 16, 8, 0}, key(METRO_W_WUP, l), true, 0));
      if (m->Fp != F) chk(metro::launch_fill_bf16(L.wdown, static_cast<int64_t>(d) * m->Fp, 0, 0));
      chk(metro::launch_init_normal(L.wdown, m->Fp, d, F, in_order, key(METRO_W_WDOWN, l), true, 0));
    }
    if (r == hipSuccess) r = hipDeviceSynchronize();
    if (r != hipSuccess) return bail(hip_fail(nullptr, r, "weight initialisation"));
  }
  *out = m;
  return METRO_OK;
}

void metro_destroy_model(metro_model* m) {
  if (!m) return;
  (void)hipSetDevice(m->device);
  (void)hipDeviceSynchronize();
  free_model(m);
}

metro_status metro_load_weight(metro_model* m, int32_t id, int32_t layer, const uint16_t* src, int64_t n) {
  g_err.clear();
  metro_status st = check_live(m);
  if (st != METRO_OK) return st;
  if (!src) return fail(METRO_E_INVAL, "host_bf16 is NULL");
  const metro_config& c = m->cfg;
  const int64_t d = c.d_model, F = c.ffn_dim, V = c.vocab;
  const bool global = id == METRO_W_EMBED || id == METRO_W_FINAL_NORM || id == METRO_W_LM_HEAD;
  if (id < METRO_W_EMBED || id > METRO_W_WDOWN) return fail(METRO_E_INVAL, "unknown weight id %d", id);
  if (!global && (layer < 0 || layer >= c.n_layers)) return fail(METRO_E_INVAL, "layer %d out of range", layer);
  HIP_TRY(m, hipSetDevice(m->device));
  // destination: (base, rows, cols, dst row stride); logical row r goes to
  // row map_row({grp, 16, shift, half}, r)
  uint16_t* base = nullptr;
  int64_t rows = 0, cols = 0, ld = 0, grp = 16, shift = 0, half = 0;
  const Layer* L = global ? nullptr : &m->layers[layer];
  switch (id) {
    case METRO_W_EMBED: base = m->embed; rows = V; cols = d; break;
    case METRO_W_LM_HEAD: base = m->lm_head; rows = V; cols = d; break;
    case METRO_W_FINAL_NORM: base = m->final_norm; rows = 1; cols = d; break;
    case METRO_W_ATTN_NORM: base = L->attn_norm; rows = 1; cols = d; break;
    case METRO_W_FFN_NORM: base = L->ffn_norm; rows = 1; cols = d; break;
    case METRO_W_WQ: base = L->wqkv; rows = m->q_dim; cols = d; half = c.head_dim / 2; break;
    case METRO_W_WK: base = L->wqkv; rows = m->kv_dim; cols = d; shift = m->q_dim; half = c.head_dim / 2; break;
    case METRO_W_WV:
      base = L->wqkv;
      rows = m->kv_dim;
      cols = d;
      shift = m->q_dim + m->kv_dim;
      half = c.head_dim / 2;
      break;
    case METRO_W_WO: base = L->wo; rows = d; cols = m->q_dim; break;
    case METRO_W_WGATE: base = L->wgu; rows = F; cols = d; grp = 8; break;
    case METRO_W_WUP: base = L->wgu; rows = F; cols = d; grp = 8; shift = 8; break;
    case METRO_W_WDOWN: base = L->wdown; rows = d; cols = F; ld = m->Fp; break;
  }
  if (ld == 0) ld = cols;
  if (n != rows * cols)
    return fail(METRO_E_INVAL, "weight %d: %lld elements given, %lld expected", id, (long long)n,
                (long long)(rows * cols));
  if (rows == 1 || id == METRO_W_EMBED) {  // norms and the embedding table stay row-major
    HIP_TRY(m, hipMemcpy(base, src, rows * cols * 2, hipMemcpyHostToDevice));
    return METRO_OK;
  }
  // projections: row-major upload into a staging buffer, then rearranged into
  // MFMA operand order at their rows
  uint16_t* stage = nullptr;
  HIP_TRY(m, hipMalloc(&stage, rows * cols * 2));
  hipError_t e = hipMemcpy(stage, src, rows * cols * 2, hipMemcpyHostToDevice);
  if (e == hipSuccess)
    e = metro::launch_pack_weight(stage, cols, static_cast<int>(rows), static_cast<int>(cols), base,
                                  static_cast<int>(ld),
                                  {static_cast<int>(grp), 16, static_cast<int>(shift), static_cast<int>(half)},
                                  nullptr);
  if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
  (void)hipFree(stage);
  if (e != hipSuccess) return hip_fail(m, e, "weight upload");
  return METRO_OK;
}

metro_status metro_model_get_info(const metro_model* m, metro_model_info* info) {
  g_err.clear();
  if (!m || !info) return fail(METRO_E_INVAL, "NULL argument");
  info->weight_bytes = static_cast<int64_t>(m->weight_bytes);
  info->scratch_bytes = static_cast<int64_t>(m->scratch_bytes);
  info->kv_pool_bytes = static_cast<int64_t>(m->kv_bytes);
  info->kv_bytes_per_token = 2LL * m->cfg.n_kv_heads * m->cfg.head_dim * 2 * m->cfg.n_layers;
  info->n_pages = m->n_pages;
  info->free_pages = m->seqs->pool().n_free();
  info->open_seqs = m->seqs->open_count();
  info->device = m->device;
  return METRO_OK;
}

metro_status metro_seq_open(metro_model* m, int64_t* seq) {
  g_err.clear();
  metro_status st = check_live(m);
  if (st != METRO_OK) return st;
  if (!seq) return fail(METRO_E_INVAL, "seq is NULL");
  const int r = m->seqs->open(seq);
  if (r != METRO_OK) return fail(static_cast<metro_status>(r), "%s", m->seqs->error().c_str());
  return METRO_OK;
}

metro_status metro_seq_open_cached(metro_model* m, const int32_t* tokens, int32_t n_tokens, int64_t* seq,
                                   int32_t* n_cached) {
  g_err.clear();
  metro_status st = check_live(m);
  if (st != METRO_OK) return st;
  if (!seq || !n_cached) return fail(METRO_E_INVAL, "NULL argument");
  const int r = m->seqs->open_cached(tokens, n_tokens, seq, n_cached);
  if (r != METRO_OK) return fail(static_cast<metro_status>(r), "%s", m->seqs->error().c_str());
  return METRO_OK;
}

metro_status metro_prefix_cache(metro_model* m, int32_t max_pages) {
  g_err.clear();
  metro_status st = check_live(m);
  if (st != METRO_OK) return st;
  const int r = m->seqs->set_prefix_cache(max_pages);
  if (r != METRO_OK) return fail(static_cast<metro_status>(r), "%s", m->seqs->error().c_str());
  return METRO_OK;
}

metro_status metro_prefix_cache_get_stats(const metro_model* m, metro_prefix_cache_stats* out) {
  g_err.clear();
  if (!m || !out) return fail(METRO_E_INVAL, "NULL argument");
  const metro::PrefixCacheStats st = m->seqs->prefix_cache_stats();
  out->pages = st.pages;
  out->limit = st.limit;
  out->lookup_tokens = st.lookup_tokens;
  out->hit_tokens = st.hit_tokens;
  out->inserted = st.inserted;
  out->evicted = st.evicted;
  return METRO_OK;
}

metro_status metro_seq_fork(metro_model* m, int64_t src, int32_t n_tokens, void* stream, int64_t* seq) {
  g_err.clear();
  metro_status st = check_live(m);
  if (st != METRO_OK) return st;
  if (!seq) return fail(METRO_E_INVAL, "seq is NULL");
  int32_t cs = -1, cd = -1;
  const int r = m->seqs->fork(src, n_tokens, seq, &cs, &cd);
  if (r != METRO_OK) return fail(static_cast<metro_status>(r), "%s", m->seqs->error().c_str());
  if (cs >= 0) {
    HIP_TRY(m, hipSetDevice(m->device));
    HIP_TRY(m, metro::launch_page_copy(m->kv, m->layer_stride, m->page_elems, m->cfg.n_layers, cs, cd,
                                       static_cast<hipStream_t>(stream)));
  }
  return METRO_OK;
}

metro_status metro_seq_close(metro_model* m, int64_t seq) {
  g_err.clear();
  if (!m) return fail(METRO_E_INVAL, "model is NULL");
  const int r = m->seqs->close(seq);
  if (r != METRO_OK) return fail(static_cast<metro_status>(r), "%s", m->seqs->error().c_str());
  return METRO_OK;
}

metro_status metro_seq_length(const metro_model* m, int64_t seq, int32_t* length) {
  g_err.clear();
  if (!m || !length) return fail(METRO_E_INVAL, "NULL argument");
  const metro::Sequence* s = m->seqs->find(seq);
  if (!s) return fail(METRO_E_SEQ, "unknown sequence %lld", (long long)seq);
  *length = s->length;
  return METRO_OK;
}

metro_status metro_seq_pages(const metro_model* m, int64_t seq, int32_t* pages, int32_t cap, int32_t* n_pages) {
  g_err.clear();
  if (!m || !n_pages || (cap > 0 && !pages)) return fail(METRO_E_INVAL, "NULL argument");
  const metro::Sequence* s = m->seqs->find(seq);
  if (!s) return fail(METRO_E_SEQ, "unknown sequence %lld", (long long)seq);
  const int32_t n = static_cast<int32_t>(s->pages.size());
  for (int32_t i = 0; i < std::min(n, cap); ++i) pages[i] = s->pages[i];
  *n_pages = n;
  return METRO_OK;
}

metro_status metro_prefill_chunk(metro_model* m, int32_t n_items, const int64_t* seqs, const int32_t* cu,
                                 const int32_t* tokens, float* logits, int32_t* next_tok, void* stream) {
  g_err.clear();
  metro_status st = check_live(m);
  if (st != METRO_OK) return st;
  const metro_config& c = m->cfg;
  if (n_items <= 0) return fail(METRO_E_INVAL, "n_items must be positive");
  if (n_items > c.max_batch) return fail(METRO_E_CAPACITY, "n_items %d > max_batch %d", n_items, c.max_batch);
  if (!seqs || !cu || !tokens) return fail(METRO_E_INVAL, "NULL argument");
  if (cu[0] != 0) return fail(METRO_E_INVAL, "cu_tokens[0] must be 0");
  std::vector<int32_t> add(n_items);
  for (int i = 0; i < n_items; ++i) {
    add[i] = cu[i + 1] - cu[i];
    if (add[i] < 1) return fail(METRO_E_INVAL, "item %d has %d tokens", i, add[i]);
  }
  const int T = cu[n_items];
  if (T > c.max_tokens) return fail(METRO_E_CAPACITY, "%d tokens > max_tokens %d", T, c.max_tokens);
  for (int t = 0; t < T; ++t)
    if (tokens[t] < 0 || tokens[t] >= c.vocab) return fail(METRO_E_INVAL, "token %d at %d out of range", tokens[t], t);
  HIP_TRY(m, hipSetDevice(m->device));
  Desc d;
  st = take_ring(m, &d);
  if (st != METRO_OK) return st;
  const int r = m->seqs->reserve(seqs, add.data(), n_items);
  if (r != METRO_OK) return fail(static_cast<metro_status>(r), "%s", m->seqs->error().c_str());

  int32_t* tok = d.put(T);
  int32_t* pos = d.put(T);
  int32_t* slot = d.put(T);
  int32_t* last = d.put(n_items);
  std::memcpy(tok, tokens, sizeof(int32_t) * T);
  int64_t bt_total = 0;
  for (int i = 0; i < n_items; ++i) bt_total += m->seqs->find(seqs[i])->pages.size();
  int32_t* bt = d.put(bt_total);
  int32_t* item_bt = d.put(n_items);
  const int tpb = metro::prefill_tokens_per_block(m->group);
  const int64_t n_blocks = prefill_blocks(n_items, cu, tpb, nullptr);
  int32_t* blocks = d.put(3 * n_blocks);
  prefill_blocks(n_items, cu, tpb, blocks);
  int64_t bo = 0;
  for (int i = 0; i < n_items; ++i) {
    const metro::Sequence* s = m->seqs->find(seqs[i]);
    std::copy(s->pages.begin(), s->pages.end(), bt + bo);
    item_bt[i] = static_cast<int32_t>(bo);
    for (int t = cu[i]; t < cu[i + 1]; ++t) {
      const int p = s->length + (t - cu[i]);
      pos[t] = p;
      slot[t] = s->pages[p / 16] * 16 + p % 16;
    }
    last[i] = cu[i + 1] - 1;
    bo += s->pages.size();
  }
  m->cur_phase = 1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  st = upload_ring(m, d, s);
  if (st != METRO_OK) return st;
  auto dev = [&](const int32_t* hp) { return m->desc_dev + (hp - d.host); };
  metro::PrefillAttnArgs pa{};
  pa.q = m->q;
  pa.out = m->o;
  pa.blocks = dev(blocks);
  pa.item_bt = dev(item_bt);
  pa.pos = dev(pos);
  pa.bt = dev(bt);
  pa.n_blocks = static_cast<int>(n_blocks);
  pa.nq = c.n_heads;
  pa.nkv = c.n_kv_heads;
  pa.hd = c.head_dim;
  pa.scale = 1.0f / std::sqrt(static_cast<float>(c.head_dim));
  int xp = 0;
  st = launch_layers(m, T, dev(tok), dev(pos), dev(slot), nullptr, &pa, &xp, s);
  if (st != METRO_OK) return st;
  if (xp > 0)
    LAUNCH(m, METRO_K_GEMM_DOWN, s,
           metro::launch_reduce_parts(m->parts, xp, T, c.d_model, metro::kEpiAddF32, m->x, c.d_model, s));
  LAUNCH(m, METRO_K_EMBED, s, metro::launch_gather_rows(m->x, c.d_model, dev(last), n_items, m->xr, s));
  st = launch_head(m, m->xr, n_items, 0, logits, next_tok, s);
  if (st != METRO_OK) return st;
  m->seqs->commit(seqs, add.data(), n_items);
  m->seqs->record_prefill(seqs, cu, tokens, n_items);
  return METRO_OK;
}

metro_status metro_decode_step(metro_model* m, int32_t B, const int64_t* seqs, const int32_t* tokens_dev,
                               float* logits, int32_t* next_tok, void* stream) {
  g_err.clear();
  metro_status st = check_live(m);
  if (st != METRO_OK) return st;
  const metro_config& c = m->cfg;
  if (B <= 0) return fail(METRO_E_INVAL, "batch must be positive");
  if (B > c.max_batch) return fail(METRO_E_CAPACITY, "batch %d > max_batch %d", B, c.max_batch);
  if (!seqs || !tokens_dev) return fail(METRO_E_INVAL, "NULL argument");
  HIP_TRY(m, hipSetDevice(m->device));
  Desc d;
  st = take_ring(m, &d);
  if (st != METRO_OK) return st;
  std::vector<int32_t> add(B, 1);
  const int r = m->seqs->reserve(seqs, add.data(), B);
  if (r != METRO_OK) return fail(static_cast<metro_status>(r), "%s", m->seqs->error().c_str());

  int32_t* pos = d.put(B);
  int32_t* slot = d.put(B);
  int64_t bt_total = 0;
  for (int i = 0; i < B; ++i) bt_total += m->seqs->find(seqs[i])->pages.size();
  int32_t* bt = d.put(bt_total);
  int32_t* row_ctx = d.put(B);
  int32_t* row_q = d.put(B);
  int32_t* row_bt = d.put(B);
  int32_t* row_work = d.put(B);
  int32_t* row_nsplit = d.put(B);
  int64_t bo = 0;
  int32_t n_work = 0;
  for (int i = 0; i < B; ++i) {
    const metro::Sequence* s = m->seqs->find(seqs[i]);
    const int p = s->length;
    pos[i] = p;
    slot[i] = s->pages[p / 16] * 16 + p % 16;
    std::copy(s->pages.begin(), s->pages.end(), bt + bo);
    row_ctx[i] = p + 1;
    row_q[i] = i;
    row_bt[i] = static_cast<int32_t>(bo);
    row_work[i] = n_work;
    row_nsplit[i] = decode_splits(p + 1);
    n_work += row_nsplit[i];
    bo += s->pages.size();
  }
  int32_t* work = d.put(2 * static_cast<int64_t>(n_work));
  for (int i = 0, w = 0; i < B; ++i)
    for (int sp = 0; sp < row_nsplit[i]; ++sp, ++w) {
      work[2 * w] = i;
      work[2 * w + 1] = sp;
    }
  m->cur_phase = 2;
  hipStream_t s = static_cast<hipStream_t>(stream);
  st = upload_ring(m, d, s);
  if (st != METRO_OK) return st;
  auto dev = [&](const int32_t* hp) { return m->desc_dev + (hp - d.host); };
  metro::AttnArgs a{};
  a.q = m->q;
  a.work = dev(work);
  a.row_ctx = dev(row_ctx);
  a.row_qrow = dev(row_q);
  a.row_bt = dev(row_bt);
  a.row_work = dev(row_work);
  a.row_nsplit = dev(row_nsplit);
  a.bt = dev(bt);
  a.part = m->attn_part;
  a.out = m->o;
  a.n_work = n_work;
  a.rows = B;
  a.nq = c.n_heads;
  a.nkv = c.n_kv_heads;
  a.hd = c.head_dim;
  a.scale = 1.0f / std::sqrt(static_cast<float>(c.head_dim));
  int xp = 0;
  st = launch_layers(m, B, tokens_dev, dev(pos), dev(slot), &a, nullptr, &xp, s);
  if (st != METRO_OK) return st;
  st = launch_head(m, m->x, B, xp, logits, next_tok, s);
  if (st != METRO_OK) return st;
  m->seqs->commit(seqs, add.data(), B);
  m->seqs->record_unknown(seqs, B);
  return METRO_OK;
}

metro_status metro_profile_start(metro_model* m, int32_t cls, int32_t phase) {
  g_err.clear();
  metro_status st = check_live(m);
  if (st != METRO_OK) return st;
  if (cls < METRO_K_EMBED || cls > METRO_K_ARGMAX || cls == 5 || phase < 0 || phase > 2)
    return fail(METRO_E_INVAL, "profile: bad kernel class %d or phase %d", cls, phase);
  HIP_TRY(m, hipSetDevice(m->device));
  if (m->prof_ev.empty()) {
    m->prof_ev.resize(2 * kProfPairs, nullptr);
    m->prof_used.assign(kProfPairs, 0);
    for (auto& e : m->prof_ev) HIP_TRY(m, hipEventCreate(&e));
  }
  for (int i = 0; i < kProfPairs; ++i) m->prof_used[i] = 0;
  m->prof_cls = cls;
  m->prof_phase = phase;
  m->prof_next = 0;
  m->prof_ms = 0.0;
  m->prof_count = 0;
  return METRO_OK;
}

metro_status metro_profile_stop(metro_model* m, double* total_ms, int64_t* launches) {
  g_err.clear();
  metro_status st = check_live(m);
  if (st != METRO_OK) return st;
  if (!total_ms || !launches) return fail(METRO_E_INVAL, "NULL argument");
  if (!m->prof_ev.empty()) {
    for (int i = 0; i < kProfPairs; ++i) {
      st = prof_harvest(m, i);
      if (st != METRO_OK) return st;
    }
  }
  *total_ms = m->prof_ms;
  *launches = m->prof_count;
  m->prof_cls = -1;
  return METRO_OK;
}

// ---------------------------------------------------------------------------
// Single-op entry points (include/metro_ops.h)
// ---------------------------------------------------------------------------

metro_status metro_op_pack_weight(const uint16_t* W_rowmajor, int32_t ld, int32_t N, int32_t K, int32_t Kp,
                                  uint16_t* W_packed, void* stream) {
  g_err.clear();
  if (!W_rowmajor || !W_packed || N <= 0 || N % 16 || Kp <= 0 || Kp % 128 || K <= 0 || K > Kp || ld < K)
    return fail(METRO_E_INVAL, "pack_weight: bad shape (N %% 16, Kp %% 128, 0 < K <= Kp, ld >= K required)");
  hipError_t e =
      metro::launch_pack_weight(W_rowmajor, ld, N, K, W_packed, Kp, metro::kRowsInOrder,
                                static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(nullptr, e, "launch_pack_weight");
  return METRO_OK;
}

// whether p (if given) is not a multiple of a bytes
static bool misaligned(const void* p, uintptr_t a) { return p && reinterpret_cast<uintptr_t>(p) % a != 0; }

metro_status metro_op_gemm(const uint16_t* X, int32_t ldx, const uint16_t* W, int32_t Kp, int32_t M, int32_t N,
                           int32_t epilogue, float* out_f32, uint16_t* out_bf16, int32_t ldo, float* workspace,
                           void* stream) {
  g_err.clear();
  if (!X || !W || M < 0 || N <= 0 || Kp <= 0 || Kp % 128 || N % 32 || ldx < Kp)
    return fail(METRO_E_INVAL, "gemm: bad shape (Kp %% 128, N %% 32, ldx >= Kp required)");
  if (epilogue == metro::kEpiSwiGLU ? !out_bf16 : !out_f32) return fail(METRO_E_INVAL, "gemm: output is NULL");
  if ((epilogue == metro::kEpiSwiGLU ? ldo < N / 2 : ldo < N) || ldo % 4)
    return fail(METRO_E_INVAL, "gemm: bad ldo");
  // the kernels move X and W in 16-byte pieces and store 4 outputs at a time
  if (ldx % 8 || misaligned(X, 16) || misaligned(W, 16) || misaligned(out_f32, 16) || misaligned(out_bf16, 8) ||
      misaligned(workspace, 16))
    return fail(METRO_E_INVAL, "gemm: X, W and workspace must be 16-byte aligned, ldx a multiple of 8, out_f32 "
                               "16-byte and out_bf16 8-byte aligned");
  int parts = 0;
  hipError_t e = metro::launch_gemm(X, ldx, W, Kp, M, N, epilogue, out_f32, out_bf16, ldo, workspace,
                                    8LL * M * N, &parts,
                                    static_cast<hipStream_t>(stream));
  if (e == hipSuccess && parts > 0)
    e = metro::launch_reduce_parts(workspace, parts, M, N, epilogue, out_f32, ldo, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(nullptr, e, "launch_gemm");
  return METRO_OK;
}

metro_status metro_op_gemm_plan(int32_t M, int32_t N, int32_t Kp, int32_t epilogue, int32_t has_workspace,
                                int32_t* kind, int32_t* k_slices, int32_t* tail_split) {
  g_err.clear();
  if (!kind || !k_slices || !tail_split || M <= 0 || N <= 0 || Kp <= 0 || Kp % 128 || N % 32 ||
      epilogue < metro::kEpiStoreF32 || epilogue > metro::kEpiSwiGLU)
    return fail(METRO_E_INVAL, "gemm plan: bad shape (Kp %% 128, N %% 32) or epilogue");
  const metro::GemmPlan p = metro::plan_gemm(M, N, Kp, epilogue, has_workspace ? 8LL * M * N : 0);
  *kind = static_cast<int32_t>(p.kind);
  *k_slices = p.ks;
  *tail_split = p.tail_split;
  return METRO_OK;
}

metro_status metro_op_rmsnorm(float* x, const uint16_t* g, float eps, uint16_t* h, int32_t rows, int32_t d,
                              void* stream) {
  g_err.clear();
  if (!x || !g || !h || rows < 0 || d <= 0 || d % 4 || d > metro::kRmsNormMaxDim)
    return fail(METRO_E_INVAL, "rmsnorm: bad arguments");
  if (misaligned(x, 16) || misaligned(g, 8) || misaligned(h, 8))
    return fail(METRO_E_INVAL, "rmsnorm: x must be 16-byte aligned, g and h 8-byte aligned");
  hipError_t e = metro::launch_rmsnorm(x, d, g, eps, h, d, rows, d, nullptr, 0, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(nullptr, e, "launch_rmsnorm");
  return METRO_OK;
}

// Device copy of the host descriptor arrays of one attention op call (and
// room for split states), freed when the op returns.
struct OpBuffer {
  void* p = nullptr;
  ~OpBuffer() {
    if (p) (void)hipFree(p);
  }
};

metro_status check_attn_shape(int32_t nq, int32_t nkv, int32_t hd, int32_t n_pages, const void* q, const void* kv,
                              const void* out) {
  if (hd != 64 && hd != 128) return fail(METRO_E_INVAL, "attention: head_dim must be 64 or 128");
  if (misaligned(q, 16) || misaligned(kv, 16) || misaligned(out, 8))
    return fail(METRO_E_INVAL, "attention: q and kv must be 16-byte aligned, out 8-byte aligned");
  if (nkv <= 0 || nq <= 0 || nq % nkv) return fail(METRO_E_INVAL, "attention: n_heads %% n_kv_heads != 0");
  const int g = nq / nkv;
  if (g != 1 && g != 2 && g != 4 && g != 8) return fail(METRO_E_INVAL, "attention: group size must be 1, 2, 4 or 8");
  if (n_pages <= 0) return fail(METRO_E_INVAL, "attention: n_pages must be positive");
  return METRO_OK;
}

metro_status metro_op_attn_decode(const uint16_t* q, const uint16_t* kv, int32_t n_pages, int32_t nq, int32_t nkv,
                                  int32_t hd, int32_t rows, const int32_t* ctx, const int32_t* block_tables,
                                  uint16_t* out, void* stream) {
  g_err.clear();
  metro_status st = check_attn_shape(nq, nkv, hd, n_pages, q, kv, out);
  if (st != METRO_OK) return st;
  if (rows < 0 || (rows > 0 && (!q || !kv || !ctx || !block_tables || !out)))
    return fail(METRO_E_INVAL, "attn_decode: NULL argument or rows < 0");
  if (rows == 0) return METRO_OK;
  // descriptor arrays, in the order of the model's decode call
  std::vector<int32_t> row_ctx(rows), row_q(rows), row_bt(rows), row_work(rows), row_nsplit(rows), work, bt;
  int64_t bo = 0;
  int32_t n_work = 0;
  for (int i = 0; i < rows; ++i) {
    if (ctx[i] < 1) return fail(METRO_E_INVAL, "attn_decode: row %d sees %d keys", i, ctx[i]);
    const int np = (ctx[i] + 15) / 16;
    for (int j = 0; j < np; ++j) {
      const int32_t id = block_tables[bo + j];
      if (id < 0 || id >= n_pages) return fail(METRO_E_INVAL, "attn_decode: page id %d out of range", id);
      bt.push_back(id);
    }
    row_ctx[i] = ctx[i];
    row_q[i] = i;
    row_bt[i] = static_cast<int32_t>(bo);
    row_work[i] = n_work;
    row_nsplit[i] = decode_splits(ctx[i]);
    for (int sp = 0; sp < row_nsplit[i]; ++sp) {
      work.push_back(i);
      work.push_back(sp);
    }
    n_work += row_nsplit[i];
    bo += np;
  }
  const int g = nq / nkv;
  std::vector<int32_t> host;
  auto put = [&](const std::vector<int32_t>& v) {
    const size_t off = host.size();
    host.insert(host.end(), v.begin(), v.end());
    host.resize((host.size() + 63) / 64 * 64, 0);
    return off;
  };
  const size_t o_work = put(work), o_ctx = put(row_ctx), o_q = put(row_q), o_bt = put(row_bt), o_rw = put(row_work),
               o_ns = put(row_nsplit), o_tab = put(bt);
  const size_t part_floats = static_cast<size_t>(n_work) * nkv * g * (hd + 2);
  OpBuffer buf;
  HIP_TRY(nullptr, hipMalloc(&buf.p, host.size() * 4 + part_floats * 4 + 256));
  int32_t* dev = static_cast<int32_t*>(buf.p);
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIP_TRY(nullptr, hipMemcpyAsync(dev, host.data(), host.size() * 4, hipMemcpyHostToDevice, s));
  metro::AttnArgs a{};
  a.q = q;
  a.kv = kv;
  a.work = dev + o_work;
  a.row_ctx = dev + o_ctx;
  a.row_qrow = dev + o_q;
  a.row_bt = dev + o_bt;
  a.row_work = dev + o_rw;
  a.row_nsplit = dev + o_ns;
  a.bt = dev + o_tab;
  a.part = reinterpret_cast<float*>(dev + host.size());
  a.out = out;
  a.n_work = n_work;
  a.rows = rows;
  a.nq = nq;
  a.nkv = nkv;
  a.hd = hd;
  a.scale = 1.0f / std::sqrt(static_cast<float>(hd));
  HIP_TRY(nullptr, metro::launch_attn_decode(a, s));
  if (n_work > rows) HIP_TRY(nullptr, metro::launch_attn_combine(a, s));
  HIP_TRY(nullptr, hipStreamSynchronize(s));
  return METRO_OK;
}

metro_status metro_op_attn_decode_noalloc(const uint16_t* q, const uint16_t* kv, int32_t n_pages, int32_t nq,
                                          int32_t nkv, int32_t hd, int32_t rows, const int32_t* ctx,
                                          const int32_t* block_tables, uint16_t* out, void* stream) {
  g_err.clear();
  metro_status st = check_attn_shape(nq, nkv, hd, n_pages, q, kv, out);
  if (st != METRO_OK) return st;
  if (rows < 0 || (rows > 0 && (!q || !kv || !ctx || !block_tables || !out)))
    return fail(METRO_E_INVAL, "attn_decode_noalloc: NULL argument or rows < 0");
  if (rows == 0) return METRO_OK;
  // sizes and checks on the host, without building anything
  int64_t pages = 0, n_work = 0;
  for (int i = 0; i < rows; ++i) {
    if (ctx[i] < 1) return fail(METRO_E_INVAL, "attn_decode_noalloc: row %d sees %d keys", i, ctx[i]);
    const int np = (ctx[i] + 15) / 16;
    for (int j = 0; j < np; ++j) {
      const int32_t id = block_tables[pages + j];
      if (id < 0 || id >= n_pages) return fail(METRO_E_INVAL, "attn_decode_noalloc: page id %d out of range", id);
    }
    pages += np;
    n_work += decode_splits(ctx[i]);
  }
  auto span = [](int64_t ints) { return (ints * 4 + 255) / 256 * 256; };
  const int g = nq / nkv;
  const int64_t part_bytes = n_work * nkv * g * (hd + 2) * 4;
  const int64_t need = 5 * span(rows) + span(pages) + span(2 * n_work) + part_bytes;
  if (need > static_cast<int64_t>(kScratchBytes))
    return fail(METRO_E_CAPACITY, "attn_decode_noalloc: %lld scratch bytes needed, %zu available",
                (long long)need, kScratchBytes);
  void* base = nullptr;
  st = scratch_on_current_device(&base);
  if (st != METRO_OK) return st;
  char* at = static_cast<char*>(base);
  auto take = [&](int64_t bytes) {
    char* p = at;
    at += bytes;
    return p;
  };
  int32_t* d_ctx = reinterpret_cast<int32_t*>(take(span(rows)));
  int32_t* d_q = reinterpret_cast<int32_t*>(take(span(rows)));
  int32_t* d_bto = reinterpret_cast<int32_t*>(take(span(rows)));
  int32_t* d_work0 = reinterpret_cast<int32_t*>(take(span(rows)));
  int32_t* d_ns = reinterpret_cast<int32_t*>(take(span(rows)));
  int32_t* d_bt = reinterpret_cast<int32_t*>(take(span(pages)));
  int32_t* d_work = reinterpret_cast<int32_t*>(take(span(2 * n_work)));
  float* d_part = reinterpret_cast<float*>(take(part_bytes));
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIP_TRY(nullptr, hipMemcpyAsync(d_ctx, ctx, rows * 4, hipMemcpyHostToDevice, s));
  HIP_TRY(nullptr, hipMemcpyAsync(d_bt, block_tables, pages * 4, hipMemcpyHostToDevice, s));
  hipLaunchKernelGGL(describe_decode_kernel, dim3(1), dim3(64), 0, s, d_ctx, rows, d_q, d_bto, d_work0, d_ns,
                     d_work);
  HIP_TRY(nullptr, hipGetLastError());
  metro::AttnArgs a{};
  a.q = q;
  a.kv = kv;
  a.work = d_work;
  a.row_ctx = d_ctx;
  a.row_qrow = d_q;
  a.row_bt = d_bto;
  a.row_work = d_work0;
  a.row_nsplit = d_ns;
  a.bt = d_bt;
  a.part = d_part;
  a.out = out;
  a.n_work = static_cast<int>(n_work);
  a.rows = rows;
  a.nq = nq;
  a.nkv = nkv;
  a.hd = hd;
  a.scale = 1.0f / std::sqrt(static_cast<float>(hd));
  HIP_TRY(nullptr, metro::launch_attn_decode(a, s));
  if (n_work > rows) HIP_TRY(nullptr, metro::launch_attn_combine(a, s));
  return METRO_OK;
}

metro_status metro_op_attn_prefill(const uint16_t* q, const uint16_t* kv, int32_t n_pages, int32_t nq, int32_t nkv,
                                   int32_t hd, int32_t n_items, const int32_t* cu_q, const int32_t* ctx_before,
                                   const int32_t* block_tables, uint16_t* out, void* stream) {
  g_err.clear();
  metro_status st = check_attn_shape(nq, nkv, hd, n_pages, q, kv, out);
  if (st != METRO_OK) return st;
  if (n_items < 0 || (n_items > 0 && (!q || !kv || !cu_q || !ctx_before || !block_tables || !out)))
    return fail(METRO_E_INVAL, "attn_prefill: NULL argument or n_items < 0");
  if (n_items == 0) return METRO_OK;
  if (cu_q[0] != 0) return fail(METRO_E_INVAL, "attn_prefill: cu_q[0] must be 0");
  std::vector<int32_t> pos, item_bt(n_items), bt;
  int64_t bo = 0;
  for (int i = 0; i < n_items; ++i) {
    const int c = cu_q[i + 1] - cu_q[i];
    if (c < 1 || ctx_before[i] < 0) return fail(METRO_E_INVAL, "attn_prefill: item %d has %d queries after %d keys",
                                                i, c, ctx_before[i]);
    for (int t = 0; t < c; ++t) pos.push_back(ctx_before[i] + t);
    const int np = (ctx_before[i] + c + 15) / 16;
    for (int j = 0; j < np; ++j) {
      const int32_t id = block_tables[bo + j];
      if (id < 0 || id >= n_pages) return fail(METRO_E_INVAL, "attn_prefill: page id %d out of range", id);
      bt.push_back(id);
    }
    item_bt[i] = static_cast<int32_t>(bo);
    bo += np;
  }
  const int tpb = metro::prefill_tokens_per_block(nq / nkv);
  std::vector<int32_t> blocks(3 * prefill_blocks(n_items, cu_q, tpb, nullptr));
  prefill_blocks(n_items, cu_q, tpb, blocks.data());
  std::vector<int32_t> host;
  auto put = [&](const std::vector<int32_t>& v) {
    const size_t off = host.size();
    host.insert(host.end(), v.begin(), v.end());
    host.resize((host.size() + 63) / 64 * 64, 0);
    return off;
  };
  const size_t o_pos = put(pos), o_ibt = put(item_bt), o_bt = put(bt), o_blk = put(blocks);
  OpBuffer buf;
  HIP_TRY(nullptr, hipMalloc(&buf.p, host.size() * 4 + 256));
  int32_t* dev = static_cast<int32_t*>(buf.p);
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIP_TRY(nullptr, hipMemcpyAsync(dev, host.data(), host.size() * 4, hipMemcpyHostToDevice, s));
  metro::PrefillAttnArgs a{};
  a.q = q;
  a.kv = kv;
  a.out = out;
  a.blocks = dev + o_blk;
  a.item_bt = dev + o_ibt;
  a.pos = dev + o_pos;
  a.bt = dev + o_bt;
  a.n_blocks = static_cast<int>(blocks.size() / 3);
  a.nq = nq;
  a.nkv = nkv;
  a.hd = hd;
  a.scale = 1.0f / std::sqrt(static_cast<float>(hd));
  HIP_TRY(nullptr, metro::launch_attn_prefill(a, s));
  HIP_TRY(nullptr, hipStreamSynchronize(s));
  return METRO_OK;
}

metro_status metro_op_argmax(const float* logits, int32_t rows, int32_t vocab, int32_t* out, void* stream) {
  g_err.clear();
  if (!logits || !out || rows < 0 || vocab <= 0 || vocab % 4) return fail(METRO_E_INVAL, "argmax: bad arguments");
  hipError_t e = metro::launch_argmax(logits, vocab, rows, out, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(nullptr, e, "launch_argmax");
  return METRO_OK;
}

}  // extern "C"
