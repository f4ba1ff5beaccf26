/*
 * metro.h -- C ABI of libmetro.so: batched Llama-style forward pass (chunked
 * prefill + greedy decode) over many agents' paged KV caches, on one AMD
 * Instinct MI355X (gfx950).
 *
 * Why this boundary.  AI Metropolis (arXiv 2411.03519) spends about 95% of a
 * multi-agent simulation in LLM inference (§1) and gains its speed-up by
 * letting more ready agents share one inference batch (§1, §3.2).  Each agent
 * issues LLM requests from its own thread through a thin shim to a serving
 * engine, the simulation engine being decoupled from it (§3.6); a
 * worker runs the requests of a ready cluster together (§3.1, Algorithm 3);
 * generation has a fixed length with no end-of-sequence stop (§4.1, replay
 * with ignore_eos); requests are never preempted mid-inference (§3.5); and a
 * common prompt prefix may be shared (§4.1, prefix caching).  This header is
 * that shim's lower half: one sequence handle per agent request, calls that
 * run a batch of ready requests, results returned as logits and greedy tokens.
 *
 * The network is the public Llama decoder (RMSNorm, rotary embedding in the
 * rotate-half pairing, grouped-query attention with contiguous head groups,
 * SwiGLU feed-forward, untied LM head, no biases), the model family the paper
 * serves (§4.1, Llama-3 8B and 70B).
 *
 * Numerics.  Weights, the KV cache and every GEMM activation operand are
 * bfloat16; products accumulate in fp32; the residual stream, RMS statistics,
 * attention scores, softmax and attention accumulation are fp32; logits are
 * fp32.  Greedy choice = lowest index among the maximal fp32 logits.
 * Batch dependence: a projection's kernel and k split are chosen from the
 * number of rows of the call, so a sequence's results depend on how many
 * others share its call by fp32 rounding (at Llama-3-8B widths, depth 2,
 * logits move by up to a few 1e-2 between batch sizes, the size of the fp32
 * noise itself); calls of equal row count give bitwise equal rows whatever
 * the other sequences are, and page placement never changes a result.
 *
 * Conventions for every call below.
 *  - Return value: METRO_OK or a negative metro_status; metro_last_error()
 *    then returns a thread-local message naming what failed.
 *  - Host state is all-or-nothing: a call that fails with any status other
 *    than METRO_E_HIP changes no sequence and no page.
 *  - METRO_E_HIP (a HIP runtime error or a failed launch) poisons the model:
 *    every later call on it returns METRO_E_HIP; only metro_destroy_model is
 *    still valid.
 *  - Device pointers are plain HIP device addresses on the model's device;
 *    host pointers are ordinary host memory, read during the call only.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Device work is
 *    enqueued asynchronously; outputs are valid once the stream has reached the
 *    call.  A model is not thread-safe, and all calls on one model must be
 *    ordered on one stream (the model owns one set of scratch buffers).
 */
#ifndef METRO_H
#define METRO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define METRO_ABI_VERSION 2

typedef enum metro_status {
  METRO_OK = 0,
  METRO_E_INVAL = -1,     /* bad argument: null pointer, bad shape, token id, duplicate sequence */
  METRO_E_NOMEM = -2,     /* a device or host allocation failed */
  METRO_E_NOPAGES = -3,   /* the KV page pool cannot hold the call's new tokens */
  METRO_E_SEQ = -4,       /* unknown or closed sequence handle */
  METRO_E_CAPACITY = -5,  /* a configured maximum (batch, tokens, context, sequences) exceeded */
  METRO_E_HIP = -6        /* HIP runtime error; the model is poisoned */
} metro_status;

/* Model shape and capacity.  Requirements (else METRO_E_INVAL):
 * d_model % 128 == 0; head_dim is 64 or 128; n_heads % n_kv_heads == 0;
 * n_heads / n_kv_heads in {1, 2, 4, 8}; n_heads*head_dim % 128 == 0;
 * ffn_dim % 16 == 0; vocab % 32 == 0;
 * page_size == 16; all counts > 0. */
typedef struct metro_config {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_heads;        /* query heads */
  int32_t n_kv_heads;     /* key/value heads (GQA groups) */
  int32_t head_dim;
  int32_t ffn_dim;
  int32_t vocab;
  float rope_base;        /* RoPE theta base, e.g. 1e4 or 5e5 */
  float rms_eps;          /* RMSNorm epsilon, e.g. 1e-5 */
  int32_t page_size;      /* tokens per KV page; must be 16 */
  int32_t max_batch;      /* max sequences (items) in one call */
  int32_t max_tokens;     /* max new tokens summed over the items of one call */
  int32_t max_context;    /* max tokens held by one sequence */
  int32_t max_seqs;       /* max sequences open at once */
  int64_t kv_pool_bytes;  /* bytes of HBM for KV pages; 0 = all free memory
                             left after weights and scratch, minus 2 GiB */
} metro_config;

/* Weight tensors.  Every matrix is row-major [out, in] bf16, as in the Llama
 * checkpoints: EMBED and LM_HEAD [vocab, d_model]; WQ [n_heads*head_dim,
 * d_model]; WK, WV [n_kv_heads*head_dim, d_model]; WO [d_model,
 * n_heads*head_dim]; WGATE, WUP [ffn_dim, d_model]; WDOWN [d_model, ffn_dim];
 * the three norms are [d_model] gains. */
typedef enum metro_weight_id {
  METRO_W_EMBED = 0,
  METRO_W_FINAL_NORM = 1,
  METRO_W_LM_HEAD = 2,
  METRO_W_ATTN_NORM = 3,   /* per layer from here on */
  METRO_W_WQ = 4,
  METRO_W_WK = 5,
  METRO_W_WV = 6,
  METRO_W_WO = 7,
  METRO_W_FFN_NORM = 8,
  METRO_W_WGATE = 9,
  METRO_W_WUP = 10,
  METRO_W_WDOWN = 11
} metro_weight_id;

typedef struct metro_model metro_model; /* opaque */

typedef struct metro_model_info {
  int64_t weight_bytes;     /* device bytes of packed weights */
  int64_t scratch_bytes;    /* device bytes of activation scratch */
  int64_t kv_pool_bytes;    /* device bytes of the KV page pool */
  int64_t kv_bytes_per_token; /* all layers, K and V */
  int32_t n_pages;          /* pages in the pool */
  int32_t free_pages;       /* pages referenced by no sequence and not held by the prefix cache */
  int32_t open_seqs;
  int32_t device;           /* HIP device ordinal */
} metro_model_info;

/* ABI version of the loaded library (METRO_ABI_VERSION it was built with). */
int32_t metro_abi_version(void);

/* Thread-local message for the last failing call on this thread ("" if none). */
const char* metro_last_error(void);

/* Static name of a status code. */
const char* metro_status_name(int32_t status);

/* Create a model of the Llama family the paper serves (§4.1: Llama-3 8B and
 * 70B) on the current HIP device.  Allocates the packed weights, the
 * KV page pool and scratch sized for cfg's maxima.  Every weight is filled on
 * the device from a counter-based generator keyed by init_seed: matrices with
 * N(0, 0.02) values rounded to bf16, norm gains with 1.0 (the random
 * initialisation used when no checkpoint is loaded).  metro_load_weight then
 * replaces any tensor.  On success *out owns everything; free it with
 * metro_destroy_model.  Debugging: with the environment variable
 * METRO_SYNC_CHECK set to a non-zero integer when the model is created, every
 * kernel launch of the model is followed by a wait on its stream and an error
 * check, so that a failing kernel is reported (E_HIP, metro_last_error) by
 * the launch that ran it; results are unchanged, calls become synchronous.
 * Errors: E_INVAL (cfg), E_NOMEM, E_HIP. */
metro_status metro_create_model(const metro_config* cfg, uint64_t init_seed, metro_model** out);

/* Free every device and host resource of the model (NULL is a no-op).
 * Synchronises the device first. */
void metro_destroy_model(metro_model* model);

/* Copy one weight tensor from host bf16 (uint16 storage) into the model's
 * packed device layout.  layer is ignored (pass -1) for EMBED, FINAL_NORM and
 * LM_HEAD.  n_elems must equal the tensor's element count.  Synchronous.
 * Errors: E_INVAL (id, layer, count, null), E_HIP. */
metro_status metro_load_weight(metro_model* model, int32_t weight_id, int32_t layer,
                               const uint16_t* host_bf16, int64_t n_elems);

metro_status metro_model_get_info(const metro_model* model, metro_model_info* info);

/* Open an empty sequence: the context of one agent's LLM request (§3.1: a
 * worker issues the requests of the agents of a ready cluster).  With the
 * prefix cache on, the pages its prefills fill are entered in the cache.
 * Errors: E_CAPACITY (max_seqs open). */
metro_status metro_seq_open(metro_model* model, int64_t* seq);

/* Automatic prefix caching: the common-prompt-prefix cache of the serving
 * engine (§4.1; the paper reports about 20% more throughput with it on).
 *
 * A page (16 positions) enters the cache once a prefill has filled it while
 * every earlier token of its sequence also came from prefills (the host has
 * seen them all).  It is keyed by its 16 token ids and the cached page before
 * it, so a key stands for the exact token prefix up to the page's end; a hit
 * is never approximate.  metro_seq_open_cached attaches the longest chain of
 * cached pages that matches a prompt, by reference; the caller then prefills
 * only the rest.  A decode step, whose tokens live on the device, ends a
 * sequence's entries; forked sequences enter none.
 *
 * The cache holds one reference per cached page.  Pages that only the cache
 * holds are reclaimed when a call needs pages and too few are free, and when
 * entering a page would exceed max_pages: least recently used first, a page
 * never before the cached pages that continue it.  When two sequences fill
 * equal prefixes, the first one's page stays cached and the second keeps a
 * reference to it until it closes.
 *
 * max_pages > 0 turns the cache on (or changes its limit, evicting down to it
 * where it can); 0 turns it off and releases every cached page.  Off by
 * default.  Host bookkeeping only; no device work.  Errors: E_INVAL. */
metro_status metro_prefix_cache(metro_model* model, int32_t max_pages);

typedef struct metro_prefix_cache_stats {
  int32_t pages;            /* pages the cache holds */
  int32_t limit;            /* max_pages (0 = off) */
  int64_t lookup_tokens;    /* prompt tokens offered to metro_seq_open_cached */
  int64_t hit_tokens;       /* of which attached from the cache */
  int64_t inserted;         /* pages entered so far */
  int64_t evicted;          /* pages released so far */
} metro_prefix_cache_stats;

metro_status metro_prefix_cache_get_stats(const metro_model* model, metro_prefix_cache_stats* stats);

/* Open a sequence for a prompt tokens[0 .. n_tokens) (host int32) and attach
 * the longest chain of cached pages matching its first tokens, at most
 * n_tokens - 1 of them, so that at least one token is left for the prefill
 * that returns the prompt's next-token logits.  *n_cached receives the number
 * of tokens attached (a multiple of 16; 0 with the cache off); the sequence
 * starts at that length and the caller prefills tokens[*n_cached ..).
 * Errors: E_INVAL (NULL, n_tokens < 0), E_CAPACITY (max_seqs open). */
metro_status metro_seq_open_cached(metro_model* model, const int32_t* tokens, int32_t n_tokens, int64_t* seq,
                                   int32_t* n_cached);

/* Open a new sequence whose first n_tokens positions are those of src
 * (0 < n_tokens <= length of src).  Whole pages are shared by reference (never
 * written again by either sequence); a partly filled last page is copied on
 * `stream`.  This is the by-reference sharing of a common prompt prefix
 * (§4.1, prefix caching).
 * The new sequence enters no pages in the prefix cache.
 * Errors: E_SEQ, E_INVAL, E_CAPACITY, E_NOPAGES, E_HIP. */
metro_status metro_seq_fork(metro_model* model, int64_t src, int32_t n_tokens, void* stream,
                            int64_t* seq);

/* Close a sequence and drop its page references.  Errors: E_SEQ. */
metro_status metro_seq_close(metro_model* model, int64_t seq);

/* Tokens currently held by a sequence.  Errors: E_SEQ. */
metro_status metro_seq_length(const metro_model* model, int64_t seq, int32_t* length);

/* The sequence's block table: page ids for positions 16*i .. 16*i+15.  Writes
 * min(cap, n) ids to pages (may be NULL when cap == 0) and n to *n_pages. */
metro_status metro_seq_pages(const metro_model* model, int64_t seq, int32_t* pages, int32_t cap,
                             int32_t* n_pages);

/* Chunked prefill: append a chunk of prompt tokens to each of n_items
 * sequences and run the forward pass over all of them in one batch (the
 * prompts of a ready cluster's requests served together, §3.1 and
 * Algorithm 3; more ready agents make larger batches, §3.2).
 *   seqs      host [n_items] distinct open sequences
 *   cu_tokens host [n_items+1] prefix sums: item i owns tokens[cu[i] .. cu[i+1])
 *             (cu[0] == 0, each item >= 1 token, cu[n_items] <= max_tokens)
 *   tokens    host int32 token ids in [0, vocab)
 *   logits    device fp32 [n_items, vocab] or NULL: logits of each item's last
 *             new position
 *   next_tok  device int32 [n_items] or NULL: greedy token of that position
 * Positions are appended at length .. length+c-1 of each sequence.  Pages for
 * the new tokens are taken from the pool for all items or none (reclaiming
 * pages only the prefix cache holds when too few are free).
 * Errors: E_INVAL, E_SEQ, E_CAPACITY, E_NOPAGES, E_HIP. */
metro_status metro_prefill_chunk(metro_model* model, int32_t n_items, const int64_t* seqs,
                                 const int32_t* cu_tokens, const int32_t* tokens, float* logits,
                                 int32_t* next_tok, void* stream);

/* One decode step: append one token to each of `batch` sequences and return
 * the next-token distribution of each (one token for every ready agent's
 * running request, §3.2; generation runs a fixed number of steps with no
 * end-of-sequence stop, as in the replay of §4.1).
 *   seqs       host [batch] distinct open sequences, each of length >= 1
 *   tokens_dev device int32 [batch] token ids (e.g. the previous step's
 *              next_tok); an id outside [0, vocab) turns that row's outputs
 *              into NaN logits and next_tok -1 instead of faulting
 *   logits     device fp32 [batch, vocab] or NULL
 *   next_tok   device int32 [batch] or NULL
 * Errors: E_INVAL, E_SEQ, E_CAPACITY, E_NOPAGES, E_HIP. */
metro_status metro_decode_step(metro_model* model, int32_t batch, const int64_t* seqs,
                               const int32_t* tokens_dev, float* logits, int32_t* next_tok,
                               void* stream);

/* Kernel classes of the forward pass, for launch timing. */
typedef enum metro_kernel_class {
  METRO_K_EMBED = 0,
  METRO_K_RMSNORM = 1,
  METRO_K_GEMM_QKV = 2,
  METRO_K_ROPE_KV = 3,
  METRO_K_ATTENTION = 4,   /* decode attention includes the merge of context splits */
  METRO_K_GEMM_O = 6,
  METRO_K_GEMM_GATE_UP = 7,
  METRO_K_GEMM_DOWN = 8,
  METRO_K_LM_HEAD = 9,
  METRO_K_ARGMAX = 10
} metro_kernel_class;

/* Launch timing (instrumentation).  After metro_profile_start, every launch
 * of kernel_class in the given phase (0 = any call, 1 = prefill_chunk,
 * 2 = decode_step) is bracketed by a pair of HIP events on the call's stream;
 * metro_profile_stop waits for the recorded events and returns the summed
 * GPU time between each pair and the number of launches timed, then turns
 * timing off.  Only one class is timed at a time; starting again resets the
 * sums.  Errors: E_INVAL (class, phase, NULL), E_HIP. */
metro_status metro_profile_start(metro_model* model, int32_t kernel_class, int32_t phase);
metro_status metro_profile_stop(metro_model* model, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* METRO_H */
