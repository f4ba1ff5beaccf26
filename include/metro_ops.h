/*
 * metro_ops.h -- single kernels of libmetro.so's forward pass, exported so
 * that each can be checked on its own against a CPU reference.  The model
 * entry points in metro.h are what a serving loop calls; these run one step
 * of it on caller-owned device buffers.
 *
 * All pointers are device pointers on the current HIP device; work is
 * enqueued on `stream` (a hipStream_t, NULL = default stream).  Return value
 * and metro_last_error() as in metro.h; a launch failure returns METRO_E_HIP.
 */
#ifndef METRO_OPS_H
#define METRO_OPS_H

#include <stdint.h>

#include "metro.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Weight layout of the projection GEMMs.  W_packed receives the bf16 matrix
 * W [N, Kp] (W[n, k] = W_rowmajor[n * ld + k] for k < K, 0 for K <= k < Kp) in
 * matrix-core operand order: 16 x 32 tiles (16 rows, 32 columns), tiles
 * row-major over (n / 16, k / 32), tile (tn, tk) stored as 64 chunks of 8
 * elements in the order c = r + 16 g, chunk c = W[16 tn + r][32 tk + 8 g ..
 * 8 g + 7]; i.e. W[n, k] sits at element
 *   ((n/16 * Kp/32 + k/32) * 64 + n%16 + 16 * ((k/8)%4)) * 8 + k%8.
 * W_rowmajor: device bf16 [N, ld], ld >= K; W_packed: device bf16, N * Kp
 * elements, not overlapping W_rowmajor.  N % 16 == 0, Kp % 128 == 0,
 * 0 < K <= Kp.  Errors: E_INVAL for shapes outside these rules or NULL. */
metro_status metro_op_pack_weight(const uint16_t* W_rowmajor, int32_t ld, int32_t N, int32_t K, int32_t Kp,
                                  uint16_t* W_packed, void* stream);

/* Projection GEMM of the Llama block (QKV, O, gate/up, down, LM head):
 *   acc[m, n] = sum_k X[m, k] * W[n, k]   (bf16 operands, fp32 accumulation)
 * X: bf16 [M, ldx] row-major, the first Kp columns used; W: bf16 [N, Kp] in
 * the layout metro_op_pack_weight writes; Kp % 128 == 0, N % 32 == 0,
 * ldx % 8 == 0; X, W, workspace and out_f32 16-byte aligned, out_bf16 8-byte
 * aligned (E_INVAL otherwise: the kernels move 16-byte pieces).
 * epilogue:
 *   0  out_f32[m*ldo + n]  = acc[m, n]
 *   1  out_f32[m*ldo + n] += acc[m, n]                       (residual add)
 *   2  W rows come in blocks of 16 = 8 gate rows then the 8 up rows of the
 *      same features (block b: gate_j, j = 8b .. 8b+7, then up_j);
 *      out_bf16[m*ldo + j] = bf16(silu(gate_j) * up_j), j < N/2
 *      (SwiGLU, Shazeer 2020).
 * workspace: NULL, or device fp32 [8][M][N]; when given, a decode-sized GEMM
 * (M <= 1024, epilogue 0 or 1) may run the k-split form the model uses (slices in
 * the workspace, then summed in slice order into the output), and a larger one
 * (any epilogue) may split the 256 x 256 tiles of its last, partly filled
 * round of workgroups over k the same way.  Its contents on return are
 * unspecified.
 * Errors: E_INVAL for shapes outside these rules or a NULL operand. */
metro_status metro_op_gemm(const uint16_t* X, int32_t ldx, const uint16_t* W, int32_t Kp, int32_t M, int32_t N,
                           int32_t epilogue, float* out_f32, uint16_t* out_bf16, int32_t ldo, float* workspace,
                           void* stream);

/* The kernels metro_op_gemm would run for a product (the model chooses by the
 * same rules), for inspection and tests; host only, no device work.
 * has_workspace: nonzero as for a non-NULL workspace.  *kind: 0 decode kernel
 * (weight streaming, up to 64 rows), 1 tiled with 128 x 128 blocks, 2 tiled
 * with 256 (W rows) x 128 blocks, 3 tiled with 256 x 256 blocks.  *k_slices:
 * k slices of every block (> 1 only with a workspace); *tail_split: k slices
 * of each block of the last, partly filled round of workgroups (1: none).
 * Counts compute units of the current device (256 when there is none).
 * Errors: E_INVAL (shape rules of metro_op_gemm, NULL outputs). */
metro_status metro_op_gemm_plan(int32_t M, int32_t N, int32_t Kp, int32_t epilogue, int32_t has_workspace,
                                int32_t* kind, int32_t* k_slices, int32_t* tail_split);

/* RMSNorm (Zhang & Sennrich 2019): h[r, :] = bf16(x[r, :] / sqrt(mean(x[r, :]^2)
 * + eps) * g), x fp32 [rows, d], g bf16 [d], h bf16 [rows, d], d % 4 == 0, d <= 8192;
 * x 16-byte aligned, g and h 8-byte aligned (E_INVAL otherwise). */
metro_status metro_op_rmsnorm(float* x, const uint16_t* g, float eps, uint16_t* h, int32_t rows, int32_t d,
                              void* stream);

/* Greedy choice: out[r] = lowest index of the maximum of logits[r, :] (fp32
 * [rows, vocab], vocab % 4 == 0); NaN values are skipped, -1 if none is left. */
metro_status metro_op_argmax(const float* logits, int32_t rows, int32_t vocab, int32_t* out, void* stream);

/* KV pages as the attention kernels read them (the layout of one layer's slab
 * of the model's pool): page p holds 16 consecutive positions; its bytes are
 * [K | V][kv_head][tile], a tile being 16 keys x head_dim bf16 in matrix-core
 * operand order:
 *   K tile:   key r, dim e  at ((e/32 * 4 + (e/8)%4) * 16 + r) * 8 + e%8
 *   V^T tile: dim e, key r  at ((e/32 * 4 + r/4) * 16 + e%16) * 8 + ((e/16)%2) * 4 + r%4
 * so that element (page, K|V = c, head h, ...) sits at
 *   page * (2 * n_kv_heads * 16 * head_dim) + (c * n_kv_heads + h) * 16 * head_dim + offset.
 * Page ids index this array (0 <= id < n_pages). */

/* Decode attention of the model's forward pass (grouped-query, causal, paged;
 * the attention of the Llama decoder the paper serves, §4.1): for each row i
 * and query head j, with kv head h = j / (nq / nkv) and keys t = 0 .. ctx[i]-1
 * of the row's pages,
 *   out[i, j, :] = bf16( sum_t softmax_t(q[i, j, :] . K[t, h, :] / sqrt(hd)) V[t, h, :] )
 * with fp32 scores, softmax and accumulation (the weights enter the bf16
 * matrix cores as a bf16 pair hi + lo).  Rows of more than 128 pages are cut
 * into 128-page work items whose states are merged in order, as in the model.
 *   q            device bf16 [rows, nq, hd], 16-byte aligned
 *   kv           device bf16, n_pages pages in the layout above, 16-byte aligned
 *   ctx          host int32 [rows], >= 1
 *   block_tables host int32, row after row: ceil(ctx[i] / 16) page ids each
 *   out          device bf16 [rows, nq * hd], 8-byte aligned
 * hd is 64 or 128; nq / nkv is 1, 2, 4 or 8.  Allocates and frees device
 * memory for its descriptors and split states and returns after the kernels
 * have finished on `stream` (a test entry point, not for serving loops).
 * Errors: E_INVAL (shapes, NULL, page id out of range), E_HIP. */
metro_status metro_op_attn_decode(const uint16_t* q, const uint16_t* kv, int32_t n_pages, int32_t nq, int32_t nkv,
                                  int32_t hd, int32_t rows, const int32_t* ctx, const int32_t* block_tables,
                                  uint16_t* out, void* stream);

/* Chunked-prefill attention of the model's forward pass: item i has
 * c_i = cu_q[i+1] - cu_q[i] queries (rows cu_q[i] .. cu_q[i+1]-1 of q and
 * out) at positions ctx_before[i] .. ctx_before[i] + c_i - 1, and its pages
 * hold keys 0 .. ctx_before[i] + c_i - 1 (the chunk's own keys included).
 * The query at position p sees keys 0 .. p (causal), otherwise as
 * metro_op_attn_decode.
 *   q            device bf16 [cu_q[n_items], nq, hd]
 *   cu_q         host int32 [n_items + 1], cu_q[0] = 0, each item >= 1 query
 *   ctx_before   host int32 [n_items], >= 0
 *   block_tables host int32, item after item: ceil((ctx_before[i] + c_i) / 16) ids
 *   out          device bf16 [cu_q[n_items], nq * hd]
 * Synchronous as metro_op_attn_decode.  Errors: E_INVAL, E_HIP. */
metro_status metro_op_attn_prefill(const uint16_t* q, const uint16_t* kv, int32_t n_pages, int32_t nq, int32_t nkv,
                                   int32_t hd, int32_t n_items, const int32_t* cu_q, const int32_t* ctx_before,
                                   const int32_t* block_tables, uint16_t* out, void* stream);

/* metro_op_attn_decode for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels and results, with the descriptors and split
 * states in a fixed device array of 64 MiB that the library holds on each GPU
 * it runs on until the process ends, instead of a per-call allocation.  No
 * hipMalloc or hipFree, no allocating library call.  Arguments as for
 * metro_op_attn_decode (ctx and block_tables are host arrays, copied to the
 * device on `stream`).  Asynchronous: out is valid once `stream` has reached
 * the call.  Every call on one GPU uses that GPU's array, so calls that
 * overlap on one GPU (other streams or host threads) race; calls ordered on
 * one stream do not.  Needs 5 * rows + pages + 2 * work items int32 (each
 * rounded up to 256 bytes) plus work items * nkv * (nq / nkv) * (hd + 2) fp32,
 * a work item being up to 128 pages of one row.
 * Errors: E_INVAL as metro_op_attn_decode, E_CAPACITY when that exceeds the
 * array, E_HIP. */
metro_status metro_op_attn_decode_noalloc(const uint16_t* q, const uint16_t* kv, int32_t n_pages, int32_t nq,
                                          int32_t nkv, int32_t hd, int32_t rows, const int32_t* ctx,
                                          const int32_t* block_tables, uint16_t* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* METRO_OPS_H */
