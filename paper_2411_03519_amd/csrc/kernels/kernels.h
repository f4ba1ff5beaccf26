// Host-side launchers of the gfx950 kernels used by the runtime.
// Shapes are checked by the runtime before any launch; the launchers assume
// them (see each kernel's comment for what it requires).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace metro {

// --- launch timing ----------------------------------------------------------

// Events that the kernel dispatches of one launcher call record their start
// and end into (hipExtLaunchKernel puts them on the dispatch packet, so the
// interval is the kernels' execution, as a kernel trace reports it).  Set by
// the runtime around one launcher call while that kernel class is timed; null
// otherwise.  The first dispatch records the start; every dispatch records the
// end, so a launcher that issues a second kernel (the fixup of a split GEMM)
// is timed from the start of its first kernel to the end of its last.
struct LaunchEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};
extern thread_local LaunchEvents launch_events;

template <typename F, typename... Args>
inline void launch_kernel(F kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, Args... args) {
  hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, launch_events.start, launch_events.stop, 0u, args...);
  launch_events.start = nullptr;
}

// --- elementwise / row kernels (elementwise.hip) ---------------------------

// x[t, :] = E[tok[t], :] as fp32; a token outside [0, vocab) gives a NaN row.
hipError_t launch_embed(const int32_t* tok, const uint16_t* embed, int vocab, int d, float* x, int T,
                        hipStream_t s);

// h[r, :] = bf16(x[r, :] * rsqrt(mean(x[r, :]^2) + eps) * g); d % 4 == 0,
// d <= kRmsNormMaxDim.  With 0 < n_parts <= 8 the row first takes the pending
// GEMM slices: x[r, :] += sum_s parts[s][r][:] (slice stride rows*d), written
// back to x.  hipErrorInvalidValue outside these limits.
constexpr int kRmsNormMaxDim = 8192;
hipError_t launch_rmsnorm(float* x, int ldx, const uint16_t* g, float eps, uint16_t* h, int ldh, int rows, int d,
                          const float* parts, int n_parts, hipStream_t s);

// RoPE (rotate-half) on q and k of qkv [T, (nq+2nkv)*hd] fp32 at positions
// pos[t]; q -> bf16 [T, nq*hd]; k, v -> bf16 into the KV slot slot[t]
// (page*16 + offset) of this layer's slab (K row-major, V transposed).
// rope is [max_pos][hd/2] (cos, sin).
// With n_parts > 0, qkv is the first of n_parts slices [T][(nq+2nkv)hd] to sum.
hipError_t launch_rope_kv(const float* qkv, int n_parts, int T, int nq, int nkv, int hd, const int32_t* pos,
                          const int32_t* slot, const float2* rope, uint16_t* q, uint16_t* kv_layer,
                          hipStream_t s);

// out[i, :] = x[rows[i], :]
hipError_t launch_gather_rows(const float* x, int d, const int32_t* rows, int n, float* out, hipStream_t s);

// out[r] = lowest index of the maximum of logits[r, :]; -1 if the row has no
// non-NaN value.
hipError_t launch_argmax(const float* logits, int vocab, int rows, int32_t* out, hipStream_t s);

// Row placement of a weight matrix in its packed buffer: source row r goes to
// row map_row(m, r).  With half > 0 each head of 2*half rows is first
// interleaved for the rotate-half RoPE: blocks of 8 rows of the head's first
// half, each followed by the 8 matching rows of its second half, so that dims
// d and d + half meet in lanes l and l + 32 of a 16-row MFMA tile (half % 8
// == 0).  Then rows go in groups of `group` to blocks of `block` rows, offset
// by `shift` (gate/up: groups of 8 into blocks of 16, the up rows shifted by 8).
struct RowMap {
  int group, block, shift, half;
};
constexpr RowMap kRowsInOrder{16, 16, 0, 0};

// row of dim d (0 <= d < 2*half) of a head in the rotate-half interleave
__host__ __device__ __forceinline__ int rope_pair_row(int d, int half) {
  const int e = d < half ? d : d - half;
  return (e / 8) * 16 + (d < half ? 0 : 8) + e % 8;
}

__host__ __device__ __forceinline__ int64_t map_row(const RowMap& m, int64_t r) {
  if (m.half > 0) {
    const int64_t hd = 2 * m.half, d = r % hd;
    r = r - d + rope_pair_row(static_cast<int>(d), m.half);
  }
  return (r / m.group) * m.block + m.shift + r % m.group;
}

// Random initialisation of one logical weight tensor [rows, cols]: logical
// row r goes to row map_row(map, r) of the destination, which is row-major
// with row stride ld, or, with packed, in MFMA operand order (packed_offset)
// with ld = Kp.  Values are 0.02 * N(0, 1) from a SplitMix64-keyed Box-Muller
// draw, rounded to bf16.
hipError_t launch_init_normal(uint16_t* dst, int64_t ld, int rows, int cols, RowMap map, uint64_t key, bool packed,
                              hipStream_t s);

// Row-major bf16 [rows, cols] (row stride ld_src, device) -> rows map_row(map, r)
// of a packed [*, Kp] weight; columns cols .. Kp-1 are written as zero.
hipError_t launch_pack_weight(const uint16_t* src, int64_t ld_src, int rows, int cols, uint16_t* dst, int Kp,
                              RowMap map, hipStream_t s);
hipError_t launch_fill_bf16(uint16_t* dst, int64_t n, uint16_t value, hipStream_t s);

// Copy page src to page dst in every layer (page_elems bf16 per layer).
hipError_t launch_page_copy(uint16_t* pool, int64_t layer_stride, int64_t page_elems, int layers, int src,
                            int dst, hipStream_t s);

// --- GEMMs (gemm.hip) -------------------------------------------------------

enum GemmEpilogue {
  kEpiStoreF32 = 0,  // out_f32[m, n] = acc
  kEpiAddF32 = 1,    // out_f32[m, n] += acc   (residual stream)
  kEpiSwiGLU = 2,    // W rows in blocks of 16 = 8 gate rows, then the 8 up
                     // rows of the same features:
                     // out_bf16[m, j] = bf16(silu(gate_j) * up_j), N = 2 * F
  kEpiRopeKV = 3,    // QKV projection with W rows in the rotate-half
                     // interleave of RowMap: RoPE on q and k, q to its
                     // buffer, k and v to the row's KV cache slot
};

// Where the QKV epilogue puts its results (launch_gemm_rope_kv).
struct RopeKV {
  const int32_t* pos;   // [M] position of each row
  const int32_t* slot;  // [M] KV cache slot of each row (page * 16 + offset)
  const float2* rope;   // [max_context][hd / 2] (cos, sin)
  uint16_t* q;          // [M, nq, hd] bf16, rotated
  uint16_t* kv;         // this layer's slab of the KV pool
  int nq, nkv, hd;
};

// Y = X[M, Kp] (bf16, row stride ldx) x W[N, Kp]^T (bf16 in MFMA operand
// order, packed_offset; Kp % 128 == 0, N % 32 == 0), fp32 accumulation, then
// the epilogue.
// ldo is the row stride of the output in elements.  `part` is an fp32
// workspace of part_cap floats (or null).  With it a decode-sized GEMM
// (M <= kSplitMaxRows, fp32 epilogue) may split K over workgroups: it then
// writes *n_parts > 0 slices part[s][m][n] ([ks][M][N], ks <= 8) instead of
// applying the epilogue, and the consumer sums them in slice order.  A larger
// one with 256-row tiles (any epilogue) may split only the tiles of its last,
// partly filled round (up to CUs * 256 * 256 floats of part), and completes
// them itself (*n_parts stays 0).
// Kernel choice (plan_gemm): up to 64 rows the weight-streaming decode GEMM;
// then the tiled GEMM with 128 x 128 blocks (narrow products up to
// kMidMaxRows rows, wide ones while they fit the CUs), 256 (W rows) x 128
// blocks (wide products at up to 256 rows otherwise, narrow ones of up to 128
// rows that 128 x 128 blocks would leave mostly idle), or 256 x 256 blocks.
enum class GemmKind { kSkinny, kMid, kWide, kBig };
struct GemmPlan {
  GemmKind kind;
  int nt;          // row tiles per wave (decode kernel)
  int ks;          // k slices of every tile
  int tail_split;  // k slices of each tile from tail_first on (1: none)
  int tail_first;
};
constexpr int kMidMaxRows = 1000;
constexpr int kSplitMaxRows = 1024;
GemmPlan plan_gemm(int M, int N, int Kp, int epilogue, int64_t part_cap);
hipError_t launch_gemm(const uint16_t* X, int ldx, const uint16_t* W, int Kp, int M, int N, int epilogue,
                       float* out_f32, uint16_t* out_bf16, int ldo, float* part, int64_t part_cap, int* n_parts,
                       hipStream_t s);
// QKV projection (N = (nq + 2 nkv) * hd) with RoPE and the KV cache write in
// its epilogue, in place of launch_gemm + launch_rope_kv, for the shapes
// gemm_rope_kv_fused accepts: up to kRopeKVMaxRows rows (decode kernel), or
// the batches plan_gemm gives 256 x 256 tiles (prefill chunks); K is not split,
// so no slice sums are left.  hipErrorInvalidValue for other shapes.
constexpr int kRopeKVMaxRows = 64;
bool gemm_rope_kv_fused(int M, int N, int Kp);
hipError_t launch_gemm_rope_kv(const uint16_t* X, int ldx, const uint16_t* W, int Kp, int M, int N, const RopeKV& rk,
                               hipStream_t s);
// Apply the fp32 epilogue to KS slices: out (=|+=) sum_s part[s].
hipError_t launch_reduce_parts(const float* part, int KS, int M, int N, int epilogue, float* out, int ldo,
                               hipStream_t s);

// --- attention (attention.hip) ---------------------------------------------

// KV page layout per (layer, page, kv head): a K tile then a V^T tile of 16
// keys x hd (layouts in common.h).
struct AttnArgs {
  const uint16_t* q;        // [rows_total, nq, hd] bf16 (row = query token)
  const uint16_t* kv;       // this layer's slab of the KV pool
  const int32_t* work;      // [n_work][2]: (row, split)
  const int32_t* row_ctx;   // [rows]: keys visible to the row (0 .. ctx-1)
  const int32_t* row_qrow;  // [rows]: row of q / out for this row
  const int32_t* row_bt;    // [rows]: offset of the row's block table in bt
  const int32_t* row_work;  // [rows]: first work item of the row
  const int32_t* row_nsplit;// [rows]: work items of the row
  const int32_t* bt;        // block tables
  float* part;              // [n_work][nkv][group][hd + 2] fp32 split states
  uint16_t* out;            // [rows_total, nq*hd] bf16
  int n_work, rows, nq, nkv, hd;
  float scale;              // 1/sqrt(hd)
};

// Decode attention: one workgroup per (work item, kv head), a work item being
// up to kDecodePagesPerSplit pages of one row.  Rows of one split are final;
// the others leave (max, sum, output) states for launch_attn_combine.
constexpr int kDecodePagesPerSplit = 128;
hipError_t launch_attn_decode(const AttnArgs& a, hipStream_t s);
hipError_t launch_attn_combine(const AttnArgs& a, hipStream_t s);

struct PrefillAttnArgs {
  const uint16_t* q;        // [T, nq, hd] bf16
  const uint16_t* kv;       // this layer's slab of the KV pool
  uint16_t* out;            // [T, nq*hd] bf16
  const int32_t* blocks;    // [n_blocks][3]: (item, first row, rows) of a query block
  const int32_t* item_bt;   // [items]: offset of the item's block table in bt
  const int32_t* pos;       // [T]: absolute position of each row
  const int32_t* bt;        // block tables
  int n_blocks, nq, nkv, hd;
  float scale;
};

// Causal flash attention of prefill rows over their sequence's pages (which
// already hold this call's keys).  Query blocks hold prefill_tokens_per_block
// consecutive rows of one item.
hipError_t launch_attn_prefill(const PrefillAttnArgs& a, hipStream_t s);
int prefill_tokens_per_block(int group);

}  // namespace metro
