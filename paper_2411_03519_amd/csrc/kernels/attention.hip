// Paged grouped-query attention on gfx950 with MFMA.
//
// KV page layout (per layer, page, kv head): K and V^T tiles of 16 keys x hd
// in the layouts of common.h (k_tile_offset, vt_tile_offset), bf16: every
// matrix-core operand is one 16-byte load per lane and every load instruction
// reads 1 KiB of a tile contiguously.
//
//   scores  S^T[key][q] = sum_d K[key][d] Q[q][d]       v_mfma_f32_16x16x32_bf16
//           A = K rows (16 keys), B = Q^T (16 query columns)
//   output  O^T[d][q] += sum_key V^T[d][key] P^T[key][q] v_mfma_f32_16x16x16_bf16
//           (decode, one page) or 16x16x32 over a page pair (prefill)
//
// The MFMA output of S^T leaves lane l with keys 4(l/16)+i of query column
// l%16, which is exactly the B operand the P.V product needs, so the softmax
// runs in registers with no lane shuffles except the two cross-row steps of
// the row maximum.  The query columns are the (token, head) pairs of one GQA
// group, so a K/V page is read once per group.
//
// Precision: scores, the running max/sum and the output accumulators are fp32.
// P enters the bf16 matrix core as hi = bf16(p) plus lo = bf16(p - hi) (two
// MFMAs), which keeps p to about 16 significant bits.
//
// Decode: one workgroup per (work item, kv head), a work item being up to 128
// pages of one row, so that long rows spread over several CUs; its waves take
// the pages round-robin and merge through LDS in wave order.  Rows of several
// work items leave their states in a workspace and a small kernel merges them
// in split order (an agent-scope fence in every workgroup, which an in-kernel
// merge would need, costs L2 write-backs on the multi-XCD chip).  The split
// count depends on the row's own context length only, never on the batch.
//
// Prefill (flash attention): one workgroup = (query block, kv head); the K and
// V pages of the block's visible context go through LDS in pairs, by direct
// loads into a 4-stage ring (three pairs in flight while one is consumed), and
// are shared by the eight waves (two per SIMD); causal masking per element.
#include "common.h"
#include "kernels.h"

namespace metro {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegBig = -1.0e30f;

typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma_k32(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma_k16(uint2 a, uint2 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, a), __builtin_bit_cast(s16x4, b), c,
                                                   0, 0, 0);
}

// 2^x by the hardware instruction (v_exp_f32, about 1 ulp).  exp2f adds a
// range fix-up (compare, two selects, ldexp) that only matters for results
// below 2^-126; here x = s - m <= 0 is a softmax exponent, and such a weight
// is below half an ulp of the running sum (>= 1) and of any output that the
// weight-1 key contributes to, so it changes no result.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// p -> (hi, lo) bf16 pairs packed two per word
__device__ __forceinline__ void split_bf16(float p0, float p1, uint32_t& hi, uint32_t& lo) {
  hi = pack_bf16x2(p0, p1);
  lo = pack_bf16x2(p0 - lo_bf16(hi), p1 - hi_bf16(hi));
}

// Keys past the end of a context sit in slots of the last page that no call
// has written (or that hold a closed sequence's values): their softmax weight
// is 0, but 0 times a NaN or Inf bit pattern there would still poison the
// output, so their V values are zeroed.  Decode: in the operand of the row's
// partly filled last page, which is taken outside the page ring so the ring
// holds no extra registers; a V^T operand word holds the bf16 values of two
// consecutive keys k, k + 1 of one dim (k in the low half), and
// keep_below(w, k, n) keeps those below n.  Prefill: in LDS, for the last
// page pair of a query block.
__device__ __forceinline__ uint32_t keep_below(uint32_t w, int k, int n) {
  return k + 1 < n ? w : (k < n ? (w & 0xffffu) : 0u);
}

// ===========================================================================
// Decode
// ===========================================================================

// One workgroup of kDecodeWaves waves per (row, kv head); wave w takes pages
// w, w + kDecodeWaves, ...  The wave's page ids are read once into one VGPR
// (lane j holds the id of the wave's j-th page, 64 pages per pass) so the page
// loop never waits on a memory lookup; PD pages of K/V are kept in flight in
// a register ring.  The waves' (max, sum, output) states are merged through
// LDS in wave order.  Probes over 25 and 200 rows of ~1300-token contexts
// (8 kv heads, scattered pages): 16 waves with two pages in flight (128
// VGPRs) took 26.9 us at 25 rows against 28.1 for 8 waves x 2 and 27.9 for
// 16 x 1; at 200 rows 16 x 1 (102 VGPRs) took 212 us against 218 for 8 x 2
// and 220 for 16 x 2 -- a deeper ring pays while the grid is too small to
// fill the CUs twice over, more resident waves pay once it is not.  Smaller
// splits than 128 pages only moved time into the combine kernel.
constexpr int kDecodeWaves = 16;
constexpr int kDecodeRing2MaxWaves = 512 * 16;  // waves of the grid up to which PD = 2

template <int HD, int G, int NW, int PD, int PS = kDecodePagesPerSplit>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(4))) void attn_decode_kernel(AttnArgs a) {
  constexpr int KQ = HD / 32;  // score MFMAs per page
  constexpr int NT = HD / 16;  // output tiles (pairs share one 16-byte V load)
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int wi = blockIdx.x / a.nkv, h = blockIdx.x % a.nkv;
  const int row = a.work[2 * wi], split = a.work[2 * wi + 1];
  const int ctx = a.row_ctx[row];
  const int qrow = a.row_qrow[row];
  const int p0 = split * PS;
  const int32_t* bt = a.bt + a.row_bt[row] + p0;
  const int n_pages = min(ceil_div(ctx, kPage) - p0, PS);  // pages of this split
  const float qscale = a.scale * kLog2e;

  // Q^T operand: column col = head h*G + col (zero beyond the group); MFMA i
  // takes dims 32i + 8grp .. +7, matching the K tile layout.
  uint4 qf[KQ];
#pragma unroll
  for (int i = 0; i < KQ; ++i) qf[i] = make_uint4(0, 0, 0, 0);
  if (col < G) {
    const uint16_t* qp = a.q + (static_cast<size_t>(qrow) * a.nq + h * G + col) * HD;
#pragma unroll
    for (int i = 0; i < KQ; ++i) qf[i] = *reinterpret_cast<const uint4*>(qp + 32 * i + 8 * grp);
  }

  f32x4 o[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = kNegBig, l = 0.f;

  uint4 kf[PD][KQ];
  uint4 vf[PD][NT / 2];
  const size_t koff = kv_offset(0, 0, a.nkv, h, 0, HD, 0), voff = kv_offset(0, 1, a.nkv, h, 0, HD, 0);
  const size_t pstride = static_cast<size_t>(2) * a.nkv * kPage * HD;
  auto load_page = [&](int sl, int page) {
    const uint16_t* kp = a.kv + static_cast<size_t>(page) * pstride + koff;
    const uint16_t* vp = a.kv + static_cast<size_t>(page) * pstride + voff;
#pragma unroll
    for (int i = 0; i < KQ; ++i) kf[sl][i] = *reinterpret_cast<const uint4*>(kp + 512 * i + 8 * lane);
#pragma unroll
    for (int c = 0; c < NT / 2; ++c) vf[sl][c] = *reinterpret_cast<const uint4*>(vp + 512 * c + 8 * lane);
  };

  // One page: scores, online softmax, P.V.  `last` marks the row's partly
  // filled last page: keys from ctx on get no weight and V = 0.
  auto page_step = [&](const uint4* kp, uint4* vp, int p, bool last) __attribute__((always_inline)) {
    f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < KQ; ++i) s = mfma_k32(kp[i], qf[i], s);
    float sv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) sv[r] = (!last || p * kPage + 4 * grp + r < ctx) ? s[r] * qscale : -INFINITY;
    float mp = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    mp = fmaxf(mp, __shfl_xor(mp, 16, kWave));
    mp = fmaxf(mp, __shfl_xor(mp, 32, kWave));
    const float mn = fmaxf(m, mp);
    const float corr = exp2f(m - mn);
    m = mn;
    float pv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) pv[r] = exp2_hw(sv[r] - mn);
    l = l * corr + ((pv[0] + pv[1]) + (pv[2] + pv[3]));
    uint2 hi, lo;
    split_bf16(pv[0], pv[1], hi.x, lo.x);
    split_bf16(pv[2], pv[3], hi.y, lo.y);
    if (last) {
      const int n = ctx - p * kPage, k0 = 4 * grp;
#pragma unroll
      for (int c = 0; c < NT / 2; ++c) {
        vp[c].x = keep_below(vp[c].x, k0, n);
        vp[c].y = keep_below(vp[c].y, k0 + 2, n);
        vp[c].z = keep_below(vp[c].z, k0, n);
        vp[c].w = keep_below(vp[c].w, k0 + 2, n);
      }
    }
#pragma unroll
    for (int c = 0; c < NT / 2; ++c) {
      const uint2 v0 = make_uint2(vp[c].x, vp[c].y), v1 = make_uint2(vp[c].z, vp[c].w);
      o[2 * c] *= corr;
      o[2 * c] = mfma_k16(v0, hi, o[2 * c]);
      o[2 * c] = mfma_k16(v0, lo, o[2 * c]);
      o[2 * c + 1] *= corr;
      o[2 * c + 1] = mfma_k16(v1, hi, o[2 * c + 1]);
      o[2 * c + 1] = mfma_k16(v1, lo, o[2 * c + 1]);
    }
  };

  // Full pages go through the register ring; a partly filled last page of the
  // row (in this split) is taken afterwards by the wave it falls to, so the
  // ring carries no masking.  Each wave's pages and their order are the same
  // either way.
  const bool part_last = (ctx % kPage) != 0 && p0 + n_pages == ceil_div(ctx, kPage);
  const int n_full = n_pages - (part_last ? 1 : 0);
  const int np = wave < n_full ? (n_full - wave + NW - 1) / NW : 0;
  for (int j0 = 0; j0 < np; j0 += 64) {
    const int nj = min(64, np - j0);
    // lane j: id of the wave's page j0 + j
    const int pid = lane < nj ? bt[wave + NW * (j0 + lane)] : 0;
#pragma unroll
    for (int sl = 0; sl < PD; ++sl) load_page(sl, __builtin_amdgcn_readlane(pid, min(sl, nj - 1)));
    for (int base = 0; base < nj; base += PD) {
#pragma unroll
      for (int sl = 0; sl < PD; ++sl) {
        const int it = base + sl;
        if (it < nj) page_step(kf[sl], vf[sl], p0 + wave + NW * (j0 + it), false);
        load_page(sl, __builtin_amdgcn_readlane(pid, min(it + PD, nj - 1)));
      }
    }
  }
  if (part_last && wave == n_full % NW) {
    load_page(0, bt[n_full]);
    page_step(kf[0], vf[0], p0 + n_full, true);
  }
  l += __shfl_xor(l, 16, kWave);
  l += __shfl_xor(l, 32, kWave);

  // merge the waves in order
  __shared__ float sm[NW][G], sl_[NW][G];
  __shared__ float so[NW][HD][G];
  if (col < G) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) so[wave][16 * t + 4 * grp + i][col] = o[t][i];
    if (grp == 0) {
      sm[wave][col] = m;
      sl_[wave][col] = l;
    }
  }
  __syncthreads();
  const bool whole = a.row_nsplit[row] == 1;
  for (int idx = threadIdx.x; idx < G * HD; idx += blockDim.x) {
    const int g = idx / HD, d = idx % HD;
    float M = sm[0][g];
#pragma unroll
    for (int w = 1; w < NW; ++w) M = fmaxf(M, sm[w][g]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float f = exp2f(sm[w][g] - M);
      L += sl_[w][g] * f;
      O += so[w][d][g] * f;
    }
    if (whole) {
      a.out[(static_cast<size_t>(qrow) * a.nq + h * G + g) * HD + d] = f32_to_bf16(O / L);
    } else {
      float* pp = a.part + ((static_cast<size_t>(wi) * a.nkv + h) * G + g) * (HD + 2);
      pp[d] = O;
      if (d == 0) {
        pp[HD] = M;
        pp[HD + 1] = L;
      }
    }
  }
}

// Merge the split states of each (row, query head) in split order.  One block
// of hd threads per (row, head); rows with a single split are already final.
__global__ __launch_bounds__(128) void attn_combine_kernel(AttnArgs a) {
  const int row = blockIdx.x / a.nq, j = blockIdx.x % a.nq;
  const int ns = a.row_nsplit[row];
  if (ns == 1) return;
  const int G = a.nq / a.nkv, hd = a.hd;
  const int h = j / G, g = j % G;
  const int w0 = a.row_work[row];
  const int d = threadIdx.x;
  auto state = [&](int s2) { return a.part + ((static_cast<size_t>(w0 + s2) * a.nkv + h) * G + g) * (hd + 2); };
  float M = kNegBig;
  for (int s2 = 0; s2 < ns; ++s2) M = fmaxf(M, state(s2)[hd]);
  float L = 0.f, O = 0.f;
  for (int s2 = 0; s2 < ns; ++s2) {
    const float* pp = state(s2);
    const float f = exp2f(pp[hd] - M);
    L += pp[hd + 1] * f;
    O += pp[d] * f;
  }
  a.out[(static_cast<size_t>(a.row_qrow[row]) * a.nq + j) * hd + d] = f32_to_bf16(O / L);
}

// Zero the V^T entries of keys n0 and beyond in the two V^T page tiles of a
// prefill stage (2 x 16 keys x HD bf16 in LDS), one 32-bit word (two keys of
// one dim) per step.  Out of line: inlined, its index arithmetic raised the
// register count of the whole kernel.
template <int HD>
__device__ __attribute__((noinline)) void zero_v_past(uint32_t* vt, int n0, int tid, int nthreads) {
  constexpr int kWordsPerPage = kPage * HD / 2;
  for (int w = tid; w < 2 * kWordsPerPage; w += nthreads) {
    const int pg = w / kWordsPerPage, in = w % kWordsPerPage;
    // word in of a tile: element pair 2*in, 2*in + 1 = keys 4g + 2j, +1 of dim e
    const int j = in & 1, g = (in >> 6) & 3;   // (((e/32)*4 + g)*16 + e%16)*8 + u*4 + (2j|2j+1)
    const int k = pg * kPage + 4 * g + 2 * j;
    uint32_t v = vt[w];
    if (k >= n0) v = 0u;
    else if (k + 1 >= n0) v &= 0xffffu;
    vt[w] = v;
  }
}

// ===========================================================================
// Prefill (flash attention over pages)
// ===========================================================================

// Query columns of one 16-wide MFMA tile: 16/G tokens x G heads.
// Waves x query tiles per wave (16 tiles = 256 query columns per block): at
// head dim 128, 16 waves (four per SIMD) of one tile each, since 8 waves of
// two tiles (208 VGPRs) left only two waves per SIMD to hide the latency of
// each tile's chain of score MFMAs, softmax and output MFMAs; at head dim 64
// a page tile is too small to split over 16 waves, so 8 waves of two tiles.
template <int HD>
struct PrefillShape {
  static constexpr int NW = HD >= 128 ? 16 : 8, NQ = 16 / NW;
};
constexpr int kPrefillTilesPerBlock = 16;
constexpr int kPrefillPageIds = 512;  // page ids staged in LDS (contexts up to 8192 keys)

template <int HD, int G, int NW, int NQ>
__global__ __launch_bounds__(NW * 64) void attn_prefill_kernel(PrefillAttnArgs a) {
  constexpr int KQ = HD / 32;
  constexpr int NT = HD / 16;
  constexpr int TPT = 16 / G;         // tokens per tile
  constexpr int TPW = NQ * TPT;       // tokens per wave
  constexpr int PCH = kPage * HD / 8;  // 16-byte chunks of one K (or V^T) page tile
  constexpr int WPT = NW / 4;         // waves bringing each of the 4 tiles of a stage
  constexpr int LPW = PCH / WPT / 64;  // direct loads per wave per stage
  constexpr int NS = 4;               // stages of the LDS ring
  static_assert(NW % 4 == 0 && PCH % (WPT * 64) == 0, "the waves share each tile evenly");
  // stage = one page pair: [K page 0, K page 1, V^T page 0, V^T page 1]
  __shared__ uint4 ring[NS][4][PCH];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15, grp = lane >> 4;
  const int bi = blockIdx.x / a.nkv, h = blockIdx.x % a.nkv;
  const int item = a.blocks[3 * bi], row0 = a.blocks[3 * bi + 1], nrows = a.blocks[3 * bi + 2];
  const int32_t* bt = a.bt + a.item_bt[item];
  const int last_pos = a.pos[row0 + nrows - 1];
  const int first_pos = a.pos[row0];
  const int n_pages = last_pos / kPage + 1;
  const int n_pairs = (n_pages + 1) / 2;
  const float qscale = a.scale * kLog2e;

  // this lane's query column in each tile
  int qpos[NQ], qrow[NQ];
  bool qok[NQ];
  uint4 qf[NQ][KQ];
#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    const int tok = wave * TPW + n * TPT + col / G;
    qok[n] = tok < nrows;
    qrow[n] = row0 + (qok[n] ? tok : 0);
    qpos[n] = qok[n] ? a.pos[qrow[n]] : -1;
    const uint16_t* qp = a.q + (static_cast<size_t>(qrow[n]) * a.nq + h * G + col % G) * HD + 8 * grp;
#pragma unroll
    for (int i = 0; i < KQ; ++i)
      qf[n][i] = qok[n] ? *reinterpret_cast<const uint4*>(qp + 32 * i) : make_uint4(0, 0, 0, 0);
  }

  f32x4 o[NQ][NT];
  float m[NQ], l[NQ];
#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    m[n] = kNegBig;
    l[n] = 0.f;
#pragma unroll
    for (int t = 0; t < NT; ++t) o[n][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // Waves WPT*t .. WPT*t + WPT-1 bring the parts of tile t of every stage:
  // the K (t < 2) or V^T (t >= 2) tile of page 2*pair + (t & 1).  The absent
  // second page of an odd count is stood in for by the last page: finite
  // values, all of its keys masked.
  const int tile = wave / WPT, piece = wave % WPT;
  const size_t part = kv_offset(0, tile >> 1, a.nkv, h, 0, HD, 0) + piece * (PCH / WPT) * 8;
  const size_t pstride = static_cast<size_t>(2) * a.nkv * kPage * HD;
  // The block's page ids go to LDS once, so that a stage's load issue waits
  // on an LDS read rather than on a block-table load from memory (pages past
  // the table's capacity are still read from the block table).
  __shared__ int32_t page_ids[kPrefillPageIds];
  for (int i = tid; i < min(n_pages, kPrefillPageIds); i += NW * 64) page_ids[i] = bt[i];
  __syncthreads();
  auto issue = [&](int pair) __attribute__((always_inline)) {
    const int pi = min(2 * pair + (tile & 1), n_pages - 1);
    const int id = pi < kPrefillPageIds ? page_ids[pi] : bt[pi];
    const uint16_t* src = a.kv + static_cast<size_t>(id) * pstride + part + 8 * lane;
    const uint32_t dst = lds_address(&ring[pair % NS][tile][piece * (PCH / WPT)]);
#pragma unroll
    for (int c = 0; c < LPW; ++c) lds_load16(src + 512 * c, dst + 1024 * c);
  };

  issue(0);
  if (n_pairs > 1) issue(1);
  if (n_pairs > 2) issue(2);
  for (int pair = 0; pair < n_pairs; ++pair) {
    // this pair's tiles have landed once at most the later pairs' loads are
    // outstanding; then every wave's part is in LDS after the barrier, and the
    // stage read in the previous iteration is free for pair + 3
    const int later = min(n_pairs - 1 - pair, 2);
    if (later == 2) wait_vmcnt<2 * LPW>();
    else if (later == 1) wait_vmcnt<LPW>();
    else wait_vmcnt<0>();
    lds_barrier();
    if (pair + 3 < n_pairs) issue(pair + 3);
    const uint4(*st)[PCH] = ring[pair % NS];
    // Keys past the block's last position (never written, or the stand-in
    // page of an odd count) get V = 0 in the stage before any wave reads it:
    // only the last pair can hold them, so only it pays the extra barrier.
    if (const int n0 = last_pos + 1 - 2 * pair * kPage; n0 < 2 * kPage) {
      zero_v_past<HD>(reinterpret_cast<uint32_t*>(&ring[pair % NS][2][0]), n0, tid, NW * 64);
      __syncthreads();
    }

    // K operand of both pages (A of S^T): key row col, dims 32i + 8grp .. +7;
    // V^T operand over the pair: dims of tile t, keys 4grp .. 4grp+3 of each
    // page (held for all query tiles when the wave has several, else read
    // from LDS as each output tile needs it)
    uint4 kf[2][KQ];
#pragma unroll
    for (int pg = 0; pg < 2; ++pg)
#pragma unroll
      for (int i = 0; i < KQ; ++i) kf[pg][i] = st[pg][64 * i + lane];
    auto vt_operand = [&](int t) __attribute__((always_inline)) {
      const int vo = 128 * (t >> 1) + 2 * lane + (t & 1);  // in 8-byte units
      const uint2 va = reinterpret_cast<const uint2*>(st[2])[vo];
      const uint2 vb = reinterpret_cast<const uint2*>(st[3])[vo];
      return make_uint4(va.x, va.y, vb.x, vb.y);
    };
    uint4 vf[NQ > 1 ? NT : 1];
    if constexpr (NQ > 1) {
#pragma unroll
      for (int t = 0; t < NT; ++t) vf[t] = vt_operand(t);
    }

    // keys of this pair visible to every query of the block: no mask needed
    const bool all_visible = (2 * pair + 2) * kPage - 1 <= first_pos;
#pragma unroll
    for (int n = 0; n < NQ; ++n) {
      float sv[2][4];  // raw scores q.k
#pragma unroll
      for (int pg = 0; pg < 2; ++pg) {
        f32x4 sc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < KQ; ++i) sc = mfma_k32(kf[pg][i], qf[n][i], sc);
#pragma unroll
        for (int r = 0; r < 4; ++r) sv[pg][r] = sc[r];
      }
      if (!all_visible) {
#pragma unroll
        for (int pg = 0; pg < 2; ++pg)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if ((2 * pair + pg) * kPage + 4 * grp + r > qpos[n]) sv[pg][r] = -INFINITY;
      }
      // The reference max m only moves when some column's max exceeds it by
      // more than 8 (a factor 2^8): o and l carry the same scale, so their
      // quotient is unchanged, and p = 2^(s - m) stays below 2^8.  Whether any
      // score does is read off the exponents s*scale - m themselves, so the
      // column maxima (a cross-lane reduction) are formed only when m moves.
      float e[2][4];
      bool grow = false;
#pragma unroll
      for (int pg = 0; pg < 2; ++pg)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          e[pg][r] = fmaf(sv[pg][r], qscale, -m[n]);
          grow |= e[pg][r] > 8.f;
        }
      if (__any(grow)) {
        float mp = fmaxf(fmaxf(fmaxf(sv[0][0], sv[0][1]), fmaxf(sv[0][2], sv[0][3])),
                         fmaxf(fmaxf(sv[1][0], sv[1][1]), fmaxf(sv[1][2], sv[1][3])));
        mp = max_xor32(max_xor16(mp)) * qscale;  // in log2 units
        const float mn = fmaxf(m[n], mp);
        const float corr = exp2f(m[n] - mn);
        m[n] = mn;
        l[n] *= corr;
#pragma unroll
        for (int t = 0; t < NT; ++t) o[n][t] *= corr;
#pragma unroll
        for (int pg = 0; pg < 2; ++pg)
#pragma unroll
          for (int r = 0; r < 4; ++r) e[pg][r] = fmaf(sv[pg][r], qscale, -m[n]);
      }
      float pv[2][4];
      float ps = 0.f;
#pragma unroll
      for (int pg = 0; pg < 2; ++pg)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          pv[pg][r] = exp2_hw(e[pg][r]);
          ps += pv[pg][r];
        }
      l[n] += ps;
      // P^T operand over the page pair: k-slot 8grp+j is key 4grp+j of page
      // j/4, the order of the V^T operand
      uint4 hi, lo;
      split_bf16(pv[0][0], pv[0][1], hi.x, lo.x);
      split_bf16(pv[0][2], pv[0][3], hi.y, lo.y);
      split_bf16(pv[1][0], pv[1][1], hi.z, lo.z);
      split_bf16(pv[1][2], pv[1][3], hi.w, lo.w);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const uint4 v = NQ > 1 ? vf[NQ > 1 ? t : 0] : vt_operand(t);
        o[n][t] = mfma_k32(v, hi, o[n][t]);
        o[n][t] = mfma_k32(v, lo, o[n][t]);
      }
    }
  }

#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    const float L = sum_xor32(sum_xor16(l[n]));
    if (!qok[n]) continue;
    const float inv = 1.0f / L;
    uint16_t* op = a.out + (static_cast<size_t>(qrow[n]) * a.nq + h * G + col % G) * HD;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      uint2 w;
      w.x = pack_bf16x2(o[n][t][0] * inv, o[n][t][1] * inv);
      w.y = pack_bf16x2(o[n][t][2] * inv, o[n][t][3] * inv);
      *reinterpret_cast<uint2*>(op + 16 * t + 4 * grp) = w;
    }
  }
}

// ===========================================================================

template <int HD, int G, int NW>
static hipError_t launch_decode_g(bool ring2, dim3 grid, dim3 block, const AttnArgs& a, hipStream_t s) {
  if (ring2)
    launch_kernel((attn_decode_kernel<HD, G, NW, 2>), grid, block, 0, s, a);
  else
    launch_kernel((attn_decode_kernel<HD, G, NW, 1>), grid, block, 0, s, a);
  return hipGetLastError();
}

template <int HD>
static hipError_t launch_decode_hd(const AttnArgs& a, hipStream_t s) {
  constexpr int NW = kDecodeWaves;
  const dim3 grid(a.n_work * a.nkv), block(NW * 64);
  const bool ring2 = static_cast<int64_t>(a.n_work) * a.nkv * NW <= kDecodeRing2MaxWaves;
  switch (a.nq / a.nkv) {
    case 1: return launch_decode_g<HD, 1, NW>(ring2, grid, block, a, s);
    case 2: return launch_decode_g<HD, 2, NW>(ring2, grid, block, a, s);
    case 4: return launch_decode_g<HD, 4, NW>(ring2, grid, block, a, s);
    case 8: return launch_decode_g<HD, 8, NW>(ring2, grid, block, a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attn_combine(const AttnArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  launch_kernel(attn_combine_kernel, dim3(a.rows * a.nq), dim3(a.hd), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_attn_decode(const AttnArgs& a, hipStream_t s) {
  if (a.n_work <= 0) return hipSuccess;
  if (a.hd == 128) return launch_decode_hd<128>(a, s);
  if (a.hd == 64) return launch_decode_hd<64>(a, s);
  return hipErrorInvalidValue;
}

template <int HD>
static hipError_t launch_prefill_hd(const PrefillAttnArgs& a, hipStream_t s) {
  const dim3 grid(a.n_blocks * a.nkv), block(PrefillShape<HD>::NW * 64);
  switch (a.nq / a.nkv) {
    case 1: launch_kernel((attn_prefill_kernel<HD, 1, PrefillShape<HD>::NW, PrefillShape<HD>::NQ>), grid, block, 0, s, a); break;
    case 2: launch_kernel((attn_prefill_kernel<HD, 2, PrefillShape<HD>::NW, PrefillShape<HD>::NQ>), grid, block, 0, s, a); break;
    case 4: launch_kernel((attn_prefill_kernel<HD, 4, PrefillShape<HD>::NW, PrefillShape<HD>::NQ>), grid, block, 0, s, a); break;
    case 8: launch_kernel((attn_prefill_kernel<HD, 8, PrefillShape<HD>::NW, PrefillShape<HD>::NQ>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attn_prefill(const PrefillAttnArgs& a, hipStream_t s) {
  if (a.n_blocks <= 0) return hipSuccess;
  if (a.hd == 128) return launch_prefill_hd<128>(a, s);
  if (a.hd == 64) return launch_prefill_hd<64>(a, s);
  return hipErrorInvalidValue;
}

int prefill_tokens_per_block(int group) { return kPrefillTilesPerBlock * 16 / group; }

}  // namespace metro
