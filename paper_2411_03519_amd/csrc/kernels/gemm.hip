// bf16 MFMA GEMMs of the Llama projections on gfx950 (v_mfma_f32_16x16x32_bf16,
// fp32 accumulation):  Y[M, N] = X[M, K] . W[N, K]^T  + fused epilogue.
//
// Operand convention.  The MFMA computes D = A . B with A 16x32 (rows = output
// features n, i.e. W rows) and B 32x16 (columns = activation rows m).  Lane l
// supplies A[l%16][8(l/16) .. 8(l/16)+7] and B[8(l/16) .. +7][l%16] and
// receives D[4(l/16) + i][l%16], i = 0..3: four consecutive output features of
// one activation row, so every epilogue store is a contiguous 16-byte (fp32)
// or 8-byte (bf16) vector.
//
// W is stored in exactly that A-operand order (packed_offset in common.h): a
// 16 x 32 tile of W is 1 KiB, lane l's 16 bytes at offset 16l, so a wave
// loading an A operand from HBM issues one contiguous 1 KiB read.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace metro {

__device__ __forceinline__ f32x4 mfma16(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

__device__ __forceinline__ float silu_f32(float z) { return z / (1.0f + expf(-z)); }

// Epilogue for one 16x16 accumulator tile: lane holds features n .. n+3 of row m.
template <int EPI>
__device__ __forceinline__ void store_tile(f32x4 v, int m, int n, float* __restrict__ outf, int ldo) {
  float4* p = reinterpret_cast<float4*>(outf + static_cast<size_t>(m) * ldo + n);
  if (EPI == kEpiStoreF32) {
    *p = make_float4(v[0], v[1], v[2], v[3]);
  } else {
    float4 o = *p;
    o.x += v[0];
    o.y += v[1];
    o.z += v[2];
    o.w += v[3];
    *p = o;
  }
}

// gate/up tiles of the same 16 features -> bf16(silu(gate) * up)
__device__ __forceinline__ void store_swiglu(f32x4 gt, f32x4 up, int m, int j, uint16_t* __restrict__ outb,
                                             int ldo) {
  uint2 o;
  o.x = pack_bf16x2(silu_f32(gt[0]) * up[0], silu_f32(gt[1]) * up[1]);
  o.y = pack_bf16x2(silu_f32(gt[2]) * up[2], silu_f32(gt[3]) * up[3]);
  *reinterpret_cast<uint2*>(outb + static_cast<size_t>(m) * ldo + j) = o;
}

// ---------------------------------------------------------------------------
// Skinny GEMM (M <= 16*MT, decode batches).  Streaming W from HBM is the cost,
// and every W row tile needs the activation rows of its k range, so each wave
// owns NT row tiles (16*NT rows of W) to keep those activation reads well
// below the W bytes.  A workgroup of NW waves owns the 16*NT rows and a k
// slice (grid.y = KS slices); wave w takes the 128-wide k blocks w, w+NW, ...
// of the slice.  A block is 4 packed 16 x 32 tiles per row tile, i.e. 4 KiB
// contiguous in W, read as four 1 KiB wave loads.
// Partial tiles of the 8 waves are summed through LDS in wave order; with
// KS > 1 the slice sums go to part[slice][m][n] and the consumer kernel adds
// the slices (in slice order) where it reads the result.
// ---------------------------------------------------------------------------
// q / k / v of one row for dims d0 .. d0+3 (a) and d0+half .. (b) of a head
// whose features start at column f0 of the QKV product
__device__ __forceinline__ void store_rope_kv(f32x4 a, f32x4 b, int m, int head, int d0, const RopeKV& rk) {
  const int hd = rk.hd, half = hd / 2;
  const int sl = rk.slot[m], page = sl / kPage, off = sl % kPage;
  if (head < rk.nq + rk.nkv) {
    const float2* c = rk.rope + static_cast<size_t>(rk.pos[m]) * half + d0;
    f32x4 ra, rb;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float2 cs = c[i];
      ra[i] = a[i] * cs.x - b[i] * cs.y;
      rb[i] = a[i] * cs.y + b[i] * cs.x;
    }
    if (head < rk.nq) {
      uint16_t* dst = rk.q + (static_cast<size_t>(m) * rk.nq + head) * hd;
      *reinterpret_cast<uint2*>(dst + d0) = make_uint2(pack_bf16x2(ra[0], ra[1]), pack_bf16x2(ra[2], ra[3]));
      *reinterpret_cast<uint2*>(dst + d0 + half) = make_uint2(pack_bf16x2(rb[0], rb[1]), pack_bf16x2(rb[2], rb[3]));
    } else {
      // dims d0 .. d0+3 (d0 % 4 == 0) are 4 consecutive elements of the K
      // tile: one 8-byte store each for the two halves
      uint16_t* kt = rk.kv + kv_offset(page, 0, rk.nkv, head - rk.nq, 0, hd, 0);
      *reinterpret_cast<uint2*>(kt + k_tile_offset(off, d0)) =
          make_uint2(pack_bf16x2(ra[0], ra[1]), pack_bf16x2(ra[2], ra[3]));
      *reinterpret_cast<uint2*>(kt + k_tile_offset(off, d0 + half)) =
          make_uint2(pack_bf16x2(rb[0], rb[1]), pack_bf16x2(rb[2], rb[3]));
    }
  } else {
    uint16_t* vt = rk.kv + kv_offset(page, 1, rk.nkv, head - rk.nq - rk.nkv, 0, hd, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      vt[vt_tile_offset(d0 + i, off)] = f32_to_bf16(a[i]);
      vt[vt_tile_offset(d0 + i + half, off)] = f32_to_bf16(b[i]);
    }
  }
}

template <int MT, int NT, int EPI, int PF, int NW>
__global__ __launch_bounds__(NW * 64) void gemm_skinny_kernel(const uint16_t* __restrict__ X, int ldx,
                                                              const uint16_t* __restrict__ W, int Kp, int M, int N,
                                                              float* __restrict__ outf, uint16_t* __restrict__ outb,
                                                              int ldo, float* __restrict__ part, RopeKV rk) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * 16 * NT;
  const int KS = gridDim.y, slice = blockIdx.y;
  const int kslice = Kp / KS, k0 = slice * kslice;

  f32x4 acc[NT][MT];
#pragma unroll
  for (int a = 0; a < NT; ++a)
#pragma unroll
    for (int b = 0; b < MT; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  // packed tile (n0/16 + nt, k0/32) of W, this lane's chunk
  const uint16_t* wrow[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
    wrow[nt] = W + (static_cast<size_t>(n0 / 16 + nt) * (Kp / 32) + k0 / 32) * 512 + lane * 8;
  const uint16_t* xrow[MT];
  bool xok[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * 16 + r;
    xok[mt] = m < M;
    xrow[mt] = X + static_cast<size_t>(xok[mt] ? m : 0) * ldx + k0 + 8 * g;
  }

  // the wave's k blocks are wave, wave + NW, ...; PF of them are in flight in a
  // register ring whose slots are refilled right after use (clamped, so every
  // load is unconditional and each block waits only for its own loads)
  const int nkb = kslice / 128;
  const int nb = wave < nkb ? (nkb - wave + NW - 1) / NW : 0;
  if (nb > 0) {
    uint4 wv[PF][NT][4], xv[PF][MT][4];
    auto load = [&](int sl, int j) {
      const int k = (wave + NW * j) * 128;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) wv[sl][nt][i] = *reinterpret_cast<const uint4*>(wrow[nt] + (k / 32 + i) * 512);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          xv[sl][mt][i] = xok[mt] ? *reinterpret_cast<const uint4*>(xrow[mt] + k + 32 * i) : make_uint4(0, 0, 0, 0);
    };
#pragma unroll
    for (int sl = 0; sl < PF; ++sl) load(sl, min(sl, nb - 1));
    for (int base = 0; base < nb; base += PF) {
#pragma unroll
      for (int sl = 0; sl < PF; ++sl) {
        const int it = base + sl;
        if (it < nb) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
              for (int mt = 0; mt < MT; ++mt) acc[nt][mt] = mfma16(wv[sl][nt][i], xv[sl][mt][i], acc[nt][mt]);
        }
        if (PF > 1) load(sl, min(it + PF, nb - 1));
        else if (it + 1 < nb) load(sl, it + 1);
      }
    }
  }

  __shared__ f32x4 red[NW][NT * MT][kWave];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) red[wave][nt * MT + mt][lane] = acc[nt][mt];
  __syncthreads();

  const int m_lane = r;  // activation row within a 16-row tile
  const int n_lane = 4 * g;
  if (EPI == kEpiSwiGLU) {
    // Tile nt holds the gate (rows 0..7) and up (rows 8..15) projections of
    // features 8 (n0/16 + nt) .. +7: lane l < 32 has gate rows 4(l/16) .. +3
    // and lane l + 32 the matching up rows, which a 32-lane swap brings together.
    for (int t = wave; t < NT * MT; t += NW) {
      f32x4 sum = red[0][t][lane];
#pragma unroll
      for (int w = 1; w < NW; ++w) sum += red[w][t][lane];
      f32x4 gt, up;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const auto pr = __builtin_amdgcn_permlane32_swap(__float_as_uint(sum[i]), __float_as_uint(sum[i]), false, false);
        gt[i] = __uint_as_float(pr[0]);  // from lane l % 32
        up[i] = __uint_as_float(pr[1]);  // from lane l % 32 + 32
      }
      const int nt = t / MT, mt = t % MT;
      const int m = mt * 16 + m_lane;
      if (lane < 32 && m < M) store_swiglu(gt, up, m, 8 * (n0 / 16 + nt) + n_lane, outb, ldo);
    }
  } else if (EPI == kEpiRopeKV) {
    // Tile nt holds dims 8j .. 8j+7 (rows 0..7) and the matching dims of the
    // head's second half (rows 8..15) of one head, j = its 16-row tile within
    // the head: as for SwiGLU, a 32-lane swap brings each pair together.
    for (int t = wave; t < NT * MT; t += NW) {
      f32x4 sum = red[0][t][lane];
#pragma unroll
      for (int w = 1; w < NW; ++w) sum += red[w][t][lane];
      f32x4 a, b;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const auto pr = __builtin_amdgcn_permlane32_swap(__float_as_uint(sum[i]), __float_as_uint(sum[i]), false, false);
        a[i] = __uint_as_float(pr[0]);  // dim d (lane l % 32)
        b[i] = __uint_as_float(pr[1]);  // dim d + hd/2 (lane l % 32 + 32)
      }
      const int nt = t / MT, mt = t % MT;
      const int m = mt * 16 + m_lane;
      const int f0 = n0 + nt * 16;
      if (lane < 32 && m < M) store_rope_kv(a, b, m, f0 / rk.hd, 8 * ((f0 % rk.hd) / 16) + n_lane, rk);
    }
  } else {
    for (int t = wave; t < NT * MT; t += NW) {
      f32x4 sum = red[0][t][lane];
#pragma unroll
      for (int w = 1; w < NW; ++w) sum += red[w][t][lane];
      const int nt = t / MT, mt = t % MT;
      const int m = mt * 16 + m_lane;
      if (m >= M) continue;
      if (KS > 1)
        store_tile<kEpiStoreF32>(sum, m, n0 + nt * 16 + n_lane, part + static_cast<size_t>(slice) * M * N, N);
      else
        store_tile<EPI>(sum, m, n0 + nt * 16 + n_lane, outf, ldo);
    }
  }
}

// out[m, n] (=|+=) sum over slices of part[s][m][n], in slice order
template <int EPI>
__global__ __launch_bounds__(256) void reduce_parts_kernel(const float* __restrict__ part, int KS, int M, int N,
                                                           float* __restrict__ out, int ldo) {
  const int64_t n4 = static_cast<int64_t>(M) * N / 4;
  for (int64_t e = blockIdx.x * 256ll + threadIdx.x; e < n4; e += static_cast<int64_t>(gridDim.x) * 256) {
    const int m = static_cast<int>((4 * e) / N), n = static_cast<int>((4 * e) % N);
    float4 s = reinterpret_cast<const float4*>(part)[e];
    for (int k = 1; k < KS; ++k) {
      const float4 v = reinterpret_cast<const float4*>(part + static_cast<size_t>(k) * M * N)[e];
      s.x += v.x;
      s.y += v.y;
      s.z += v.z;
      s.w += v.w;
    }
    float4* o = reinterpret_cast<float4*>(out + static_cast<size_t>(m) * ldo + n);
    if (EPI == kEpiAddF32) {
      const float4 x = *o;
      s.x += x.x;
      s.y += x.y;
      s.z += x.z;
      s.w += x.w;
    }
    *o = s;
  }
}

// ---------------------------------------------------------------------------
// Tiled GEMM (prefill chunks, large decode batches), bound by the matrix
// cores.  Block tile 256 (n, rows of W) x 256 (m, activation rows); 8 waves in
// 4 x 2 (two per SIMD), each 64 x 128 = 2 x 4 tiles of
// v_mfma_f32_32x32x16_bf16 (A = W rows, B = activation rows).  Lane l
// supplies A[l%32][8(l/32) .. +7] and B[8(l/32) .. +7][l%32] and receives D
// rows 8q + 4(l/32) + i (q = 0..3, i = 0..3) of column l%32: four consecutive
// output features of one activation row per q.
//
// Operands reach LDS by direct loads (global_load_lds_dwordx4: each lane's 16
// bytes land at LDS base + 16 * lane), through a ring of NS stages (Big: 5 of
// 32-wide k); the loads of the later stages are in flight while one is
// consumed, with no staging registers.  In LDS the weights keep their packed 16 x 32 tiles in
// lane order, so every MFMA operand read by 16 lanes is 256 contiguous bytes,
// free of bank conflicts.  Activations in 32-wide k stages are gathered into
// the same form (64 contiguous bytes of each of 16 rows per wave load); in
// 64-wide k stages one wave load takes 8 whole rows of the stage (8 x 128
// bytes, whole cache lines) into a 1 KiB block whose 16-byte chunks are
// XOR-swizzled by row (act_chunk_slot), which keeps the operand reads free of
// bank conflicts: 8 consecutive rows of one k chunk fall in 8 distinct
// 16-byte slots of a 128-byte bank period (8B gate/up at M=128: 71.7 -> 66.3
// us against half-line loads; agent trace 12.3-12.5k -> 12.8k tokens/s).
// The stage consumed in step kt is refilled (with stage kt + NS - 1) in step
// kt + 1, after the barrier that every wave passes only once done reading it.
// ---------------------------------------------------------------------------
// Tile shapes: WN x WM waves, each TN x TM tiles of 32 x 32, NS stages of
// KT 32-wide k tiles in the LDS ring.  Big: 256 x 256 blocks for long prefill
// chunks.  Mid: 128 x 128 blocks for batches of 65 to a few hundred rows: 8
// waves of 64 x 32 (two per SIMD) and a ring of 4 stages of 64-wide k (128
// KiB).  At these sizes the k loop itself was the cost: with every global
// load skipped the former Mid tile (4 waves of 64 x 64, 5 stages of 32-wide
// k) still took 28 of its 62 us for the 8B gate/up at M=128, and the loads
// added to that rather than hiding under it (ring depths 5, 8 and 9 all gave
// the same time); stages twice as wide halve the barriers per unit of work
// and the second wave per SIMD covers one wave's waits.  In the model: agent
// trace 12.16k -> 12.56k tokens/s, fixed batch of 100 +5%, 70B at B=128
// 2.55k -> 2.62k.
// KT: 32-wide k tiles per stage (1, or 2 for 64-wide stages: half the
// barriers per unit of work).
template <int WN_, int WM_, int TN_, int TM_, int NS_, int KT_ = 1>
struct TileShape {
  static constexpr int WN = WN_, WM = WM_, TN = TN_, TM = TM_, NS = NS_, KT = KT_;
  static constexpr int WAVES = WN * WM, NTH = WAVES * 64;
  static constexpr int BN = WN * TN * 32, BM = WM * TM * 32;  // block tile
  static constexpr int WT = BN / 16, XT = BM / 16;            // 16 x 32 tiles per k tile
  static constexpr int LPW = KT * (WT + XT) / WAVES;          // direct loads per wave per stage
  static_assert((KT * (WT + XT)) % WAVES == 0, "the waves share the tiles of a stage evenly");
  static_assert(NS >= 3, "the pipeline keeps a stage in use, one landed and loads in flight");
  static_assert(KT == 1 || KT == 2 || KT == 4, "stages of 32, 64 or 128 k");
};
using BigTile = TileShape<4, 2, 2, 4, 5>;
using MidTile = TileShape<2, 4, 2, 1, 4, 2>;
// Wide: 256 rows of W x 128 activation rows, 8 waves of 64 x 64, 5 stages
// (120 KiB), for wide products at up to 256 rows when 128 x 128 tiles would be
// too many for one round: against 256 x 256 tiles it does no matrix work on
// absent rows at M <= 128 (70B gate/up at M=128 in a probe: 202 against 267
// us; the LM head at M=80: 225 against 268) and gives twice the workgroups at
// M = 129..256 (8B gate/up at M=192: 78 against 91 us).
using WideTile = TileShape<4, 2, 2, 2, 5>;

__device__ __forceinline__ f32x16 mfma32(uint4 a, uint4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// Slot of 16-byte chunk c of tile row `row` within that row's 128 bytes of a
// swizzled activation block (64-wide k stages); the map is its own inverse,
// so it also gives the chunk held in slot c.  The 8 rows of a block put one
// chunk into 8 distinct slots of a 128-byte bank period, and rows of the next
// block into the other half of a 256-byte one.
__device__ __forceinline__ int act_chunk_slot(int c, int row) { return c ^ (row & 7) ^ ((row >> 3) & 1); }

// wait until at most PER * min(later, MAXC) direct loads of this wave are outstanding
template <int PER, int MAXC>
__device__ __forceinline__ void wait_later_stages(int later) {
  if constexpr (MAXC > 0) {
    if (later >= MAXC) {
      wait_vmcnt<PER * MAXC>();
      return;
    }
    wait_later_stages<PER, MAXC - 1>(later);
  } else {
    wait_vmcnt<0>();
  }
}

// Grouped tile order: tiles in launch order sweep groups of kGroupM m-tiles,
// m fastest within a group, so the ~256 blocks in flight cover a compact
// patch of tiles and share their W and X tiles through the caches.
template <class S>
__host__ __device__ __forceinline__ void tile_origin(int t, int M, int N, int& m0, int& n0) {
  constexpr int kGroupM = 16;
  const int mt = (M + S::BM - 1) / S::BM, nt = (N + S::BN - 1) / S::BN;
  const int group = t / (kGroupM * nt);
  const int first_m = group * kGroupM;
  const int gm = min(mt - first_m, kGroupM);
  const int in = t % (kGroupM * nt);
  n0 = (in / gm) * S::BN;
  m0 = (first_m + in % gm) * S::BM;
}

// Workgroups are handed to the 8 XCDs in turn (workgroup b to XCD b % 8), and
// each XCD has its own L2.  Work item of workgroup b (of `total`) such that
// every XCD gets a contiguous run of the work list: in tile_origin order the
// row tiles that read the same W columns are neighbours, so they run on one
// XCD and share its L2 instead of each fetching W through the fabric.  In the
// model (agent trace, 8B) this gained 2.5%; for prefill-sized 256 x 256 grids
// it cost 1% and is not applied there.
__device__ __forceinline__ int xcd_contiguous(int b, int total) {
  constexpr int kXcds = 8;
  const int q = total / kXcds, r = total % kXcds, x = b % kXcds, s = b / kXcds;
  return x * q + min(x, r) + s;
}

// Work of one workgroup.  Without a tail split the grid's tiles x k slices
// (slice-major list, tiles in tile_origin order) are spread over the XCDs by
// xcd_contiguous (256 x 256 tiles: only up to kSplitMaxRows rows; above, the
// list in grid order).  With one (tail_split = S > 1), workgroups x <
// tail_first take tile x over all of K, and the last tiles, which would leave
// most CUs idle in the final round, are cut into S k slices each: workgroup
// tail_first + u takes slice u % S of tile tail_first + u / S and stores its
// fp32 sums to part[u][BM][BN] for gemm_tail_fixup_kernel.
template <class S, int EPI>
__global__ __launch_bounds__(S::NTH) void gemm_tiled_kernel(const uint16_t* __restrict__ X, int ldx,
                                                            const uint16_t* __restrict__ W, int Kp, int M, int N,
                                                            float* __restrict__ outf, uint16_t* __restrict__ outb,
                                                            int ldo, float* __restrict__ part, int tail_first,
                                                            int tail_split, RopeKV rk) {
  constexpr int WM = S::WM, TN = S::TN, TM = S::TM, NS = S::NS, LPW = S::LPW, KT = S::KT;
  __shared__ uint4 wring[NS][KT * S::WT * 64];  // per stage and k tile: WT tiles of 16 x 32 (1 KiB each)
  __shared__ uint4 xring[NS][KT * S::XT * 64];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave / WM, wm = wave % WM;  // the wave's (TN*32) x (TM*32) tile
  const int lr = lane & 31, lh = lane >> 5;

  // tile and k range (each slice a multiple of 128)
  int tile = blockIdx.x, KS = gridDim.y, slice = blockIdx.y, unit = -1;
  if (tail_split > 1 && tile >= tail_first) {
    unit = tile - tail_first;
    tile = tail_first + unit / tail_split;
    KS = tail_split;
    slice = unit % tail_split;
  } else if (tail_split == 1 && (S::BM * S::BN < 256 * 256 || M <= kSplitMaxRows)) {
    const int i = xcd_contiguous(blockIdx.y * gridDim.x + blockIdx.x, gridDim.x * gridDim.y);
    slice = i / gridDim.x;
    tile = i % gridDim.x;
  }
  const int kspan = Kp / KS, k0 = slice * kspan;
  const int nk = kspan / (32 * KT);
  int m0, n0;
  tile_origin<S>(tile, M, N, m0, n0);

  // Wave w loads tiles w*LPW .. w*LPW + LPW - 1 of the list [W tiles, X
  // tiles] of every stage.  Rows past N or M re-read the last valid row:
  // finite values whose products only reach outputs that are not stored.
  const uint16_t* src[LPW];
  uint32_t dst[LPW];
  int src_step[LPW];       // elements per 32-wide k tile
  uint32_t dst_step[LPW];  // bytes per stage of the operand's ring
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int t = wave * LPW + j;  // [k tile 0: W tiles .. k tile KT-1: W tiles][the same for X]
    if (t < KT * S::WT) {
      const int kk = t / S::WT, wt = t % S::WT;
      const int rt = min(n0 / 16 + wt, N / 16 - 1);
      src[j] = W + (static_cast<size_t>(rt) * (Kp / 32) + k0 / 32 + kk) * 512 + lane * 8;
      dst[j] = lds_address(&wring[0][0]) + t * 1024;
      src_step[j] = 512 * KT;
      dst_step[j] = KT * S::WT * 1024;
    } else {
      const int u = t - KT * S::WT, kk = u / S::XT, tx = u % S::XT;
      if constexpr (KT == 2) {
        // block u: rows 8u .. 8u+7 of the tile, all 64 k of the stage; lane l
        // fills slot l % 8 of row 8u + l / 8
        const int row = min(m0 + 8 * u + (lane >> 3), M - 1);
        src[j] = X + static_cast<size_t>(row) * ldx + k0 + 8 * act_chunk_slot(lane & 7, 8 * u + (lane >> 3));
        (void)kk;
        (void)tx;
      } else {
        const int row = min(m0 + 16 * tx + (lane & 15), M - 1);
        src[j] = X + static_cast<size_t>(row) * ldx + k0 + 32 * kk + 8 * (lane >> 4);
      }
      dst[j] = lds_address(&xring[0][0]) + u * 1024;
      src_step[j] = 32 * KT;
      dst_step[j] = KT * S::XT * 1024;
    }
  }
  auto issue = [&](int kt) __attribute__((always_inline)) {
    const uint32_t stage = kt % NS;
#pragma unroll
    for (int j = 0; j < LPW; ++j) lds_load16(src[j] + kt * src_step[j], dst[j] + stage * dst_step[j]);
  };

  f32x16 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // operand fragments of the 16-wide k half ks (0 .. 2 KT - 1) of stage kt
  auto read_frags = [&](int kt, int ks, uint4 (&af)[TN], uint4 (&bf)[TM]) __attribute__((always_inline)) {
    const uint4* ws = wring[kt % NS] + (ks >> 1) * S::WT * 64;
    const int q = 16 * (2 * (ks & 1) + lh);  // chunk of the lane's 8 k values within a tile
#pragma unroll
    for (int i = 0; i < TN; ++i) {
      const int row = wn * TN * 32 + i * 32 + lr;
      af[i] = ws[(row >> 4) * 64 + (row & 15) + q];
    }
    if constexpr (KT == 2) {
      const uint4* xs = xring[kt % NS];
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int row = wm * TM * 32 + j * 32 + lr;
        bf[j] = xs[(row >> 3) * 64 + (row & 7) * 8 + act_chunk_slot(2 * ks + lh, row)];
      }
    } else {
      const uint4* xs = xring[kt % NS] + (ks >> 1) * S::XT * 64;
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int row = wm * TM * 32 + j * 32 + lr;
        bf[j] = xs[(row >> 4) * 64 + (row & 15) + q];
      }
    }
  };
  auto mfmas = [&](const uint4 (&af)[TN], const uint4 (&bf)[TM]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j) acc[i][j] = mfma32(af[i], bf[j], acc[i][j]);
  };
  auto mfmas_row = [&](int i, const uint4 (&af)[TN], const uint4 (&bf)[TM]) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = mfma32(af[i], bf[j], acc[i][j]);
  };

  // Software pipeline across the barrier: the fragments of the first k half
  // of step kt + 1 are read while the second half of step kt multiplies, so
  // no wave waits on LDS after a barrier.  The barrier of step kt sits
  // between its two halves: past it, every wave's loads of stage kt + 1 have
  // landed and every wave has consumed stage kt - 1, whose slot then takes
  // stage kt + NS - 1.
#pragma unroll
  for (int p = 0; p < NS - 1; ++p)
    if (p < nk) issue(p);
  wait_later_stages<LPW, NS - 2>(nk - 1);
  lds_barrier();
  uint4 a0[TN], b0[TM], a1[TN], b1[TM];
  read_frags(0, 0, a0, b0);
  // halves 0 .. 2 KT - 2 of stage kt, each multiplied while the next is read;
  // the last one is left in a1, b1
  auto inner_halves = [&](int kt) __attribute__((always_inline)) {
#pragma unroll
    for (int h = 0; h + 1 < 2 * KT; h += 2) {
      read_frags(kt, h + 1, a1, b1);
      mfmas(a0, b0);
      if (h + 2 < 2 * KT) {
        read_frags(kt, h + 2, a0, b0);
        mfmas(a1, b1);
      }
    }
  };
  // (the last step is peeled: a loop exit between the halves would merge
  // control flow there and make the compiler's LDS waits cover the reads
  // issued for the next step)
  for (int kt = 0; kt + 1 < nk; ++kt) {
    inner_halves(kt);
    // stage kt + 1 has landed once only the loads of stages kt + 2 .. are
    // outstanding
    wait_later_stages<LPW, NS - 3>(nk - 2 - kt);
    __builtin_amdgcn_sched_barrier(0);
    lds_barrier();
    __builtin_amdgcn_sched_barrier(0);
    // the first row of MFMAs goes ahead of the load issue, so the matrix pipe
    // is fed while the wave computes addresses
    mfmas_row(0, a1, b1);
    __builtin_amdgcn_sched_barrier(0);
    if (kt + NS - 1 < nk) issue(kt + NS - 1);
    read_frags(kt + 1, 0, a0, b0);
#pragma unroll
    for (int i = 1; i < TN; ++i) mfmas_row(i, a1, b1);
  }
  inner_halves(nk - 1);
  mfmas(a1, b1);

  // Fully unrolled (acc must stay in registers).  Slice sums are stored raw:
  // to part[slice][m][n] with KS > 1, to part[unit][m - m0][n - n0] for a
  // tail unit.  The residual add first loads all 4 * TN float4 of one 32-row
  // group of activation rows, then adds and stores them (one round trip per
  // group rather than per value); the scheduling barrier keeps the compiler
  // from hoisting every group's loads at once.
  if constexpr (EPI == kEpiRopeKV) {
    // (launched without k slices) each 16-row block of a 32-row tile holds 8
    // dims of a head's first half, then the matching 8 of its second half in
    // the rotate-half interleave: the lane's rows 8q + 4(l/32) + i of q = 0, 2
    // pair with those of q = 1, 3 in the same lane
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      const int m = m0 + wm * TM * 32 + j * 32 + lr;
      if (m >= M) continue;
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int nb = n0 + wn * TN * 32 + i * 32;
        if (nb >= N) continue;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int r0 = nb + 16 * u;  // first W row of the 16-row block
          const f32x4 a{acc[i][j][8 * u], acc[i][j][8 * u + 1], acc[i][j][8 * u + 2], acc[i][j][8 * u + 3]};
          const f32x4 b{acc[i][j][8 * u + 4], acc[i][j][8 * u + 5], acc[i][j][8 * u + 6], acc[i][j][8 * u + 7]};
          store_rope_kv(a, b, m, r0 / rk.hd, 8 * ((r0 % rk.hd) / 16) + 4 * lh, rk);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    return;
  }
  const bool raw = KS > 1;
  float* const pout = unit >= 0 ? part + static_cast<size_t>(unit) * S::BM * S::BN
                      : raw     ? part + static_cast<size_t>(slice) * M * N
                                : outf;
  const int pld = unit >= 0 ? S::BN : raw ? N : ldo;
  const int om = unit >= 0 ? m0 : 0, on = unit >= 0 ? n0 : 0;  // origin of pout
  if (EPI == kEpiAddF32 && !raw) {
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      const int m = m0 + wm * TM * 32 + j * 32 + lr;
      if (m >= M) continue;
      float4 r[TN][4];
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int nb = min(n0 + wn * TN * 32 + i * 32, N - 32);  // in bounds; stored only if < N
#pragma unroll
        for (int q = 0; q < 4; ++q)
          r[i][q] = *reinterpret_cast<const float4*>(outf + static_cast<size_t>(m) * ldo + nb + 8 * q + 4 * lh);
      }
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int nb = n0 + wn * TN * 32 + i * 32;
        if (nb >= N) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float4 v = r[i][q];
          v.x += acc[i][j][4 * q];
          v.y += acc[i][j][4 * q + 1];
          v.z += acc[i][j][4 * q + 2];
          v.w += acc[i][j][4 * q + 3];
          *reinterpret_cast<float4*>(outf + static_cast<size_t>(m) * ldo + nb + 8 * q + 4 * lh) = v;
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int m = m0 + wm * TM * 32 + j * 32 + lr;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < TN; ++i) {
      const int nb = n0 + wn * TN * 32 + i * 32;  // 32-row tile of W
      if (nb >= N) continue;
      if (EPI == kEpiSwiGLU && !raw) {
        // the tile is two 16-row blocks of 8 gate rows then the 8 matching up
        // rows: the lane's rows 8q + 4(l/32) + i of q = 0, 2 (gate) pair with
        // those of q = 1, 3 (up) in the same lane
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const f32x4 gt{acc[i][j][8 * q], acc[i][j][8 * q + 1], acc[i][j][8 * q + 2], acc[i][j][8 * q + 3]};
          const f32x4 up{acc[i][j][8 * q + 4], acc[i][j][8 * q + 5], acc[i][j][8 * q + 6], acc[i][j][8 * q + 7]};
          store_swiglu(gt, up, m, 8 * (nb / 16 + q) + 4 * lh, outb, ldo);
          __builtin_amdgcn_sched_barrier(0);
        }
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x4 v{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
          if (raw)
            store_tile<kEpiStoreF32>(v, m - om, nb + 8 * q + 4 * lh - on, pout, pld);
          else
            store_tile<EPI>(v, m, nb + 8 * q + 4 * lh, pout, pld);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  }
}

// Tail tiles of a product split by gemm_tiled_kernel: out (=|+=) the sum of
// each tile's `split` slice sums, added in slice order.  Workgroup (t, y)
// covers rows 4y .. 4y+3 of tail tile t, a thread 4 consecutive columns.
template <class S, int EPI>
__global__ __launch_bounds__(256) void gemm_tail_fixup_kernel(const float* __restrict__ part, int tail_first,
                                                              int split, int M, int N, float* __restrict__ out,
                                                              int ldo) {
  constexpr int kCols = S::BN / 4;  // threads per tile row
  static_assert(256 % kCols == 0 && S::BM % (256 / kCols) == 0, "rows of a tile split evenly");
  const int i = blockIdx.y * (256 / kCols) + threadIdx.x / kCols;
  const int j = 4 * (threadIdx.x % kCols);
  int m0, n0;
  tile_origin<S>(tail_first + blockIdx.x, M, N, m0, n0);
  const int m = m0 + i, n = n0 + j;
  if (m >= M || n >= N) return;
  const float* p = part + static_cast<size_t>(blockIdx.x) * split * S::BM * S::BN + i * S::BN + j;
  float4 a = *reinterpret_cast<const float4*>(p);
  for (int sl = 1; sl < split; ++sl) {
    const float4 v = *reinterpret_cast<const float4*>(p + static_cast<size_t>(sl) * S::BM * S::BN);
    a.x += v.x;
    a.y += v.y;
    a.z += v.z;
    a.w += v.w;
  }
  store_tile<EPI>(f32x4{a.x, a.y, a.z, a.w}, m, n, out, ldo);
}

// The same for the gate/up product: a tile's BN rows of W are BN/16 blocks of
// 8 gate rows then the 8 matching up rows; output column j of the tile (of
// BN/2) takes gate row 16(j/8) + j%8 and up row 16(j/8) + 8 + j%8, summed over
// the slices in slice order, then out_bf16[m][n0/2 + j] = bf16(silu(gate) *
// up).  Workgroup (t, y) covers rows 8y .. 8y+7 of tail tile t, a thread 4
// consecutive output columns.
template <class S>
__global__ __launch_bounds__(256) void gemm_tail_fixup_swiglu_kernel(const float* __restrict__ part, int tail_first,
                                                                     int split, int M, int N,
                                                                     uint16_t* __restrict__ out, int ldo) {
  constexpr int kCols = S::BN / 8;  // threads per tile row (4 of the BN/2 output columns each)
  static_assert(256 % kCols == 0 && S::BM % (256 / kCols) == 0, "rows of a tile split evenly");
  const int i = blockIdx.y * (256 / kCols) + threadIdx.x / kCols;
  const int j = 4 * (threadIdx.x % kCols);
  const int wg = 16 * (j / 8) + j % 8;  // gate row of output column j within the tile
  int m0, n0;
  tile_origin<S>(tail_first + blockIdx.x, M, N, m0, n0);
  const int m = m0 + i;
  if (m >= M || n0 + wg >= N) return;
  const float* p = part + static_cast<size_t>(blockIdx.x) * split * S::BM * S::BN + i * S::BN + wg;
  float4 g = *reinterpret_cast<const float4*>(p);
  float4 u = *reinterpret_cast<const float4*>(p + 8);
  for (int sl = 1; sl < split; ++sl) {
    const float* q = p + static_cast<size_t>(sl) * S::BM * S::BN;
    const float4 gv = *reinterpret_cast<const float4*>(q);
    const float4 uv = *reinterpret_cast<const float4*>(q + 8);
    g.x += gv.x;
    g.y += gv.y;
    g.z += gv.z;
    g.w += gv.w;
    u.x += uv.x;
    u.y += uv.y;
    u.z += uv.z;
    u.w += uv.w;
  }
  store_swiglu(f32x4{g.x, g.y, g.z, g.w}, f32x4{u.x, u.y, u.z, u.w}, m, n0 / 2 + j, out, ldo);
}

// ---------------------------------------------------------------------------

constexpr int kSkinnyPF = 1;                // k blocks in flight per wave
constexpr int kSkinnyWaves = 8;             // waves per workgroup (k split inside it)

// Row tiles per wave of the decode kernel: 4 (64 rows) amortises the
// activation reads best, but for short, narrow products (QKV-sized) 2 tiles
// and twice the workgroups finish sooner (11.0 vs 12.9 us at N=6144, K=4096),
// and the gate/up product, which cannot split K, takes 7 where that makes the
// workgroups a multiple of the 256 CUs (448 -> 256 at the 8B shape: 46.3 ->
// 42.5 us).
static int skinny_tiles(int N, int Kp, int epilogue) {
  if (epilogue == kEpiSwiGLU && (N / 16) % (7 * 256) == 0) return 7;
  if (N % 64) return 2;
  return N <= 8192 && Kp <= 4096 ? 2 : 4;
}

// Decode kernel: workgroups split K while fewer than `target` cover the
// product; slices stay multiples of 128, and the slice sums (ks * M * N fp32,
// written and read again) stay within a quarter of the weight bytes (N * Kp
// bf16), i.e. 8 * ks * M <= Kp.
static int gemm_k_splits(int blocks, int target, int M, int Kp) {
  int ks = 1;
  while (blocks * ks < target && ks < 8 && (Kp / (2 * ks)) % 128 == 0 && 8 * (2 * ks) * M <= Kp) ks *= 2;
  return ks;
}

// Tiled kernels: the most k slices (a power of two up to 8, slices multiples
// of 128) whose workgroups still fit one round of the CUs, with slice sums up
// to half the weight bytes (4 * ks * M <= Kp).  At M = 80..256 the narrow
// 8B/70B products ran fastest with one round of workgroups (8B O at M=200: 4
// slices, 256 workgroups, 26 us; 2 slices 30 us; 8B down at M=200: 4 slices
// 50 us, 8 slices over 512 workgroups 57 us); in the model this took the
// agent trace from 11.7k to 12.2k tokens/s and the 70B step (B=128) from
// 2.47k to 2.57k against the former rule (fewer than 512 workgroups for
// 128 x 128 tiles, slice sums within a quarter of the weights).
static int tiled_k_splits(int tiles, int cus, int M, int Kp) {
  int ks = 1;
  while (ks < 8 && tiles * (2 * ks) <= cus && (Kp / (2 * ks)) % 128 == 0 && 4 * (2 * ks) * M <= Kp) ks *= 2;
  return ks;
}

// Compute units of the current device (256 on MI355X), cached per device.
static int device_cus() {
  static int cache[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

// Kernel choice, from probes over M = 80 .. 12800 at the Llama-3-8B and 70B
// shapes: the decode kernel up to 64 rows; then 128 x 128 tiles (more blocks)
// for narrow products, and for wide ones up to 192 rows while their tiles
// number at most the CUs (in the 70B model at M=128 gate/up took 242 us as 448
// such tiles against 203 us as 224 of 256 x 256, although cache-cold probes
// had ranked them the other way); else 256 x 128 tiles for wide products up to
// 128 rows, or up to 256 while they number at most the CUs, and for narrow
// products of up to 128 rows that 128 x 128 tiles leave mostly idle; 256 x 256
// tiles for the rest and for long prefill chunks.
GemmPlan plan_gemm(int M, int N, int Kp, int epilogue, int64_t part_cap) {
  GemmPlan p{GemmKind::kBig, 4, 1, 1, 0};
  const bool can_split = part_cap > 0;
  const bool split = can_split && epilogue != kEpiSwiGLU && M <= kSplitMaxRows;
  if (M <= 64) {
    p.kind = GemmKind::kSkinny;
    p.nt = skinny_tiles(N, Kp, epilogue);
    if (split) p.ks = gemm_k_splits(N / (16 * p.nt), p.nt == 2 ? 512 : 256, M, Kp);
    while (p.ks > 1 && static_cast<int64_t>(p.ks) * M * N > part_cap) p.ks /= 2;
    return p;
  }
  auto tiles_of = [&](int bn, int bm) { return ((N + bn - 1) / bn) * ((M + bm - 1) / bm); };
  const int mid_tiles = tiles_of(MidTile::BN, MidTile::BM), wide_tiles = tiles_of(WideTile::BN, WideTile::BM);
  const int cus = device_cus();
  if (N >= 16384) {  // wide products: gate/up and the LM head
    if (M <= 192 && mid_tiles <= cus)
      p.kind = GemmKind::kMid;
    else if (M <= WideTile::BM || (M <= 2 * WideTile::BM && wide_tiles <= cus))
      p.kind = GemmKind::kWide;
    else
      p.kind = GemmKind::kBig;
  } else {
    p.kind = M <= kMidMaxRows ? GemmKind::kMid : GemmKind::kBig;
  }
  const int kind_tiles = p.kind == GemmKind::kMid    ? mid_tiles
                         : p.kind == GemmKind::kWide ? wide_tiles
                                                     : tiles_of(BigTile::BN, BigTile::BM);
  if (split) p.ks = tiled_k_splits(kind_tiles, cus, M, Kp);
  // Narrow products of up to 128 rows whose 128 x 128 tiles fill under three
  // quarters of the CUs even with k slices take 256 x 128 tiles when those
  // reach at least as many workgroups (70B QKV at M=128: 40 tiles x 4 slices,
  // 55 us, against 80 x 2 of 128 x 128, 63 us, in a probe; larger batches
  // were not measured with this rule and keep 128 x 128 tiles).
  if (split && p.kind == GemmKind::kMid && M <= WideTile::BM && 4 * mid_tiles * p.ks < 3 * cus) {
    const int wks = tiled_k_splits(wide_tiles, cus, M, Kp);
    if (wide_tiles * wks >= mid_tiles * p.ks) {
      p.kind = GemmKind::kWide;
      p.ks = wks;
    }
  }
  const int bn = p.kind == GemmKind::kMid ? MidTile::BN : p.kind == GemmKind::kWide ? WideTile::BN : BigTile::BN;
  const int bm = p.kind == GemmKind::kMid ? MidTile::BM : p.kind == GemmKind::kWide ? WideTile::BM : BigTile::BM;
  const int tiles = tiles_of(bn, bm);
  while (p.ks > 1 && static_cast<int64_t>(p.ks) * M * N > part_cap) p.ks /= 2;  // slice sums fit the workspace
  // Last round of 256-row tiles (one workgroup per CU): with r tiles left for
  // C CUs, cut each into S k slices (S a power of two, r * S <= C, slices
  // multiples of 128), so that round takes 1/S of a tile's time; the fixup
  // kernel adds the slices.
  if (p.kind != GemmKind::kMid && p.ks == 1 && can_split) {
    const int r = tiles % cus;
    int sp = 1;
    while (r > 0 && sp < 8 && r * (2 * sp) <= cus && (Kp / (2 * sp)) % 128 == 0) sp *= 2;
    if (sp > 1 && static_cast<int64_t>(r) * sp * bm * bn <= part_cap) {
      p.tail_split = sp;
      p.tail_first = tiles - r;
    }
  }
  return p;
}


template <int MT, int NT, int EPI>
static void launch_skinny(const uint16_t* X, int ldx, const uint16_t* W, int Kp, int M, int N, float* outf,
                          uint16_t* outb, int ldo, float* part, int ks, hipStream_t s) {
  // 7 row tiles: 4 waves, so that the cross-wave reduction buffer fits in LDS
  constexpr int NW = NT == 7 ? 4 : kSkinnyWaves;
  launch_kernel((gemm_skinny_kernel<MT, NT, EPI, kSkinnyPF, NW>), dim3(N / (16 * NT), ks), dim3(NW * 64), 0, s, X,
                ldx, W, Kp, M, N, outf, outb, ldo, part, RopeKV{});
}

template <int NT, int EPI>
static void launch_skinny_m(const uint16_t* X, int ldx, const uint16_t* W, int Kp, int M, int N, float* outf,
                            uint16_t* outb, int ldo, float* part, int ks, hipStream_t s) {
  if (M <= 16)
    launch_skinny<1, NT, EPI>(X, ldx, W, Kp, M, N, outf, outb, ldo, part, ks, s);
  else if (M <= 32)
    launch_skinny<2, NT, EPI>(X, ldx, W, Kp, M, N, outf, outb, ldo, part, ks, s);
  else
    launch_skinny<4, NT, EPI>(X, ldx, W, Kp, M, N, outf, outb, ldo, part, ks, s);
}

template <class S, int EPI>
static void launch_tiled(const uint16_t* X, int ldx, const uint16_t* W, int Kp, int M, int N, float* outf,
                         uint16_t* outb, int ldo, float* part, int ks, hipStream_t s, int tail_split = 1,
                         int tail_first = 0) {
  const int tiles = ((N + S::BN - 1) / S::BN) * ((M + S::BM - 1) / S::BM);
  const int blocks = tail_split > 1 ? tail_first + (tiles - tail_first) * tail_split : tiles;
  launch_kernel((gemm_tiled_kernel<S, EPI>), dim3(blocks, ks), dim3(S::NTH), 0, s, X, ldx, W, Kp, M, N, outf, outb,
                ldo, part, tail_first, tail_split, RopeKV{});
  if (tail_split > 1) {
    if constexpr (EPI == kEpiSwiGLU)
      launch_kernel((gemm_tail_fixup_swiglu_kernel<S>), dim3(tiles - tail_first, S::BM / (2048 / S::BN)),
                    dim3(256), 0, s, part, tail_first, tail_split, M, N, outb, ldo);
    else
      launch_kernel((gemm_tail_fixup_kernel<S, EPI>), dim3(tiles - tail_first, S::BM / (1024 / S::BN)), dim3(256),
                    0, s, part, tail_first, tail_split, M, N, outf, ldo);
  }
}

template <int EPI>
static hipError_t launch_epi(const GemmPlan& p, const uint16_t* X, int ldx, const uint16_t* W, int Kp, int M, int N,
                             float* outf, uint16_t* outb, int ldo, float* part, hipStream_t s) {
  switch (p.kind) {
    case GemmKind::kSkinny:
      if (p.nt == 7)
        launch_skinny_m<7, EPI>(X, ldx, W, Kp, M, N, outf, outb, ldo, part, p.ks, s);
      else if (p.nt == 4)
        launch_skinny_m<4, EPI>(X, ldx, W, Kp, M, N, outf, outb, ldo, part, p.ks, s);
      else
        launch_skinny_m<2, EPI>(X, ldx, W, Kp, M, N, outf, outb, ldo, part, p.ks, s);
      break;
    case GemmKind::kMid:
      launch_tiled<MidTile, EPI>(X, ldx, W, Kp, M, N, outf, outb, ldo, part, p.ks, s);
      break;
    case GemmKind::kWide:
      launch_tiled<WideTile, EPI>(X, ldx, W, Kp, M, N, outf, outb, ldo, part, p.ks, s, p.tail_split, p.tail_first);
      break;
    case GemmKind::kBig:
      launch_tiled<BigTile, EPI>(X, ldx, W, Kp, M, N, outf, outb, ldo, part, p.ks, s, p.tail_split, p.tail_first);
      break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(const uint16_t* X, int ldx, const uint16_t* W, int Kp, int M, int N, int epilogue,
                       float* out_f32, uint16_t* out_bf16, int ldo, float* part, int64_t part_cap, int* n_parts,
                       hipStream_t s) {
  *n_parts = 0;
  if (M <= 0) return hipSuccess;
  const GemmPlan p = plan_gemm(M, N, Kp, epilogue, part != nullptr ? part_cap : 0);
  if (p.ks > 1) *n_parts = p.ks;
  switch (epilogue) {
    case kEpiStoreF32:
      return launch_epi<kEpiStoreF32>(p, X, ldx, W, Kp, M, N, out_f32, out_bf16, ldo, part, s);
    case kEpiAddF32:
      return launch_epi<kEpiAddF32>(p, X, ldx, W, Kp, M, N, out_f32, out_bf16, ldo, part, s);
    case kEpiSwiGLU:
      return launch_epi<kEpiSwiGLU>(p, X, ldx, W, Kp, M, N, out_f32, out_bf16, ldo, part, s);
    default:
      return hipErrorInvalidValue;
  }
}

// 2 row tiles per wave, 4 waves, K whole: 14.4 us at M=25, N=6144, K=4096
// (with 4 k slices the product alone takes 13.1 us, but the slice sums then
// cost a RoPE kernel of 5.2 us)
bool gemm_rope_kv_fused(int M, int N, int Kp) {
  return M <= kRopeKVMaxRows || plan_gemm(M, N, Kp, kEpiStoreF32, 0).kind == GemmKind::kBig;
}

hipError_t launch_gemm_rope_kv(const uint16_t* X, int ldx, const uint16_t* W, int Kp, int M, int N, const RopeKV& rk,
                               hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (!gemm_rope_kv_fused(M, N, Kp) || N != (rk.nq + 2 * rk.nkv) * rk.hd || rk.hd % 32 || N % 32)
    return hipErrorInvalidValue;
  if (M > kRopeKVMaxRows) {  // 256 x 256 tiles over all of K (no workspace: no split of the last round)
    const int tiles = ((N + BigTile::BN - 1) / BigTile::BN) * ((M + BigTile::BM - 1) / BigTile::BM);
    launch_kernel((gemm_tiled_kernel<BigTile, kEpiRopeKV>), dim3(tiles, 1), dim3(BigTile::NTH), 0, s, X, ldx, W, Kp,
                  M, N, nullptr, nullptr, 0, nullptr, 0, 1, rk);
    return hipGetLastError();
  }
  constexpr int NT = 2, NW = 4;
  auto go = [&](auto mt) {
    constexpr int MT = decltype(mt)::value;
    launch_kernel((gemm_skinny_kernel<MT, NT, kEpiRopeKV, kSkinnyPF, NW>), dim3(N / (16 * NT), 1), dim3(NW * 64), 0,
                  s, X, ldx, W, Kp, M, N, nullptr, nullptr, 0, nullptr, rk);
  };
  if (M <= 16)
    go(std::integral_constant<int, 1>{});
  else if (M <= 32)
    go(std::integral_constant<int, 2>{});
  else
    go(std::integral_constant<int, 4>{});
  return hipGetLastError();
}

hipError_t launch_reduce_parts(const float* part, int KS, int M, int N, int epilogue, float* out, int ldo,
                               hipStream_t s) {
  const int64_t n4 = static_cast<int64_t>(M) * N / 4;
  const int grid = static_cast<int>(std::min<int64_t>((n4 + 255) / 256, 4096));
  if (epilogue == kEpiAddF32)
    launch_kernel((reduce_parts_kernel<kEpiAddF32>), dim3(grid), dim3(256), 0, s, part, KS, M, N, out, ldo);
  else
    launch_kernel((reduce_parts_kernel<kEpiStoreF32>), dim3(grid), dim3(256), 0, s, part, KS, M, N, out, ldo);
  return hipGetLastError();
}

}  // namespace metro
