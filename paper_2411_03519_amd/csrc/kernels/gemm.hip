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
// Any fixed permutation of the reduction index is allowed as long as A and B
// use the same one; the skinny kernel uses this to let each lane read 64
// contiguous bytes of a W row per 128-wide k block.
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
// Skinny GEMM (M <= 16*MT, decode batches).  Weight streaming is the cost, so
// one workgroup of 8 waves owns 16*NT rows of W and the whole K: wave w takes
// the 128-wide k blocks w, w+8, ... (so the 8 waves read adjacent 256-byte
// runs of each row), partial tiles are summed through LDS in a fixed order.
// Lane (r = l%16, g = l/16) reads W[n0 + r][kb*128 + 32g .. +31] and the same
// 32 k of its activation row; MFMA i of the block consumes elements 8i .. 8i+7.
// ---------------------------------------------------------------------------
template <int MT, int NT, int EPI>
__global__ __launch_bounds__(512) void gemm_skinny_kernel(const uint16_t* __restrict__ X, int ldx,
                                                          const uint16_t* __restrict__ W, int Kp, int M,
                                                          float* __restrict__ outf, uint16_t* __restrict__ outb,
                                                          int ldo) {
  constexpr int NW = 8;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * 16 * NT;

  f32x4 acc[NT][MT];
#pragma unroll
  for (int a = 0; a < NT; ++a)
#pragma unroll
    for (int b = 0; b < MT; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const uint16_t* wrow[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) wrow[nt] = W + static_cast<size_t>(n0 + nt * 16 + r) * Kp + g * 32;
  const uint16_t* xrow[MT];
  bool xok[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * 16 + r;
    xok[mt] = m < M;
    xrow[mt] = X + static_cast<size_t>(xok[mt] ? m : 0) * ldx + g * 32;
  }

  const int nkb = Kp / 128;
  for (int kb = wave; kb < nkb; kb += NW) {
    const int k = kb * 128;
    uint4 wv[NT][4], xv[MT][4];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) wv[nt][i] = *reinterpret_cast<const uint4*>(wrow[nt] + k + 8 * i);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        xv[mt][i] = xok[mt] ? *reinterpret_cast<const uint4*>(xrow[mt] + k + 8 * i) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[nt][mt] = mfma16(wv[nt][i], xv[mt][i], acc[nt][mt]);
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
    // NT == 2: tile 0 holds gate features, tile 1 up features of block n0/32
    for (int mt = wave; mt < MT; mt += NW) {
      f32x4 gs = red[0][mt][lane], us = red[0][MT + mt][lane];
#pragma unroll
      for (int w = 1; w < NW; ++w) {
        gs += red[w][mt][lane];
        us += red[w][MT + mt][lane];
      }
      const int m = mt * 16 + m_lane;
      if (m < M) store_swiglu(gs, us, m, (n0 / 32) * 16 + n_lane, outb, ldo);
    }
  } else {
    for (int t = wave; t < NT * MT; t += NW) {
      f32x4 s = red[0][t][lane];
#pragma unroll
      for (int w = 1; w < NW; ++w) s += red[w][t][lane];
      const int nt = t / MT, mt = t % MT;
      const int m = mt * 16 + m_lane;
      if (m < M) store_tile<EPI>(s, m, n0 + nt * 16 + n_lane, outf, ldo);
    }
  }
}

// ---------------------------------------------------------------------------
// Tiled GEMM (M > 64: prefill chunks, large decode batches).  Block tile
// 128 (m) x 128 (n) x 64 (k), 4 waves in 2x2, each wave 64x64 = 4x4 MFMA
// tiles.  Tiles are staged through LDS (double buffered, rows padded by 16 B);
// the next k tile is fetched into registers while the current one is used.
// ---------------------------------------------------------------------------
constexpr int TBM = 128, TBN = 128, TBK = 64, TPAD = 8;

template <int EPI>
__global__ __launch_bounds__(256) void gemm_tiled_kernel(const uint16_t* __restrict__ X, int ldx,
                                                         const uint16_t* __restrict__ W, int Kp, int M, int N,
                                                         float* __restrict__ outf, uint16_t* __restrict__ outb,
                                                         int ldo) {
  __shared__ uint16_t xs[2][TBM][TBK + TPAD];
  __shared__ uint16_t ws[2][TBN][TBK + TPAD];
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int r = lane & 15, g = lane >> 4;
  const int wm = wave >> 1, wn = wave & 1;  // wave's 64x64 quadrant
  const int m0 = blockIdx.y * TBM, n0 = blockIdx.x * TBN;

  // global -> register staging: 1024 16-byte chunks per operand tile, 4 per thread
  const int lrow = tid >> 3, lcol = (tid & 7) * 8;
  uint4 xr[4], wr[4];
  auto fetch = [&](int k) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + lrow + 32 * i;
      xr[i] = m < M ? *reinterpret_cast<const uint4*>(X + static_cast<size_t>(m) * ldx + k + lcol)
                    : make_uint4(0, 0, 0, 0);
      const int n = n0 + lrow + 32 * i;
      wr[i] = n < N ? *reinterpret_cast<const uint4*>(W + static_cast<size_t>(n) * Kp + k + lcol)
                    : make_uint4(0, 0, 0, 0);
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<uint4*>(&xs[buf][lrow + 32 * i][lcol]) = xr[i];
      *reinterpret_cast<uint4*>(&ws[buf][lrow + 32 * i][lcol]) = wr[i];
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = Kp / TBK;
  fetch(0);
  stash(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) fetch((kt + 1) * TBK);
#pragma unroll
    for (int kc = 0; kc < TBK / 32; ++kc) {
      uint4 af[4], bf[4];
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
        af[nt] = *reinterpret_cast<const uint4*>(&ws[buf][wn * 64 + nt * 16 + r][kc * 32 + g * 8]);
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
        bf[mt] = *reinterpret_cast<const uint4*>(&xs[buf][wm * 64 + mt * 16 + r][kc * 32 + g * 8]);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) acc[nt][mt] = mfma16(af[nt], bf[mt], acc[nt][mt]);
    }
    if (kt + 1 < nk) stash(buf ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
    const int m = m0 + wm * 64 + mt * 16 + r;
    if (m >= M) continue;
    if (EPI == kEpiSwiGLU) {
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const int nb = n0 + wn * 64 + p * 32;  // 32-row (gate, up) block
        if (nb < N) store_swiglu(acc[2 * p][mt], acc[2 * p + 1][mt], m, (nb / 32) * 16 + 4 * g, outb, ldo);
      }
    } else {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int n = n0 + wn * 64 + nt * 16;
        if (n < N) store_tile<EPI>(acc[nt][mt], m, n + 4 * g, outf, ldo);
      }
    }
  }
}

// ---------------------------------------------------------------------------

template <int EPI>
static hipError_t launch_epi(const uint16_t* X, int ldx, const uint16_t* W, int Kp, int M, int N, float* outf,
                             uint16_t* outb, int ldo, hipStream_t s) {
  if (M <= 64) {
    // SwiGLU needs a (gate, up) pair per workgroup
    constexpr int NT = 2;
    const dim3 grid(N / (16 * NT));
    if (M <= 16)
      hipLaunchKernelGGL((gemm_skinny_kernel<1, NT, EPI>), grid, dim3(512), 0, s, X, ldx, W, Kp, M, outf, outb, ldo);
    else if (M <= 32)
      hipLaunchKernelGGL((gemm_skinny_kernel<2, NT, EPI>), grid, dim3(512), 0, s, X, ldx, W, Kp, M, outf, outb, ldo);
    else
      hipLaunchKernelGGL((gemm_skinny_kernel<4, NT, EPI>), grid, dim3(512), 0, s, X, ldx, W, Kp, M, outf, outb, ldo);
  } else {
    const dim3 grid((N + TBN - 1) / TBN, (M + TBM - 1) / TBM);
    hipLaunchKernelGGL((gemm_tiled_kernel<EPI>), grid, dim3(256), 0, s, X, ldx, W, Kp, M, N, outf, outb, ldo);
  }
  return hipGetLastError();
}

hipError_t launch_gemm(const uint16_t* X, int ldx, const uint16_t* W, int Kp, int M, int N, int epilogue,
                       float* out_f32, uint16_t* out_bf16, int ldo, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  switch (epilogue) {
    case kEpiStoreF32:
      return launch_epi<kEpiStoreF32>(X, ldx, W, Kp, M, N, out_f32, out_bf16, ldo, s);
    case kEpiAddF32:
      return launch_epi<kEpiAddF32>(X, ldx, W, Kp, M, N, out_f32, out_bf16, ldo, s);
    case kEpiSwiGLU:
      return launch_epi<kEpiSwiGLU>(X, ldx, W, Kp, M, N, out_f32, out_bf16, ldo, s);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace metro
