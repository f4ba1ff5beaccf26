// Paged grouped-query attention on gfx950 (decode rows, and prefill rows in
// this first version): one work item = (row, split of the row's pages) for one
// kv head, computing the G query heads that share that kv head, so each K/V
// page is read once per group.
//
// Layout.  A page holds 16 positions; per layer and kv head its K tile and V
// tile are each a contiguous [16][hd] bf16 block.  Lane (tg, dg) of a wave
// owns dims 8dg .. 8dg+7 of token rows tg, tg+TPL, ...: one 16-byte load per
// row, and each load instruction of the wave covers TPL whole rows (1 KiB,
// fully coalesced).
//
// Softmax is the online (streaming) form in fp32 with scores pre-multiplied
// by log2(e) so exp2 can be used; the four waves of a workgroup take pages
// round-robin and are merged through LDS; rows whose context spans several
// splits leave (max, sum, unnormalised output) partials for the combine
// kernel.  The number of splits depends on the context length only.
#include "common.h"
#include "kernels.h"

namespace metro {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegBig = -1.0e30f;

template <int HD, int G>
__global__ __launch_bounds__(256) void attn_paged_kernel(AttnArgs a) {
  constexpr int DL = HD / 8;        // lanes per token row
  constexpr int TPL = kWave / DL;   // token rows per load instruction
  constexpr int TPW = kPage / TPL;  // token rows per lane per page
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int dg = lane % DL, tg = lane / DL;
  const int wi = blockIdx.x / a.nkv, h = blockIdx.x % a.nkv;
  const int row = a.work[2 * wi], split = a.work[2 * wi + 1];
  const int ctx = a.row_ctx[row];
  const int qrow = a.row_qrow[row];
  const int32_t* bt = a.bt + a.row_bt[row];
  const int n_pages = ceil_div(ctx, kPage);
  const int p_begin = split * a.pages_per_split;
  const int p_end = min(n_pages, p_begin + a.pages_per_split);

  const float qscale = a.scale * kLog2e;
  float qv[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint4 w = *reinterpret_cast<const uint4*>(
        a.q + (static_cast<size_t>(qrow) * a.nq + h * G + g) * HD + dg * 8);
    const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      qv[g][2 * e] = lo_bf16(ww[e]) * qscale;
      qv[g][2 * e + 1] = hi_bf16(ww[e]) * qscale;
    }
  }

  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = kNegBig;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[g][e] = 0.f;
  }

  for (int p = p_begin + wave; p < p_end; p += 4) {
    const int page = bt[p];
    const uint16_t* kb = a.kv + kv_offset(page, 0, a.nkv, h, 0, HD, dg * 8);
    const uint16_t* vb = a.kv + kv_offset(page, 1, a.nkv, h, 0, HD, dg * 8);
    uint4 kw[TPW], vw[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      kw[j] = *reinterpret_cast<const uint4*>(kb + (j * TPL + tg) * HD);
      vw[j] = *reinterpret_cast<const uint4*>(vb + (j * TPL + tg) * HD);
    }
    float s[TPW][G];
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      const uint32_t kk[4] = {kw[j].x, kw[j].y, kw[j].z, kw[j].w};
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          d += qv[g][2 * e] * lo_bf16(kk[e]);
          d += qv[g][2 * e + 1] * hi_bf16(kk[e]);
        }
        s[j][g] = d;
      }
    }
#pragma unroll
    for (int o = 1; o < DL; o <<= 1)
#pragma unroll
      for (int j = 0; j < TPW; ++j)
#pragma unroll
        for (int g = 0; g < G; ++g) s[j][g] += __shfl_xor(s[j][g], o, kWave);
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      const int pos = p * kPage + j * TPL + tg;
      if (pos >= ctx) {
#pragma unroll
        for (int g = 0; g < G; ++g) s[j][g] = -INFINITY;
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mp = s[0][g];
#pragma unroll
      for (int j = 1; j < TPW; ++j) mp = fmaxf(mp, s[j][g]);
#pragma unroll
      for (int o = DL; o < kWave; o <<= 1) mp = fmaxf(mp, __shfl_xor(mp, o, kWave));
      const float mn = fmaxf(m[g], mp);
      const float corr = exp2f(m[g] - mn);
      m[g] = mn;
      l[g] *= corr;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[g][e] *= corr;
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
        const float pj = exp2f(s[j][g] - mn);
        l[g] += pj;
        const uint32_t vv[4] = {vw[j].x, vw[j].y, vw[j].z, vw[j].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[g][2 * e] += pj * lo_bf16(vv[e]);
          acc[g][2 * e + 1] += pj * hi_bf16(vv[e]);
        }
      }
    }
  }

  // sum over the token groups of the wave (all share the wave's running max)
#pragma unroll
  for (int o = DL; o < kWave; o <<= 1) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      l[g] += __shfl_xor(l[g], o, kWave);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[g][e] += __shfl_xor(acc[g][e], o, kWave);
    }
  }

  __shared__ float sm[4][G], sl[4][G];
  __shared__ float sacc[4][G][HD];
  if (tg == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int e = 0; e < 8; ++e) sacc[wave][g][dg * 8 + e] = acc[g][e];
      if (dg == 0) {
        sm[wave][g] = m[g];
        sl[wave][g] = l[g];
      }
    }
  }
  __syncthreads();

  const int nsplit = a.row_nsplit[row];
  for (int idx = threadIdx.x; idx < G * HD; idx += blockDim.x) {
    const int g = idx / HD, d = idx % HD;
    float M = sm[0][g];
#pragma unroll
    for (int w = 1; w < 4; ++w) M = fmaxf(M, sm[w][g]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = exp2f(sm[w][g] - M);
      L += sl[w][g] * f;
      O += sacc[w][g][d] * f;
    }
    if (nsplit == 1) {
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

// Merge the split partials of each (row, query head).  One block of hd
// threads per (row, head); rows with a single split were already written.
__global__ __launch_bounds__(128) void attn_combine_kernel(AttnArgs a) {
  const int row = blockIdx.x / a.nq, j = blockIdx.x % a.nq;
  const int ns = a.row_nsplit[row];
  if (ns == 1) return;
  const int G = a.nq / a.nkv;
  const int h = j / G, g = j % G;
  const int hd = a.hd;
  const int w0 = a.row_work[row];
  const int d = threadIdx.x;
  auto part = [&](int s) { return a.part + ((static_cast<size_t>(w0 + s) * a.nkv + h) * G + g) * (hd + 2); };
  float M = kNegBig;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, part(s)[hd]);
  float L = 0.f, O = 0.f;
  for (int s = 0; s < ns; ++s) {
    const float* pp = part(s);
    const float f = exp2f(pp[hd] - M);
    L += pp[hd + 1] * f;
    O += pp[d] * f;
  }
  a.out[(static_cast<size_t>(a.row_qrow[row]) * a.nq + j) * hd + d] = f32_to_bf16(O / L);
}

template <int HD>
static hipError_t launch_hd(const AttnArgs& a, hipStream_t s) {
  const dim3 grid(a.n_work * a.nkv);
  switch (a.nq / a.nkv) {
    case 1: hipLaunchKernelGGL((attn_paged_kernel<HD, 1>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((attn_paged_kernel<HD, 2>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((attn_paged_kernel<HD, 4>), grid, dim3(256), 0, s, a); break;
    case 8: hipLaunchKernelGGL((attn_paged_kernel<HD, 8>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attn_paged(const AttnArgs& a, hipStream_t s) {
  if (a.n_work <= 0) return hipSuccess;
  if (a.hd == 128) return launch_hd<128>(a, s);
  if (a.hd == 64) return launch_hd<64>(a, s);
  return hipErrorInvalidValue;
}

hipError_t launch_attn_combine(const AttnArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(attn_combine_kernel, dim3(a.rows * a.nq), dim3(a.hd), 0, s, a);
  return hipGetLastError();
}

}  // namespace metro
