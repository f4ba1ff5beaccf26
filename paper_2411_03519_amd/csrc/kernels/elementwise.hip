// Row-wise and elementwise kernels of the forward pass (gfx950, wave64):
// embedding gather, RMSNorm, RoPE + paged KV write, row gather, greedy argmax,
// plus weight initialisation and page copy used by the runtime.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace metro {

thread_local LaunchEvents launch_events;

// ---------------------------------------------------------------------------
// Embedding gather: x[t, :] = fp32(E[tok[t], :]).  One block per token.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void embed_kernel(const int32_t* __restrict__ tok,
                                                    const uint16_t* __restrict__ E, int vocab, int d,
                                                    float* __restrict__ x) {
  const int t = blockIdx.x;
  const int id = tok[t];
  float* xr = x + static_cast<size_t>(t) * d;
  if (id < 0 || id >= vocab) {
    for (int i = threadIdx.x; i < d; i += blockDim.x) xr[i] = __builtin_nanf("");
    return;
  }
  const uint4* er = reinterpret_cast<const uint4*>(E + static_cast<size_t>(id) * d);
  for (int i = threadIdx.x; i < d / 8; i += blockDim.x) {
    uint4 w = er[i];
    float4 a = make_float4(lo_bf16(w.x), hi_bf16(w.x), lo_bf16(w.y), hi_bf16(w.y));
    float4 b = make_float4(lo_bf16(w.z), hi_bf16(w.z), lo_bf16(w.w), hi_bf16(w.w));
    reinterpret_cast<float4*>(xr)[2 * i] = a;
    reinterpret_cast<float4*>(xr)[2 * i + 1] = b;
  }
}

hipError_t launch_embed(const int32_t* tok, const uint16_t* embed, int vocab, int d, float* x, int T,
                        hipStream_t s) {
  if (T <= 0) return hipSuccess;
  launch_kernel(embed_kernel, dim3(T), dim3(256), 0, s, tok, embed, vocab, d, x);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// RMSNorm: h = bf16(x * rsqrt(mean(x^2) + eps) * g).  One block per row; each
// thread owns VPT float4 of the row and first issues all its loads (x, g and
// the n_parts k-slice sums of the GEMM that produced the residual), so the
// row costs one memory round trip; the slices are added in slice order and
// the updated residual is written back.
// ---------------------------------------------------------------------------
constexpr int kMaxParts = 8;

template <int NTH, int VPT>
__global__ __launch_bounds__(NTH) void rmsnorm_kernel(float* __restrict__ x, int ldx, const uint16_t* __restrict__ g,
                                                      float eps, uint16_t* __restrict__ h, int ldh, int d,
                                                      const float* __restrict__ parts, int n_parts, int rows) {
  const int r = blockIdx.x, n4 = d / 4;
  float4* xr = reinterpret_cast<float4*>(x + static_cast<size_t>(r) * ldx);
  const uint2* gr = reinterpret_cast<const uint2*>(g);
  const float4* pr = reinterpret_cast<const float4*>(parts + static_cast<size_t>(r) * d);
  const size_t stride = static_cast<size_t>(rows) * d / 4;
  float4 v[VPT], pv[VPT][kMaxParts];
  uint2 gw[VPT];
#pragma unroll
  for (int j = 0; j < VPT; ++j) {
    const int i = threadIdx.x + j * NTH;
    if (i < n4) {
      v[j] = xr[i];
      gw[j] = gr[i];
#pragma unroll
      for (int k = 0; k < kMaxParts; ++k)
        if (k < n_parts) pv[j][k] = pr[k * stride + i];
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < VPT; ++j) {
    const int i = threadIdx.x + j * NTH;
    if (i >= n4) continue;
    if (n_parts > 0) {
      float4 sum = pv[j][0];
#pragma unroll
      for (int k = 1; k < kMaxParts; ++k)
        if (k < n_parts) {
          sum.x += pv[j][k].x;
          sum.y += pv[j][k].y;
          sum.z += pv[j][k].z;
          sum.w += pv[j][k].w;
        }
      v[j].x += sum.x;
      v[j].y += sum.y;
      v[j].z += sum.z;
      v[j].w += sum.w;
      xr[i] = v[j];
    }
    ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
  }
  ss = wave_sum(ss);
  constexpr int NWV = NTH / 64;
  __shared__ float red[NWV];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < NWV; ++w) tot += red[w];
  const float inv = rsqrtf(tot / static_cast<float>(d) + eps);
  uint2* hr = reinterpret_cast<uint2*>(h + static_cast<size_t>(r) * ldh);
#pragma unroll
  for (int j = 0; j < VPT; ++j) {
    const int i = threadIdx.x + j * NTH;
    if (i >= n4) continue;
    uint2 o;
    o.x = pack_bf16x2(v[j].x * inv * lo_bf16(gw[j].x), v[j].y * inv * hi_bf16(gw[j].x));
    o.y = pack_bf16x2(v[j].z * inv * lo_bf16(gw[j].y), v[j].w * inv * hi_bf16(gw[j].y));
    hr[i] = o;
  }
}

hipError_t launch_rmsnorm(float* x, int ldx, const uint16_t* g, float eps, uint16_t* h, int ldh, int rows, int d,
                          const float* parts, int n_parts, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (n_parts > kMaxParts || d % 4) return hipErrorInvalidValue;
  const int n4 = d / 4;
  auto go = [&](auto nth, auto vpt) {
    constexpr int NTH = decltype(nth)::value, VPT = decltype(vpt)::value;
    launch_kernel((rmsnorm_kernel<NTH, VPT>), dim3(rows), dim3(NTH), 0, s, x, ldx, g, eps, h, ldh, d, parts, n_parts,
                  rows);
  };
  if (n4 <= 256)
    go(std::integral_constant<int, 256>{}, std::integral_constant<int, 1>{});
  else if (n4 <= 1024)
    go(std::integral_constant<int, 1024>{}, std::integral_constant<int, 1>{});
  else if (n4 <= 2048)
    go(std::integral_constant<int, 1024>{}, std::integral_constant<int, 2>{});
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// RoPE on q and k (rotate-half pairs (i, i + hd/2)), bf16 rounding, and the
// write of k and v into their page slot (tile layouts in common.h).  One
// wave per (token, head) of the nq + 2 nkv heads; lane j < hd/2 takes the pair
// (j, j + hd/2).  The qkv value is the sum of the GEMM's k slices in slice
// order when the GEMM was split.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void rope_kv_kernel(const float* __restrict__ qkv, int n_parts, int T, int nq,
                                                     int nkv, int hd, const int32_t* __restrict__ pos,
                                                     const int32_t* __restrict__ slot,
                                                     const float2* __restrict__ rope, uint16_t* __restrict__ q,
                                                     uint16_t* __restrict__ kv) {
  const int nh = nq + 2 * nkv;
  const int t = blockIdx.x / nh, head = blockIdx.x % nh;
  const int half = hd / 2;
  const int width = nh * hd;
  const float* row = qkv + static_cast<size_t>(t) * width + head * hd;
  const size_t pstride = static_cast<size_t>(T) * width;
  auto val = [&](int i) {
    float v = row[i];
    for (int k = 1; k < n_parts; ++k) v += row[k * pstride + i];
    return v;
  };
  const int j = threadIdx.x;
  if (j >= half) return;
  const int sl = slot[t];
  const int page = sl / kPage, off = sl % kPage;
  // columns of a head come in the rotate-half interleave of its W rows
  const float a = val(rope_pair_row(j, half)), b = val(rope_pair_row(j + half, half));
  if (head < nq + nkv) {
    const float2 c = rope[static_cast<size_t>(pos[t]) * half + j];
    const uint16_t ra = f32_to_bf16(a * c.x - b * c.y);
    const uint16_t rb = f32_to_bf16(a * c.y + b * c.x);
    if (head < nq) {
      uint16_t* dst = q + static_cast<size_t>(t) * nq * hd + head * hd;
      dst[j] = ra;
      dst[j + half] = rb;
    } else {
      uint16_t* kt = kv + kv_offset(page, 0, nkv, head - nq, 0, hd, 0);
      kt[k_tile_offset(off, j)] = ra;
      kt[k_tile_offset(off, j + half)] = rb;
    }
  } else {
    uint16_t* vt = kv + kv_offset(page, 1, nkv, head - nq - nkv, 0, hd, 0);
    vt[vt_tile_offset(j, off)] = f32_to_bf16(a);
    vt[vt_tile_offset(j + half, off)] = f32_to_bf16(b);
  }
}

hipError_t launch_rope_kv(const float* qkv, int n_parts, int T, int nq, int nkv, int hd, const int32_t* pos,
                          const int32_t* slot, const float2* rope, uint16_t* q, uint16_t* kv_layer,
                          hipStream_t s) {
  if (T <= 0) return hipSuccess;
  launch_kernel(rope_kv_kernel, dim3(T * (nq + 2 * nkv)), dim3(64), 0, s, qkv, n_parts, T, nq, nkv, hd, pos,
                     slot, rope, q, kv_layer);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Row gather (the last position of each prefill item).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gather_rows_kernel(const float* __restrict__ x, int d,
                                                          const int32_t* __restrict__ rows,
                                                          float* __restrict__ out) {
  const float4* src = reinterpret_cast<const float4*>(x + static_cast<size_t>(rows[blockIdx.x]) * d);
  float4* dst = reinterpret_cast<float4*>(out + static_cast<size_t>(blockIdx.x) * d);
  for (int i = threadIdx.x; i < d / 4; i += blockDim.x) dst[i] = src[i];
}

hipError_t launch_gather_rows(const float* x, int d, const int32_t* rows, int n, float* out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  launch_kernel(gather_rows_kernel, dim3(n), dim3(256), 0, s, x, d, rows, out);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Greedy argmax over fp32 logits: lowest index among the maxima, NaN skipped.
// One block of 1024 threads per row; each thread issues kArgmaxBatch float4
// loads before comparing any, so a 128k-entry row costs four memory round
// trips instead of one per load (23.8 -> about 5 us for 25 rows of 128256).
// ---------------------------------------------------------------------------
struct ArgBest {
  float v;
  int i;
};

__device__ __forceinline__ ArgBest arg_better(ArgBest a, ArgBest b) {
  if (b.i < 0) return a;
  if (a.i < 0) return b;
  if (b.v > a.v || (b.v == a.v && b.i < a.i)) return b;
  return a;
}

constexpr int kArgmaxBatch = 8;

__global__ __launch_bounds__(1024) void argmax_kernel(const float* __restrict__ logits, int vocab,
                                                      int32_t* __restrict__ out) {
  const float4* row = reinterpret_cast<const float4*>(logits + static_cast<size_t>(blockIdx.x) * vocab);
  const int n4 = vocab / 4;
  ArgBest b{0.f, -1};
  // a thread visits j = tid, tid + 1024, ... in increasing order, so the
  // strict comparison keeps its lowest index among equal values
  for (int j0 = threadIdx.x; j0 < n4; j0 += kArgmaxBatch * 1024) {
    float4 v[kArgmaxBatch];
#pragma unroll
    for (int u = 0; u < kArgmaxBatch; ++u) {
      const int j = j0 + u * 1024;
      v[u] = j < n4 ? row[j] : make_float4(__builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""),
                                           __builtin_nanf(""));
    }
#pragma unroll
    for (int u = 0; u < kArgmaxBatch; ++u) {
      const int j = j0 + u * 1024;
      const float e[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (e[k] == e[k] && (b.i < 0 || e[k] > b.v)) b = ArgBest{e[k], 4 * j + k};
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    ArgBest other{__shfl_xor(b.v, o, kWave), __shfl_xor(b.i, o, kWave)};
    b = arg_better(b, other);
  }
  __shared__ float sv[16];
  __shared__ int si[16];
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sv[w] = b.v;
    si[w] = b.i;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    ArgBest r{sv[0], si[0]};
    for (int k = 1; k < 16; ++k) r = arg_better(r, ArgBest{sv[k], si[k]});
    out[blockIdx.x] = r.i;
  }
}

hipError_t launch_argmax(const float* logits, int vocab, int rows, int32_t* out, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  launch_kernel(argmax_kernel, dim3(rows), dim3(1024), 0, s, logits, vocab, out);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight initialisation: SplitMix64 (Steele, Lea & Flood 2014) as a
// counter-based hash of (key, element index) -> two uniforms -> Box-Muller
// (one normal per element) -> 0.02 * z -> bf16.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t splitmix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

__global__ __launch_bounds__(256) void init_normal_kernel(uint16_t* __restrict__ dst, int64_t ld, int rows,
                                                          int cols, RowMap map, uint64_t key, bool packed) {
  const int64_t n = static_cast<int64_t>(rows) * cols;
  for (int64_t e = blockIdx.x * 256ll + threadIdx.x; e < n; e += static_cast<int64_t>(gridDim.x) * 256) {
    const int r = static_cast<int>(e / cols), c = static_cast<int>(e % cols);
    const uint64_t h = splitmix64(key + static_cast<uint64_t>(e + 1) * 0x9e3779b97f4a7c15ull);
    const float u1 = (static_cast<float>(h >> 40) + 1.0f) * (1.0f / 16777216.0f);  // (0, 1]
    const float u2 = static_cast<float>((h >> 16) & 0xffffffull) * (1.0f / 16777216.0f);  // [0, 1)
    const float z = sqrtf(-2.0f * logf(u1)) * cosf(6.283185307179586f * u2);
    const int64_t pr = map_row(map, r);
    dst[packed ? packed_offset(pr, c, ld) : pr * ld + c] = f32_to_bf16(0.02f * z);
  }
}

hipError_t launch_init_normal(uint16_t* dst, int64_t ld, int rows, int cols, RowMap map, uint64_t key, bool packed,
                              hipStream_t s) {
  const int64_t n = static_cast<int64_t>(rows) * cols;
  const int64_t blocks = (n + 255) / 256;
  const int grid = static_cast<int>(blocks < 65536 ? blocks : 65536);
  launch_kernel(init_normal_kernel, dim3(grid), dim3(256), 0, s, dst, ld, rows, cols, map, key, packed);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Row-major bf16 weight -> MFMA operand order (packed_offset): one thread per
// 8-element chunk (row r, k .. k+7) of the destination's Kp columns, logical
// row r going to row map_row(map, r); k >= cols is zero.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void pack_weight_kernel(const uint16_t* __restrict__ src, int64_t ld_src,
                                                          int rows, int cols, uint16_t* __restrict__ dst, int Kp,
                                                          RowMap map) {
  const int kc = Kp / 8;
  const int64_t n = static_cast<int64_t>(rows) * kc;
  for (int64_t e = blockIdx.x * 256ll + threadIdx.x; e < n; e += static_cast<int64_t>(gridDim.x) * 256) {
    const int r = static_cast<int>(e / kc), k = static_cast<int>(e % kc) * 8;
    uint16_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = k + j < cols ? src[r * ld_src + k + j] : 0;
    const int64_t pr = map_row(map, r);
    uint4 o;
    o.x = v[0] | (static_cast<uint32_t>(v[1]) << 16);
    o.y = v[2] | (static_cast<uint32_t>(v[3]) << 16);
    o.z = v[4] | (static_cast<uint32_t>(v[5]) << 16);
    o.w = v[6] | (static_cast<uint32_t>(v[7]) << 16);
    *reinterpret_cast<uint4*>(dst + packed_offset(pr, k, Kp)) = o;
  }
}

hipError_t launch_pack_weight(const uint16_t* src, int64_t ld_src, int rows, int cols, uint16_t* dst, int Kp,
                              RowMap map, hipStream_t s) {
  const int64_t n = static_cast<int64_t>(rows) * (Kp / 8);
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  launch_kernel(pack_weight_kernel, dim3(static_cast<int>(blocks < 65536 ? blocks : 65536)), dim3(256), 0, s, src,
                ld_src, rows, cols, dst, Kp, map);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void fill_bf16_kernel(uint16_t* __restrict__ dst, int64_t n, uint16_t v) {
  for (int64_t e = blockIdx.x * 256ll + threadIdx.x; e < n; e += static_cast<int64_t>(gridDim.x) * 256) dst[e] = v;
}

hipError_t launch_fill_bf16(uint16_t* dst, int64_t n, uint16_t value, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  launch_kernel(fill_bf16_kernel, dim3(static_cast<int>(blocks < 65536 ? blocks : 65536)), dim3(256), 0, s,
                     dst, n, value);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Page copy across all layers (partial last page of a forked prefix).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void page_copy_kernel(uint16_t* __restrict__ pool, int64_t layer_stride,
                                                        int64_t page_elems, int src, int dst) {
  uint16_t* base = pool + static_cast<size_t>(blockIdx.x) * layer_stride;
  const uint4* s = reinterpret_cast<const uint4*>(base + static_cast<size_t>(src) * page_elems);
  uint4* d = reinterpret_cast<uint4*>(base + static_cast<size_t>(dst) * page_elems);
  for (int64_t i = threadIdx.x; i < page_elems / 8; i += 256) d[i] = s[i];
}

hipError_t launch_page_copy(uint16_t* pool, int64_t layer_stride, int64_t page_elems, int layers, int src,
                            int dst, hipStream_t s) {
  launch_kernel(page_copy_kernel, dim3(layers), dim3(256), 0, s, pool, layer_stride, page_elems, src, dst);
  return hipGetLastError();
}

}  // namespace metro
