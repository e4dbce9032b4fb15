// The per-token core product z'_t = Sigma_{i(t)} z_t (App. D, middle step;
// Sec. 3.1: Sigma_i is the only per-LoRA matrix), and the split-K reduction
// of the fused GEMM.
//
// Core product.  Tokens arrive sorted by (cluster, adapter), so tokens of one
// LoRA are contiguous.  The sort cuts the sorted positions into items: runs
// of one adapter, at most kSigmaChunk long.  A workgroup takes one item,
// stages that adapter's Sigma_i in LDS once (fp32, rows padded to r+1 words
// so that lanes reading one column hit distinct banks) and produces every
// output of the item's tokens with a fixed ascending-order fp32 dot product.
// z_t is first summed over the shrink's k-splits in fixed order.  No atomics:
// the result is bitwise reproducible.  With Sigma == null (uncompressed path)
// the stage only sums and converts.
#include "cts_internal.h"

namespace cts {
namespace {

constexpr int kSigThreads = 256;
constexpr int kSigMaxR = 128;
constexpr int kPerThread = kSigmaChunk * kSigMaxR / kSigThreads;   // z elements per thread

template <typename TI> __device__ __forceinline__ float ld(const TI* p, int64_t i);
template <> __device__ __forceinline__ float ld<float>(const float* p, int64_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld<bf16_t>(const bf16_t* p, int64_t i) { return bf16_to_f32(p[i].bits); }

template <typename TI> __device__ __forceinline__ void st(TI* p, int64_t i, float v);
template <> __device__ __forceinline__ void st<float>(float* p, int64_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st<bf16_t>(bf16_t* p, int64_t i, float v) { p[i].bits = f32_to_bf16(v); }

template <typename TI>
__global__ __launch_bounds__(kSigThreads) void sigma_kernel(const float* __restrict__ zpart, int S,
                                                            int T, int r,
                                                            const int32_t* __restrict__ sorted_aid,
                                                            int n, const int32_t* __restrict__ items,
                                                            const int32_t* __restrict__ n_items,
                                                            const TI* __restrict__ Sigma,
                                                            TI* __restrict__ zp) {
  __shared__ float z[kSigmaChunk * kSigMaxR];
  __shared__ float sig[kSigMaxR * (kSigMaxR + 1)];

  const int item = blockIdx.x;
  if (item >= n_items[0]) return;
  const int tid = threadIdx.x;
  const int lo = items[item], hi = items[item + 1];
  const int cnt = (hi - lo) * r;   // outputs of this item

  // Sigma_a -> LDS (independent loads, issued before the partial sums)
  const int ld_sig = r + 1;
  if (Sigma != nullptr) {
    int a = sorted_aid[lo];
    a = a < 0 ? 0 : (a >= n ? n - 1 : a);
    const TI* sa = Sigma + static_cast<int64_t>(a) * r * r;
    for (int e = tid; e < r * r; e += kSigThreads) sig[(e / r) * ld_sig + (e % r)] = ld<TI>(sa, e);
  }
  // z = sum over k-splits, fixed order; the kPerThread loads of one split are independent
  float acc[kPerThread];
#pragma unroll
  for (int u = 0; u < kPerThread; ++u) acc[u] = 0.f;
  const int64_t split_stride = static_cast<int64_t>(T) * r;
  const float* zbase = zpart + static_cast<int64_t>(lo) * r;
  for (int q = 0; q < S; ++q) {
#pragma unroll
    for (int u = 0; u < kPerThread; ++u) {
      const int e = tid + u * kSigThreads;
      if (e < cnt) acc[u] += zbase[q * split_stride + e];
    }
  }
#pragma unroll
  for (int u = 0; u < kPerThread; ++u) {
    const int e = tid + u * kSigThreads;
    if (e < cnt) z[e] = acc[u];
  }
  __syncthreads();

  TI* out = zp + static_cast<int64_t>(lo) * r;
  if (Sigma == nullptr) {
    for (int e = tid; e < cnt; e += kSigThreads) st<TI>(out, e, z[e]);
    return;
  }
  for (int e = tid; e < cnt; e += kSigThreads) {
    const int i = e / r, c = e % r;
    const float* srow = sig + c * ld_sig;
    const float* zi = z + i * r;
    float d = 0.f;
    for (int q = 0; q < r; ++q) d = fmaf(srow[q], zi[q], d);
    st<TI>(out, e, d);
  }
}

template <int OUT_BF16>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, int S,
                                                            int N, int M,
                                                            const int32_t* __restrict__ perm,
                                                            void* __restrict__ out, int64_t ldo) {
  constexpr int V = OUT_BF16 ? 8 : 4;
  const int cpr = M / V;
  const int64_t c = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (c >= static_cast<int64_t>(N) * cpr) return;
  const int j = static_cast<int>(c / cpr), m = static_cast<int>(c % cpr) * V;
  float acc[V];
#pragma unroll
  for (int v = 0; v < V; ++v) acc[v] = 0.f;
  for (int s = 0; s < S; ++s) {
    const float* src = part + (static_cast<int64_t>(s) * N + j) * M + m;
#pragma unroll
    for (int v = 0; v < V; v += 4) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(src + v);
      acc[v] += x[0]; acc[v + 1] += x[1]; acc[v + 2] += x[2]; acc[v + 3] += x[3];
    }
  }
  const int64_t row = perm ? perm[j] : j;
  if (OUT_BF16) {
    uint4 w;
    w.x = f32_to_bf16(acc[0]) | (static_cast<uint32_t>(f32_to_bf16(acc[1])) << 16);
    w.y = f32_to_bf16(acc[2]) | (static_cast<uint32_t>(f32_to_bf16(acc[3])) << 16);
    w.z = f32_to_bf16(acc[4 % V]) | (static_cast<uint32_t>(f32_to_bf16(acc[5 % V])) << 16);
    w.w = f32_to_bf16(acc[6 % V]) | (static_cast<uint32_t>(f32_to_bf16(acc[7 % V])) << 16);
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(out) + row * ldo + m) = w;
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(out) + row * ldo + m) =
        f32x4{acc[0], acc[1], acc[2], acc[3]};
  }
}

}  // namespace

hipError_t launch_sigma(const float* zpart, int S, int T, int r, const int32_t* sorted_aid, int n,
                        const int32_t* items, const int32_t* n_items, int max_items,
                        const void* Sigma, void* zp, int in_dtype, hipStream_t stream) {
  dim3 grid(max_items);
  if (in_dtype == 0)
    hipLaunchKernelGGL(sigma_kernel<float>, grid, dim3(kSigThreads), 0, stream, zpart, S, T, r,
                       sorted_aid, n, items, n_items, static_cast<const float*>(Sigma),
                       static_cast<float*>(zp));
  else
    hipLaunchKernelGGL(sigma_kernel<bf16_t>, grid, dim3(kSigThreads), 0, stream, zpart, S, T, r,
                       sorted_aid, n, items, n_items, static_cast<const bf16_t*>(Sigma),
                       static_cast<bf16_t*>(zp));
  return hipGetLastError();
}

hipError_t launch_splitk_reduce(const float* part, int S, int N, int M, const int32_t* perm,
                                void* out, int64_t ldo, int out_dtype, hipStream_t stream) {
  const int V = out_dtype == 1 ? 8 : 4;
  const int64_t chunks = static_cast<int64_t>(N) * (M / V);
  dim3 grid(static_cast<unsigned>((chunks + 255) / 256));
  if (out_dtype == 1)
    hipLaunchKernelGGL(splitk_reduce_kernel<1>, grid, dim3(256), 0, stream, part, S, N, M, perm, out, ldo);
  else
    hipLaunchKernelGGL(splitk_reduce_kernel<0>, grid, dim3(256), 0, stream, part, S, N, M, perm, out, ldo);
  return hipGetLastError();
}

}  // namespace cts
