// The per-token core product z'_t = Sigma_{i(t)} z_t (App. D, middle step;
// Sec. 3.1: Sigma_i is the only per-LoRA matrix), and the split-K reduction
// of the fused GEMM.
//
// Sigma stage.  Tokens arrive sorted by (cluster, adapter), so tokens of one
// LoRA are contiguous: a workgroup walks its TB sorted positions run by run,
// stages each run's Sigma_i in LDS once (fp32, rows padded to r+1 words so
// that lanes reading one column hit distinct banks), and computes one output
// element per thread with a fixed ascending-order fp32 dot product.  z_t is
// first reduced over the shrink's k-splits in fixed order.  No atomics: the
// result is bitwise reproducible.  With Sigma == null (uncompressed path) the
// stage only reduces and converts.
#include "cts_internal.h"

namespace cts {
namespace {

constexpr int kSigThreads = 256;
constexpr int kSigMaxR = 128;

template <typename TI> __device__ __forceinline__ float ld(const TI* p, int64_t i);
template <> __device__ __forceinline__ float ld<float>(const float* p, int64_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld<bf16_t>(const bf16_t* p, int64_t i) { return bf16_to_f32(p[i].bits); }

template <typename TI> __device__ __forceinline__ void st(TI* p, int64_t i, float v);
template <> __device__ __forceinline__ void st<float>(float* p, int64_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st<bf16_t>(bf16_t* p, int64_t i, float v) { p[i].bits = f32_to_bf16(v); }

template <typename TI, int TB>
__global__ __launch_bounds__(kSigThreads) void sigma_kernel(const float* __restrict__ zpart, int S,
                                                            int T, int r,
                                                            const int32_t* __restrict__ sorted_aid,
                                                            int n, const TI* __restrict__ Sigma,
                                                            TI* __restrict__ zp) {
  __shared__ float z[TB * kSigMaxR];
  __shared__ float sig[kSigMaxR * (kSigMaxR + 1)];
  __shared__ int32_t aid[TB];

  const int tid = threadIdx.x;
  const int j0 = blockIdx.x * TB;
  const int tb = min(TB, T - j0);

  for (int i = tid; i < tb; i += kSigThreads) {
    int a = sorted_aid ? sorted_aid[j0 + i] : 0;
    aid[i] = a < 0 ? 0 : (a >= n ? n - 1 : a);
  }
  for (int e = tid; e < tb * r; e += kSigThreads) {
    const int i = e / r, c = e % r;
    const int64_t off = static_cast<int64_t>(j0 + i) * r + c;
    float s = 0.f;
    for (int q = 0; q < S; ++q) s += zpart[static_cast<int64_t>(q) * T * r + off];
    z[i * r + c] = s;
  }
  __syncthreads();

  if (Sigma == nullptr) {
    for (int e = tid; e < tb * r; e += kSigThreads)
      st<TI>(zp, static_cast<int64_t>(j0) * r + e, z[e]);
    return;
  }

  const int ld_sig = r + 1;
  int cur = 0;
  while (cur < tb) {
    const int a = aid[cur];
    int end = cur + 1;
    while (end < tb && aid[end] == a) ++end;
    const TI* sa = Sigma + static_cast<int64_t>(a) * r * r;
    for (int e = tid; e < r * r; e += kSigThreads) sig[(e / r) * ld_sig + (e % r)] = ld<TI>(sa, e);
    __syncthreads();
    for (int e = tid; e < (end - cur) * r; e += kSigThreads) {
      const int i = cur + e / r, c = e % r;
      const float* srow = sig + c * ld_sig;
      const float* zi = z + i * r;
      float acc = 0.f;
      for (int q = 0; q < r; ++q) acc = fmaf(srow[q], zi[q], acc);
      st<TI>(zp, static_cast<int64_t>(j0 + i) * r + c, acc);
    }
    __syncthreads();
    cur = end;
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
                        const void* Sigma, void* zp, int in_dtype, hipStream_t stream) {
  constexpr int TB = 8;
  dim3 grid((T + TB - 1) / TB);
  if (in_dtype == 0)
    hipLaunchKernelGGL((sigma_kernel<float, TB>), grid, dim3(kSigThreads), 0, stream, zpart, S, T, r,
                       sorted_aid, n, static_cast<const float*>(Sigma), static_cast<float*>(zp));
  else
    hipLaunchKernelGGL((sigma_kernel<bf16_t, TB>), grid, dim3(kSigThreads), 0, stream, zpart, S, T, r,
                       sorted_aid, n, static_cast<const bf16_t*>(Sigma), static_cast<bf16_t*>(zp));
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
