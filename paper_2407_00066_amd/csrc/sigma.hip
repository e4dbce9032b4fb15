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
#include "cts.h"
#include "cts_internal.h"

namespace cts {
namespace {

constexpr int kSigThreads = 256;
// MAXR: the largest rank a kernel instance takes (64 or 128).  LDS rows are
// MAXR + 4 floats: 16-byte aligned, and lanes reading one column of 16 rows
// (4 consecutive k each) land on distinct banks.

template <typename TI> struct Vec16;
template <> struct Vec16<float> {          // 4 floats per 16 bytes
  static constexpr int N = 4;
  __device__ static __forceinline__ void widen(const uint4& v, float* o) {
    o[0] = __uint_as_float(v.x); o[1] = __uint_as_float(v.y);
    o[2] = __uint_as_float(v.z); o[3] = __uint_as_float(v.w);
  }
};
template <> struct Vec16<bf16_t> {         // 8 bf16 per 16 bytes
  static constexpr int N = 8;
  __device__ static __forceinline__ void widen(const uint4& v, float* o) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = bf16_to_f32(static_cast<uint16_t>(w[i] & 0xffffu));
      o[2 * i + 1] = bf16_to_f32(static_cast<uint16_t>(w[i] >> 16));
    }
  }
};

template <typename TI> __device__ __forceinline__ void st(TI* p, int64_t i, float v);
template <> __device__ __forceinline__ void st<float>(float* p, int64_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st<bf16_t>(bf16_t* p, int64_t i, float v) { p[i].bits = f32_to_bf16(v); }

template <typename TI> __device__ __forceinline__ float ld(const TI* p, int64_t i);
template <> __device__ __forceinline__ float ld<float>(const float* p, int64_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld<bf16_t>(const bf16_t* p, int64_t i) { return bf16_to_f32(p[i].bits); }

// Diagonal Sigma_i (Sec. 3.1, eq. JD-Diag; App. F: no batched product is
// needed): z'_t[c] = sigma_i[c] z_t[c], an elementwise scale.  Same items and
// the same fixed-order split sum as sigma_kernel; no LDS.
template <typename TI>
__global__ __launch_bounds__(kSigThreads) void sigma_diag_kernel(const float* __restrict__ zpart, int S,
                                                                 int T, int r,
                                                                 const int32_t* __restrict__ sorted_aid,
                                                                 int n, const int32_t* __restrict__ items,
                                                                 const int32_t* __restrict__ n_items,
                                                                 const TI* __restrict__ sigma,
                                                                 TI* __restrict__ zp,
                                                                 const int32_t* __restrict__ sorted_seg,
                                                                 const int32_t* __restrict__ seg_rank,
                                                                 int32_t* __restrict__ sorted_rank,
                                                                 const int32_t* __restrict__ split_dev,
                                                                 const int32_t* __restrict__ item_aid) {
  const int item = blockIdx.x;
  // the item's bounds and adapter are read with the item count (the grid
  // covers max_items items; the arrays hold max_items + 1 entries)
  const int n_it = n_items[0];
  const int lo = items[item], hi = items[item + 1];
  const int a_it = item_aid[item];
  // the shrink's split count (read from a valid address either way)
  const int s_dev = (split_dev ? split_dev : n_items)[0];
  // all five loads before the exit test: one round trip, not a chain
  asm volatile("" ::"s"(lo), "s"(hi), "s"(a_it), "s"(s_dev));
  if (item >= n_it) return;
  if (split_dev) S = min(s_dev, S);
  const int tid = threadIdx.x;
  const int cnt = (hi - lo) * r;
  const int rk = seg_rank ? seg_rank_of(seg_rank, sorted_seg[lo], r) : r;   // a multiple of 8
  if (sorted_rank && tid < hi - lo) sorted_rank[lo + tid] = rk;
  int a = a_it;
  a = a < 0 ? 0 : (a >= n ? n - 1 : a);
  const TI* sa = sigma + static_cast<int64_t>(a) * r;
  const int64_t split_stride = static_cast<int64_t>(T) * r;
  const float* zbase = zpart + static_cast<int64_t>(lo) * r;
  TI* out = zp + static_cast<int64_t>(lo) * r;
  for (int e4 = tid * 4; e4 < cnt; e4 += kSigThreads * 4) {
    const int c = e4 % r;                                  // r % 8 == 0: c..c+3 in one row
    const bool in_rank = c < rk;                           // and all four, or none, below rk
    float s[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) s[v] = in_rank ? ld<TI>(sa, c + v) : 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int q = 0; in_rank && q < S; q += 16) {
      f32x4 w[16];
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (q + u < S) w[u] = *reinterpret_cast<const f32x4*>(zbase + (q + u) * split_stride + e4);
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (q + u < S) acc += w[u];
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) st<TI>(out, e4 + v, s[v] * acc[v]);
  }
}

// Several modules in one launch (blockIdx.y = module m): module m's Sigma
// is sigma[m], and its z and z' are the columns [m r, m r + r) of rows ldz
// apart.
struct SigmaMods {
  const void* sigma[CTS_MAX_MODULES];
};

// ZB: split partials whose loads are in flight together per thread (the
// host picks the smallest of 8, 16 or 32 that covers the split; fewer
// registers mean more workgroups resident when there are many items)
template <typename TI, int MAXR, int ZB>
__global__ __launch_bounds__(kSigThreads) void sigma_kernel(const float* __restrict__ zpart, int S,
                                                            int T, int r,
                                                            const int32_t* __restrict__ sorted_aid,
                                                            int n, const int32_t* __restrict__ items,
                                                            const int32_t* __restrict__ n_items,
                                                            const TI* __restrict__ Sigma,
                                                            TI* __restrict__ zp,
                                                            const int32_t* __restrict__ sorted_seg,
                                                            const int32_t* __restrict__ seg_rank,
                                                            int32_t* __restrict__ sorted_rank, int ldz,
                                                            const int32_t* __restrict__ split_dev,
                                                            const SigmaMods mods, int nmod,
                                                            const int32_t* __restrict__ item_aid) {
  constexpr int kSigLd = MAXR + 4;
  __shared__ __attribute__((aligned(16))) float z[kSigmaChunk * kSigLd];
  __shared__ __attribute__((aligned(16))) float sig[MAXR * kSigLd];

  const int item = blockIdx.x;
  // the item's bounds and adapter are read with the item count (the grid
  // covers max_items items; the arrays hold max_items + 1 entries)
  const int n_it = n_items[0];
  const int lo = items[item], hi = items[item + 1];
  const int a_it = item_aid[item];
  // the shrink's split count (read from a valid address either way)
  const int s_dev = (split_dev ? split_dev : n_items)[0];
  // all five loads before the exit test: one round trip, not a chain
  asm volatile("" ::"s"(lo), "s"(hi), "s"(a_it), "s"(s_dev));
  if (item >= n_it) return;
  if (nmod > 0) {
    const int m = blockIdx.y;
    Sigma = static_cast<const TI*>(mods.sigma[m]);
    zpart += static_cast<int64_t>(m) * r;
    zp += static_cast<int64_t>(m) * r;
  }
  // pieces the shrink actually split the reduction into (at most S)
  if (split_dev) S = min(s_dev, S);
  const int tid = threadIdx.x;
  const int nt = hi - lo;                 // tokens of this item (<= kSigmaChunk), one adapter
  const int cnt = nt * r;                 // outputs of this item
  // rank of the item's segment (a multiple of 8): Sigma's entries past it and
  // z's are neither read nor used; they stage as zeros
  const int rk = seg_rank ? seg_rank_of(seg_rank, sorted_seg[lo], r) : r;
  if (sorted_rank && tid < nt) sorted_rank[lo + tid] = rk;

  // Loads first, uses after: this thread's split partials (they depend on
  // the item only) and its 16-byte pieces of Sigma_a (on the adapter) are
  // all in flight before the first is waited for.  z = sum over the
  // shrink's k-splits in fixed order; 4 consecutive values per thread and
  // round, ZB splits' loads in flight at a time.  Rows of zpart and zp are
  // ldz apart (ldz = r, or the stacked rank of several modules).
  const int64_t split_stride = static_cast<int64_t>(T) * ldz;
  const float* zbase = zpart + static_cast<int64_t>(lo) * ldz;
  constexpr int ZR = (kSigmaChunk * MAXR / 4 + kSigThreads - 1) / kSigThreads;   // rounds of 4 values
  f32x4 zacc[ZR];
  f32x4 zv[ZR][ZB];
#pragma unroll
  for (int u = 0; u < ZR; ++u) zacc[u] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto zload = [&](int q) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < ZR; ++u) {
      const int e4 = (tid + u * kSigThreads) * 4;
      const bool ok = e4 < cnt && e4 % r < rk;
      const int64_t zo = static_cast<int64_t>(e4 / r) * ldz + e4 % r;
#pragma unroll
      for (int w = 0; w < ZB; ++w)
        if (ok && q + w < S) zv[u][w] = *reinterpret_cast<const f32x4*>(zbase + (q + w) * split_stride + zo);
    }
  };
  auto zsum = [&](int q) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < ZR; ++u) {
      const int e4 = (tid + u * kSigThreads) * 4;
      const bool ok = e4 < cnt && e4 % r < rk;
#pragma unroll
      for (int w = 0; w < ZB; ++w)
        if (ok && q + w < S) zacc[u] += zv[u][w];
    }
  };
  zload(0);

  // Sigma_a -> LDS as fp32
  if (Sigma != nullptr) {
    int a = a_it;
    a = a < 0 ? 0 : (a >= n ? n - 1 : a);
    constexpr int V = Vec16<TI>::N;
    constexpr int PER = (MAXR * MAXR / V + kSigThreads - 1) / kSigThreads;
    const uint4* sa = reinterpret_cast<const uint4*>(Sigma + static_cast<int64_t>(a) * r * r);
    const int nv = r * r / V;
    uint4 raw[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = tid + u * kSigThreads;
      const int row = (e * V) / r, col = (e * V) % r;
      raw[u] = (e < nv && row < rk && col < rk) ? sa[e] : uint4{0u, 0u, 0u, 0u};
    }
    zsum(0);
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = tid + u * kSigThreads;
      if (e < nv) {
        float w[V];
        Vec16<TI>::widen(raw[u], w);
        const int row = (e * V) / r, col = (e * V) % r;     // V consecutive columns, col % V == 0
#pragma unroll
        for (int q = 0; q < V; q += 4)
          *reinterpret_cast<f32x4*>(sig + row * kSigLd + col + q) = f32x4{w[q], w[q + 1], w[q + 2], w[q + 3]};
      }
    }
  } else {
    zsum(0);
  }
  // splits past the first 16
  for (int q = ZB; q < S; q += ZB) {
    zload(q);
    zsum(q);
  }
#pragma unroll
  for (int u = 0; u < ZR; ++u) {
    const int e4 = (tid + u * kSigThreads) * 4;
    if (e4 < cnt) {
      const int i = e4 / r, c = e4 % r;
      *reinterpret_cast<f32x4*>(z + i * kSigLd + c) = zacc[u];
    }
  }
  __syncthreads();

  TI* out = zp + static_cast<int64_t>(lo) * ldz;
  if (Sigma == nullptr) {
    for (int e = tid; e < cnt; e += kSigThreads)
      st<TI>(out, static_cast<int64_t>(e / r) * ldz + e % r, z[(e / r) * kSigLd + e % r]);
    return;
  }
  // z'[i][c] = sum_q Sigma[c][q] z[i][q] on the fp32 matrix cores: one
  // 16x16x4 MFMA step multiplies the item's (up to 16) token rows by 16
  // columns of Sigma^T over 4 k; wave w takes column blocks w, w+4, ...
  // A lane reads one z value (row l%16, k l/16) and one Sigma value (row =
  // output column l%16, k l/16) per step.  Rows past the item's tokens and
  // columns past r read stale LDS and are never stored (an output depends
  // only on its own row of z and its own row of Sigma).
  const int lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 15, fk = lane >> 4;
  for (int cb = wave; cb * 16 < r; cb += kSigThreads / 64) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    const float* zr = z + fr * kSigLd + fk;
    const float* sr = sig + (cb * 16 + fr) * kSigLd + fk;
    for (int q = 0; q < r; q += 4)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(zr[q], sr[q], acc, 0, 0, 0);
    const int c = cb * 16 + fr;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int i = 4 * fk + v;
      if (i < nt && c < r) st<TI>(out, static_cast<int64_t>(i) * ldz + c, acc[v]);
    }
  }
}

template <int OUT_BF16>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, int S,
                                                            int N, int M,
                                                            const int32_t* __restrict__ perm,
                                                            void* __restrict__ out, int64_t ldo,
                                                            const SplitkMods mods) {
  constexpr int V = OUT_BF16 ? 8 : 4;
  const int cpr = M / V;
  const int64_t c = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (c >= static_cast<int64_t>(N) * cpr) return;
  const int j = static_cast<int>(c / cpr), mc = static_cast<int>(c % cpr) * V;
  // several modules: columns [col[q], col[q+1]) of the partials are module
  // q's output (each a multiple of 8 wide, so a chunk lies in one module)
  int m = mc;
  if (mods.n > 0) {
    int q = 0;
#pragma unroll
    for (int u = 1; u < kMaxGemmModules; ++u) q += (u < mods.n && mc >= mods.col[u]) ? 1 : 0;
    out = mods.out[q];
    ldo = mods.ldo[q];
    m = mc - mods.col[q];
  }
  const int64_t row = perm ? perm[j] : j;     // read with the partials
  float acc[V];
#pragma unroll
  for (int v = 0; v < V; ++v) acc[v] = 0.f;
  // the partials are summed in piece order; four pieces' loads go out before
  // their sums, so a launch waits for one round trip per four pieces (not one
  // per piece)
  const float* src0 = part + static_cast<int64_t>(j) * M + mc;
  const int64_t pstride = static_cast<int64_t>(N) * M;
  int s = 0;
  for (; s + 4 <= S; s += 4) {
    f32x4 x[4][V / 4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < V / 4; ++v)
        x[u][v] = *reinterpret_cast<const f32x4*>(src0 + (s + u) * pstride + 4 * v);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < V / 4; ++v) {
        acc[4 * v] += x[u][v][0]; acc[4 * v + 1] += x[u][v][1];
        acc[4 * v + 2] += x[u][v][2]; acc[4 * v + 3] += x[u][v][3];
      }
  }
  for (; s < S; ++s) {
#pragma unroll
    for (int v = 0; v < V / 4; ++v) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(src0 + s * pstride + 4 * v);
      acc[4 * v] += x[0]; acc[4 * v + 1] += x[1]; acc[4 * v + 2] += x[2]; acc[4 * v + 3] += x[3];
    }
  }
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
                        const void* Sigma, void* zp, int in_dtype, hipStream_t stream,
                        bool diag, const int32_t* sorted_seg, const int32_t* seg_rank,
                        int32_t* sorted_rank, int ldz, const int32_t* split_dev,
                        const void* const* sigmas, int nmod, const int32_t* item_aid) {
  if (seg_rank && !sorted_seg) return hipErrorInvalidValue;
  if (!item_aid) return hipErrorInvalidValue;
  if (sorted_rank && !seg_rank) return hipErrorInvalidValue;
  if (ldz <= 0) ldz = r;
  if (ldz != r && (diag || ldz < r || ldz % 4)) return hipErrorInvalidValue;
  if (nmod < 0 || nmod > CTS_MAX_MODULES || (nmod > 0 && (!sigmas || diag || ldz < nmod * r)))
    return hipErrorInvalidValue;
  SigmaMods mods{};
  for (int m = 0; m < nmod; ++m) mods.sigma[m] = sigmas[m];
  dim3 grid(max_items, nmod > 0 ? nmod : 1);
  if (diag && Sigma) {
    if (in_dtype == 0)
      hipLaunchKernelGGL(sigma_diag_kernel<float>, grid, dim3(kSigThreads), 0, stream, zpart, S, T, r,
                         sorted_aid, n, items, n_items, static_cast<const float*>(Sigma),
                         static_cast<float*>(zp), sorted_seg, seg_rank, sorted_rank, split_dev, item_aid);
    else
      hipLaunchKernelGGL(sigma_diag_kernel<bf16_t>, grid, dim3(kSigThreads), 0, stream, zpart, S, T, r,
                         sorted_aid, n, items, n_items, static_cast<const bf16_t*>(Sigma),
                         static_cast<bf16_t*>(zp), sorted_seg, seg_rank, sorted_rank, split_dev, item_aid);
    return hipGetLastError();
  }
  if (r > 128) return hipErrorInvalidValue;
  // S: the most pieces the shrink may have split into (the device-chosen
  // split is at most S)
  const int zb = S <= 8 ? 8 : (S <= 16 || r > 64) ? 16 : 32;
#define CTS_SIGMA_LAUNCH(TI_, MAXR_, ZB_)                                                              \
  hipLaunchKernelGGL((sigma_kernel<TI_, MAXR_, ZB_>), grid, dim3(kSigThreads), 0, stream, zpart, S, T, r, \
                     sorted_aid, n, items, n_items, static_cast<const TI_*>(Sigma), static_cast<TI_*>(zp), \
                     sorted_seg, seg_rank, sorted_rank, ldz, split_dev, mods, nmod, item_aid)
  if (in_dtype == 0 && r <= 64) {
    if (zb == 8) CTS_SIGMA_LAUNCH(float, 64, 8);
    else if (zb == 16) CTS_SIGMA_LAUNCH(float, 64, 16);
    else CTS_SIGMA_LAUNCH(float, 64, 32);
  } else if (in_dtype == 0) {
    if (zb == 8) CTS_SIGMA_LAUNCH(float, 128, 8);
    else CTS_SIGMA_LAUNCH(float, 128, 16);
  } else if (r <= 64) {
    if (zb == 8) CTS_SIGMA_LAUNCH(bf16_t, 64, 8);
    else if (zb == 16) CTS_SIGMA_LAUNCH(bf16_t, 64, 16);
    else CTS_SIGMA_LAUNCH(bf16_t, 64, 32);
  } else {
    if (zb == 8) CTS_SIGMA_LAUNCH(bf16_t, 128, 8);
    else CTS_SIGMA_LAUNCH(bf16_t, 128, 16);
  }
#undef CTS_SIGMA_LAUNCH
  return hipGetLastError();
}

hipError_t launch_splitk_reduce(const float* part, int S, int N, int M, const int32_t* perm,
                                void* out, int64_t ldo, int out_dtype, hipStream_t stream,
                                const SplitkMods* mods) {
  const int V = out_dtype == 1 ? 8 : 4;
  SplitkMods md{};
  if (mods) {
    if (mods->n < 1 || mods->n > kMaxGemmModules || mods->col[0] != 0 || mods->col[mods->n] != M)
      return hipErrorInvalidValue;
    for (int q = 0; q < mods->n; ++q)
      if (mods->col[q + 1] <= mods->col[q] || mods->col[q] % 8) return hipErrorInvalidValue;
    md = *mods;
  }
  const int64_t chunks = static_cast<int64_t>(N) * (M / V);
  dim3 grid(static_cast<unsigned>((chunks + 255) / 256));
  if (out_dtype == 1)
    hipLaunchKernelGGL(splitk_reduce_kernel<1>, grid, dim3(256), 0, stream, part, S, N, M, perm, out, ldo, md);
  else
    hipLaunchKernelGGL(splitk_reduce_kernel<0>, grid, dim3(256), 0, stream, part, S, N, M, perm, out, ldo, md);
  return hipGetLastError();
}

}  // namespace cts
