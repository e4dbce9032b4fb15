// Token bucketing: a stable LSD radix sort of the token indices by the
// composite key (cluster << bits_n | adapter), done by one 1024-thread
// workgroup entirely in LDS.  The token index is the implicit last key
// (stability), so the order is the unique (cluster, adapter, token) order.
//
// Grouping tokens by cluster is what turns the shared-basis products into
// contiguous GEMM segments: every LoRA of cluster k uses U_k, V_k (Sec. 3.2).
//
// Per radix pass (digit of <= 8 bits), each of the 16 waves owns a contiguous
// run of tokens.  A wave ranks equal digits inside each 64-token chunk with
// one ballot per digit bit (lanes with identical digits get identical
// ballot-and masks), so ranking needs no atomics and is deterministic:
//   1) count walk:   per-wave digit histogram in LDS,
//   2) scan:         exclusive scan over (digit, wave) in digit-major order,
//   3) scatter walk: position = running base + rank among equal digits.
#include "cts_internal.h"

namespace cts {
namespace {

constexpr int kWaves = kSortThreads / 64;
constexpr int kRadix = 256;

__device__ __forceinline__ uint64_t match_digit(uint32_t d, bool valid, int dbits) {
  uint64_t m = __ballot(valid);
  for (int b = 0; b < dbits; ++b) {
    const bool bit = (d >> b) & 1u;
    const uint64_t bb = __ballot(bit);
    m &= bit ? bb : ~bb;
  }
  return m;
}

__global__ __launch_bounds__(kSortThreads) void sort_kernel(
    const int32_t* __restrict__ adapter_id, const int32_t* __restrict__ cluster_of, int T, int n,
    int K, int bits_n, int bits_k, int32_t* __restrict__ perm, int32_t* __restrict__ offs,
    int32_t* __restrict__ sorted_seg, int32_t* __restrict__ sorted_aid,
    int32_t* __restrict__ items, int32_t* __restrict__ n_items, int32_t* __restrict__ ctiles,
    int32_t* __restrict__ n_ctiles) {
  __shared__ uint32_t key[kSortMaxT];
  __shared__ uint32_t buf0[kSortMaxT];
  __shared__ uint32_t buf1[kSortMaxT];
  __shared__ uint32_t hist[kWaves * kRadix];
  __shared__ uint32_t tot[kRadix];
  __shared__ uint32_t incl[kRadix];
  __shared__ uint32_t wsum[4];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  for (int t = tid; t < T; t += kSortThreads) {
    int a = adapter_id[t];
    a = a < 0 ? 0 : (a >= n ? n - 1 : a);
    int c = cluster_of ? cluster_of[a] : a;
    c = c < 0 ? 0 : (c >= K ? K - 1 : c);
    key[t] = (static_cast<uint32_t>(c) << bits_n) | static_cast<uint32_t>(a);
    buf0[t] = static_cast<uint32_t>(t);
  }
  __syncthreads();

  const int total_bits = bits_n + bits_k;
  const int passes = (total_bits + 7) / 8;
  const int dbits = passes ? (total_bits + passes - 1) / passes : 0;
  const uint32_t dmask = (1u << dbits) - 1u;
  const int R = 1 << dbits;
  const int chunks = (T + 63) / 64;
  const int cpw = (chunks + kWaves - 1) / kWaves;
  const int seg_lo = wave * cpw * 64;
  const int seg_hi = min(T, seg_lo + cpw * 64);
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));

  uint32_t* in = buf0;
  uint32_t* out = buf1;
  for (int p = 0; p < passes; ++p) {
    const int shift = p * dbits;
    for (int i = tid; i < kWaves * kRadix; i += kSortThreads) hist[i] = 0;
    __syncthreads();

    // 1) count walk (wave-private histogram rows; leaders have distinct digits)
    for (int b = seg_lo; b < seg_hi; b += 64) {
      const int idx = b + lane;
      const bool valid = idx < seg_hi;
      const uint32_t item = valid ? in[idx] : 0u;
      const uint32_t d = valid ? ((key[item] >> shift) & dmask) : 0u;
      const uint64_t peers = match_digit(d, valid, dbits);
      if (valid && lane == __ffsll(static_cast<unsigned long long>(peers)) - 1)
        hist[wave * kRadix + d] += static_cast<uint32_t>(__popcll(peers));
    }
    __syncthreads();

    // 2) exclusive scan in (digit, wave) order
    if (tid < R) {
      uint32_t s = 0;
      for (int w = 0; w < kWaves; ++w) s += hist[w * kRadix + tid];
      tot[tid] = s;
    }
    __syncthreads();
    if (tid < kRadix) {
      uint32_t v = (tid < R) ? tot[tid] : 0u;
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t u = __shfl_up(v, off);
        if (lane >= off) v += u;
      }
      incl[tid] = v;
      if (lane == 63) wsum[wave] = v;
    }
    __syncthreads();
    if (tid < R) {
      uint32_t run = incl[tid] - tot[tid];
      for (int w = 0; w < wave; ++w) run += wsum[w];
      for (int w = 0; w < kWaves; ++w) {
        const uint32_t h = hist[w * kRadix + tid];
        hist[w * kRadix + tid] = run;
        run += h;
      }
    }
    __syncthreads();

    // 3) scatter walk
    for (int b = seg_lo; b < seg_hi; b += 64) {
      const int idx = b + lane;
      const bool valid = idx < seg_hi;
      const uint32_t item = valid ? in[idx] : 0u;
      const uint32_t d = valid ? ((key[item] >> shift) & dmask) : 0u;
      const uint64_t peers = match_digit(d, valid, dbits);
      if (valid) {
        const uint32_t base = hist[wave * kRadix + d];
        out[base + static_cast<uint32_t>(__popcll(peers & lt_mask))] = item;
        if (lane == __ffsll(static_cast<unsigned long long>(peers)) - 1)
          hist[wave * kRadix + d] = base + static_cast<uint32_t>(__popcll(peers));
      }
    }
    __syncthreads();
    uint32_t* tmp = in; in = out; out = tmp;
  }

  // outputs; out[] is free scratch now: sorted cluster values for the offsets
  const uint32_t amask = (1u << bits_n) - 1u;
  for (int j = tid; j < T; j += kSortThreads) {
    const uint32_t t = in[j];
    const uint32_t k = key[t];
    perm[j] = static_cast<int32_t>(t);
    out[j] = k >> bits_n;
    if (sorted_seg) sorted_seg[j] = static_cast<int32_t>(k >> bits_n);
    if (sorted_aid) sorted_aid[j] = static_cast<int32_t>(k & amask);
  }
  __syncthreads();

  // Compaction of run starts, in order (ballot + wave prefix): a sorted
  // position starts an entry when it starts a kChunk-aligned window or its
  // key (masked by kmask) differs from the previous position's.
  auto compact_starts = [&](uint32_t kmask, int chunk, int32_t* outp, int32_t* outn) {
    uint32_t done = 0;
    for (int base = 0; base < T; base += kSortThreads) {
      const int j = base + tid;
      bool st = false;
      if (j < T) st = (j % chunk == 0) || ((key[in[j]] & kmask) != (key[in[j - 1]] & kmask));
      const uint64_t bal = __ballot(st);
      if (lane == 0) hist[wave] = static_cast<uint32_t>(__popcll(bal));
      __syncthreads();
      uint32_t before = 0, total = 0;
      for (int w = 0; w < kWaves; ++w) {
        const uint32_t c = hist[w];
        before += (w < wave) ? c : 0u;
        total += c;
      }
      if (st) outp[done + before + static_cast<uint32_t>(__popcll(bal & lt_mask))] = j;
      done += total;
      __syncthreads();
    }
    if (tid == 0) {
      outp[done] = T;
      outn[0] = static_cast<int32_t>(done);
    }
  };
  // core-product items: runs of one adapter, cut at kSigmaChunk windows
  if (items) compact_starts(amask, kSigmaChunk, items, n_items);
  // segment tiles: runs of one cluster, cut at kSegTile windows
  if (ctiles) compact_starts(~amask, kSegTile, ctiles, n_ctiles);
  for (int k = tid; k <= K; k += kSortThreads) {
    int lo = 0, hi = T;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (out[mid] < static_cast<uint32_t>(k)) lo = mid + 1; else hi = mid;
    }
    offs[k] = lo;
  }
}

int ceil_log2(int v) {
  int b = 0;
  while ((1 << b) < v) ++b;
  return b;
}

}  // namespace

hipError_t launch_sort(const int32_t* adapter_id, const int32_t* cluster_of, int T, int n, int K,
                       int32_t* perm, int32_t* offs, int32_t* sorted_seg, int32_t* sorted_aid,
                       int32_t* items, int32_t* n_items, int32_t* ctiles, int32_t* n_ctiles,
                       hipStream_t stream) {
  const int bits_n = ceil_log2(n);
  const int bits_k = cluster_of ? ceil_log2(K) : 0;  // key is the adapter alone when K == n
  hipLaunchKernelGGL(sort_kernel, dim3(1), dim3(kSortThreads), 0, stream, adapter_id, cluster_of,
                     T, n, K, bits_n, bits_k, perm, offs, sorted_seg, sorted_aid, items, n_items,
                     ctiles, n_ctiles);
  return hipGetLastError();
}

}  // namespace cts
