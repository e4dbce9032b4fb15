// Token bucketing: a stable LSD radix sort of the token indices by the
// composite key (cluster << bits_n | adapter), done by one 1024-thread
// workgroup entirely in LDS.  (key, token) pairs move together and the token
// index is the implicit last key (stability), so the order is the unique
// (cluster, adapter, token) order.
//
// Grouping tokens by cluster is what turns the shared-basis products into
// contiguous GEMM segments: every LoRA of cluster k uses U_k, V_k (Sec. 3.2).
//
// Per 8-bit radix pass, each of the 16 waves owns a contiguous run of
// 64-token chunks.  Inside a chunk, a lane finds the lanes holding the same
// digit with ballots (deterministic, no atomics): first one ballot per
// distinct digit of the chunk (tokens of one request share an adapter, so a
// chunk usually holds one to three digits), then, if more than eight distinct
// digits remain, one ballot per digit bit.  The count walk records each
// token's offset inside its (wave, digit) group; an exclusive scan in
// (digit, wave) order turns the group sizes into bases; the scatter walk
// writes every pair to base + offset.
//
// After the last pass one blocked scan compacts, in sorted order, the starts
// of the Sigma-stage items (runs of one adapter cut at kSigmaChunk) and of
// the shrink's segment tiles (runs of one cluster cut at kSegTile).
#include "cts_internal.h"

namespace cts {
namespace {

constexpr int kRadixBits = 8;
constexpr int kRadix = 1 << kRadixBits;
// run path: at most this many runs (its all-pairs ranking costs R^2 / 1024
// compares per thread; past a few hundred runs the radix passes are cheaper)
constexpr int kMaxRuns = 256;

// One workgroup of NT threads sorts at most MAXT tokens: 1024 threads for up
// to kSortMaxT, 256 threads (cheaper barriers) for up to 2048.
template <int NT> struct SortCfg {
  static constexpr int W = NT / 64;                          // waves
  static constexpr int MAXT = NT == 1024 ? kSortMaxT : 2048;
  static constexpr int MC = MAXT / 64 / W;                   // chunks per wave, at most
  static constexpr int TPD = NT / kRadix;                    // scan threads per digit
  // cluster maps up to this size are staged in LDS (in the radix histogram)
  static constexpr int LDS_MAP = W * kRadix;
  static_assert(W * kRadix == 4 * NT, "scan: four counters per thread");
  static_assert(kMaxRuns <= NT, "run path: one run per thread");
};
constexpr int kSortSmallT = 2048;

// Lanes of this wave whose digit equals this lane's (only lanes in `valid`).
__device__ __forceinline__ uint64_t match_digit(uint32_t d, uint64_t valid, int lane) {
  uint64_t rem = valid, peers = 0;
  for (int it = 0; it < 8 && rem; ++it) {
    const int leader = __ffsll(static_cast<unsigned long long>(rem)) - 1;
    const uint32_t dl = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(d), leader));
    const uint64_t eq = __ballot(d == dl) & valid;
    if (d == dl) peers = eq;
    rem &= ~eq;
  }
  if (rem) {
    uint64_t m = valid;
#pragma unroll
    for (int b = 0; b < kRadixBits; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t bb = __ballot(bit);
      m &= bit ? bb : ~bb;
    }
    if ((rem >> lane) & 1ull) peers = m;
  }
  return peers;
}

// Exclusive scan of one value per thread over the workgroup; also returns the
// total.  Uses wsum[NW]; contains two barriers.
template <int NW>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* wsum, int lane, int wave,
                                                         uint32_t* total) {
  uint32_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t u = __shfl_up(x, off);
    if (lane >= off) x += u;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const uint32_t s = wsum[w];
    before += (w < wave) ? s : 0u;
    all += s;
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

template <int NT>
__global__ __launch_bounds__(NT) void sort_kernel(
    const int32_t* __restrict__ adapter_id, const int32_t* __restrict__ cluster_of, int T, int n,
    int K, int bits_n, int bits_k, int32_t* __restrict__ perm, int32_t* __restrict__ offs,
    int32_t* __restrict__ sorted_seg, int32_t* __restrict__ sorted_aid,
    int32_t* __restrict__ items, int32_t* __restrict__ n_items, int32_t* __restrict__ ctiles,
    int32_t* __restrict__ n_ctiles, int32_t* __restrict__ item_aid, int32_t* __restrict__ ctile_seg) {
  using C = SortCfg<NT>;
  constexpr int kWaves = C::W;
  __shared__ uint32_t kbuf[2][C::MAXT];
  __shared__ uint16_t vbuf[2][C::MAXT];
  __shared__ uint32_t hist[kWaves * kRadix];   // [wave][digit]
  __shared__ uint32_t wsum[kWaves];
  // run keys with their run index, (key << 8) | run, padded with 16 entries
  // that rank below nothing (all ones: a real entry is below 2^40)
  __shared__ __attribute__((aligned(16))) uint64_t run_key[kMaxRuns + 16];
  __shared__ uint32_t run_start[kMaxRuns + 1], run_order[kMaxRuns], run_off[kMaxRuns];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  // key layout: cluster << bits_n | adapter; without a cluster map (K == n)
  // the key is the adapter, which is also its cluster
  const int cshift = cluster_of ? bits_n : 0;

  // A cluster map of at most C::LDS_MAP entries is staged in LDS (its loads go
  // out with the adapter ids', one round trip instead of a dependent second
  // one); the run arrays' space is free until the run path below.
  const bool map_lds = cluster_of && n <= C::LDS_MAP;
  int32_t* const cmap = reinterpret_cast<int32_t*>(hist);
  if (map_lds)
    for (int i = tid; i < n; i += NT) cmap[i] = cluster_of[i];
  if (cluster_of && !map_lds) {
    for (int t = tid; t < T; t += NT) {
      int a = adapter_id[t];
      a = a < 0 ? 0 : (a >= n ? n - 1 : a);
      int c = cluster_of[a];
      c = c < 0 ? 0 : (c >= K ? K - 1 : c);
      kbuf[0][t] = static_cast<uint32_t>(a) | (static_cast<uint32_t>(c) << bits_n);
      vbuf[0][t] = static_cast<uint16_t>(t);
    }
  } else {
    for (int t = tid; t < T; t += NT) {
      int a = adapter_id[t];
      a = a < 0 ? 0 : (a >= n ? n - 1 : a);
      kbuf[0][t] = static_cast<uint32_t>(a);
      vbuf[0][t] = static_cast<uint16_t>(t);
    }
    if (map_lds) {
      __syncthreads();
      for (int t = tid; t < T; t += NT) {
        const uint32_t a = kbuf[0][t];
        int c = cmap[a];
        c = c < 0 ? 0 : (c >= K ? K - 1 : c);
        kbuf[0][t] = a | (static_cast<uint32_t>(c) << bits_n);
      }
    }
  }

  const int passes = (bits_n + bits_k + kRadixBits - 1) / kRadixBits;
  const int chunks = (T + 63) / 64;
  const int cpw = (chunks + kWaves - 1) / kWaves;
  const int seg_lo = wave * cpw * 64;
  const int seg_hi = min(T, seg_lo + cpw * 64);

  __syncthreads();
  int in = 0;

  // ---- run path -------------------------------------------------------------
  // Tokens of one request share an adapter, so the keys usually come in long
  // runs.  When there are at most kMaxRuns maximal runs of equal keys, the
  // runs themselves are ranked by (key, first token) with an all-pairs count,
  // their lengths are summed in rank order, and every token goes to its run's
  // offset plus its place in the run: the same stable order as the radix
  // passes, which run otherwise.
  {
    const int ipt = (T + NT - 1) / NT;
    const int j0 = tid * ipt, j1 = min(T, j0 + ipt);
    uint32_t cnt = 0;
    uint32_t kp = (j0 > 0 && j0 < T) ? kbuf[0][j0 - 1] : 0u;
    for (int j = j0; j < j1; ++j) {
      const uint32_t k = kbuf[0][j];
      cnt += (j == 0 || k != kp) ? 1u : 0u;
      kp = k;
    }
    uint32_t R;
    const uint32_t base = block_exclusive_scan<kWaves>(cnt, wsum, lane, wave, &R);
    if (R <= static_cast<uint32_t>(kMaxRuns)) {                  // uniform
      uint32_t r = base;
      kp = (j0 > 0 && j0 < T) ? kbuf[0][j0 - 1] : 0u;
      for (int j = j0; j < j1; ++j) {
        const uint32_t k = kbuf[0][j];
        if (j == 0 || k != kp) {
          run_start[r] = j;
          run_key[r] = (static_cast<uint64_t>(k) << 8) | r;
          ++r;
        }
        kp = k;
      }
      if (tid == 0) run_start[R] = T;
      if (tid < 16) run_key[R + tid] = ~0ull;
      __syncthreads();
      if (static_cast<uint32_t>(tid) < R) {
        // (key, first token) order is (key, run index) order, and the run
        // index makes every composite distinct: the rank is the number of
        // smaller composites.  16 per step, eight 16-byte reads in flight.
        const uint64_t kr = run_key[tid];
        uint32_t rank = 0;
        const ulong2* rk = reinterpret_cast<const ulong2*>(run_key);
        for (uint32_t q = 0; q < R; q += 16) {
          ulong2 v[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) v[i] = rk[q / 2 + i];
#pragma unroll
          for (int i = 0; i < 8; ++i) rank += (v[i].x < kr ? 1u : 0u) + (v[i].y < kr ? 1u : 0u);
        }
        run_order[rank] = tid;
      }
      __syncthreads();
      uint32_t len = 0;
      if (static_cast<uint32_t>(tid) < R) {
        const uint32_t rr = run_order[tid];
        len = run_start[rr + 1] - run_start[rr];
      }
      uint32_t tot;
      const uint32_t off = block_exclusive_scan<kWaves>(len, wsum, lane, wave, &tot);
      if (static_cast<uint32_t>(tid) < R) run_off[run_order[tid]] = off;
      __syncthreads();
      int rid = static_cast<int>(base) - 1;                      // run holding j0 - 1
      kp = (j0 > 0 && j0 < T) ? kbuf[0][j0 - 1] : 0u;
      for (int j = j0; j < j1; ++j) {
        const uint32_t k = kbuf[0][j];
        if (j == 0 || k != kp) ++rid;
        kp = k;
        const uint32_t pos = run_off[rid] + static_cast<uint32_t>(j) - run_start[rid];
        kbuf[1][pos] = k;
        vbuf[1][pos] = static_cast<uint16_t>(j);
      }
      __syncthreads();
      in = 1;
    }
  }

  const bool radix = (in == 0);
  for (int p = 0; radix && p < passes; ++p) {
    const int shift = p * kRadixBits;
#pragma unroll
    for (int i = 0; i < 4; ++i) hist[tid + i * NT] = 0;
    __syncthreads();

    // count walk: offset of each token inside its (wave, digit) group
    uint32_t kr[C::MC], dr[C::MC], pos[C::MC];
    uint16_t vr[C::MC];
#pragma unroll
    for (int c = 0; c < C::MC; ++c) {
      kr[c] = 0; dr[c] = 0; pos[c] = 0; vr[c] = 0;
      if (c < cpw) {
        const int idx = seg_lo + c * 64 + lane;
        const bool valid = idx < seg_hi;
        const uint32_t k = valid ? kbuf[in][idx] : 0u;
        const uint16_t v = valid ? vbuf[in][idx] : static_cast<uint16_t>(0);
        const uint32_t d = (k >> shift) & (kRadix - 1);
        const uint64_t peers = match_digit(d, __ballot(valid), lane);
        const uint32_t rank = static_cast<uint32_t>(__popcll(peers & lt_mask));
        // every lane of a digit group reads the count before the group's
        // lowest lane adds the group size (same wave: in order)
        const uint32_t old = valid ? hist[wave * kRadix + d] : 0u;
        if (valid && rank == 0) hist[wave * kRadix + d] = old + static_cast<uint32_t>(__popcll(peers));
        kr[c] = k; vr[c] = v; dr[c] = d; pos[c] = old + rank;
      }
    }
    __syncthreads();

    // exclusive scan in (digit, wave) order: thread owns digit tid/TPD and
    // four consecutive waves of it
    {
      const int d = tid / C::TPD, w0 = (tid % C::TPD) * 4;
      uint32_t x[4], s = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) { x[j] = hist[(w0 + j) * kRadix + d]; s += x[j]; }
      uint32_t total;
      uint32_t base = block_exclusive_scan<kWaves>(s, wsum, lane, wave, &total);
#pragma unroll
      for (int j = 0; j < 4; ++j) { hist[(w0 + j) * kRadix + d] = base; base += x[j]; }
    }
    __syncthreads();

    // scatter walk
#pragma unroll
    for (int c = 0; c < C::MC; ++c) {
      if (c < cpw) {
        const int idx = seg_lo + c * 64 + lane;
        if (idx < seg_hi) {
          const uint32_t dst = hist[wave * kRadix + dr[c]] + pos[c];
          kbuf[in ^ 1][dst] = kr[c];
          vbuf[in ^ 1][dst] = vr[c];
        }
      }
    }
    __syncthreads();
    in ^= 1;
  }

  // outputs (coalesced)
  const uint32_t amask = (1u << bits_n) - 1u;
  for (int j = tid; j < T; j += NT) {
    const uint32_t k = kbuf[in][j];
    perm[j] = static_cast<int32_t>(vbuf[in][j]);
    if (sorted_seg) sorted_seg[j] = static_cast<int32_t>(k >> cshift);
    if (sorted_aid) sorted_aid[j] = static_cast<int32_t>(k & amask);
  }

  // run starts, both lists in one blocked scan: thread tid owns positions
  // [tid*ipt, tid*ipt + ipt); counts packed as items | tiles << 16 (each
  // total is at most T + 1 <= 8193)
  if (items || ctiles) {
    const int ipt = (T + NT - 1) / NT;
    const int j0 = tid * ipt, j1 = min(T, j0 + ipt);
    uint32_t cnt = 0;
    uint32_t kp = (j0 > 0 && j0 < T) ? kbuf[in][j0 - 1] : 0u;
    for (int j = j0; j < j1; ++j) {
      const uint32_t k = kbuf[in][j];
      const bool si = (j % kSigmaChunk == 0) || k != kp;
      const bool sc = (j % kSegTile == 0) || (k >> cshift) != (kp >> cshift);
      cnt += (si ? 1u : 0u) + (sc ? 0x10000u : 0u);
      kp = k;
    }
    uint32_t total;
    uint32_t base = block_exclusive_scan<kWaves>(cnt, wsum, lane, wave, &total);
    uint32_t bi = base & 0xffffu, bc = base >> 16;
    kp = (j0 > 0 && j0 < T) ? kbuf[in][j0 - 1] : 0u;
    for (int j = j0; j < j1; ++j) {
      const uint32_t k = kbuf[in][j];
      const bool si = (j % kSigmaChunk == 0) || k != kp;
      const bool sc = (j % kSegTile == 0) || (k >> cshift) != (kp >> cshift);
      if (si && items) {
        items[bi] = j;
        if (item_aid) item_aid[bi] = static_cast<int32_t>(k & amask);
      }
      if (sc && ctiles) {
        ctiles[bc] = j;
        if (ctile_seg) ctile_seg[bc] = static_cast<int32_t>(k >> cshift);
      }
      bi += si ? 1u : 0u;
      bc += sc ? 1u : 0u;
      kp = k;
    }
    if (tid == 0) {
      if (items) { items[total & 0xffffu] = T; n_items[0] = static_cast<int32_t>(total & 0xffffu); }
      if (ctiles) { ctiles[total >> 16] = T; n_ctiles[0] = static_cast<int32_t>(total >> 16); }
    }
  }

  // cluster offsets: first sorted position whose cluster is >= k
  for (int k = tid; k <= K; k += NT) {
    int lo = 0, hi = T;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if ((kbuf[in][mid] >> cshift) < static_cast<uint32_t>(k)) lo = mid + 1; else hi = mid;
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
                       hipStream_t stream, int32_t* item_aid, int32_t* ctile_seg) {
  const int bits_n = ceil_log2(n);
  const int bits_k = cluster_of ? ceil_log2(K) : 0;  // key is the adapter alone when K == n
  if (T <= kSortSmallT)
    hipLaunchKernelGGL(sort_kernel<256>, dim3(1), dim3(256), 0, stream, adapter_id, cluster_of,
                       T, n, K, bits_n, bits_k, perm, offs, sorted_seg, sorted_aid, items, n_items,
                       ctiles, n_ctiles, item_aid, ctile_seg);
  else
    hipLaunchKernelGGL(sort_kernel<1024>, dim3(1), dim3(1024), 0, stream, adapter_id, cluster_of,
                       T, n, K, bits_n, bits_k, perm, offs, sorted_seg, sorted_aid, items, n_items,
                       ctiles, n_ctiles, item_aid, ctile_seg);
  return hipGetLastError();
}

}  // namespace cts
