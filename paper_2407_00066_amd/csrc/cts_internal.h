// Internal declarations shared by the HIP translation units of libcts.
// Nothing here is part of the public ABI (see include/cts.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cts {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// bfloat16 storage type: raw bits, converted explicitly.
struct bf16_t { uint16_t bits; };

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// float -> bfloat16, round to nearest, ties to even; NaN stays NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// ---------------------------------------------------------------- bucketing
constexpr int kSortThreads = 1024;
constexpr int kSortMaxT = 8192;

// Tokens of one adapter handled together by the core-product stage.
constexpr int kSigmaChunk = 16;

// Upper bound of the number of core-product items for T tokens and n adapters.
inline int max_sigma_items(int T, int n) {
  return (T + kSigmaChunk - 1) / kSigmaChunk + (n < T ? n : T);
}

// Token columns of one shrink tile: a run of one cluster inside a kSegTile
// window of sorted positions.
constexpr int kSegTile = 64;
// Batches of at most this many tokens are bucketed inside the shrink kernel
// (no separate sort launch).
constexpr int kFuseSortMaxT = 2 * 64;
inline int max_seg_tiles(int T, int nseg) {
  return (T + kSegTile - 1) / kSegTile + (nseg < T ? nseg : T);
}

// Sorts tokens by (cluster, adapter, token).  Writes perm[T] and offs[K+1];
// optionally sorted_seg[T] (cluster of each sorted position), sorted_aid[T]
// (adapter of each sorted position) and the core-product items: items[0..c)
// are the sorted positions where a run of one adapter starts or crosses a
// multiple of kSigmaChunk, items[c] = T, and n_items[0] = c; likewise the
// segment tiles ctiles/n_ctiles for runs of one cluster and kSegTile.
// Optionally item_aid[i] (the adapter of item i) and ctile_seg[i] (the
// cluster of tile i), so that the later stages need not look them up
// through the sorted positions.
// cluster_of may be null (every adapter its own cluster, K == n).
hipError_t launch_sort(const int32_t* adapter_id, const int32_t* cluster_of, int T, int n, int K,
                       int32_t* perm, int32_t* offs, int32_t* sorted_seg, int32_t* sorted_aid,
                       int32_t* items, int32_t* n_items, int32_t* ctiles, int32_t* n_ctiles,
                       hipStream_t stream, int32_t* item_aid = nullptr, int32_t* ctile_seg = nullptr);

// ----------------------------------------------------- segmented MFMA GEMM
// Modules one fused-GEMM launch can hold.
constexpr int kMaxGemmModules = 8;
// out[j][m] (m < M rows of the weight operand, j < N sorted token positions) =
//     sum_k A0[m][k] * B0[map(j)][k]                       (dense phase, K0)
//   + sum_k A1_{seg(j)}[m][k] * B1[map1(j)][k]             (segment phase, K1)
// where seg(j) = sorted_seg[j] and A1_s = A1 + s * seg_stride_a1.
// map(j) = perm[j]; map1(j) = perm[j] if b1_gather else j.
// Output: part != null -> fp32 partials part[ks][j][m] for split ks;
//         else out[perm[j]][m] (out_perm) or out[j][m], element type out_dtype.
// Every operand (and every segment of A1) must be smaller than 2^31 bytes:
// a0_bytes, b0_bytes, a1_seg_bytes and b1_bytes bound the buffer loads.
struct GemmParams {
  int M, N;
  const void* A0; int64_t lda0; const void* B0; int64_t ldb0; int K0;
  const void* A1; int64_t seg_stride_a1; int64_t lda1; const void* B1; int64_t ldb1; int K1;
  uint32_t a0_bytes, b0_bytes, a1_seg_bytes, b1_bytes;
  int b1_gather;
  const int32_t* perm;        // [N] sorted position -> token
  const int32_t* sorted_seg;  // [N] sorted position -> segment (cluster / adapter)
  // optional rank of each segment: the segment phase of segment s reads only
  // its first rank_of(s) elements of the reduction (rank_of: see seg_rank_of)
  const int32_t* seg_rank;
  // with seg_rank: the rank of each sorted position's segment, as seg_rank_of
  // gives it ([N], written by the core-product stage); the LDS-ring tiles
  // read their columns' ranks from here
  const int32_t* sorted_rank;
  int ksplit;
  float* part;
  void* out; int64_t ldo; int out_perm; int out_dtype;
  // optional explicit token tiles: tile t covers sorted positions
  // [tile_start[t], tile_start[t+1]) (at most the tile width); n_tiles[0]
  // tiles exist and the grid is sized for max_tiles (the rest exit at once)
  const int32_t* tile_start; const int32_t* n_tiles; int max_tiles;
  // optional segment of each explicit tile (else sorted_seg[tile_start[t]])
  const int32_t* tile_seg;
  // optional bucketing inside the kernel (token-tile mode, N <= kFuseSortMaxT;
  // fs_adapter != null): every workgroup sorts the N tokens by (cluster,
  // adapter, token) in LDS and takes its tile, perm and segments from there;
  // workgroup 0 also writes perm, sorted_seg, sorted_aid and the core-product
  // items exactly as launch_sort would (ids clamped the same way).  perm,
  // sorted_seg, tile_start and n_tiles are then unused.
  const int32_t* fs_adapter; const int32_t* fs_cluster;   // fs_cluster null: key = adapter
  int fs_n, fs_K, fs_bits_n;
  int32_t* fs_perm; int32_t* fs_seg; int32_t* fs_aid; int32_t* fs_items; int32_t* fs_nitems;
  int32_t* fs_item_aid;   // optional: the adapter of each core-product item
  // token-tile mode of the LDS-ring tiles: split_target > 0 makes the split
  // along k follow the tile count n known on the device: S = min(ksplit,
  // ceil(split_target / (ceil(M / BM) n))) pieces.  The grid is then sized
  // ceil(M / BM) max_tiles + split_target (enough for every n) and workgroup
  // 0 writes S to split_out[0] for the core-product stage.
  int split_target; int32_t* split_out;
  // m-tiles per group of the XCD-aware tile order (set by the launcher)
  int group_m;
  // Several modules in one launch (n_mod > 0; LDS-ring tiles, no token
  // tiles): module m owns the grid's row tiles [mod_rt[m], mod_rt[m+1]),
  // mod_rt[m+1] - mod_rt[m] = ceil(mod_M[m] / BM), and its M, A0, A1, B1,
  // out, ldo and operand sizes replace the fields above.  Its split partials
  // are the columns [mod_col[m], mod_col[m] + mod_M[m]) of rows part_ld floats
  // apart (0: M).
  int n_mod;
  int mod_rt[kMaxGemmModules + 1];
  int mod_M[kMaxGemmModules], mod_col[kMaxGemmModules];
  const void* mod_A0[kMaxGemmModules];
  const void* mod_A1[kMaxGemmModules];
  const void* mod_B1[kMaxGemmModules];
  void* mod_out[kMaxGemmModules];
  int64_t mod_ldo[kMaxGemmModules];
  uint32_t mod_a0_bytes[kMaxGemmModules], mod_a1_seg_bytes[kMaxGemmModules], mod_b1_bytes[kMaxGemmModules];
  int64_t part_ld;
};

// Tile shapes of the segmented GEMM (BM x BN x BK).  Large 256x256x64, Wide
// 256x128x64, Mid 128x128x64, Narrow 128x64x128, Decode 64x64x128 and Shrink
// 64x64x64 load their k-tiles straight into LDS; Small 64x64x64 stages them
// in registers; F32 is the fp32 path.  Explicit token tiles are taken by
// the 64-wide ones (Decode, Shrink, Small, F32).
enum class Tile { Large, Wide, Narrow, Decode, Shrink, Mid, Small, F32 };
hipError_t launch_seg_gemm(const GemmParams& p, int in_dtype, Tile tile, hipStream_t stream);
void tile_dims(Tile tile, int* BM, int* BN, int* BK);

// Rank of segment s from a caller's rank table: clamped to [0, kmax] and
// rounded down to a multiple of 8 (16-byte chunks never straddle it).
__device__ __forceinline__ int seg_rank_of(const int32_t* seg_rank, int s, int kmax) {
  int v = seg_rank[s];
  v = v < 0 ? 0 : (v > kmax ? kmax : v);
  return v & ~7;
}

// ------------------------------------------------------------- Sigma stage
// zp[j][c] = sum_{c'} Sigma_{aid(j)}[c][c'] * (sum_s zpart[s][j][c'])  (Sigma may be null:
// then zp = sum_s zpart).  With diag, Sigma is [n][r] (the diagonals) and
// zp[j][c] = Sigma_{aid(j)}[c] * (sum_s zpart[s][j][c]).  With seg_rank, the
// position's segment sorted_seg[j] has rank rk = seg_rank_of(seg_rank, .., r):
// only c, c' < rk are read (Sigma's leading block, z's first rk entries) and
// zp[j][c >= rk] = 0, and sorted_rank (if not null) receives rk for every
// position j.  Rounded to the input type.  One workgroup per item of the
// sort (max_items workgroups are launched; the extra ones exit).  ldz (0 =
// r): row stride of zpart's rows and of zp (full Sigma only), for the slice
// of one module in Z stacked over several modules.
hipError_t launch_sigma(const float* zpart, int S, int T, int r, const int32_t* sorted_aid, int n,
                        const int32_t* items, const int32_t* n_items, int max_items,
                        const void* Sigma, void* zp, int in_dtype, hipStream_t stream,
                        bool diag = false, const int32_t* sorted_seg = nullptr,
                        const int32_t* seg_rank = nullptr, int32_t* sorted_rank = nullptr,
                        int ldz = 0, const int32_t* split_dev = nullptr,
                        const void* const* sigmas = nullptr, int nmod = 0,
                        const int32_t* item_aid = nullptr);

// Records stage event i of the profiling aid (cts_set_stage_events) on s when
// it is on; a no-op otherwise.
hipError_t stage_mark(int i, hipStream_t s);

// Outputs of several modules' split partials reduced in one launch: the
// partials' columns [col[q], col[q+1]) (multiples of 8, col[0] = 0,
// col[n] = M) go to module q's output out[q] with rows ldo[q] apart.
struct SplitkMods {
  int n;
  int col[kMaxGemmModules + 1];
  void* out[kMaxGemmModules];
  int64_t ldo[kMaxGemmModules];
};

// y[perm[j]][m] = sum_s part[s][j][m], converted to out_dtype (with mods:
// into the module that owns column m, at its column m - col[q]).
hipError_t launch_splitk_reduce(const float* part, int S, int N, int M, const int32_t* perm,
                                void* out, int64_t ldo, int out_dtype, hipStream_t stream,
                                const SplitkMods* mods = nullptr);

}  // namespace cts
