// C entry points of libcts: argument validation (pure host code, no HIP call
// before every check has passed), workspace planning and the launch
// sequence of the layer:
//   1. bucketing          tokens sorted by (cluster, adapter)         sort.hip
//   2. shrink             Z  = V_k^T X per cluster segment (fp32)     gemm.hip
//   3. core               Z' = Sigma_i Z per token                     sigma.hip
//   4. fused base + up    Y  = W X + U_k Z' scattered to token order   gemm.hip
//   (5. split-K reduce    only when the fused GEMM is split along k)   sigma.hip
// The uncompressed comparison path runs the same stages with one segment per
// adapter, V_k^T -> A_i, U_k -> B_i and no core product.
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <vector>

#include "cts.h"
#include "cts_internal.h"

// Scratch memory of cts_apply_noalloc: one static array per device (each
// GPU the library runs on holds its own copy until the process ends); it
// stands in for the workspace argument of cts_apply.
__device__ __align__(256) unsigned char scratch[CTS_NOALLOC_SCRATCH_BYTES];

namespace {

using cts::Tile;

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct Plan {
  int elt, out_elt;
  int rank, nseg;
  Tile main_tile, shrink_tile;
  int main_split, shrink_split;
  int max_items, max_ctiles;
  size_t off_perm, off_seg, off_aid, off_srank, off_offs, off_items, off_nitems, off_ctiles, off_nctiles,
      off_iaid, off_cseg, off_ssplit, off_zpart, off_zp, off_ypart, total;
};

constexpr uint64_t kMaxOperandBytes = 0x7fffffffull;   // buffer-load offsets are 31-bit

int ceil_div(int64_t a, int64_t b) { return static_cast<int>((a + b - 1) / b); }

// The shrink's split along d_in for `rank` rank rows.  When the tiles come
// from the separate sort (bf16, T > kFuseSortMaxT) the split follows the
// tile count on the device: 512 workgroups, at least 8 k-tiles each, and
// this returns the most it could use (the split for the fewest tiles,
// ceil(T / 64)).  Otherwise (fp32, or the bucketing inside the shrink) it is
// fixed: 256 (bf16) or 512 (fp32) workgroups over an estimate of the tiles
// (token tiles plus half of the possible segment starts), at least 2
// k-tiles each.
constexpr int kShrinkAdaptiveTarget = 512;

bool shrink_adaptive(int T, Tile t) { return t == Tile::Shrink && T > cts::kFuseSortMaxT; }

int shrink_split_of(int T, int rank, int nseg, int d_in, Tile t) {
  int BM, BN, BK;
  cts::tile_dims(t, &BM, &BN, &BK);
  const bool adaptive = shrink_adaptive(T, t);
  const int expect = ceil_div(std::max(T, 1), BN) + (adaptive ? 0 : std::min(nseg, std::max(T, 1)) / 2);
  const int tiles = ceil_div(rank, BM) * std::max(expect, 1);
  const int nk = ceil_div(d_in, BK);
  const int target = adaptive ? kShrinkAdaptiveTarget : (t == Tile::F32 ? 512 : 256);
  const int kmin = adaptive ? 8 : 2;
  return std::max(1, std::min(std::min(ceil_div(target, tiles), std::max(1, nk / kmin)), 64));
}

// Batches of more than kSortMaxT tokens (the one-workgroup bucketing's
// limit) run as consecutive pieces of near-equal size, each at most
// kSortMaxT tokens and a complete layer call of its own: y_t depends on
// token t alone (its x_t and its adapter), so the pieces' rows are the
// batch's rows.  The first `rem` pieces hold q + 1 tokens, the rest q.
struct Pieces { int n, q, rem; };

Pieces pieces_of(int T) {
  Pieces pc;
  pc.n = T <= cts::kSortMaxT ? 1 : ceil_div(T, cts::kSortMaxT);
  pc.q = T / pc.n;
  pc.rem = T % pc.n;
  return pc;
}

// Runs fn(piece problem, first token) over the pieces of p->T in token order;
// stops at the first status that is not CTS_OK.
template <typename F> int for_pieces(const cts_problem* p, F&& fn) {
  const Pieces pc = pieces_of(p->T);
  cts_problem q = *p;
  int t0 = 0;
  for (int i = 0; i < pc.n; ++i) {
    q.T = pc.q + (i < pc.rem ? 1 : 0);
    const int rc = fn(q, static_cast<size_t>(t0));
    if (rc != CTS_OK) return rc;
    t0 += q.T;
  }
  return CTS_OK;
}

// Validates the sizes of `p` (T <= kSortMaxT) for the compressed
// (compressed=true) or the uncompressed path and fills the launch plan.
// Pure host arithmetic.
int plan_piece(const cts_problem* p, bool compressed, Plan* pl) {
  if (!p) return CTS_ERR_INVALID_ARG;
  if (p->T < 0 || p->d_in < 1 || p->d_out < 1 || p->n_adapters < 1) return CTS_ERR_INVALID_ARG;
  if (compressed && (p->r < 1 || p->n_clusters < 1)) return CTS_ERR_INVALID_ARG;
  if (!compressed && p->r_lora < 1) return CTS_ERR_INVALID_ARG;
  if (p->dtype != CTS_F32 && p->dtype != CTS_BF16) return CTS_ERR_UNSUPPORTED;
  if (p->out_dtype != CTS_F32 && p->out_dtype != CTS_BF16) return CTS_ERR_UNSUPPORTED;
  if (p->dtype == CTS_F32 && p->out_dtype != CTS_F32) return CTS_ERR_UNSUPPORTED;
  if (p->T > cts::kSortMaxT) return CTS_ERR_UNSUPPORTED;   // a piece
  if (p->d_in % 8 || p->d_out % 8) return CTS_ERR_UNSUPPORTED;
  if (p->n_adapters > 65536) return CTS_ERR_UNSUPPORTED;
  pl->elt = p->dtype == CTS_BF16 ? 2 : 4;
  pl->out_elt = p->out_dtype == CTS_BF16 ? 2 : 4;
  if (compressed) {
    if (p->n_clusters > 65536) return CTS_ERR_UNSUPPORTED;
    if (p->r % 8 || p->r > 128) return CTS_ERR_UNSUPPORTED;
    pl->rank = p->r;
    pl->nseg = p->n_clusters;
  } else {
    const int q = 16 / pl->elt;
    if (p->r_lora % q || p->r_lora > 128) return CTS_ERR_UNSUPPORTED;
    pl->rank = p->r_lora;
    pl->nseg = p->n_adapters;
  }

  const int T = p->T;
  int BM, BN, BK;
  // fused GEMM tile and k split.  Prefill-sized batches: 256x256 tiles.
  // Smaller batches are bound by the weight stream and by how often each
  // compute unit re-reads its operands from L2: 256x128 tiles when they alone
  // give most compute units work or the reduction is long, else 128x128
  // tiles while they still give at least 128 tiles, else 128x64 tiles, and
  // 64x64 for decode batches; each split along k up to one round of 256
  // workgroups (partials summed afterwards).
  auto tiles_of = [&](Tile t) {
    int bm, bn, bk;
    cts::tile_dims(t, &bm, &bn, &bk);
    return ceil_div(p->d_out, bm) * ceil_div(std::max(T, 1), bn);
  };
  int max_split = 1;
  if (p->dtype == CTS_F32) {
    pl->main_tile = Tile::F32;
  } else if (T >= 2048) {
    pl->main_tile = Tile::Large;
  } else if (T > 64 && (tiles_of(Tile::Wide) >= 192 || p->d_in >= 8192)) {
    pl->main_tile = Tile::Wide;
    max_split = 8;
  } else if (T > 64 && tiles_of(Tile::Mid) >= 128) {
    pl->main_tile = Tile::Mid;
    max_split = 4;
  } else if (T > 64) {
    pl->main_tile = Tile::Narrow;
    max_split = 4;
  } else {
    pl->main_tile = Tile::Decode;
    max_split = 4;
  }
  cts::tile_dims(pl->main_tile, &BM, &BN, &BK);
  {
    const int tiles = tiles_of(pl->main_tile);
    const int nk = ceil_div(p->d_in, BK);
    // no more workgroups than one round over the compute units
    const int s = std::min(std::min(std::max(1, 256 / tiles), max_split), std::max(1, nk / 4));
    pl->main_split = std::max(1, s);
  }
  // shrink: one workgroup per (cluster segment tile of <= kSegTile tokens,
  // 64 rank rows), split along d_in so that about 256 (bf16) or 512 (fp32)
  // workgroups run; the Sigma stage sums the split partials.  The bf16
  // shrink takes its split from the tile count on the device (at most
  // shrink_split, the split for the fewest tiles T can make); the fp32 one
  // from an estimate of the tile count.
  pl->shrink_tile = (p->dtype == CTS_F32) ? Tile::F32 : Tile::Shrink;
  cts::tile_dims(pl->shrink_tile, &BM, &BN, &BK);
  pl->max_ctiles = cts::max_seg_tiles(T, pl->nseg);
  pl->shrink_split = shrink_split_of(T, pl->rank, pl->nseg, p->d_in, pl->shrink_tile);
  pl->max_items = cts::max_sigma_items(T, p->n_adapters);

  // every operand a kernel reads through a buffer resource must stay below 2^31 bytes
  const uint64_t e = pl->elt;
  const uint64_t seg_v = static_cast<uint64_t>(pl->rank) * p->d_in * e;
  const uint64_t seg_u = static_cast<uint64_t>(p->d_out) * pl->rank * e;
  if (static_cast<uint64_t>(T) * p->d_in * e > kMaxOperandBytes ||
      static_cast<uint64_t>(p->d_out) * p->d_in * e > kMaxOperandBytes ||
      seg_v > kMaxOperandBytes || seg_u > kMaxOperandBytes)
    return CTS_ERR_UNSUPPORTED;

  size_t off = 0;
  pl->off_perm = off;  off = align_up(off + 4ull * T);
  pl->off_seg = off;   off = align_up(off + 4ull * T);
  pl->off_aid = off;   off = align_up(off + 4ull * T);
  pl->off_srank = off; off = align_up(off + 4ull * T);
  pl->off_offs = off;  off = align_up(off + 4ull * (pl->nseg + 1));
  pl->off_items = off; off = align_up(off + 4ull * (pl->max_items + 1));
  pl->off_nitems = off; off = align_up(off + 4);
  pl->off_ctiles = off; off = align_up(off + 4ull * (pl->max_ctiles + 1));
  pl->off_nctiles = off; off = align_up(off + 4);
  pl->off_iaid = off;  off = align_up(off + 4ull * (pl->max_items + 1));
  pl->off_cseg = off;  off = align_up(off + 4ull * (pl->max_ctiles + 1));
  pl->off_ssplit = off; off = align_up(off + 4);
  pl->off_zpart = off; off = align_up(off + 4ull * pl->shrink_split * T * pl->rank);
  pl->off_zp = off;    off = align_up(off + static_cast<size_t>(pl->elt) * T * pl->rank);
  pl->off_ypart = off;
  if (pl->main_split > 1) off = align_up(off + 4ull * pl->main_split * T * p->d_out);
  pl->total = off;
  return CTS_OK;
}

// The plan of p: for a batch of pieces, the plan of its largest piece, with
// a workspace that also fits the smaller piece size.
int make_plan(const cts_problem* p, bool compressed, Plan* pl) {
  if (!p) return CTS_ERR_INVALID_ARG;
  if (p->T <= cts::kSortMaxT) return plan_piece(p, compressed, pl);
  const Pieces pc = pieces_of(p->T);
  cts_problem q = *p;
  q.T = pc.q + (pc.rem ? 1 : 0);
  int rc = plan_piece(&q, compressed, pl);
  if (rc != CTS_OK || !pc.rem) return rc;
  Plan small;
  q.T = pc.q;
  rc = plan_piece(&q, compressed, &small);
  if (rc != CTS_OK) return rc;
  pl->total = std::max(pl->total, small.total);
  return CTS_OK;
}

// Stage-boundary events of the profiling aid (null when off).
hipEvent_t g_stage_events[CTS_N_STAGE_EVENTS] = {};
bool g_stage_on = false;

hipError_t mark(int i, hipStream_t s) {
  return (g_stage_on && g_stage_events[i]) ? hipEventRecord(g_stage_events[i], s) : hipSuccess;
}

// The bucketing cts_sort_by_cluster leaves in its workspace (perm is its own
// argument): each sorted position's cluster and adapter, the core-product
// items and their count, the shrink tiles and their count.
struct BucketLayout { size_t seg, aid, items, nitems, ctiles, nctiles, iaid, cseg, total; };

bool bucket_layout(int T, int n, int K, BucketLayout* L) {
  if (T < 0 || n < 1 || K < 1 || T > cts::kSortMaxT || n > 65536 || K > 65536) return false;
  size_t off = 0;
  L->seg = off;     off = align_up(off + 4ull * T);
  L->aid = off;     off = align_up(off + 4ull * T);
  L->items = off;   off = align_up(off + 4ull * (cts::max_sigma_items(T, n) + 1));
  L->nitems = off;  off = align_up(off + 4);
  L->ctiles = off;  off = align_up(off + 4ull * (cts::max_seg_tiles(T, K) + 1));
  L->nctiles = off; off = align_up(off + 4);
  L->iaid = off;    off = align_up(off + 4ull * (cts::max_sigma_items(T, n) + 1));
  L->cseg = off;    off = align_up(off + 4ull * (cts::max_seg_tiles(T, K) + 1));
  L->total = off;
  return true;
}

struct Range { const void* p; size_t bytes; };

// Every float array is read or written in 16-byte vectors: its address must be
// a multiple of 16 (ids: of 4).
bool misaligned(const void* ptr, uintptr_t a) {
  return (reinterpret_cast<uintptr_t>(ptr) & (a - 1)) != 0;
}

bool overlap(Range a, Range b) {
  if (!a.p || !b.p || !a.bytes || !b.bytes) return false;
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a.p), b0 = reinterpret_cast<uintptr_t>(b.p);
  return a0 < b0 + b.bytes && b0 < a0 + a.bytes;
}

// y must not overlap any input or the workspace; the workspace must not
// overlap any input.
bool any_overlap(Range y, Range ws, const Range* in, int n_in) {
  if (overlap(y, ws)) return true;
  for (int i = 0; i < n_in; ++i)
    if (overlap(y, in[i]) || overlap(ws, in[i])) return true;
  return false;
}

int run_layer(const cts_problem* p, const Plan& pl, bool compressed, const void* x,
              const int32_t* adapter_id, const int32_t* cluster_of, const void* W,
              const void* Ubasis, const void* Vbasis, const void* Sigma, void* y, void* workspace,
              hipStream_t stream, bool sigma_diag = false, const int32_t* seg_rank = nullptr) {
  char* ws = static_cast<char*>(workspace);
  int32_t* perm = reinterpret_cast<int32_t*>(ws + pl.off_perm);
  int32_t* sseg = reinterpret_cast<int32_t*>(ws + pl.off_seg);
  int32_t* said = reinterpret_cast<int32_t*>(ws + pl.off_aid);
  int32_t* srank = reinterpret_cast<int32_t*>(ws + pl.off_srank);
  int32_t* offs = reinterpret_cast<int32_t*>(ws + pl.off_offs);
  int32_t* items = reinterpret_cast<int32_t*>(ws + pl.off_items);
  int32_t* n_items = reinterpret_cast<int32_t*>(ws + pl.off_nitems);
  int32_t* ctiles = reinterpret_cast<int32_t*>(ws + pl.off_ctiles);
  int32_t* n_ctiles = reinterpret_cast<int32_t*>(ws + pl.off_nctiles);
  int32_t* iaid = reinterpret_cast<int32_t*>(ws + pl.off_iaid);
  int32_t* cseg = reinterpret_cast<int32_t*>(ws + pl.off_cseg);
  float* zpart = reinterpret_cast<float*>(ws + pl.off_zpart);
  void* zp = ws + pl.off_zp;
  float* ypart = reinterpret_cast<float*>(ws + pl.off_ypart);
  const int T = p->T, rank = pl.rank;

  hipError_t e = mark(0, stream);
  if (e != hipSuccess) return CTS_ERR_HIP;
  // small bf16 batches are bucketed inside the shrink kernel (one launch less)
  const bool fuse_sort = T <= cts::kFuseSortMaxT && pl.shrink_tile == Tile::Shrink;
  if (!fuse_sort) {
    e = cts::launch_sort(adapter_id, compressed ? cluster_of : nullptr, T, p->n_adapters,
                         pl.nseg, perm, offs, sseg, said, items, n_items, ctiles, n_ctiles, stream, iaid, cseg);
    if (e != hipSuccess) return CTS_ERR_HIP;
  }
  if (mark(1, stream) != hipSuccess) return CTS_ERR_HIP;

  cts::GemmParams g{};
  g.M = rank; g.N = T;
  g.A0 = nullptr; g.K0 = 0;
  g.A1 = Vbasis; g.seg_stride_a1 = static_cast<int64_t>(rank) * p->d_in; g.lda1 = p->d_in;
  g.B1 = x; g.ldb1 = p->d_in; g.K1 = p->d_in; g.b1_gather = 1;
  g.a0_bytes = 0; g.b0_bytes = 0;
  g.a1_seg_bytes = static_cast<uint32_t>(static_cast<uint64_t>(rank) * p->d_in * pl.elt);
  g.b1_bytes = static_cast<uint32_t>(static_cast<uint64_t>(T) * p->d_in * pl.elt);
  g.perm = perm; g.sorted_seg = sseg;
  g.ksplit = pl.shrink_split; g.part = zpart;
  g.tile_start = ctiles; g.n_tiles = n_ctiles; g.max_tiles = pl.max_ctiles; g.tile_seg = cseg;
  int32_t* ssplit = nullptr;
  if (shrink_adaptive(T, pl.shrink_tile)) {
    ssplit = reinterpret_cast<int32_t*>(ws + pl.off_ssplit);
    g.split_target = kShrinkAdaptiveTarget; g.split_out = ssplit;
  }
  if (fuse_sort) {
    g.tile_start = nullptr; g.n_tiles = nullptr; g.tile_seg = nullptr;
    g.fs_item_aid = iaid;
    g.fs_adapter = adapter_id; g.fs_cluster = compressed ? cluster_of : nullptr;
    g.fs_n = p->n_adapters; g.fs_K = pl.nseg;
    int bits_n = 0;
    while ((1 << bits_n) < p->n_adapters) ++bits_n;
    g.fs_bits_n = bits_n;
    g.fs_perm = perm; g.fs_seg = sseg; g.fs_aid = said; g.fs_items = items; g.fs_nitems = n_items;
  }
  e = cts::launch_seg_gemm(g, p->dtype, pl.shrink_tile, stream);
  if (e != hipSuccess || mark(2, stream) != hipSuccess) return CTS_ERR_HIP;

  e = cts::launch_sigma(zpart, pl.shrink_split, T, rank, said, p->n_adapters, items, n_items,
                        pl.max_items, compressed ? Sigma : nullptr, zp, p->dtype, stream, sigma_diag,
                        sseg, seg_rank, seg_rank ? srank : nullptr, 0, ssplit, nullptr, 0, iaid);
  if (e != hipSuccess || mark(3, stream) != hipSuccess) return CTS_ERR_HIP;

  cts::GemmParams f{};
  f.M = p->d_out; f.N = T;
  f.A0 = W; f.lda0 = p->d_in; f.B0 = x; f.ldb0 = p->d_in; f.K0 = p->d_in;
  f.A1 = Ubasis; f.seg_stride_a1 = static_cast<int64_t>(p->d_out) * rank; f.lda1 = rank;
  f.B1 = zp; f.ldb1 = rank; f.K1 = rank; f.b1_gather = 0;
  f.a0_bytes = static_cast<uint32_t>(static_cast<uint64_t>(p->d_out) * p->d_in * pl.elt);
  f.b0_bytes = static_cast<uint32_t>(static_cast<uint64_t>(T) * p->d_in * pl.elt);
  f.a1_seg_bytes = static_cast<uint32_t>(static_cast<uint64_t>(p->d_out) * rank * pl.elt);
  f.b1_bytes = static_cast<uint32_t>(static_cast<uint64_t>(T) * rank * pl.elt);
  f.perm = perm; f.sorted_seg = sseg; f.seg_rank = seg_rank;
  f.sorted_rank = seg_rank ? srank : nullptr;
  f.ksplit = pl.main_split;
  f.part = pl.main_split > 1 ? ypart : nullptr;
  f.out = y; f.ldo = p->d_out; f.out_perm = 1; f.out_dtype = p->out_dtype;
  e = cts::launch_seg_gemm(f, p->dtype, pl.main_tile, stream);
  if (e != hipSuccess || mark(4, stream) != hipSuccess) return CTS_ERR_HIP;

  if (pl.main_split > 1) {
    e = cts::launch_splitk_reduce(ypart, pl.main_split, T, p->d_out, perm, y, p->d_out,
                                  p->out_dtype, stream);
    if (e != hipSuccess) return CTS_ERR_HIP;
  }
  return mark(5, stream) == hipSuccess ? CTS_OK : CTS_ERR_HIP;
}

}  // namespace

namespace cts {
hipError_t stage_mark(int i, hipStream_t s) { return mark(i, s); }
}  // namespace cts


extern "C" {

const char* cts_status_string(int status) {
  switch (status) {
    case CTS_OK: return "CTS_OK";
    case CTS_ERR_INVALID_ARG: return "CTS_ERR_INVALID_ARG: invalid argument";
    case CTS_ERR_UNSUPPORTED: return "CTS_ERR_UNSUPPORTED: outside the supported limits";
    case CTS_ERR_WORKSPACE: return "CTS_ERR_WORKSPACE: workspace too small";
    case CTS_ERR_HIP: return "CTS_ERR_HIP: HIP runtime or launch failure";
    case CTS_ERR_BAD_IDS: return "CTS_ERR_BAD_IDS: adapter or cluster id out of range";
    default: return "CTS_ERR_UNKNOWN";
  }
}

size_t cts_workspace_size(const cts_problem* p) {
  Plan pl;
  return make_plan(p, true, &pl) == CTS_OK ? pl.total : 0;
}

size_t cts_workspace_size_uncompressed(const cts_problem* p) {
  Plan pl;
  return make_plan(p, false, &pl) == CTS_OK ? pl.total : 0;
}

int cts_workspace_bucketing(const cts_problem* p, int32_t compressed, size_t* offsets) {
  if (!offsets) return CTS_ERR_INVALID_ARG;
  Plan pl;
  const int rc = make_plan(p, compressed != 0, &pl);
  if (rc != CTS_OK) return rc;
  if (p->T > cts::kSortMaxT) return CTS_ERR_UNSUPPORTED;   // each piece buckets on its own
  offsets[0] = pl.off_perm;
  offsets[1] = pl.off_seg;
  offsets[2] = pl.off_aid;
  offsets[3] = pl.off_items;
  offsets[4] = pl.off_nitems;
  return CTS_OK;
}

size_t cts_bucketing_size(int32_t T, int32_t n, int32_t K) {
  BucketLayout L;
  return bucket_layout(T, n, K, &L) ? L.total : 0;
}

int cts_sort_by_cluster(const int32_t* adapter_id, const int32_t* cluster_of, int32_t T, int32_t n,
                        int32_t K, int32_t* perm, int32_t* cluster_offsets, void* workspace,
                        size_t workspace_bytes, void* stream) {
  if (T < 0 || n < 1 || K < 1 || !cluster_offsets) return CTS_ERR_INVALID_ARG;
  if (!cluster_of && K != n) return CTS_ERR_INVALID_ARG;
  if (T > 0 && (!adapter_id || !perm)) return CTS_ERR_INVALID_ARG;
  if (misaligned(adapter_id, 4) || misaligned(cluster_of, 4) || misaligned(perm, 4) ||
      misaligned(cluster_offsets, 4) || misaligned(workspace, 16))
    return CTS_ERR_INVALID_ARG;
  if (T > cts::kSortMaxT || n > 65536 || K > 65536) return CTS_ERR_UNSUPPORTED;
  BucketLayout L;
  bucket_layout(T, n, K, &L);
  if (workspace && workspace_bytes < L.total) return CTS_ERR_WORKSPACE;
  const Range out[3] = {{perm, 4ull * T}, {cluster_offsets, 4ull * (K + 1)},
                        {workspace, workspace ? L.total : 0}};
  const Range in[2] = {{adapter_id, 4ull * T}, {cluster_of, cluster_of ? 4ull * n : 0}};
  for (int a = 0; a < 3; ++a)
    for (int b = a + 1; b < 3; ++b)
      if (overlap(out[a], out[b])) return CTS_ERR_INVALID_ARG;
  for (const Range& o : out)
    for (const Range& i : in)
      if (overlap(o, i)) return CTS_ERR_INVALID_ARG;
  char* ws = static_cast<char*>(workspace);
  auto at = [&](size_t off) { return ws ? reinterpret_cast<int32_t*>(ws + off) : nullptr; };
  const hipError_t e = cts::launch_sort(adapter_id, cluster_of, T, n, K, perm, cluster_offsets, at(L.seg),
                                        at(L.aid), at(L.items), at(L.nitems), at(L.ctiles), at(L.nctiles),
                                        static_cast<hipStream_t>(stream), at(L.iaid), at(L.cseg));
  return e == hipSuccess ? CTS_OK : CTS_ERR_HIP;
}

namespace {

// Device address of the current device's copy of `scratch`, looked up once
// per device (hipGetSymbolAddress with that device current) and kept.  The
// array's name is a host-side stand-in in host code: only this address may
// be handed to kernels.
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

int scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return CTS_ERR_HIP;
  if (dev >= kMaxDevices) return CTS_ERR_UNSUPPORTED;
  void* ptr = g_scratch[dev].load(std::memory_order_acquire);
  if (!ptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    ptr = g_scratch[dev].load(std::memory_order_relaxed);
    if (!ptr) {
      if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return CTS_ERR_HIP;
      g_scratch[dev].store(ptr, std::memory_order_release);
    }
  }
  *out = ptr;
  return CTS_OK;
}

// workspace == nullptr with noalloc: the call runs in this device's static
// scratch array (the problem's workspace must fit in it).
int apply_compressed(const cts_problem* p, const void* x, const int32_t* adapter_id,
                     const int32_t* cluster_of, const void* W, const void* U, const void* Vt,
                     const void* Sigma, void* y, void* workspace, size_t workspace_bytes, void* stream,
                     bool sigma_diag, const int32_t* rank_of_cluster = nullptr, bool ranked = false,
                     bool noalloc = false) {
  Plan pl;
  const int rc = make_plan(p, true, &pl);
  if (rc != CTS_OK) return rc;
  if (p->T == 0) return CTS_OK;
  if (!x || !adapter_id || !cluster_of || !W || !U || !Vt || !Sigma || !y || (!workspace && !noalloc))
    return CTS_ERR_INVALID_ARG;
  for (const void* q : {x, W, U, Vt, Sigma, static_cast<const void*>(y), static_cast<const void*>(workspace)})
    if (misaligned(q, 16)) return CTS_ERR_INVALID_ARG;
  if (misaligned(adapter_id, 4) || misaligned(cluster_of, 4)) return CTS_ERR_INVALID_ARG;
  if (ranked && (!rank_of_cluster || misaligned(rank_of_cluster, 4))) return CTS_ERR_INVALID_ARG;
  if (noalloc ? pl.total > CTS_NOALLOC_SCRATCH_BYTES : workspace_bytes < pl.total)
    return noalloc ? CTS_ERR_UNSUPPORTED : CTS_ERR_WORKSPACE;
  const size_t e = pl.elt;
  const size_t T = p->T, di = p->d_in, dout = p->d_out, r = p->r, n = p->n_adapters, K = p->n_clusters;
  const Range in[8] = {{x, T * di * e}, {adapter_id, 4 * T}, {cluster_of, 4 * n},
                       {W, dout * di * e}, {U, K * dout * r * e}, {Vt, K * r * di * e},
                       {Sigma, n * (sigma_diag ? 1 : r) * r * e},
                       {rank_of_cluster, ranked ? 4 * K : 0}};
  // (the static scratch array is an allocation of its own: no caller array
  // can overlap it)
  if (any_overlap({y, T * dout * pl.out_elt}, {workspace, noalloc ? 0 : workspace_bytes}, in, 8))
    return CTS_ERR_INVALID_ARG;
  if (noalloc) {
    const int sc = scratch_of_current_device(&workspace);
    if (sc != CTS_OK) return sc;
  }
  return for_pieces(p, [&](const cts_problem& q, size_t t0) {
    Plan pq;
    const int rq = make_plan(&q, true, &pq);
    if (rq != CTS_OK) return rq;
    return run_layer(&q, pq, true, static_cast<const char*>(x) + t0 * di * e, adapter_id + t0, cluster_of, W,
                     U, Vt, Sigma, static_cast<char*>(y) + t0 * dout * pl.out_elt, workspace,
                     static_cast<hipStream_t>(stream), sigma_diag, ranked ? rank_of_cluster : nullptr);
  });
}

}  // namespace

int cts_apply(const cts_problem* p, const void* x, const int32_t* adapter_id,
              const int32_t* cluster_of, const void* W, const void* U, const void* Vt,
              const void* Sigma, void* y, void* workspace, size_t workspace_bytes, void* stream) {
  return apply_compressed(p, x, adapter_id, cluster_of, W, U, Vt, Sigma, y, workspace,
                          workspace_bytes, stream, false);
}

int cts_apply_noalloc(const cts_problem* p, const void* x, const int32_t* adapter_id,
                      const int32_t* cluster_of, const void* W, const void* U, const void* Vt,
                      const void* Sigma, void* y, void* stream) {
  return apply_compressed(p, x, adapter_id, cluster_of, W, U, Vt, Sigma, y, nullptr, 0, stream, false,
                          nullptr, false, true);
}

int cts_apply_diag(const cts_problem* p, const void* x, const int32_t* adapter_id,
                   const int32_t* cluster_of, const void* W, const void* U, const void* Vt,
                   const void* sigma, void* y, void* workspace, size_t workspace_bytes,
                   void* stream) {
  return apply_compressed(p, x, adapter_id, cluster_of, W, U, Vt, sigma, y, workspace,
                          workspace_bytes, stream, true);
}

int cts_apply_ranked(const cts_problem* p, const void* x, const int32_t* adapter_id,
                     const int32_t* cluster_of, const void* W, const void* U, const void* Vt,
                     const void* Sigma, const int32_t* rank_of_cluster, void* y, void* workspace,
                     size_t workspace_bytes, void* stream) {
  return apply_compressed(p, x, adapter_id, cluster_of, W, U, Vt, Sigma, y, workspace,
                          workspace_bytes, stream, false, rank_of_cluster, true);
}

namespace {

// ---- several modules sharing x, the adapter ids and the cluster map
// Workgroups of a grouped multi-module launch: one round over 256 compute
// units.
constexpr int64_t kGroupedMaxWorkgroups = 256;

struct MultiPlan {
  Plan mod[CTS_MAX_MODULES];   // per-module plans (fused GEMM tile and split)
  int M, rtot, shrink_split;
  // grouped: every module's fused GEMM in one launch, with the tile and split
  // of one GEMM as wide as all the modules together (bf16 inputs, M > 1)
  bool grouped;
  Tile g_tile;
  int g_split, d_sum;
  size_t off_zpart, off_zp, off_ypart, total;
};

int multi_plan_piece(const cts_problem* p, int M, const int32_t* d_out, MultiPlan* mp) {
  if (!p || M < 1 || !d_out) return CTS_ERR_INVALID_ARG;
  if (M > CTS_MAX_MODULES) return CTS_ERR_UNSUPPORTED;
  mp->M = M;
  for (int m = 0; m < M; ++m) {
    cts_problem q = *p;
    q.d_out = d_out[m];
    const int rc = make_plan(&q, true, &mp->mod[m]);
    if (rc != CTS_OK) return rc;
  }
  const Plan& p0 = mp->mod[0];
  const int T = p->T;
  mp->rtot = M * p->r;
  if (static_cast<uint64_t>(mp->rtot) * p->d_in * p0.elt > kMaxOperandBytes) return CTS_ERR_UNSUPPORTED;
  // shrink over the stacked rank: as for one module, with M r rank rows
  mp->shrink_split = shrink_split_of(T, mp->rtot, p0.nseg, p->d_in, p0.shrink_tile);
  size_t off = p0.off_zpart;                        // the shared sort arrays of module 0's layout
  mp->off_zpart = off; off = align_up(off + 4ull * mp->shrink_split * T * mp->rtot);
  mp->off_zp = off;    off = align_up(off + static_cast<size_t>(p0.elt) * T * mp->rtot);
  mp->off_ypart = off;
  mp->d_sum = 0;
  for (int m = 0; m < M; ++m) mp->d_sum += d_out[m];
  // grouped when the one launch fits one round of workgroups over the
  // compute units (q/k/v at T = 512: 192 workgroups instead of three launches
  // and three split-K sums); two launches of a round each are kept apart
  // (gate/up at T = 512: 448 grouped workgroups were slower than 2 x 224)
  mp->grouped = false;
  if (M > 1 && p0.elt == 2) {
    cts_problem q = *p;
    q.d_out = mp->d_sum;
    Plan gp;
    if (plan_piece(&q, true, &gp) == CTS_OK) {
      int BM, BN, BK;
      cts::tile_dims(gp.main_tile, &BM, &BN, &BK);
      int64_t rt = 0;
      for (int m = 0; m < M; ++m) rt += ceil_div(d_out[m], BM);
      const int64_t wgs = rt * ceil_div(std::max(T, 1), BN) * gp.main_split;
      if (wgs <= kGroupedMaxWorkgroups) {
        mp->grouped = true;
        mp->g_tile = gp.main_tile;
        mp->g_split = gp.main_split;
      }
    }
  }
  size_t yp = 0;
  if (mp->grouped) {
    if (mp->g_split > 1) yp = 4ull * mp->g_split * T * mp->d_sum;
  } else {
    for (int m = 0; m < M; ++m)
      if (mp->mod[m].main_split > 1) yp = std::max<size_t>(yp, 4ull * mp->mod[m].main_split * T * d_out[m]);
  }
  off = align_up(off + yp);
  mp->total = off;
  return CTS_OK;
}

// As make_plan: a batch of pieces takes its largest piece's plan, with a
// workspace that also fits the smaller piece size.
int make_multi_plan(const cts_problem* p, int M, const int32_t* d_out, MultiPlan* mp) {
  if (!p) return CTS_ERR_INVALID_ARG;
  if (p->T <= cts::kSortMaxT) return multi_plan_piece(p, M, d_out, mp);
  const Pieces pc = pieces_of(p->T);
  cts_problem q = *p;
  q.T = pc.q + (pc.rem ? 1 : 0);
  int rc = multi_plan_piece(&q, M, d_out, mp);
  if (rc != CTS_OK || !pc.rem) return rc;
  MultiPlan small;
  q.T = pc.q;
  rc = multi_plan_piece(&q, M, d_out, &small);
  if (rc != CTS_OK) return rc;
  mp->total = std::max(mp->total, small.total);
  return CTS_OK;
}

// ext_perm / ext_bucket: a bucketing from cts_sort_by_cluster (then the ids
// are not read and no sort runs here).
int run_multi(const cts_problem* p, const MultiPlan& mp, const int32_t* d_out, const void* x,
              const int32_t* adapter_id, const int32_t* cluster_of, const void* const* W,
              const void* const* U, const void* Vt, const void* const* Sigma, void* const* y, void* workspace,
              hipStream_t stream, const int32_t* ext_perm = nullptr, const void* ext_bucket = nullptr,
              int64_t ldy = 0) {
  const Plan& pl = mp.mod[0];
  char* ws = static_cast<char*>(workspace);
  int32_t* perm = reinterpret_cast<int32_t*>(ws + pl.off_perm);
  int32_t* sseg = reinterpret_cast<int32_t*>(ws + pl.off_seg);
  int32_t* said = reinterpret_cast<int32_t*>(ws + pl.off_aid);
  int32_t* offs = reinterpret_cast<int32_t*>(ws + pl.off_offs);
  int32_t* items = reinterpret_cast<int32_t*>(ws + pl.off_items);
  int32_t* n_items = reinterpret_cast<int32_t*>(ws + pl.off_nitems);
  int32_t* ctiles = reinterpret_cast<int32_t*>(ws + pl.off_ctiles);
  int32_t* n_ctiles = reinterpret_cast<int32_t*>(ws + pl.off_nctiles);
  int32_t* iaid = reinterpret_cast<int32_t*>(ws + pl.off_iaid);
  int32_t* cseg = reinterpret_cast<int32_t*>(ws + pl.off_cseg);
  const bool ext = ext_perm != nullptr;
  if (ext) {
    BucketLayout L;
    bucket_layout(p->T, p->n_adapters, p->n_clusters, &L);
    char* b = static_cast<char*>(const_cast<void*>(ext_bucket));
    perm = const_cast<int32_t*>(ext_perm);
    sseg = reinterpret_cast<int32_t*>(b + L.seg);
    said = reinterpret_cast<int32_t*>(b + L.aid);
    items = reinterpret_cast<int32_t*>(b + L.items);
    n_items = reinterpret_cast<int32_t*>(b + L.nitems);
    ctiles = reinterpret_cast<int32_t*>(b + L.ctiles);
    n_ctiles = reinterpret_cast<int32_t*>(b + L.nctiles);
    iaid = reinterpret_cast<int32_t*>(b + L.iaid);
    cseg = reinterpret_cast<int32_t*>(b + L.cseg);
  }
  float* zpart = reinterpret_cast<float*>(ws + mp.off_zpart);
  char* zp = ws + mp.off_zp;
  float* ypart = reinterpret_cast<float*>(ws + mp.off_ypart);
  const int T = p->T, r = p->r, rt = mp.rtot;

  hipError_t e = mark(0, stream);
  if (e != hipSuccess) return CTS_ERR_HIP;
  const bool fuse_sort = !ext && T <= cts::kFuseSortMaxT && pl.shrink_tile == Tile::Shrink;
  if (!fuse_sort && !ext) {
    e = cts::launch_sort(adapter_id, cluster_of, T, p->n_adapters, pl.nseg, perm, offs, sseg, said, items, n_items,
                         ctiles, n_ctiles, stream, iaid, cseg);
    if (e != hipSuccess) return CTS_ERR_HIP;
  }
  if (mark(1, stream) != hipSuccess) return CTS_ERR_HIP;

  // one shrink over the stacked V_k^T of all modules: Z [T][M r]
  cts::GemmParams g{};
  g.M = rt; g.N = T;
  g.A0 = nullptr; g.K0 = 0;
  g.A1 = Vt; g.seg_stride_a1 = static_cast<int64_t>(rt) * p->d_in; g.lda1 = p->d_in;
  g.B1 = x; g.ldb1 = p->d_in; g.K1 = p->d_in; g.b1_gather = 1;
  g.a0_bytes = 0; g.b0_bytes = 0;
  g.a1_seg_bytes = static_cast<uint32_t>(static_cast<uint64_t>(rt) * p->d_in * pl.elt);
  g.b1_bytes = static_cast<uint32_t>(static_cast<uint64_t>(T) * p->d_in * pl.elt);
  g.perm = perm; g.sorted_seg = sseg;
  g.ksplit = mp.shrink_split; g.part = zpart;
  g.tile_start = ctiles; g.n_tiles = n_ctiles; g.max_tiles = pl.max_ctiles; g.tile_seg = cseg;
  int32_t* ssplit = nullptr;
  if (shrink_adaptive(T, pl.shrink_tile)) {
    ssplit = reinterpret_cast<int32_t*>(ws + pl.off_ssplit);
    g.split_target = kShrinkAdaptiveTarget; g.split_out = ssplit;
  }
  if (fuse_sort) {
    g.tile_start = nullptr; g.n_tiles = nullptr; g.tile_seg = nullptr;
    g.fs_item_aid = iaid;
    g.fs_adapter = adapter_id; g.fs_cluster = cluster_of;
    g.fs_n = p->n_adapters; g.fs_K = pl.nseg;
    int bits_n = 0;
    while ((1 << bits_n) < p->n_adapters) ++bits_n;
    g.fs_bits_n = bits_n;
    g.fs_perm = perm; g.fs_seg = sseg; g.fs_aid = said; g.fs_items = items; g.fs_nitems = n_items;
  }
  e = cts::launch_seg_gemm(g, p->dtype, pl.shrink_tile, stream);
  if (e != hipSuccess || mark(2, stream) != hipSuccess) return CTS_ERR_HIP;

  // core product of every module on its slice of Z (rows M r apart), one launch
  e = cts::launch_sigma(zpart, mp.shrink_split, T, r, said, p->n_adapters, items, n_items, pl.max_items, Sigma[0],
                        zp, p->dtype, stream, false, sseg, nullptr, nullptr, rt, ssplit, Sigma, mp.M, iaid);
  if (e != hipSuccess) return CTS_ERR_HIP;
  if (mark(3, stream) != hipSuccess) return CTS_ERR_HIP;

  if (mp.grouped) {
    // one launch: module m's row tiles follow module m-1's
    int BM, BN, BK;
    cts::tile_dims(mp.g_tile, &BM, &BN, &BK);
    cts::GemmParams f{};
    f.M = d_out[0]; f.N = T;
    f.A0 = W[0]; f.lda0 = p->d_in; f.B0 = x; f.ldb0 = p->d_in; f.K0 = p->d_in;
    f.A1 = U[0]; f.lda1 = r; f.B1 = zp; f.ldb1 = rt; f.K1 = r; f.b1_gather = 0;
    f.b0_bytes = static_cast<uint32_t>(static_cast<uint64_t>(T) * p->d_in * pl.elt);
    f.perm = perm; f.sorted_seg = sseg;
    f.ksplit = mp.g_split;
    f.part = mp.g_split > 1 ? ypart : nullptr;
    f.part_ld = mp.d_sum;
    f.out = y[0]; f.ldo = ldy > 0 ? ldy : d_out[0]; f.out_perm = 1; f.out_dtype = p->out_dtype;
    f.n_mod = mp.M;
    cts::SplitkMods sm{};
    sm.n = mp.M;
    int rt_acc = 0, col = 0;
    for (int m = 0; m < mp.M; ++m) {
      const int dm = d_out[m];
      f.mod_rt[m] = rt_acc;
      f.mod_M[m] = dm;
      f.mod_col[m] = col;
      f.mod_A0[m] = W[m];
      f.mod_a0_bytes[m] = static_cast<uint32_t>(static_cast<uint64_t>(dm) * p->d_in * pl.elt);
      f.mod_A1[m] = U[m];
      f.mod_a1_seg_bytes[m] = static_cast<uint32_t>(static_cast<uint64_t>(dm) * r * pl.elt);
      f.mod_B1[m] = zp + static_cast<size_t>(m) * r * pl.elt;
      f.mod_b1_bytes[m] =
          static_cast<uint32_t>((static_cast<uint64_t>(T) * rt - static_cast<uint64_t>(m) * r) * pl.elt);
      f.mod_out[m] = y[m];
      f.mod_ldo[m] = ldy > 0 ? ldy : dm;
      sm.col[m] = col;
      sm.out[m] = y[m];
      sm.ldo[m] = f.mod_ldo[m];
      rt_acc += (dm + BM - 1) / BM;
      col += dm;
    }
    f.mod_rt[mp.M] = rt_acc;
    sm.col[mp.M] = col;
    f.a0_bytes = f.mod_a0_bytes[0]; f.a1_seg_bytes = f.mod_a1_seg_bytes[0]; f.b1_bytes = f.mod_b1_bytes[0];
    e = cts::launch_seg_gemm(f, p->dtype, mp.g_tile, stream);
    if (e != hipSuccess) return CTS_ERR_HIP;
    if (mp.g_split > 1) {
      e = cts::launch_splitk_reduce(ypart, mp.g_split, T, mp.d_sum, perm, nullptr, 0, p->out_dtype, stream, &sm);
      if (e != hipSuccess) return CTS_ERR_HIP;
    }
    if (mark(4, stream) != hipSuccess) return CTS_ERR_HIP;
    return mark(5, stream) == hipSuccess ? CTS_OK : CTS_ERR_HIP;
  }

  // fused W_m X + U_k^(m) Z'^(m) per module
  for (int m = 0; m < mp.M; ++m) {
    const Plan& pm = mp.mod[m];
    const int dm = d_out[m];
    cts::GemmParams f{};
    f.M = dm; f.N = T;
    f.A0 = W[m]; f.lda0 = p->d_in; f.B0 = x; f.ldb0 = p->d_in; f.K0 = p->d_in;
    f.A1 = U[m]; f.seg_stride_a1 = static_cast<int64_t>(dm) * r; f.lda1 = r;
    f.B1 = zp + static_cast<size_t>(m) * r * pl.elt; f.ldb1 = rt; f.K1 = r; f.b1_gather = 0;
    f.a0_bytes = static_cast<uint32_t>(static_cast<uint64_t>(dm) * p->d_in * pl.elt);
    f.b0_bytes = static_cast<uint32_t>(static_cast<uint64_t>(T) * p->d_in * pl.elt);
    f.a1_seg_bytes = static_cast<uint32_t>(static_cast<uint64_t>(dm) * r * pl.elt);
    f.b1_bytes = static_cast<uint32_t>((static_cast<uint64_t>(T) * rt - static_cast<uint64_t>(m) * r) * pl.elt);
    f.perm = perm; f.sorted_seg = sseg;
    f.ksplit = pm.main_split;
    f.part = pm.main_split > 1 ? ypart : nullptr;
    const int64_t ldm = ldy > 0 ? ldy : dm;              // output row stride (packed: the slices' total)
    f.out = y[m]; f.ldo = ldm; f.out_perm = 1; f.out_dtype = p->out_dtype;
    e = cts::launch_seg_gemm(f, p->dtype, pm.main_tile, stream);
    if (e != hipSuccess) return CTS_ERR_HIP;
    if (pm.main_split > 1) {
      e = cts::launch_splitk_reduce(ypart, pm.main_split, T, dm, perm, y[m], ldm, p->out_dtype, stream);
      if (e != hipSuccess) return CTS_ERR_HIP;
    }
  }
  if (mark(4, stream) != hipSuccess) return CTS_ERR_HIP;
  return mark(5, stream) == hipSuccess ? CTS_OK : CTS_ERR_HIP;
}

}  // namespace

size_t cts_workspace_size_multi(const cts_problem* p, int32_t M, const int32_t* d_out) {
  MultiPlan mp;
  return make_multi_plan(p, M, d_out, &mp) == CTS_OK ? mp.total : 0;
}

namespace {

// The checks of cts_apply_multi and cts_apply_multi_sorted: either the ids
// (adapter_id, cluster_of) or a bucketing (perm, bucket of bucket_bytes).
// ypk != null: the packed output of cts_apply_multi_packed (module m's
// columns at the sum of the earlier d_out, rows ldy elements apart) instead of
// the array y.
int apply_multi_checked(const cts_problem* p, int32_t M, const int32_t* d_out, const void* x,
                        const int32_t* adapter_id, const int32_t* cluster_of, const int32_t* perm,
                        const void* bucket, size_t bucket_bytes, const void* const* W, const void* const* U,
                        const void* Vt, const void* const* Sigma, void* const* y, void* workspace,
                        size_t workspace_bytes, void* stream, void* ypk = nullptr, int32_t ldy = 0) {
  MultiPlan mp;
  const int rc = make_multi_plan(p, M, d_out, &mp);
  if (rc != CTS_OK) return rc;
  void* yp[CTS_MAX_MODULES];
  int64_t cols = 0;
  for (int m = 0; m < M; ++m) cols += d_out[m];
  if (ypk) {
    // columns of module m: [c_m, c_m + d_out[m]), c_m a multiple of 8 (d_out
    // is); rows ldy elements apart, a multiple of 8 (16-byte rows)
    if (ldy < cols || ldy % 8) return CTS_ERR_INVALID_ARG;
    int64_t c = 0;
    for (int m = 0; m < M; ++m) {
      yp[m] = static_cast<char*>(ypk) + c * mp.mod[m].out_elt;
      c += d_out[m];
    }
    y = yp;
  }
  if (p->T == 0) return CTS_OK;
  const bool sorted = perm != nullptr || bucket != nullptr;
  if (sorted ? (!perm || !bucket) : (!adapter_id || !cluster_of)) return CTS_ERR_INVALID_ARG;
  if (!x || !W || !U || !Vt || !Sigma || !y || !workspace) return CTS_ERR_INVALID_ARG;
  BucketLayout L{};
  if (sorted) {
    if (p->T > cts::kSortMaxT) return CTS_ERR_UNSUPPORTED;
    bucket_layout(p->T, p->n_adapters, p->n_clusters, &L);
    if (misaligned(perm, 4) || misaligned(bucket, 16)) return CTS_ERR_INVALID_ARG;
    if (bucket_bytes < L.total) return CTS_ERR_WORKSPACE;
  }
  for (int m = 0; m < M; ++m)
    if (!W[m] || !U[m] || !Sigma[m] || !y[m] || misaligned(W[m], 16) || misaligned(U[m], 16) ||
        misaligned(Sigma[m], 16) || misaligned(y[m], 16))
      return CTS_ERR_INVALID_ARG;
  for (const void* q : {x, Vt, static_cast<const void*>(workspace)})
    if (misaligned(q, 16)) return CTS_ERR_INVALID_ARG;
  if (misaligned(adapter_id, 4) || misaligned(cluster_of, 4)) return CTS_ERR_INVALID_ARG;
  if (workspace_bytes < mp.total) return CTS_ERR_WORKSPACE;
  const size_t e = mp.mod[0].elt;
  const size_t T = p->T, di = p->d_in, r = p->r, n = p->n_adapters, K = p->n_clusters;
  // every output against the workspace, every input and the other outputs
  std::vector<Range> in = {{x, T * di * e}, {Vt, K * static_cast<size_t>(mp.rtot) * di * e}};
  if (sorted) {
    in.push_back({perm, 4 * T});
    in.push_back({bucket, L.total});
  } else {
    in.push_back({adapter_id, 4 * T});
    in.push_back({cluster_of, 4 * n});
  }
  for (int m = 0; m < M; ++m) {
    const size_t dm = d_out[m];
    in.push_back({W[m], dm * di * e});
    in.push_back({U[m], K * dm * r * e});
    in.push_back({Sigma[m], n * r * r * e});
  }
  if (ypk) {
    // the packed slices are disjoint by construction: one range for all
    const Range yr{ypk, (T - 1) * static_cast<size_t>(ldy) * mp.mod[0].out_elt +
                            static_cast<size_t>(cols) * mp.mod[0].out_elt};
    if (any_overlap(yr, {workspace, workspace_bytes}, in.data(), static_cast<int>(in.size())))
      return CTS_ERR_INVALID_ARG;
  } else {
    for (int m = 0; m < M; ++m) {
      const Range ym{y[m], T * static_cast<size_t>(d_out[m]) * mp.mod[m].out_elt};
      if (any_overlap(ym, {workspace, workspace_bytes}, in.data(), static_cast<int>(in.size())))
        return CTS_ERR_INVALID_ARG;
      for (int k = 0; k < m; ++k)
        if (overlap(ym, {y[k], T * static_cast<size_t>(d_out[k]) * mp.mod[k].out_elt})) return CTS_ERR_INVALID_ARG;
    }
  }
  const int64_t ld = ypk ? ldy : 0;
  if (sorted)   // one bucketing of the whole batch (cts_sort_by_cluster: T <= kSortMaxT)
    return run_multi(p, mp, d_out, x, nullptr, nullptr, W, U, Vt, Sigma, y, workspace,
                     static_cast<hipStream_t>(stream), perm, bucket, ld);
  return for_pieces(p, [&](const cts_problem& q, size_t t0) {
    MultiPlan mq;
    const int rq = make_multi_plan(&q, M, d_out, &mq);
    if (rq != CTS_OK) return rq;
    void* yq[CTS_MAX_MODULES];
    for (int m = 0; m < M; ++m)
      yq[m] = static_cast<char*>(y[m]) + t0 * static_cast<size_t>(ld > 0 ? ld : d_out[m]) * mp.mod[m].out_elt;
    return run_multi(&q, mq, d_out, static_cast<const char*>(x) + t0 * di * e, adapter_id + t0, cluster_of, W,
                     U, Vt, Sigma, yq, workspace, static_cast<hipStream_t>(stream), nullptr, nullptr, ld);
  });
}

}  // namespace

int cts_apply_multi(const cts_problem* p, int32_t M, const int32_t* d_out, const void* x,
                    const int32_t* adapter_id, const int32_t* cluster_of, const void* const* W,
                    const void* const* U, const void* Vt, const void* const* Sigma, void* const* y,
                    void* workspace, size_t workspace_bytes, void* stream) {
  return apply_multi_checked(p, M, d_out, x, adapter_id, cluster_of, nullptr, nullptr, 0, W, U, Vt, Sigma, y,
                             workspace, workspace_bytes, stream);
}

int cts_apply_multi_sorted(const cts_problem* p, int32_t M, const int32_t* d_out, const int32_t* perm,
                           const void* bucketing, size_t bucketing_bytes, const void* x, const void* const* W,
                           const void* const* U, const void* Vt, const void* const* Sigma, void* const* y,
                           void* workspace, size_t workspace_bytes, void* stream) {
  if (p && p->T > 0 && (!perm || !bucketing)) return CTS_ERR_INVALID_ARG;
  return apply_multi_checked(p, M, d_out, x, nullptr, nullptr, perm, bucketing, bucketing_bytes, W, U, Vt,
                             Sigma, y, workspace, workspace_bytes, stream);
}

int cts_apply_multi_packed(const cts_problem* p, int32_t M, const int32_t* d_out, const int32_t* adapter_id,
                           const int32_t* cluster_of, const int32_t* perm, const void* bucketing,
                           size_t bucketing_bytes, const void* x, const void* const* W, const void* const* U,
                           const void* Vt, const void* const* Sigma, void* y, int32_t ldy, void* workspace,
                           size_t workspace_bytes, void* stream) {
  const bool ids = adapter_id || cluster_of, sorted = perm || bucketing;
  if (p && p->T > 0 && ids == sorted) return CTS_ERR_INVALID_ARG;     // exactly one of the two
  if (p && p->T > 0 && !y) return CTS_ERR_INVALID_ARG;
  return apply_multi_checked(p, M, d_out, x, adapter_id, cluster_of, perm, bucketing, bucketing_bytes, W, U, Vt,
                             Sigma, nullptr, workspace, workspace_bytes, stream, y, ldy);
}

namespace {

int apply_uncompressed(const cts_problem* p, const void* x, const int32_t* adapter_id,
                       const void* W, const void* A, const void* B, void* y, void* workspace,
                       size_t workspace_bytes, void* stream, const int32_t* rank_of_adapter,
                       bool ranked) {
  Plan pl;
  const int rc = make_plan(p, false, &pl);
  if (rc != CTS_OK) return rc;
  if (p->T == 0) return CTS_OK;
  if (!x || !adapter_id || !W || !A || !B || !y || !workspace) return CTS_ERR_INVALID_ARG;
  for (const void* q : {x, W, A, B, static_cast<const void*>(y), static_cast<const void*>(workspace)})
    if (misaligned(q, 16)) return CTS_ERR_INVALID_ARG;
  if (misaligned(adapter_id, 4)) return CTS_ERR_INVALID_ARG;
  if (ranked && (!rank_of_adapter || misaligned(rank_of_adapter, 4))) return CTS_ERR_INVALID_ARG;
  if (workspace_bytes < pl.total) return CTS_ERR_WORKSPACE;
  const size_t e = pl.elt;
  const size_t T = p->T, di = p->d_in, dout = p->d_out, rl = p->r_lora, n = p->n_adapters;
  const Range in[6] = {{x, T * di * e}, {adapter_id, 4 * T}, {W, dout * di * e},
                       {A, n * rl * di * e}, {B, n * dout * rl * e},
                       {rank_of_adapter, ranked ? 4 * n : 0}};
  if (any_overlap({y, T * dout * pl.out_elt}, {workspace, workspace_bytes}, in, 6))
    return CTS_ERR_INVALID_ARG;
  return for_pieces(p, [&](const cts_problem& q, size_t t0) {
    Plan pq;
    const int rq = make_plan(&q, false, &pq);
    if (rq != CTS_OK) return rq;
    return run_layer(&q, pq, false, static_cast<const char*>(x) + t0 * di * e, adapter_id + t0, nullptr, W, B,
                     A, nullptr, static_cast<char*>(y) + t0 * dout * pl.out_elt, workspace,
                     static_cast<hipStream_t>(stream), false, ranked ? rank_of_adapter : nullptr);
  });
}

}  // namespace

int cts_apply_uncompressed(const cts_problem* p, const void* x, const int32_t* adapter_id,
                           const void* W, const void* A, const void* B, void* y, void* workspace,
                           size_t workspace_bytes, void* stream) {
  return apply_uncompressed(p, x, adapter_id, W, A, B, y, workspace, workspace_bytes, stream,
                            nullptr, false);
}

int cts_apply_uncompressed_ranked(const cts_problem* p, const void* x, const int32_t* adapter_id,
                                  const void* W, const void* A, const void* B,
                                  const int32_t* rank_of_adapter, void* y, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  return apply_uncompressed(p, x, adapter_id, W, A, B, y, workspace, workspace_bytes, stream,
                            rank_of_adapter, true);
}

int cts_set_stage_events(void* const* events) {
  if (!events) {
    g_stage_on = false;
    return CTS_OK;
  }
  for (int i = 0; i < CTS_N_STAGE_EVENTS; ++i) g_stage_events[i] = static_cast<hipEvent_t>(events[i]);
  g_stage_on = true;
  return CTS_OK;
}

int cts_validate_ids(const cts_problem* p, const int32_t* adapter_id, const int32_t* cluster_of,
                     void* stream) {
  if (!p || p->T < 0 || p->n_adapters < 1) return CTS_ERR_INVALID_ARG;
  if (cluster_of && p->n_clusters < 1) return CTS_ERR_INVALID_ARG;
  if (p->T > 0 && !adapter_id) return CTS_ERR_INVALID_ARG;
  const size_t T = p->T, n = p->n_adapters;
  int32_t* h = static_cast<int32_t*>(malloc(4 * (T + (cluster_of ? n : 0) + 1)));
  if (!h) return CTS_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  int rc = CTS_OK;
  if (T && hipMemcpyAsync(h, adapter_id, 4 * T, hipMemcpyDeviceToHost, s) != hipSuccess) rc = CTS_ERR_HIP;
  if (rc == CTS_OK && cluster_of &&
      hipMemcpyAsync(h + T, cluster_of, 4 * n, hipMemcpyDeviceToHost, s) != hipSuccess) rc = CTS_ERR_HIP;
  if (rc == CTS_OK && hipStreamSynchronize(s) != hipSuccess) rc = CTS_ERR_HIP;
  if (rc == CTS_OK) {
    for (size_t t = 0; t < T; ++t)
      if (h[t] < 0 || h[t] >= p->n_adapters) rc = CTS_ERR_BAD_IDS;
    if (cluster_of)
      for (size_t i = 0; i < n; ++i)
        if (h[T + i] < 0 || h[T + i] >= p->n_clusters) rc = CTS_ERR_BAD_IDS;
  }
  free(h);
  return rc;
}

}  // extern "C"
