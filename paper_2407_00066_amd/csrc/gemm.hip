// Segmented MFMA GEMM used for both contractions of the layer that touch the
// weights:
//   * shrink   Z = V_k^T X       per cluster segment   (App. D, first step)
//   * fused    Y = W X + U_k Z'  base GEMM with the up-projection of every
//                                cluster segment accumulated into the same
//                                fp32 accumulators   (App. D: base term once
//                                for the batch, adapter term per token)
// The operand with rows m is a weight (W, V_k^T, U_k: k-contiguous); the
// operand with rows j is an activation in cluster-sorted order (x rows
// gathered through perm, or Z' rows).  A workgroup owns a BM x BN output tile
// and walks a flat list of BK-wide k-tiles: first the dense W tiles of its
// k-split, then, for every cluster segment that intersects its token columns,
// the k-tiles of that segment's basis with the other columns masked to zero.
//
// Global loads are raw buffer loads of 16 bytes: a row or k chunk outside
// the operand gets an out-of-range offset and reads as zero, so the loads
// carry no branches and all of a k-tile's loads are in flight together while
// earlier k-tiles are multiplied out of LDS (two register stages and two LDS
// buffers: each load has two k-tiles of compute to arrive; one barrier per
// k-tile).  LDS rows are padded by 16 bytes, which
// makes the 16-byte fragment reads of one MFMA conflict-free.
//
// Matrix cores: v_mfma_f32_32x32x16_bf16 or v_mfma_f32_16x16x32_bf16 (bf16
// in, fp32 accumulate), v_mfma_f32_16x16x4_f32 for fp32 inputs.  Both
// operands of a product use the same per-lane k assignment, so the hardware's
// internal k order does not matter; only the accumulator layout (acc_row) is
// fixed by the instruction.
#include "cts_internal.h"
#include "ldsdma.h"

namespace cts {
namespace {

// MFMA shapes.  MB x MB output block per instruction; each lane holds KG
// consecutive k of one row (A) or column (B): lane l -> row/column l % MB,
// k group l / MB.
template <typename TI, int MB> struct MfmaTraits;
template <> struct MfmaTraits<bf16_t, 16> {      // v_mfma_f32_16x16x32_bf16
  static constexpr int EPC = 8, KS = 32, KG = 8, NACC = 4;
  typedef bf16x8 frag;
  typedef f32x4 accv;
  __device__ static __forceinline__ frag ld(const bf16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }
  __device__ static __forceinline__ accv mma(frag a, frag b, accv c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct MfmaTraits<bf16_t, 32> {      // v_mfma_f32_32x32x16_bf16
  static constexpr int EPC = 8, KS = 16, KG = 8, NACC = 16;
  typedef bf16x8 frag;
  typedef f32x16 accv;
  __device__ static __forceinline__ frag ld(const bf16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }
  __device__ static __forceinline__ accv mma(frag a, frag b, accv c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct MfmaTraits<float, 16> {       // v_mfma_f32_16x16x4_f32
  static constexpr int EPC = 4, KS = 4, KG = 1, NACC = 4;
  typedef float frag;
  typedef f32x4 accv;
  __device__ static __forceinline__ frag ld(const float* p) { return *p; }
  __device__ static __forceinline__ accv mma(frag a, frag b, accv c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

// Row of accumulator element v of lane l inside an MB x MB block (the column
// is l % MB): 16x16 -> 4*(l/16) + v; 32x32 -> 8*(v/4) + 4*(l/32) + v%4.
template <int MB> __device__ __forceinline__ int acc_row(int lane, int v) {
  return MB == 16 ? 4 * (lane >> 4) + v : 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}

template <typename TI, int BM, int BN, int BK, int WM, int WN, int MB>
struct Cfg {
  static constexpr int NT = WM * WN * 64;
  static constexpr int EPC = MfmaTraits<TI, MB>::EPC;
  static constexpr int KS = MfmaTraits<TI, MB>::KS;
  static constexpr int CPR = BK / EPC;                // 16-byte chunks per tile row
  static constexpr int RPP = NT / CPR;                // tile rows covered per pass
  static constexpr int LDS_ROW = BK + EPC;            // padded row, elements
  static constexpr int CA = BM / RPP;                 // A chunks per thread
  static constexpr int CB = BN / RPP;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int FM = WTM / MB, FN = WTN / MB;
  static constexpr int AB_BYTES = 2 * (BM + BN) * LDS_ROW * (int)sizeof(TI);
  static constexpr int ST_ROW = BM + 4;               // staged fp32 row (per token)
  static constexpr int ST_BYTES = BN * ST_ROW * 4;
  static constexpr int SMEM = AB_BYTES > ST_BYTES ? AB_BYTES : ST_BYTES;
  static_assert(NT % CPR == 0 && BM % RPP == 0 && BN % RPP == 0, "chunk split");
  static_assert(WTM % MB == 0 && WTN % MB == 0 && BK % KS == 0, "tile shape");
};

__device__ __forceinline__ int split_lo(int n, int ks, int S) { return (int)((int64_t)n * ks / S); }

// XCD-aware tile order.  The dispatcher hands workgroup b to XCD b % 8, and
// each XCD has its own L2.  The linear block id is remapped so that XCD x
// owns one contiguous range of a grouped tile order (GROUP m-tiles by all
// n-tiles, column by column), i.e. a compact block of tiles whose weight rows
// and token columns stay in that XCD's L2.  The map is a bijection for any
// grid size.
constexpr int kXcds = 8;
constexpr int kGroupM = 8;
// group_m: m-tiles per group (0: kGroupM).
__device__ __forceinline__ void tile_of_block(int gm, int gn, int* mt, int* nt, int* ks, int nb_used = 0,
                                              int group_m = 0) {
  const int b = blockIdx.x;
  const int nb_mn = gm * gn;
  const int G = group_m > 0 ? group_m : kGroupM;
  // nb_mn * ksplit workgroups (the grid, or its first nb_used)
  const int nb = nb_used > 0 ? nb_used : static_cast<int>(gridDim.x);
  const int q = nb / kXcds, rem = nb % kXcds;
  const int x = b % kXcds, i = b / kXcds;
  const int L = x * q + min(x, rem) + i;
  *ks = L / nb_mn;
  const int l = L % nb_mn;
  const int per_group = G * gn;
  const int g = l / per_group;
  const int gsz = min(G, gm - g * G);               // m-tiles in this group
  const int r = l % per_group;
  *mt = g * G + r % gsz;
  *nt = r / gsz;
}

// The group size for a grid of gm x gn tiles split S ways: kGroupM when each
// XCD's share of the grid is a whole number of groups or of group columns;
// otherwise, when that share is a whole number of m-tiles with all their
// n-tiles, the share itself (one group per XCD), so that no weight row tile
// is fetched into two XCDs' L2s (e.g. 56 x 4 tiles: 7 m-tiles per XCD, not
// groups of 8 that straddle two XCDs).
int xcd_group_m(int gm, int gn, int S) {
  const int64_t nb = static_cast<int64_t>(gm) * gn * S;
  if (nb % kXcds) return kGroupM;
  const int64_t c = nb / kXcds, pg = static_cast<int64_t>(kGroupM) * gn, nmn = static_cast<int64_t>(gm) * gn;
  if (pg % c == 0 || c % pg == 0) return kGroupM;
  if (c % gn == 0 && nmn % c == 0) return static_cast<int>(c / gn);
  return kGroupM;
}

// STAGES: register stages of global loads in flight; OCC: waves per SIMD the
// register allocation must allow; MB: MFMA block (16 or 32).
template <typename TI, int BM, int BN, int BK, int WM, int WN, int STAGES, int OCC, int MB>
__global__ __launch_bounds__(WM * WN * 64, OCC) void seg_gemm_kernel(const GemmParams p) {
  using C = Cfg<TI, BM, BN, BK, WM, WN, MB>;
  using MT = MfmaTraits<TI, MB>;
  typedef typename MT::accv accv;
  typedef typename MT::frag frag;
  constexpr uint32_t ELT = sizeof(TI);
  const int gn = p.tile_start ? p.max_tiles : (p.N + BN - 1) / BN;

  __shared__ __attribute__((aligned(16))) char smem[C::SMEM];
  __shared__ int32_t t_perm[BN];
  __shared__ int32_t t_seg[BN];
  __shared__ int32_t run_start[BN + 1];
  __shared__ int32_t wave_runs[C::NT / 64];

  TI* smA = reinterpret_cast<TI*>(smem);
  TI* smB = smA + 2 * BM * C::LDS_ROW;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int mt, nt, ks;
  tile_of_block((p.M + BM - 1) / BM, gn, &mt, &nt, &ks);
  if (p.tile_start && nt >= p.n_tiles[0]) return;    // whole workgroup: no tile
  const int m0 = mt * BM;
  const int j0 = p.tile_start ? p.tile_start[nt] : nt * BN;
  const int S = p.ksplit;
  const int jn = p.tile_start ? (p.tile_start[nt + 1] - j0) : min(BN, p.N - j0);   // valid columns

  // ---- token columns of this tile: perm, segment, and segment runs -------
  for (int i = tid; i < BN; i += C::NT) {
    t_perm[i] = (i < jn) ? p.perm[j0 + i] : 0;
    t_seg[i] = (i < jn && p.sorted_seg) ? p.sorted_seg[j0 + i] : 0;
  }
  __syncthreads();
  int n_runs = 0;
  for (int base = 0; base < BN; base += C::NT) {
    const int i = base + tid;
    const bool st = (i < jn) && (i == 0 || t_seg[i] != t_seg[i - 1]);
    const uint64_t bal = __ballot(st);
    if (lane == 0) wave_runs[wave] = __popcll(bal);
    __syncthreads();
    int before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < C::NT / 64; ++w) {
      const int c = wave_runs[w];
      before += (w < wave) ? c : 0;
      total += c;
    }
    if (st) {
      const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
      run_start[n_runs + before + __popcll(bal & lt)] = i;
    }
    n_runs += total;
    __syncthreads();
  }
  if (!(p.sorted_seg && p.K1 > 0)) n_runs = 0;
  if (tid == 0) run_start[n_runs] = jn;
  __syncthreads();

  // ---- k-tile schedule ----------------------------------------------------
  const int nk0 = (p.K0 > 0) ? (p.K0 + BK - 1) / BK : 0;
  const int nk1 = (p.K1 > 0) ? (p.K1 + BK - 1) / BK : 0;
  int d_lo = 0, d_hi = 0, s_lo = 0, s_hi = 0;
  if (nk0 > 0) {
    d_lo = split_lo(nk0, ks, S); d_hi = split_lo(nk0, ks + 1, S);
    if (ks == 0) { s_lo = 0; s_hi = nk1; }
  } else {
    s_lo = split_lo(nk1, ks, S); s_hi = split_lo(nk1, ks + 1, S);
  }
  const int nd = d_hi - d_lo, ns = s_hi - s_lo;
  const int ntiles = nd + n_runs * ns;

  // ---- per-thread load coordinates (fixed for the whole kernel) ------------
  const int kc = tid % C::CPR;               // 16-byte chunk within a tile row
  const int row0 = tid / C::CPR;             // first tile row, then + RPP each

  const __amdgpu_buffer_rsrc_t rA0 = make_rsrc(p.A0, p.a0_bytes);
  const __amdgpu_buffer_rsrc_t rB0 = make_rsrc(p.B0, p.b0_bytes);
  const __amdgpu_buffer_rsrc_t rB1 = make_rsrc(p.B1, p.b1_bytes);

  // byte offsets of this thread's rows in each phase (kOob: outside the operand)
  uint32_t a0_row[C::CA], a1_row[C::CA], b0_row[C::CB], b1_row[C::CB];
  int b_jl[C::CB];
#pragma unroll
  for (int i = 0; i < C::CA; ++i) {
    const int m = m0 + row0 + i * C::RPP;
    const bool ok = m < p.M;
    a0_row[i] = ok ? static_cast<uint32_t>(m) * static_cast<uint32_t>(p.lda0) * ELT : kOob;
    a1_row[i] = ok ? static_cast<uint32_t>(m) * static_cast<uint32_t>(p.lda1) * ELT : kOob;
  }
#pragma unroll
  for (int i = 0; i < C::CB; ++i) {
    const int jl = row0 + i * C::RPP;
    const uint32_t tok = static_cast<uint32_t>(t_perm[jl]);
    const uint32_t r1 = p.b1_gather ? tok : static_cast<uint32_t>(j0 + jl);
    b_jl[i] = jl;
    b0_row[i] = tok * static_cast<uint32_t>(p.ldb0) * ELT;
    b1_row[i] = r1 * static_cast<uint32_t>(p.ldb1) * ELT;
  }

  // register stages of global loads: with S stages the loads of k-tile t+S are
  // issued while k-tile t is multiplied out of LDS
  u32x4 ra[STAGES][C::CA], rb[STAGES][C::CB];

  // load cursor: tiles are loaded strictly in order, so the position in the
  // schedule advances incrementally (no division per tile)
  int lt = 0;          // next k-tile to load
  int lq = 0;          // its segment run (segment phase)
  int lkt = s_lo;      // its k-tile within the segment phase

  // issue the loads of the next k-tile; past the end every load is out of
  // range and reads zeros, so the code has no data-dependent branches
  auto load_next = [&](u32x4 (&a)[C::CA], u32x4 (&b)[C::CB]) __attribute__((always_inline)) {
    const bool valid = lt < ntiles;
    const bool dense = lt < nd;
    const int q = min(lq, max(n_runs - 1, 0));
    const int lo = dense ? 0 : run_start[q];
    const int hi = dense ? jn : run_start[q + 1];
    const int seg = __builtin_amdgcn_readfirstlane(t_seg[lo]);
    const __amdgpu_buffer_rsrc_t rA =
        dense ? rA0
              : make_rsrc(static_cast<const char*>(p.A1) + static_cast<int64_t>(seg) * p.a1_seg_bytes,
                          p.a1_seg_bytes);
    const __amdgpu_buffer_rsrc_t rB = dense ? rB0 : rB1;
    const int kt = dense ? d_lo + lt : lkt;
    const uint32_t k = static_cast<uint32_t>(kt * BK) + kc * C::EPC;
    const int klim = dense ? p.K0 : (p.seg_rank ? seg_rank_of(p.seg_rank, seg, p.K1) : p.K1);
    // out-of-range chunks get bit 31 set (every operand is < 2^31 bytes)
    const uint32_t kmask = (valid && k < static_cast<uint32_t>(klim)) ? 0u : kOob;
    const uint32_t kb = k * ELT;
    const uint32_t span = static_cast<uint32_t>(hi - lo);
    const uint32_t dsel = dense ? 0xffffffffu : 0u;   // phase select by mask arithmetic
#pragma unroll
    for (int i = 0; i < C::CA; ++i) a[i] = load16(rA, ((a1_row[i] ^ ((a0_row[i] ^ a1_row[i]) & dsel)) + kb) | kmask);
#pragma unroll
    for (int i = 0; i < C::CB; ++i) {
      const uint32_t jmask = (static_cast<uint32_t>(b_jl[i] - lo) < span) ? 0u : kOob;
      b[i] = load16(rB, ((b1_row[i] ^ ((b0_row[i] ^ b1_row[i]) & dsel)) + kb) | kmask | jmask);
    }
    if (!dense) {
      ++lkt;
      if (lkt >= s_hi) { lkt = s_lo; ++lq; }
    }
    ++lt;
  };
  auto store_tile = [&](const u32x4 (&a)[C::CA], const u32x4 (&b)[C::CB], int buf) __attribute__((always_inline)) {
    TI* da = smA + buf * BM * C::LDS_ROW + row0 * C::LDS_ROW + kc * C::EPC;
    TI* db = smB + buf * BN * C::LDS_ROW + row0 * C::LDS_ROW + kc * C::EPC;
#pragma unroll
    for (int i = 0; i < C::CA; ++i) *reinterpret_cast<u32x4*>(da + i * C::RPP * C::LDS_ROW) = a[i];
#pragma unroll
    for (int i = 0; i < C::CB; ++i) *reinterpret_cast<u32x4*>(db + i * C::RPP * C::LDS_ROW) = b[i];
  };

  const int wm = wave / WN, wn = wave % WN;
  accv acc[C::FM][C::FN];
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j)
#pragma unroll
      for (int v = 0; v < MT::NACC; ++v) acc[i][j][v] = 0.f;

  const int frow = lane % MB, fk = (lane / MB) * MT::KG;
  auto compute = [&](int buf) __attribute__((always_inline)) {
    const TI* a = smA + buf * BM * C::LDS_ROW + (wm * C::WTM + frow) * C::LDS_ROW + fk;
    const TI* b = smB + buf * BN * C::LDS_ROW + (wn * C::WTN + frow) * C::LDS_ROW + fk;
#pragma unroll
    for (int kk = 0; kk < BK; kk += C::KS) {
      frag fa[C::FM], fb[C::FN];
#pragma unroll
      for (int i = 0; i < C::FM; ++i) fa[i] = MT::ld(a + i * MB * C::LDS_ROW + kk);
#pragma unroll
      for (int j = 0; j < C::FN; ++j) fb[j] = MT::ld(b + j * MB * C::LDS_ROW + kk);
#pragma unroll
      for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j) acc[i][j] = MT::mma(fa[i], fb[j], acc[i][j]);
    }
  };

  // prologue: k-tiles 0..STAGES-1 in flight, k-tile 0 staged in LDS buffer 0
#pragma unroll
  for (int s = 0; s < STAGES; ++s) load_next(ra[s], rb[s]);
  store_tile(ra[0], rb[0], 0);
  __syncthreads();
  // k-tile u sits in register stage u % STAGES until it is stored to LDS
  // buffer u % 2 at the end of step u-1; the loop is unrolled so that both
  // indices are compile-time constants
  constexpr int U = (STAGES % 2 == 0) ? STAGES : 2 * STAGES;
  for (int t = 0; t < ntiles; t += U) {
#pragma unroll
    for (int s = 0; s < U; ++s) {
      if (t + s >= ntiles) break;
      load_next(ra[s % STAGES], rb[s % STAGES]);                      // k-tile t+s+STAGES
      compute(s % 2);                                                  // k-tile t+s
      store_tile(ra[(s + 1) % STAGES], rb[(s + 1) % STAGES], (s + 1) % 2);  // k-tile t+s+1
      __syncthreads();
    }
  }

  // ---- epilogue: stage fp32 tile as [token][row], then 16-byte stores ------
  float* st = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
      const int col = wn * C::WTN + j * MB + lane % MB;
      const int row = wm * C::WTM + i * MB;
#pragma unroll
      for (int v = 0; v < MT::NACC; v += 4)   // 4 consecutive rows per group
        *reinterpret_cast<f32x4*>(st + col * C::ST_ROW + row + acc_row<MB>(lane, v)) =
            f32x4{acc[i][j][v], acc[i][j][v + 1], acc[i][j][v + 2], acc[i][j][v + 3]};
    }
  __syncthreads();

  if (p.part) {
    float* part = p.part + static_cast<int64_t>(ks) * p.N * p.M;
    constexpr int CPRO = BM / 4;
    for (int c = tid; c < BN * CPRO; c += C::NT) {
      const int jl = c / CPRO, mc = (c % CPRO) * 4;
      if (jl < jn && m0 + mc < p.M)
        *reinterpret_cast<f32x4*>(part + static_cast<int64_t>(j0 + jl) * p.M + m0 + mc) =
            *reinterpret_cast<const f32x4*>(st + jl * C::ST_ROW + mc);
    }
  } else if (p.out_dtype == 1) {  // bf16 out, 8 values per 16-byte store
    constexpr int CPRO = BM / 8;
    uint16_t* out = static_cast<uint16_t*>(p.out);
    for (int c = tid; c < BN * CPRO; c += C::NT) {
      const int jl = c / CPRO, mc = (c % CPRO) * 8;
      if (jl < jn && m0 + mc < p.M) {
        const float* s = st + jl * C::ST_ROW + mc;
        const f32x4 lo = *reinterpret_cast<const f32x4*>(s);
        const f32x4 hi = *reinterpret_cast<const f32x4*>(s + 4);
        uint4 v;
        v.x = f32_to_bf16(lo[0]) | (static_cast<uint32_t>(f32_to_bf16(lo[1])) << 16);
        v.y = f32_to_bf16(lo[2]) | (static_cast<uint32_t>(f32_to_bf16(lo[3])) << 16);
        v.z = f32_to_bf16(hi[0]) | (static_cast<uint32_t>(f32_to_bf16(hi[1])) << 16);
        v.w = f32_to_bf16(hi[2]) | (static_cast<uint32_t>(f32_to_bf16(hi[3])) << 16);
        const int64_t row = p.out_perm ? t_perm[jl] : static_cast<int64_t>(j0 + jl);
        *reinterpret_cast<uint4*>(out + row * p.ldo + m0 + mc) = v;
      }
    }
  } else {  // fp32 out
    constexpr int CPRO = BM / 4;
    float* out = static_cast<float*>(p.out);
    for (int c = tid; c < BN * CPRO; c += C::NT) {
      const int jl = c / CPRO, mc = (c % CPRO) * 4;
      if (jl < jn && m0 + mc < p.M) {
        const int64_t row = p.out_perm ? t_perm[jl] : static_cast<int64_t>(j0 + jl);
        *reinterpret_cast<f32x4*>(out + row * p.ldo + m0 + mc) =
            *reinterpret_cast<const f32x4*>(st + jl * C::ST_ROW + mc);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 variant with the k-tiles loaded straight into LDS.
//
// Each 16-byte buffer load writes its lane's chunk directly into LDS
// (buffer_load_dwordx4 ... lds): one wave instruction fills 1 KB, i.e. 8 tile
// rows of BK = 64 bf16 or 16 rows of BK = 32.  P LDS stages form a ring;
// k-tile t+P-1 is loaded while k-tile t is multiplied, so P-1 k-tiles of
// loads are in flight and no register holds staging data.  A lane stores
// chunk c of its row in slot c ^ key(row) (XOR swizzle; key = row % 16 for
// 256-byte rows, (row / 2) % 8 for 128-byte rows, (row / 4) % 4 for 64-byte
// rows).  The LDS serves a
// 16-byte read for 16 lanes (256 bytes, all 64 banks) per cycle, and a
// fragment read covers 16 consecutive rows at one logical chunk: with this
// key those 16 requests fall on 16 distinct bank groups.  An
// out-of-range lane (outside the operand, or a token column outside the
// current cluster segment) writes zeros.
//
// The completion of the loads and of the fragment reads is waited for
// explicitly (s_waitcnt with the exact count of loads still allowed in
// flight), and the fragment reads are issued as ds_read_b128 in inline
// assembly, so the compiler's blanket wait for LDS-writing loads before any
// LDS read does not apply.
template <int BM, int BN, int BK, int WM, int WN, int MB, int P, int DIRECT>
struct DmaCfg {
  static constexpr int NT = WM * WN * 64, NW = WM * WN;
  static constexpr int ROWB = BK * 2;                     // bytes per tile row
  static constexpr int CH = BK / 8;                       // 16-byte chunks per row
  static constexpr int RPI = 1024 / ROWB;                 // rows per 1 KB load
  static constexpr int SB = (BM + BN) * ROWB;             // bytes per stage
  static constexpr int QA = BM / RPI / NW, QB = BN / RPI / NW; // 1 KB loads per wave per k-tile
  static constexpr int LPT = QA + QB;                     // loads per thread per k-tile
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int FM = WTM / MB, FN = WTN / MB;
  static constexpr int KS = (MB == 32) ? 16 : 32;         // k per MFMA
  static constexpr int NKS = BK / KS;
  static constexpr int ST_ROW = BM + 4;
  static constexpr int ST_BYTES = BN * ST_ROW * 4;
  static constexpr int SMEM = (DIRECT || P * SB > ST_BYTES) ? P * SB : ST_BYTES;
  static_assert(BM % (RPI * NW) == 0 && BN % (RPI * NW) == 0, "load split");
  static_assert(WTM % MB == 0 && WTN % MB == 0 && BK % KS == 0, "wave tile");
  static_assert(BK == 32 || BK == 64 || BK == 128, "row width");
  static_assert((P - 2) * LPT < 64, "vmcnt range");
};

// DIRECT: the epilogue writes straight from the accumulators (4 consecutive
// output features of one token per lane) instead of staging the tile in LDS;
// used when the fp32 tile does not fit in LDS.
// PFD > 0 (rings of two or three stages): during k-tile t the workgroup also
// touches, one 4-byte load per cache line, its share of the weight rows and
// token rows of dense k-tile t + P - 1 + PFD, so that the LDS loads of that
// k-tile find them in L2.  Tiles of one XCD come in blocks of 8 row tiles
// (tile_of_block), so the 8 workgroups on one column tile each take every
// 8th token row; the WSPL workgroups on one row tile (4 with 256 tiles of
// 256x256) each take every WSPL-th weight row.
// RANKED: the segments have ranks (p.seg_rank, with each column's rank in
// p.sorted_rank): a cluster run takes only its adapter k-tiles below its
// rank, from a schedule listed in LDS.
// MODS: the launch may hold several modules (p.n_mod > 0).
template <int BM, int BN, int BK, int WM, int WN, int MB, int P, int DIRECT, int PFD = 0, int WSPL = 1,
          int FSORT = 0, int RANKED = 0, int MODS = 0>
__global__ __launch_bounds__(WM * WN * 64, 1) void seg_gemm_dma_kernel(const GemmParams p) {
  using C = DmaCfg<BM, BN, BK, WM, WN, MB, P, DIRECT>;
  static_assert(PFD == 0 || P <= 3, "prefetch wait counts cover rings of two or three stages");
  constexpr int NPF = PFD > 0 ? 1 : 0;                     // prefetch loads per wave per k-tile
  constexpr int PFW = C::NW / 2;                           // waves prefetching weight rows
  using MT = MfmaTraits<bf16_t, MB>;
  typedef typename MT::accv accv;
  constexpr uint32_t ELT = 2;

  __shared__ __attribute__((aligned(1024))) char smem[C::SMEM];
  __shared__ int32_t t_perm[BN];
  __shared__ int32_t t_seg[BN];
  __shared__ int32_t run_start[BN + 1];
  __shared__ int32_t wave_runs[C::NW];
  __shared__ uint2 sched[RANKED ? 2 * BN : 1];             // adapter k-tiles (K1 <= 2 BK)
  __shared__ int32_t t_rank[RANKED ? BN : 1];
  __shared__ int32_t n_sched_s;
  __shared__ uint32_t pf_sink[PFD > 0 ? 64 : 1];
  constexpr int FS = FSORT ? kFuseSortMaxT : 1;
  __shared__ uint64_t fs_raw[FS];                          // (key << 8) | token, in token order
  __shared__ uint32_t fs_key[FS];                          // keys, sorted
  __shared__ int32_t fs_perm[FS], fs_tile[FS + 1];
  __shared__ int32_t fs_cnt[2];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  // FSORT: bucketing of the (at most kFuseSortMaxT) tokens in LDS.  The key
  // is cluster << bits_n | adapter (the adapter alone without a cluster
  // map); the rank of token t is the number of smaller keys plus equal keys
  // of earlier tokens, the stable order of the separate sort.
  const int fs_cshift = p.fs_cluster ? p.fs_bits_n : 0;
  if (FSORT) {
    static_assert(!FSORT || (C::NT >= kFuseSortMaxT && BN >= 64), "one token per thread; 64-token tiles");
    const int T = p.N;
    // A cluster map that fits the ring's LDS (unused until the k loop) is
    // staged there: its loads go out with the adapter ids', one round trip
    // instead of a second, dependent one.
    const bool map_lds = p.fs_cluster && p.fs_n <= static_cast<int>(C::SMEM / 4);
    int32_t* const cmap = reinterpret_cast<int32_t*>(smem);
    int a = 0;
    if (tid < T) {
      a = p.fs_adapter[tid];
      a = a < 0 ? 0 : (a >= p.fs_n ? p.fs_n - 1 : a);
    }
    if (map_lds) {
      for (int i = tid; i < p.fs_n; i += C::NT) cmap[i] = p.fs_cluster[i];
      __syncthreads();
    }
    if (tid < T) {
      uint32_t key = static_cast<uint32_t>(a);
      if (p.fs_cluster) {
        int c = map_lds ? cmap[a] : p.fs_cluster[a];
        c = c < 0 ? 0 : (c >= p.fs_K ? p.fs_K - 1 : c);
        key |= static_cast<uint32_t>(c) << p.fs_bits_n;
      }
      fs_raw[tid] = (static_cast<uint64_t>(key) << 8) | static_cast<uint32_t>(tid);
    }
    __syncthreads();
    if (tid < T) {
      // the token index makes every composite distinct: the rank is the
      // number of smaller composites
      const uint64_t c = fs_raw[tid];
      int rank = 0;
      for (int j = 0; j < T; ++j) rank += fs_raw[j] < c ? 1 : 0;
      fs_perm[rank] = tid;
      fs_key[rank] = static_cast<uint32_t>(c >> 8);
    }
    __syncthreads();
    // wave 0: tile starts (a multiple of kSegTile or a new cluster) and, for
    // workgroup 0, core-product item starts (a multiple of kSigmaChunk or a
    // new key)
    if (wave == 0) {
      int nt_ = 0, ni_ = 0;
      for (int base = 0; base < T; base += 64) {
        const int j = base + lane;
        const bool valid = j < T;
        const uint32_t k = valid ? fs_key[j] : 0u;
        const uint32_t kp = (valid && j > 0) ? fs_key[j - 1] : 0u;
        const bool st = valid && (j % kSegTile == 0 || (k >> fs_cshift) != (kp >> fs_cshift));
        const bool si = valid && (j % kSigmaChunk == 0 || k != kp);
        const uint64_t bt = __ballot(st), bi = __ballot(si);
        if (st) fs_tile[nt_ + __popcll(bt & lt_mask)] = j;
        if (si && blockIdx.x == 0) {
          p.fs_items[ni_ + __popcll(bi & lt_mask)] = j;
          if (p.fs_item_aid)
            p.fs_item_aid[ni_ + __popcll(bi & lt_mask)] = static_cast<int32_t>(k & ((1u << p.fs_bits_n) - 1u));
        }
        nt_ += __popcll(bt);
        ni_ += __popcll(bi);
      }
      if (lane == 0) {
        fs_tile[nt_] = T;
        fs_cnt[0] = nt_;
        if (blockIdx.x == 0) { p.fs_items[ni_] = T; p.fs_nitems[0] = ni_; }
      }
    }
    if (blockIdx.x == 0 && tid < T) {
      const uint32_t k = fs_key[tid];
      p.fs_perm[tid] = fs_perm[tid];
      p.fs_seg[tid] = static_cast<int32_t>(k >> fs_cshift);
      p.fs_aid[tid] = static_cast<int32_t>(k & ((1u << p.fs_bits_n) - 1u));
    }
    __syncthreads();
  }
  // Token-tile mode (explicit tiles, each inside one segment): the tile's
  // segment operand becomes the dense operand (A = A1 of that segment, B = B1),
  // so the whole k loop takes the dense load path and there is no second phase.
  const bool tlist = FSORT || p.tile_start != nullptr;
  int mt, nt, ks;
  int s_pieces = p.ksplit;
  // the split along k follows the tile count only in the shrink's tile shape
  // (64 x 64 x 64); the other shapes keep the straight mapping
  constexpr bool kAdaptive = BM == 64 && BN == 64 && BK == 64;
  if (kAdaptive && tlist && p.split_target > 0) {
    // workgroups [0, gm n S) take the (row tile, tile, piece) triples, the
    // rest exit (whole workgroup, after every barrier above)
    const int gm = (p.M + BM - 1) / BM;
    const int ntl = FSORT ? fs_cnt[0] : p.n_tiles[0];
    const int per = max(gm * ntl, 1);
    s_pieces = min(max((p.split_target + per - 1) / per, 1), p.ksplit);
    if (blockIdx.x == 0 && tid == 0 && p.split_out) p.split_out[0] = s_pieces;
    const int used = gm * ntl * s_pieces;
    if (static_cast<int>(blockIdx.x) >= used) return;
    tile_of_block(gm, ntl, &mt, &nt, &ks, used);
  } else {
    const int gm_all = (MODS && !tlist && p.n_mod > 0) ? p.mod_rt[p.n_mod] : (p.M + BM - 1) / BM;
    tile_of_block(gm_all, tlist ? p.max_tiles : (p.N + BN - 1) / BN, &mt, &nt, &ks, 0, tlist ? 0 : p.group_m);
  }
  // the operands of this workgroup's module: with several modules in the
  // launch, row tiles [mod_rt[m], mod_rt[m+1]) are module m's
  const int mt_grid = mt;
  int Mv = p.M;
  const void* A0v = p.A0;
  const void* A1v = p.A1;
  const void* B1v = p.B1;
  void* outv = p.out;
  float* partv = p.part;
  int64_t ldov = p.ldo;
  uint32_t a0v_bytes = p.a0_bytes, a1_seg_bytes = p.a1_seg_bytes, b1v_bytes = p.b1_bytes;
  if (MODS && !tlist && p.n_mod > 0) {
    int mod = 0;
#pragma unroll
    for (int q = 1; q < kMaxGemmModules; ++q) mod += (q < p.n_mod && mt >= p.mod_rt[q]) ? 1 : 0;
    mod = __builtin_amdgcn_readfirstlane(mod);
    mt -= p.mod_rt[mod];
    Mv = p.mod_M[mod];
    A0v = p.mod_A0[mod]; a0v_bytes = p.mod_a0_bytes[mod];
    A1v = p.mod_A1[mod]; a1_seg_bytes = p.mod_a1_seg_bytes[mod];
    B1v = p.mod_B1[mod]; b1v_bytes = p.mod_b1_bytes[mod];
    outv = p.mod_out[mod]; ldov = p.mod_ldo[mod];
    if (partv) partv += p.mod_col[mod];
  }
  // row stride of the split partials (the modules' total width with several)
  const int64_t part_ld = (MODS && p.part_ld > 0) ? p.part_ld : Mv;
  const int S = s_pieces;
  int j0, jn;
  if (tlist) {
    // whole workgroup, after every barrier above
    if (nt >= (FSORT ? fs_cnt[0] : p.n_tiles[0])) return;
    j0 = FSORT ? fs_tile[nt] : p.tile_start[nt];
    jn = (FSORT ? fs_tile[nt + 1] : p.tile_start[nt + 1]) - j0;
  } else {
    j0 = nt * BN;
    jn = min(BN, p.N - j0);
  }
  const void* A0 = A0v;
  const void* B0 = p.B0;
  uint32_t a0_bytes = a0v_bytes, b0_bytes = p.b0_bytes;
  int64_t lda0 = p.lda0, ldb0 = p.ldb0;
  int K0 = p.K0, K1 = p.K1;
  bool b0_gather = true;
  if (tlist) {
    const int seg = FSORT ? static_cast<int>(fs_key[j0] >> fs_cshift)
                          : (p.tile_seg ? p.tile_seg[nt] : p.sorted_seg[j0]);
    A0 = static_cast<const char*>(A1v) + static_cast<int64_t>(seg) * a1_seg_bytes;
    a0_bytes = a1_seg_bytes; lda0 = p.lda1; K0 = p.K1;
    B0 = B1v; b0_bytes = b1v_bytes; ldb0 = p.ldb1; b0_gather = p.b1_gather != 0;
    K1 = 0;
  }
  const int m0 = mt * BM;
  static_assert(BN <= C::NT, "one token column per thread");

  // ---- token columns of this tile (loads only; stored to LDS below) -------
  int v_perm = 0, v_seg = 0, v_rank = 0;
  if (tid < jn) {
    if (FSORT) {
      v_perm = fs_perm[j0 + tid];
      v_seg = static_cast<int>(fs_key[j0 + tid] >> fs_cshift);
    } else {
      v_perm = p.perm[j0 + tid];
      v_seg = p.sorted_seg ? p.sorted_seg[j0 + tid] : 0;
      if (RANKED) v_rank = p.sorted_rank[j0 + tid];
    }
  }

  // ---- load mapping: this lane's row and chunk in each 1 KB load ------------
  // load j of wave w covers tile rows [RPI*(w + NW*j), +RPI) of A (j < QA) or
  // B; lane l takes row +l/CH and global chunk (l%CH) ^ key(row), stored at
  // slot l%CH.
  const int lrow = lane / C::CH;
  // the key depends on the tile row modulo 16 only, and every wave's rows
  // start at a multiple of 16 plus RPI * wave
  static_assert((C::RPI * C::NW) % 16 == 0, "swizzle period");
  const int lchunk = (lane % C::CH) ^ swz_key<BK>(C::RPI * wave + lrow);
  const uint32_t cbytes = static_cast<uint32_t>(lchunk * 16);
  const uint32_t celem = static_cast<uint32_t>(lchunk * 8);
  // Per-lane byte offsets of this lane's chunk at k = 0, for the dense (0)
  // and adapter (1) operands; kOob marks a row outside the operand (and, for
  // the dense token operand, a column outside the tile).  A k-tile adds its
  // uniform k byte offset: in the dense phase as the load's scalar offset, so
  // a full dense k-tile needs no per-lane arithmetic at all.
  uint32_t a0_v[C::QA], a1_v[C::QA], b0_v[C::QB], b1_v[C::QB];
  int b_jl[C::QB];
#pragma unroll
  for (int j = 0; j < C::QA; ++j) {
    const int m = m0 + C::RPI * (wave + C::NW * j) + lrow;
    const bool ok = m < Mv;
    a0_v[j] = ok ? static_cast<uint32_t>(m) * static_cast<uint32_t>(lda0) * ELT + cbytes : kOob;
    a1_v[j] = ok ? static_cast<uint32_t>(m) * static_cast<uint32_t>(p.lda1) * ELT + cbytes : kOob;
  }
  const __amdgpu_buffer_rsrc_t rA0 = make_rsrc(A0, a0_bytes);
  char* const smem_a = smem + wave * 1024;                  // + stage*SB + j*NW*1024
  char* const smem_b = smem + BM * C::ROWB + wave * 1024;

  // ---- dense k range of this split ----------------------------------------
  const int nk0 = (K0 > 0) ? (K0 + BK - 1) / BK : 0;
  const int nk1 = (K1 > 0) ? (K1 + BK - 1) / BK : 0;
  // With a dense phase, split ks takes its share of the dense k-tiles and the
  // cluster runs ks, ks + S, ks + 2S, ... (all of each run's k-tiles), so the
  // adapter phase is spread over the splits; without one, the splits share
  // the segment's k-tiles.
  int d_lo = 0, d_hi = 0, s_lo = 0, s_hi = 0, q_first = 0, q_step = 1;
  if (nk0 > 0) {
    d_lo = split_lo(nk0, ks, S); d_hi = split_lo(nk0, ks + 1, S);
    s_lo = 0; s_hi = nk1;
    q_first = ks; q_step = S;
  } else {
    s_lo = split_lo(nk1, ks, S); s_hi = split_lo(nk1, ks + 1, S);
  }
  const int nd = d_hi - d_lo, ns = s_hi - s_lo;
  // dense k-tiles that cover a whole BK slice: d_lo .. d_lo + nd_full - 1
  const int nd_full = nd - ((nd > 0 && d_hi * BK > K0) ? 1 : 0);
  auto dk = [&](int i) __attribute__((always_inline)) { return d_lo + i; };   // dense k-tile at position i

  // The weight rows do not depend on the token order: when the first P-1
  // k-tiles are whole dense tiles, their weight loads go out now, in flight
  // while the token columns and cluster runs are set up (the token operand's
  // loads follow once its rows are known).  With four stages the first
  // k-tile's wait below is adjusted for this order.
  const bool early = (P <= 4) && nd_full >= P - 1;
  if (early) {
#pragma unroll
    for (int st = 0; st < P - 1; ++st)
#pragma unroll
      for (int j = 0; j < C::QA; ++j)
        load16_lds(rA0, smem_a + st * C::SB + j * C::NW * 1024, a0_v[j],
                   static_cast<uint32_t>(dk(st) * BK) * ELT);
  }

  // ---- token columns: perm, segment, and segment runs ----------------------
  if (tid < BN) {
    t_perm[tid] = v_perm;
    t_seg[tid] = v_seg;
    if (RANKED) t_rank[tid] = v_rank;
  }
  __syncthreads();
  int n_runs = 0;
  for (int base = 0; base < BN; base += C::NT) {
    const int i = base + tid;
    const bool st = (i < jn) && (i == 0 || t_seg[i] != t_seg[i - 1]);
    const uint64_t bal = __ballot(st);
    if (lane == 0) wave_runs[wave] = __popcll(bal);
    __syncthreads();
    int before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < C::NW; ++w) {
      const int c = wave_runs[w];
      before += (w < wave) ? c : 0;
      total += c;
    }
    if (st) {
      const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
      run_start[n_runs + before + __popcll(bal & lt)] = i;
    }
    n_runs += total;
    __syncthreads();
  }
  if (!(p.sorted_seg && K1 > 0)) n_runs = 0;
  if (tid == 0) run_start[n_runs] = jn;
  __syncthreads();
  // this split's runs: q_first + i q_step, i < my_runs
  const int my_runs = (n_runs > q_first) ? (n_runs - q_first + q_step - 1) / q_step : 0;

  // ---- k-tile schedule: the dense tiles, then each cluster run's tiles ------
  // With ranks, run q takes only its k-tiles of this split below its rank
  // (the k-tiles past a cluster's rank are not visited).  Wave 0 lists the
  // adapter k-tiles in LDS, run by run: .x = first column | columns << 9 |
  // k-tile << 18, .y = segment | rank << 16.
  int n_sched = my_runs * ns;
  if (RANKED && my_runs > 0 && ns > 0) {
    if (wave == 0) {
      int tot = 0;
      for (int base = 0; base < my_runs; base += 64) {
        const int q = q_first + (base + lane) * q_step;
        int c = 0;
        uint32_t ex = 0, ey = 0;
        if (base + lane < my_runs) {
          const int lo = run_start[q], hi = run_start[q + 1];
          const int seg = t_seg[lo];
          const int kl = min(max(t_rank[lo], 0), K1);
          c = max(0, min(s_hi, (kl + BK - 1) / BK) - s_lo);
          ex = static_cast<uint32_t>(lo) | (static_cast<uint32_t>(hi - lo) << 9);
          ey = static_cast<uint32_t>(seg) | (static_cast<uint32_t>(kl) << 16);
        }
        int x = c;                                          // inclusive scan over the wave
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
          const int y = __shfl_up(x, d);
          if (lane >= d) x += y;
        }
        for (int i = 0; i < c; ++i)
          sched[tot + x - c + i] = make_uint2(ex | (static_cast<uint32_t>(s_lo + i) << 18), ey);
        tot += __shfl(x, 63);
      }
      if (lane == 0) n_sched_s = tot;
    }
    __syncthreads();
    n_sched = n_sched_s;
  }
  const int ntiles = nd + n_sched;

  // ---- token operand rows -------------------------------------------------
#pragma unroll
  for (int j = 0; j < C::QB; ++j) {
    const int jl = C::RPI * (wave + C::NW * j) + lrow;
    const uint32_t tok = static_cast<uint32_t>(t_perm[jl]);
    const uint32_t r1 = p.b1_gather ? tok : static_cast<uint32_t>(j0 + jl);
    b_jl[j] = jl;
    const uint32_t r0 = b0_gather ? tok : static_cast<uint32_t>(j0 + jl);
    b0_v[j] = (jl < jn) ? r0 * static_cast<uint32_t>(ldb0) * ELT + cbytes : kOob;
    b1_v[j] = r1 * static_cast<uint32_t>(p.ldb1) * ELT + cbytes;
  }
  const __amdgpu_buffer_rsrc_t rB0 = make_rsrc(B0, b0_bytes);
  const __amdgpu_buffer_rsrc_t rB1 = make_rsrc(B1v, b1v_bytes);
  int lt = 0, lq = 0, lkt = s_lo;

  // L2 prefetch: this lane's weight row or token row (kOob when none)
  uint32_t pf_v = kOob;
  const bool pf_w = __builtin_amdgcn_readfirstlane(wave) < PFW;
  if (PFD > 0) {
    static_assert(PFD == 0 || (BM % (WSPL * PFW) == 0 && BM / WSPL / PFW <= 64 &&
                               BN % (8 * PFW) == 0 && BN / 8 / PFW <= 64), "prefetch lanes");
    if (pf_w) {
      const int m = m0 + WSPL * (wave * (BM / WSPL / PFW) + lane) + (nt % WSPL);
      if (lane < BM / WSPL / PFW && m < Mv) pf_v = static_cast<uint32_t>(m) * static_cast<uint32_t>(lda0) * ELT;
    } else {
      const int jl = 8 * ((wave - PFW) * (BN / 8 / PFW) + lane) + (mt_grid & 7);
      if (lane < BN / 8 / PFW && jl < jn) {
        const uint32_t r0 = b0_gather ? static_cast<uint32_t>(t_perm[jl]) : static_cast<uint32_t>(j0 + jl);
        pf_v = r0 * static_cast<uint32_t>(ldb0) * ELT;
      }
    }
  }
  // dense k-tile ti of this split (ti counted from d_lo; past the whole
  // dense tiles the load touches nothing)
  auto prefetch = [&](int ti) __attribute__((always_inline)) {
    if (PFD > 0)
      load4_lds(pf_w ? rA0 : rB0, pf_sink, (ti < nd_full) ? pf_v : kOob,
                static_cast<uint32_t>(dk(ti) * BK) * ELT);
  };
  // Per-k-tile load state, prepared once per k-tile (the loads themselves may
  // be issued in several groups between the multiply steps).
  struct TileLoad {
    __amdgpu_buffer_rsrc_t rA, rB;
    uint32_t kk, kmask, span, dsel;   // kk: uniform k byte offset of the k-tile
    int lo;
  };
  auto prep_next = [&, jn, n_runs, n_sched, nd, ntiles, s_lo, s_hi, q_first, q_step]() __attribute__((always_inline)) {
    TileLoad L;
    const bool valid = lt < ntiles;
    uint32_t k0, klim;
    if (lt < nd) {
      // dense phase (W X): a wave-uniform branch that touches no LDS, so the
      // steady state pays no lookup latency between barrier and multiply
      L.lo = 0;
      L.span = static_cast<uint32_t>(jn);
      L.rA = rA0;
      L.rB = rB0;
      L.dsel = 0xffffffffu;
      k0 = static_cast<uint32_t>(dk(lt) * BK);
      klim = static_cast<uint32_t>(K0);
    } else if (RANKED) {
      // adapter phase with ranks: the next entry of the schedule (past its
      // end, while the ring runs dry, the loads are masked off)
      const uint2 e = sched[min(lq, max(n_sched - 1, 0))];
      const uint32_t ex = valid ? __builtin_amdgcn_readfirstlane(e.x) : 0u;
      const uint32_t ey = valid ? __builtin_amdgcn_readfirstlane(e.y) : 0u;
      L.lo = static_cast<int>(ex & 511u);
      L.span = (ex >> 9) & 511u;
      const int seg = static_cast<int>(ey & 0xffffu);
      L.rA = make_rsrc(static_cast<const char*>(A1v) + static_cast<int64_t>(seg) * a1_seg_bytes,
                       a1_seg_bytes);
      L.rB = rB1;
      L.dsel = 0u;
      k0 = (ex >> 18) * BK;
      klim = ey >> 16;
      ++lq;
    } else {
      // adapter phase (U_k Z'): one cluster run of the tile per k-tile group
      const int q = min(q_first + lq * q_step, max(n_runs - 1, 0));
      L.lo = run_start[q];
      const int hi = run_start[q + 1];
      const int seg = __builtin_amdgcn_readfirstlane(t_seg[L.lo]);
      L.rA = make_rsrc(static_cast<const char*>(A1v) + static_cast<int64_t>(seg) * a1_seg_bytes,
                       a1_seg_bytes);
      L.rB = rB1;
      L.span = static_cast<uint32_t>(hi - L.lo);
      // phase select by mask arithmetic (a conditional pick between the two
      // offset arrays would make the compiler keep them in scratch memory)
      L.dsel = 0u;
      k0 = static_cast<uint32_t>(lkt * BK);
      klim = static_cast<uint32_t>(K1);
      ++lkt;
      if (lkt >= s_hi) { lkt = s_lo; ++lq; }
    }
    L.kmask = (valid && k0 + celem < klim) ? 0u : kOob;
    L.kk = k0 * ELT;
    ++lt;
    return L;
  };
  // issue loads [g0, g1) of the k-tile (A loads first, then B) into stage st;
  // general form: any phase, per-lane k and column masks
  auto issue = [&](const TileLoad L, int st, int g0, int g1) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < C::QA; ++j)
      if (j >= g0 && j < g1)
        load16_lds(L.rA, smem_a + st * C::SB + j * C::NW * 1024,
                   ((a1_v[j] ^ ((a0_v[j] ^ a1_v[j]) & L.dsel)) + L.kk) | L.kmask);
#pragma unroll
    for (int j = 0; j < C::QB; ++j) {
      if (j + C::QA >= g0 && j + C::QA < g1) {
        const uint32_t jmask = (static_cast<uint32_t>(b_jl[j] - L.lo) < L.span) ? 0u : kOob;
        load16_lds(L.rB, smem_b + st * C::SB + j * C::NW * 1024,
                   ((b1_v[j] ^ ((b0_v[j] ^ b1_v[j]) & L.dsel)) + L.kk) | L.kmask | jmask);
      }
    }
  };
  // fast form: dense phase, whole k-tile; an out-of-range row stays at kOob
  // (plus a k offset below 2^31, still past the end of the operand)
  auto issue_fast = [&](const TileLoad L, int st, int g0, int g1) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < C::QA; ++j)
      if (j >= g0 && j < g1) load16_lds(rA0, smem_a + st * C::SB + j * C::NW * 1024, a0_v[j], L.kk);
#pragma unroll
    for (int j = 0; j < C::QB; ++j)
      if (j + C::QA >= g0 && j + C::QA < g1)
        load16_lds(rB0, smem_b + st * C::SB + j * C::NW * 1024, b0_v[j], L.kk);
  };
  auto load_next = [&](int st) __attribute__((always_inline)) {
    const TileLoad L = prep_next();
    issue(L, st, 0, C::LPT);
  };

  // ---- fragment addresses ---------------------------------------------------
  const int wm = wave / WN, wn = wave % WN;
  const int fr = lane % MB, fg = lane / MB;                 // row in block, k group
  const uint32_t smem_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));
  const uint32_t a_row_addr = smem_base + static_cast<uint32_t>((wm * C::WTM + fr) * C::ROWB);
  const uint32_t b_row_addr = smem_base + static_cast<uint32_t>(BM * C::ROWB + (wn * C::WTN + fr) * C::ROWB);
  uint32_t slot[C::NKS];                                    // swizzled chunk slot per k-step
#pragma unroll
  for (int s2 = 0; s2 < C::NKS; ++s2) {
    const int chunk = s2 * (C::KS / 8) + fg * (MT::KG / 8);
    slot[s2] = static_cast<uint32_t>(((chunk ^ swz_key<BK>(fr)) * 16));
  }

  accv acc[C::FM][C::FN];
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j)
#pragma unroll
      for (int v = 0; v < MT::NACC; ++v) acc[i][j][v] = 0.f;

  // ---- main loop --------------------------------------------------------------
  // Per k-tile t (LDS stage cur), multiply step s uses fragment buffer s % 2:
  //  * steps before the last: the MFMAs of step s are interleaved one by one
  //    with the fragment reads of step s+1 and, in the first half of the
  //    k-tile, with the loads of k-tile t+P-1;
  //  * last step: half of its MFMAs, then the wait for this lane's loads of
  //    k-tile t+1 and the workgroup barrier (after it every wave's loads of
  //    t+1 are in LDS and every wave has finished reading k-tile t-1's stage,
  //    which the next iteration overwrites), then the fragment reads of
  //    k-tile t+1's first step interleaved with the remaining MFMAs.
  // So no multiply step waits on fragment-read latency, and the barrier sits
  // behind MFMAs already issued.
  static_assert(C::NKS % 2 == 0, "fragment buffers alternate across k-tiles");
  constexpr int NM = C::FM * C::FN;                          // MFMAs per step
  constexpr int NR = C::FM + C::FN;                          // fragment reads per step
  constexpr int NLG = C::NKS > 2 ? C::NKS / 2 : 1;           // steps that issue loads
  constexpr int GPS = (C::LPT + NLG - 1) / NLG;              // loads per such step
  // issue slots per multiply step: one per MFMA or fragment read, or one per
  // load where a step has more loads than both (load-heavy, narrow tiles)
  constexpr int NSL0 = NM > NR ? NM : NR;
  constexpr int NSL = NSL0 > GPS ? NSL0 : GPS;
  static_assert(NPF == 0 || GPS < NSL, "a slot for the prefetch");
  bf16x8 fa[2][C::FM], fb[2][C::FN];
  auto read_frag = [&](int buf, int r, uint32_t sa, uint32_t sb, uint32_t sl) __attribute__((always_inline)) {
    if (r < C::FM) lds_read16(fa[buf][r], sa + sl + r * MB * C::ROWB);
    else lds_read16(fb[buf][r - C::FM], sb + sl + (r - C::FM) * MB * C::ROWB);
  };
  auto mma = [&](int buf, int m) __attribute__((always_inline)) {
    const int i = m / C::FN, j = m % C::FN;
    acc[i][j] = MT::mma(fa[buf][i], fb[buf][j], acc[i][j]);
  };

  // prefetch of the first PFD k-tiles after the ring's (waited for with them)
#pragma unroll
  for (int i = 0; i < PFD; ++i) prefetch(P - 1 + i);
  if (early) {
    // weight loads of k-tiles 0..P-2 are out; add their token loads
#pragma unroll
    for (int st = 0; st < P - 1; ++st) {
      TileLoad L;
      L.kk = static_cast<uint32_t>(dk(st) * BK) * ELT;
      issue_fast(L, st, C::QA, C::LPT);
    }
    lt = P - 1;
    wait_vmcnt<(P - 2) * C::QB>();       // k-tile 0's token loads, and all weight loads
  } else {
#pragma unroll
    for (int st = 0; st < P - 1; ++st) load_next(st);
    wait_vmcnt<(P - 2) * C::LPT>();
  }
  __builtin_amdgcn_s_barrier();
#pragma unroll
  for (int r = 0; r < NR; ++r) read_frag(0, r, a_row_addr, b_row_addr, slot[0]);

  // Dense k-tiles that cover a whole BK slice are a prefix of the schedule;
  // while the k-tile being loaded is one of them the loop runs the fast load
  // form (uniform k offset only), then the general form to the end.
  const int nfast = max(0, min(ntiles, nd_full - (P - 1)));
  int cur = 0;   // LDS stage of k-tile t
  int t = 0;
  auto ktile = [&](const TileLoad L, const bool fast) __attribute__((always_inline)) {
    int nst = cur + P - 1; if (nst >= P) nst -= P;         // stage of k-tile t+P-1
    int ncur = cur + 1; if (ncur >= P) ncur -= P;          // stage of k-tile t+1
    const uint32_t sa = a_row_addr + cur * C::SB, sb = b_row_addr + cur * C::SB;
    const uint32_t na = a_row_addr + ncur * C::SB, nb = b_row_addr + ncur * C::SB;
    auto iss = [&](int g0, int g1) __attribute__((always_inline)) {
      if (fast) issue_fast(L, nst, g0, g1);
      else issue(L, nst, g0, g1);
    };
#pragma unroll
    for (int s2 = 0; s2 < C::NKS; ++s2) {
      const int b = s2 & 1;
      wait_lgkmcnt<0>();                                   // step s2's fragments are in
#pragma unroll
      for (int i = 0; i < C::FM; ++i) pin(fa[b][i]);
#pragma unroll
      for (int j = 0; j < C::FN; ++j) pin(fb[b][j]);
      if (s2 + 1 < C::NKS) {
#pragma unroll
        for (int m = 0; m < NSL; ++m) {
          if (m < NM) mma(b, m);
          if (m < NR) read_frag(b ^ 1, m, sa, sb, slot[s2 + 1]);
          if (s2 < NLG && m < GPS) iss(s2 * GPS + m, s2 * GPS + m + 1);
          if (NPF && s2 == NLG - 1 && m == GPS) prefetch(t + P - 1 + PFD);   // after every load
          __builtin_amdgcn_sched_barrier(0);
        }
      } else {
#pragma unroll
        for (int m = 0; m < NM / 2; ++m) {
          mma(b, m);
          __builtin_amdgcn_sched_barrier(0);
        }
        // this lane's loads of k-tile t+1.  In the early order (weight loads
        // of k-tiles 0..2, then their token loads) k-tile 1's token loads
        // are followed by k-tile 2's token loads and k-tile 3's loads only.
        // With prefetches each k-tile's loads are followed by one prefetch
        // load; the prologue's go out before its ring loads.
        if (P == 4 && early && t == 0) wait_vmcnt<(P == 4 ? 2 * C::LPT - C::QA : 0)>();
        else if (P == 3 && NPF && t == 0) wait_vmcnt<(P - 2) * C::LPT + NPF>();
        else wait_vmcnt<(P - 2) * C::LPT + (P - 1) * NPF>();
        __builtin_amdgcn_s_barrier();                      // ... and every wave's
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int m = 0; m < (NM - NM / 2 > NR ? NM - NM / 2 : NR); ++m) {
          if (NM / 2 + m < NM) mma(b, NM / 2 + m);
          if (m < NR) read_frag(b ^ 1, m, na, nb, slot[0]);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    cur = ncur;
  };
  for (; t < nfast; ++t) {
    TileLoad L;                                            // dense k-tile lt, whole
    L.kk = static_cast<uint32_t>(dk(lt) * BK) * ELT;
    ++lt;
    ktile(L, true);
  }
  for (; t < ntiles; ++t) ktile(prep_next(), false);
  wait_lgkmcnt<0>();
  wait_vmcnt<0>();
  __syncthreads();

  if (DIRECT) {
    // ---- epilogue from registers: lane holds rows acc_row(v..v+3) of column l%MB
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
      const int jl = wn * C::WTN + j * MB + lane % MB;
      const bool jok = jl < jn;
      const int64_t orow = p.out_perm ? t_perm[jl] : static_cast<int64_t>(j0 + jl);
#pragma unroll
      for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int v = 0; v < MT::NACC; v += 4) {
          const int m = m0 + wm * C::WTM + i * MB + acc_row<MB>(lane, v);
          if (!jok || m >= Mv) continue;
          const f32x4 val = f32x4{acc[i][j][v], acc[i][j][v + 1], acc[i][j][v + 2], acc[i][j][v + 3]};
          if (partv) {
            *reinterpret_cast<f32x4*>(partv + (static_cast<int64_t>(ks) * p.N + j0 + jl) * part_ld + m) = val;
          } else if (p.out_dtype == 1) {
            uint2 w;
            w.x = f32_to_bf16(val[0]) | (static_cast<uint32_t>(f32_to_bf16(val[1])) << 16);
            w.y = f32_to_bf16(val[2]) | (static_cast<uint32_t>(f32_to_bf16(val[3])) << 16);
            *reinterpret_cast<uint2*>(static_cast<uint16_t*>(outv) + orow * ldov + m) = w;
          } else {
            *reinterpret_cast<f32x4*>(static_cast<float*>(outv) + orow * ldov + m) = val;
          }
        }
    }
    return;
  }

  // ---- epilogue: stage fp32 tile as [token][row], then 16-byte stores ------
  float* stg = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
      const int col = wn * C::WTN + j * MB + lane % MB;
      const int row = wm * C::WTM + i * MB;
#pragma unroll
      for (int v = 0; v < MT::NACC; v += 4)
        *reinterpret_cast<f32x4*>(stg + col * C::ST_ROW + row + acc_row<MB>(lane, v)) =
            f32x4{acc[i][j][v], acc[i][j][v + 1], acc[i][j][v + 2], acc[i][j][v + 3]};
    }
  __syncthreads();

  if (partv) {
    float* part = partv + static_cast<int64_t>(ks) * p.N * part_ld;
    constexpr int CPRO = BM / 4;
    for (int c = tid; c < BN * CPRO; c += C::NT) {
      const int jl = c / CPRO, mc = (c % CPRO) * 4;
      if (jl < jn && m0 + mc < Mv)
        *reinterpret_cast<f32x4*>(part + static_cast<int64_t>(j0 + jl) * part_ld + m0 + mc) =
            *reinterpret_cast<const f32x4*>(stg + jl * C::ST_ROW + mc);
    }
  } else if (p.out_dtype == 1) {
    constexpr int CPRO = BM / 8;
    uint16_t* out = static_cast<uint16_t*>(outv);
    for (int c = tid; c < BN * CPRO; c += C::NT) {
      const int jl = c / CPRO, mc = (c % CPRO) * 8;
      if (jl < jn && m0 + mc < Mv) {
        const float* s = stg + jl * C::ST_ROW + mc;
        const f32x4 lo = *reinterpret_cast<const f32x4*>(s);
        const f32x4 hi = *reinterpret_cast<const f32x4*>(s + 4);
        uint4 v;
        v.x = f32_to_bf16(lo[0]) | (static_cast<uint32_t>(f32_to_bf16(lo[1])) << 16);
        v.y = f32_to_bf16(lo[2]) | (static_cast<uint32_t>(f32_to_bf16(lo[3])) << 16);
        v.z = f32_to_bf16(hi[0]) | (static_cast<uint32_t>(f32_to_bf16(hi[1])) << 16);
        v.w = f32_to_bf16(hi[2]) | (static_cast<uint32_t>(f32_to_bf16(hi[3])) << 16);
        const int64_t row = p.out_perm ? t_perm[jl] : static_cast<int64_t>(j0 + jl);
        *reinterpret_cast<uint4*>(out + row * ldov + m0 + mc) = v;
      }
    }
  } else {
    constexpr int CPRO = BM / 4;
    float* out = static_cast<float*>(outv);
    for (int c = tid; c < BN * CPRO; c += C::NT) {
      const int jl = c / CPRO, mc = (c % CPRO) * 4;
      if (jl < jn && m0 + mc < Mv) {
        const int64_t row = p.out_perm ? t_perm[jl] : static_cast<int64_t>(j0 + jl);
        *reinterpret_cast<f32x4*>(out + row * ldov + m0 + mc) =
            *reinterpret_cast<const f32x4*>(stg + jl * C::ST_ROW + mc);
      }
    }
  }
}

template <int BM, int BN, int BK, int WM, int WN, int MB, int P, int DIRECT = 0, int PFD = 0,
          int WSPL = 1, int FSORT = 0, int RANKED = 0, int MODS = 0>
hipError_t launch_dma1(const GemmParams& p, hipStream_t stream) {
  const int gn = (p.tile_start || FSORT) ? p.max_tiles : (p.N + BN - 1) / BN;
  // row tiles: the modules' together when the launch holds several
  const bool mods = MODS && !(p.tile_start || FSORT) && p.n_mod > 0;
  if (!MODS && p.n_mod > 0) return hipErrorInvalidValue;
  if (mods) {
    if (p.n_mod > kMaxGemmModules || p.mod_rt[0] != 0) return hipErrorInvalidValue;
    for (int m = 0; m < p.n_mod; ++m)
      if (p.mod_rt[m + 1] - p.mod_rt[m] != (p.mod_M[m] + BM - 1) / BM) return hipErrorInvalidValue;
  }
  const int gm = mods ? p.mod_rt[p.n_mod] : (p.M + BM - 1) / BM;
  dim3 grid(gm * gn * p.ksplit);
  if ((p.tile_start || FSORT) && p.split_target > 0) {
    if (!(BM == 64 && BN == 64 && BK == 64)) return hipErrorInvalidValue;   // no adaptive split here
    // gm n S workgroups are used: fewer than gm max_tiles + split_target, and
    // at most gm max_tiles ksplit
    const int64_t gmt = (p.M + BM - 1) / BM;
    grid = dim3(static_cast<unsigned>(std::min<int64_t>(gmt * gn + p.split_target, gmt * gn * p.ksplit)));
  }
  GemmParams q = p;
  // the L2 prefetch splits its lines over groups of kGroupM row tiles
  q.group_m = (p.tile_start || FSORT || PFD > 0) ? 0 : xcd_group_m(gm, (p.N + BN - 1) / BN, p.ksplit);
  hipLaunchKernelGGL((seg_gemm_dma_kernel<BM, BN, BK, WM, WN, MB, P, DIRECT, PFD, WSPL, FSORT, RANKED, MODS>),
                     grid, dim3(WM * WN * 64), 0, stream, q);
  return hipGetLastError();
}

// A segment phase with a rank table takes the RANKED kernel; its schedule
// holds at most two k-tiles per cluster run.
template <int BM, int BN, int BK, int WM, int WN, int MB, int P, int DIRECT = 0, int PFD = 0,
          int WSPL = 1, int FSORT = 0>
hipError_t launch_dma(const GemmParams& p, hipStream_t stream) {
  const bool ranked = p.seg_rank && p.sorted_seg && p.K1 > 0 && !p.tile_start && !FSORT;
  if (p.n_mod > 0) {
    if (ranked || p.tile_start || FSORT) return hipErrorInvalidValue;
    if constexpr (FSORT == 0) return launch_dma1<BM, BN, BK, WM, WN, MB, P, DIRECT, PFD, WSPL, 0, 0, 1>(p, stream);
  }
  if (!ranked) return launch_dma1<BM, BN, BK, WM, WN, MB, P, DIRECT, PFD, WSPL, FSORT>(p, stream);
  if (p.K1 > 2 * BK || !p.sorted_rank) return hipErrorInvalidValue;
  if constexpr (FSORT == 0)
    return launch_dma1<BM, BN, BK, WM, WN, MB, P, DIRECT, PFD, WSPL, 0, 1>(p, stream);
  return hipErrorInvalidValue;
}

template <typename TI, int BM, int BN, int BK, int WM, int WN, int STAGES, int OCC, int MB = 16>
hipError_t launch_cfg(const GemmParams& p, hipStream_t stream) {
  // one linear dimension over (m-tile, n-tile, k-split), remapped in-kernel
  const int gn = p.tile_start ? p.max_tiles : (p.N + BN - 1) / BN;
  dim3 grid(((p.M + BM - 1) / BM) * gn * p.ksplit);
  hipLaunchKernelGGL((seg_gemm_kernel<TI, BM, BN, BK, WM, WN, STAGES, OCC, MB>), grid,
                     dim3(WM * WN * 64), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

// Tile shapes (BM x BN x BK: d_out rows x tokens x k; chosen by the plan from
// measurements on MI355X).  The ring tiles use 16x16x32 MFMA:
//   Large   256 x 256 x  64, 8 waves, 2-stage ring + L2 prefetch      T >= 2048
//   Wide    256 x 128 x  64, 8 waves, 3 stages     many row tiles or d_in >= 8192
//   Mid     128 x 128 x  64, 8 waves, 4 stages     >= 128 tiles
//   Narrow  128 x  64 x 128, 4 waves, 3 stages     other T > 64
//   Decode   64 x  64 x 128, 4 waves, 4 stages     T <= 64
//   Shrink   64 x  64 x  64, 4 waves, 3 stages     the V_k^T X products
//   Small    64 x  64 x  64, register-staged (bf16)
//   F32      64 x  64 x  32, register-staged, fp32 inputs
void tile_dims(Tile tile, int* BM, int* BN, int* BK) {
  switch (tile) {
    case Tile::Large: *BM = 256; *BN = 256; *BK = 64; return;
    case Tile::Wide: *BM = 256; *BN = 128; *BK = 64; return;
    case Tile::Narrow: *BM = 128; *BN = 64; *BK = 128; return;
    case Tile::Decode: *BM = 64; *BN = 64; *BK = 128; return;
    case Tile::Shrink: *BM = 64; *BN = 64; *BK = 64; return;
    case Tile::Mid: *BM = 128; *BN = 128; *BK = 64; return;
    case Tile::Small: *BM = 64; *BN = 64; *BK = 64; return;
    case Tile::F32: *BM = 64; *BN = 64; *BK = 32; return;
  }
}

hipError_t launch_seg_gemm(const GemmParams& p, int in_dtype, Tile tile, hipStream_t stream) {
  // several modules in one launch: the LDS-ring tiles only, without token tiles
  if (p.n_mod > 0 && (in_dtype == 0 || tile == Tile::Small || p.tile_start || p.fs_adapter))
    return hipErrorInvalidValue;
  // explicit token tiles (at most kSegTile columns) only with the 64-wide tiles
  if (p.tile_start &&
      !(tile == Tile::Decode || tile == Tile::Shrink || tile == Tile::Small || tile == Tile::F32))
    return hipErrorInvalidValue;
  // the split chosen on the device exists in the bf16 shrink tile only
  if (p.split_target > 0 && (in_dtype == 0 || tile != Tile::Shrink)) return hipErrorInvalidValue;
  // in-kernel bucketing exists in the bf16 shrink tile only
  if (p.fs_adapter && (in_dtype == 0 || tile != Tile::Shrink || p.N > kFuseSortMaxT || p.tile_start))
    return hipErrorInvalidValue;
  if (in_dtype == 0) return launch_cfg<float, 64, 64, 32, 2, 2, 1, 2, 16>(p, stream);
  switch (tile) {
    case Tile::Large: return launch_dma<256, 256, 64, 4, 2, 16, 2, 1, 6, 4>(p, stream);
    case Tile::Wide: return launch_dma<256, 128, 64, 4, 2, 16, 3, 1>(p, stream);
    case Tile::Narrow: return launch_dma<128, 64, 128, 4, 1, 16, 3, 1>(p, stream);
    case Tile::Decode: return launch_dma<64, 64, 128, 2, 2, 16, 4, 1>(p, stream);
    case Tile::Shrink:
      if (p.fs_adapter) return launch_dma<64, 64, 64, 2, 2, 16, 3, 1, 0, 1, 1>(p, stream);
      return launch_dma<64, 64, 64, 2, 2, 16, 3, 1>(p, stream);
    case Tile::Mid: return launch_dma<128, 128, 64, 4, 2, 16, 4, 1>(p, stream);
    default: return launch_cfg<bf16_t, 64, 64, 64, 2, 2, 2, 2, 32>(p, stream);
  }
}

}  // namespace cts
