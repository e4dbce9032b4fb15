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
// the previous k-tile is multiplied out of LDS (register prefetch, two LDS
// buffers, one barrier per k-tile).  LDS rows are padded by 16 bytes, which
// makes the 16-byte fragment reads of one MFMA conflict-free.
//
// Matrix cores: v_mfma_f32_16x16x32_bf16 (bf16 in, fp32 acc) or
// v_mfma_f32_16x16x4_f32.  Both operands of a product use the same per-lane
// k assignment, so the hardware's internal k order does not matter; the
// accumulator layout is lane l -> column l%16, rows 4*(l/16)+{0..3}.
#include "cts_internal.h"

namespace cts {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr uint32_t kOob = 0x80000000u;   // every operand is < 2^31 bytes

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           static_cast<int>(nbytes), 0x00020000);
}

__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

template <typename TI> struct MfmaTraits;
template <> struct MfmaTraits<bf16_t> {
  static constexpr int EPC = 8;   // elements per 16-byte chunk
  static constexpr int KS = 32;   // k per MFMA
  static constexpr int KG = 8;    // k per lane per MFMA
  typedef bf16x8 frag;
  __device__ static __forceinline__ frag ld(const bf16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }
  __device__ static __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct MfmaTraits<float> {
  static constexpr int EPC = 4;
  static constexpr int KS = 4;
  static constexpr int KG = 1;
  typedef float frag;
  __device__ static __forceinline__ frag ld(const float* p) { return *p; }
  __device__ static __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

template <typename TI, int BM, int BN, int BK, int WM, int WN>
struct Cfg {
  static constexpr int NT = WM * WN * 64;
  static constexpr int EPC = MfmaTraits<TI>::EPC;
  static constexpr int KS = MfmaTraits<TI>::KS;
  static constexpr int CPR = BK / EPC;                // 16-byte chunks per tile row
  static constexpr int RPP = NT / CPR;                // tile rows covered per pass
  static constexpr int LDS_ROW = BK + EPC;            // padded row, elements
  static constexpr int CA = BM / RPP;                 // A chunks per thread
  static constexpr int CB = BN / RPP;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int FM = WTM / 16, FN = WTN / 16;
  static constexpr int AB_BYTES = 2 * (BM + BN) * LDS_ROW * (int)sizeof(TI);
  static constexpr int ST_ROW = BM + 4;               // staged fp32 row (per token)
  static constexpr int ST_BYTES = BN * ST_ROW * 4;
  static constexpr int SMEM = AB_BYTES > ST_BYTES ? AB_BYTES : ST_BYTES;
  static_assert(NT % CPR == 0 && BM % RPP == 0 && BN % RPP == 0, "chunk split");
  static_assert(WTM % 16 == 0 && WTN % 16 == 0 && BK % KS == 0, "tile shape");
};

__device__ __forceinline__ int split_lo(int n, int ks, int S) { return (int)((int64_t)n * ks / S); }

template <typename TI, int BM, int BN, int BK, int WM, int WN>
__global__ __launch_bounds__(WM * WN * 64) void seg_gemm_kernel(const GemmParams p) {
  using C = Cfg<TI, BM, BN, BK, WM, WN>;
  using MT = MfmaTraits<TI>;
  typedef typename MT::frag frag;
  constexpr uint32_t ELT = sizeof(TI);

  __shared__ __attribute__((aligned(16))) char smem[C::SMEM];
  __shared__ int32_t t_perm[BN];
  __shared__ int32_t t_seg[BN];
  __shared__ int32_t run_start[BN + 1];
  __shared__ int32_t wave_runs[C::NT / 64];

  TI* smA = reinterpret_cast<TI*>(smem);
  TI* smB = smA + 2 * BM * C::LDS_ROW;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = blockIdx.x * BM;
  const int j0 = blockIdx.y * BN;
  const int ks = blockIdx.z;
  const int S = p.ksplit;
  const int jn = min(BN, p.N - j0);   // valid token columns in this tile

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

  uint32_t a0_row[C::CA], b0_row[C::CB];
#pragma unroll
  for (int i = 0; i < C::CA; ++i) {
    const int m = m0 + row0 + i * C::RPP;
    a0_row[i] = (m < p.M) ? static_cast<uint32_t>(m) * static_cast<uint32_t>(p.lda0) * ELT : kOob;
  }
#pragma unroll
  for (int i = 0; i < C::CB; ++i) {
    const int jl = row0 + i * C::RPP;
    b0_row[i] = (jl < jn) ? static_cast<uint32_t>(t_perm[jl]) * static_cast<uint32_t>(p.ldb0) * ELT : kOob;
  }

  u32x4 ra[C::CA], rb[C::CB];

  // issue the global loads of k-tile t into ra/rb
  auto load_tile = [&](int t) __attribute__((always_inline)) {
    if (t < nd) {
      const uint32_t k = static_cast<uint32_t>((d_lo + t) * BK) + kc * C::EPC;
      const bool kok = k < static_cast<uint32_t>(p.K0);
      const uint32_t kb = k * ELT;
#pragma unroll
      for (int i = 0; i < C::CA; ++i) ra[i] = load16(rA0, (kok && a0_row[i] != kOob) ? a0_row[i] + kb : kOob);
#pragma unroll
      for (int i = 0; i < C::CB; ++i) rb[i] = load16(rB0, (kok && b0_row[i] != kOob) ? b0_row[i] + kb : kOob);
    } else {
      const int q = (t - nd) / ns, kt = s_lo + (t - nd) % ns;
      const int lo = run_start[q], hi = run_start[q + 1];
      const int seg = __builtin_amdgcn_readfirstlane(t_seg[lo]);
      const __amdgpu_buffer_rsrc_t rA1 = make_rsrc(
          static_cast<const char*>(p.A1) + static_cast<int64_t>(seg) * p.a1_seg_bytes, p.a1_seg_bytes);
      const uint32_t k = static_cast<uint32_t>(kt * BK) + kc * C::EPC;
      const bool kok = k < static_cast<uint32_t>(p.K1);
      const uint32_t kb = k * ELT;
#pragma unroll
      for (int i = 0; i < C::CA; ++i) {
        const int m = m0 + row0 + i * C::RPP;
        ra[i] = load16(rA1, (kok && m < p.M) ? static_cast<uint32_t>(m) * static_cast<uint32_t>(p.lda1) * ELT + kb : kOob);
      }
#pragma unroll
      for (int i = 0; i < C::CB; ++i) {
        const int jl = row0 + i * C::RPP;
        const bool ok = kok && jl >= lo && jl < hi;
        const uint32_t row = p.b1_gather ? static_cast<uint32_t>(t_perm[jl]) : static_cast<uint32_t>(j0 + jl);
        rb[i] = load16(rB1, ok ? row * static_cast<uint32_t>(p.ldb1) * ELT + kb : kOob);
      }
    }
  };
  auto store_tile = [&](int buf) __attribute__((always_inline)) {
    TI* a = smA + buf * BM * C::LDS_ROW + row0 * C::LDS_ROW + kc * C::EPC;
    TI* b = smB + buf * BN * C::LDS_ROW + row0 * C::LDS_ROW + kc * C::EPC;
#pragma unroll
    for (int i = 0; i < C::CA; ++i) *reinterpret_cast<u32x4*>(a + i * C::RPP * C::LDS_ROW) = ra[i];
#pragma unroll
    for (int i = 0; i < C::CB; ++i) *reinterpret_cast<u32x4*>(b + i * C::RPP * C::LDS_ROW) = rb[i];
  };

  const int wm = wave / WN, wn = wave % WN;
  f32x4 acc[C::FM][C::FN];
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int frow = lane & 15, fk = (lane >> 4) * MT::KG;

  if (ntiles > 0) { load_tile(0); store_tile(0); }
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int cur = t & 1;
    if (t + 1 < ntiles) load_tile(t + 1);
    const TI* a = smA + cur * BM * C::LDS_ROW + (wm * C::WTM + frow) * C::LDS_ROW + fk;
    const TI* b = smB + cur * BN * C::LDS_ROW + (wn * C::WTN + frow) * C::LDS_ROW + fk;
#pragma unroll
    for (int kk = 0; kk < BK; kk += C::KS) {
      frag fa[C::FM], fb[C::FN];
#pragma unroll
      for (int i = 0; i < C::FM; ++i) fa[i] = MT::ld(a + i * 16 * C::LDS_ROW + kk);
#pragma unroll
      for (int j = 0; j < C::FN; ++j) fb[j] = MT::ld(b + j * 16 * C::LDS_ROW + kk);
#pragma unroll
      for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j) acc[i][j] = MT::mma(fa[i], fb[j], acc[i][j]);
    }
    if (t + 1 < ntiles) store_tile(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: stage fp32 tile as [token][row], then 16-byte stores ------
  float* st = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
      const int col = wn * C::WTN + j * 16 + (lane & 15);
      const int row = wm * C::WTM + i * 16 + (lane >> 4) * 4;
      *reinterpret_cast<f32x4*>(st + col * C::ST_ROW + row) = acc[i][j];
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

template <typename TI, int BM, int BN, int BK, int WM, int WN>
hipError_t launch_cfg(const GemmParams& p, hipStream_t stream) {
  dim3 grid((p.M + BM - 1) / BM, (p.N + BN - 1) / BN, p.ksplit);
  hipLaunchKernelGGL((seg_gemm_kernel<TI, BM, BN, BK, WM, WN>), grid, dim3(WM * WN * 64), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

void tile_dims(Tile tile, int* BM, int* BN, int* BK) {
  switch (tile) {
    case Tile::Large: *BM = 128; *BN = 128; *BK = 64; return;
    case Tile::Small: *BM = 64; *BN = 64; *BK = 64; return;
    case Tile::F32: *BM = 64; *BN = 64; *BK = 32; return;
  }
}

hipError_t launch_seg_gemm(const GemmParams& p, int in_dtype, Tile tile, hipStream_t stream) {
  if (in_dtype == 0) return launch_cfg<float, 64, 64, 32, 2, 2>(p, stream);
  if (tile == Tile::Large) return launch_cfg<bf16_t, 128, 128, 64, 2, 2>(p, stream);
  return launch_cfg<bf16_t, 64, 64, 64, 2, 2>(p, stream);
}

}  // namespace cts
