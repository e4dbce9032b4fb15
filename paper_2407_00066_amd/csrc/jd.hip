// Offline compressor: joint diagonalization of a LoRA collection by the
// eigenvalue iteration of App. A.2 and the clustering of App. A.3, fp32.
//
// One iteration from the pair (U, V) (bases as [d][r] row-major):
//   project:  P_i = A_i V, Q_i = B_i^T U          (r_l x r per LoRA, fp32 MFMA)
//             C_i = (P_i P_i^T) Q_i, D_i = (Q_i Q_i^T) P_i   (in LDS)
//   expand:   U' = sum_i B_i C_i, V' = sum_i A_i^T D_i   (fp32 MFMA, split over
//             the collection, partials summed in fixed order)
//   orthogonalize U', V' by CholeskyQR2 (Gram, Cholesky and triangular
//   inverse in one workgroup, X R^-1), and the convergence measure.
// C_i and D_i regroup the paper's chain B_i (A_i V)(V^T A_i^T)(B_i^T U) as
// B_i ((A_i V)(A_i V)^T)(B_i^T U): the same product, with r_l x r_l inner
// Gram matrices.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>
#include <vector>

#include "cts.h"
#include "cts_compress.h"
#include "cts_internal.h"

namespace cts {
namespace {

constexpr int kJT = 256;        // threads per workgroup
constexpr int kBK = 32;         // k per staged tile
constexpr int kTM = 64;         // rows per output tile
constexpr int kRMax = 128;      // largest JD rank
constexpr int kALD = kBK + 4;   // A tile, m-major: row stride (floats)
constexpr int kAML = kTM + 16;  // A tile, k-major: row stride
constexpr int kAS = (kTM * kALD > kBK * kAML) ? kTM * kALD : kBK * kAML;
// B tile (k-major, r columns): row stride.  It is 16 or 48 mod 64 floats, so
// the four k rows one MFMA reads fall on different LDS banks.
__host__ __device__ constexpr int b_ld(int r) { return r + (((r / 16) & 1) ? 32 : 16); }
// floats per staging buffer (A tile, then B tile) for rank 16 NB
template <int NB>
__host__ __device__ constexpr int stage_floats() { return kAS + kBK * b_ld(16 * NB); }
constexpr int kEpLd = kRMax + 1;   // epilogue rows (odd stride)
constexpr int kGramRows = 256;     // rows per Gram partial
constexpr int kMaxKm = 100;        // k-means iterations
constexpr int kExpIds = 2048;      // LoRA ids an expansion workgroup stages in LDS
constexpr int kMaxExpSplit = 16;   // most pieces of the collection in the expansion

__device__ __forceinline__ f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------- loaders
// A loader fills slot e (0 <= e < 512: 64 x 32 floats as float4) of the A tile
// at k0 and gives its LDS offset; a B loader fills slot e (< 8 r) of the
// 32 x r B tile.  Out-of-range slots read zeros.

// A loader is called as la(u, e, k0, off) with e = threadIdx.x + u * kJT.
static_assert(kTM * kBK / 4 / kJT == 2, "two A slots per thread");

// P_i = A_i V, with the row address of each of the thread's two A slots
// computed once (the LoRA id lookup is off the k loop): rows m = (LoRA q of
// the group, row l), k along d_in.
struct LoadLoraRowsP {
  const float* p[2];
  int off[2], kq4[2], d_in;
  __device__ LoadLoraRowsP(const float* A, const int32_t* lidx, int q0, int nq, int r_l, int d_in_)
      : d_in(d_in_) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int e = threadIdx.x + u * kJT;
      const int m = e >> 3, kq = e & 7;
      off[u] = m * kALD + 4 * kq;
      kq4[u] = 4 * kq;
      const int q = m / r_l, l = m - q * r_l;
      p[u] = (q < nq) ? A + (static_cast<int64_t>(lidx[q0 + q]) * r_l + l) * d_in + 4 * kq : nullptr;
    }
  }
  __device__ float4 operator()(int u, int, int k0, int& o) const {
    o = off[u];
    if (!p[u] || k0 + kq4[u] >= d_in) return float4{0.f, 0.f, 0.f, 0.f};
    return *reinterpret_cast<const float4*>(p[u] + k0);
  }
};

// Q_i = B_i^T U likewise: k = output row o, m = (LoRA q, column l); a LoRA's
// 32 x r_l block of rows o is contiguous.
struct LoadLoraBtP {
  const float* p[2];
  int off[2], kk[2], r_l, d_out;
  __device__ LoadLoraBtP(const float* B, const int32_t* lidx, int q0, int nq, int r_l_, int d_out_)
      : r_l(r_l_), d_out(d_out_) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int e = threadIdx.x + u * kJT;
      const int per = 8 * r_l;
      const int q = e / per, rem = e - q * per;
      const int k = rem / (r_l >> 2), l = 4 * (rem - k * (r_l >> 2));
      off[u] = k * kAML + q * r_l + l;
      kk[u] = k;
      p[u] = (q < nq) ? B + static_cast<int64_t>(lidx[q0 + q]) * d_out * r_l + static_cast<int64_t>(k) * r_l + l
                      : nullptr;
    }
  }
  __device__ float4 operator()(int u, int, int k0, int& o) const {
    o = off[u];
    if (!p[u] || k0 + kk[u] >= d_out) return float4{0.f, 0.f, 0.f, 0.f};
    return *reinterpret_cast<const float4*>(p[u] + static_cast<int64_t>(k0) * r_l);
  }
};

// U' = sum B_i C_i: rows m = output row o, k = flat (LoRA, l) index f; a
// LoRA's 64 x w block (w = min(r_l, 32) columns from l0) is read row by row.
// LoRA q of the list is ids[q - id0] (ids: the workgroup's slice of the list
// staged in LDS when kLds, read with LDS loads, else the list itself);
// r_l = 1 << lg.
template <bool kLds>
__device__ __forceinline__ int list_id(const int32_t* ids, int i) {
  if constexpr (kLds) return ((const __attribute__((address_space(3))) int32_t*)ids)[i];
  return ids[i];
}

template <bool kLds>
struct LoadExpandB {
  const float* B; const int32_t* ids; int id0, lg, r_l, d_out, o0, f_end;
  __device__ float4 operator()(int, int e, int k0, int& off) const {
    const int w = r_l < kBK ? r_l : kBK;
    const int w4 = w >> 2;
    const int j4 = e % w4, m = (e / w4) & (kTM - 1), qq = e / (w4 * kTM);
    off = m * kALD + qq * w + 4 * j4;
    const int f = k0 + qq * w + 4 * j4;       // k0: flat index of the tile
    const int o = o0 + m;
    if (f >= f_end || o >= d_out) return float4{0.f, 0.f, 0.f, 0.f};
    const int q = f >> lg, l = f & (r_l - 1);
    const int64_t base = static_cast<int64_t>(list_id<kLds>(ids, q - id0)) * d_out * r_l;
    return *reinterpret_cast<const float4*>(B + base + static_cast<int64_t>(o) * r_l + l);
  }
};

// V' = sum A_i^T D_i: k = flat (LoRA, l), m = input column c.
template <bool kLds>
struct LoadExpandA {
  const float* A; const int32_t* ids; int id0, lg, r_l, d_in, c0, f_end;
  __device__ float4 operator()(int, int e, int k0, int& off) const {
    const int kk = e >> 4, m4 = e & 15;
    off = kk * kAML + 4 * m4;
    const int f = k0 + kk, c = c0 + 4 * m4;
    if (f >= f_end || c >= d_in) return float4{0.f, 0.f, 0.f, 0.f};
    const int q = f >> lg, l = f & (r_l - 1);
    const int64_t row = static_cast<int64_t>(list_id<kLds>(ids, q - id0)) * r_l + l;
    return *reinterpret_cast<const float4*>(A + row * d_in + c);
  }
};

// B tile: rows k of an [K][r] array (a basis, or C / D rows).
struct LoadRowsR {
  const float* X; int r, K;
  __device__ float4 operator()(int, int e, int k0, int& off) const {
    const int r4 = r >> 2;
    const int kk = e / r4, n = 4 * (e - kk * r4);
    off = kk * b_ld(r) + n;
    const int k = k0 + kk;
    if (k >= K) return float4{0.f, 0.f, 0.f, 0.f};
    return *reinterpret_cast<const float4*>(X + static_cast<int64_t>(k) * r + n);
  }
};

// acc[nb] += A(rows 16 w + ..., k) B(k, 16 nb + ...) over k in [k_begin,
// k_end), tiles of 32 double-buffered through registers; NB = r / 16 column
// blocks.  Lane l of wave w holds rows 16 w + 4 (l / 16) + v, column
// 16 nb + l % 16 of block nb.
template <int NB, bool AKM, typename LA, typename LB>
__device__ void tile_gemm(float* smem, int k_begin, int k_end, const LA& la, const LB& lb, f32x4 (&acc)[NB]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 15, fk = lane >> 4;
  constexpr int R = 16 * NB;
  constexpr int NBS = 8 * R;                              // B float4 slots
  constexpr int NAQ = kTM * kBK / 4 / kJT;                // 2 A slots per thread
  constexpr int NBQ = (NBS + kJT - 1) / kJT;              // 1..4 B slots per thread
  // two register sets: while k-tile t is multiplied from LDS, the loads of
  // k-tiles t+1 (issued one step earlier) and t+2 are in flight
  float4 ra[2][NAQ], rb[2][NBQ];
  int oa[2][NAQ], ob[2][NBQ];
  const int nt = (k_end - k_begin + kBK - 1) / kBK;
  auto fetch = [&](int t, float4 (&ra_)[NAQ], float4 (&rb_)[NBQ], int (&oa_)[NAQ], int (&ob_)[NBQ]) {
    const int k0 = k_begin + t * kBK;
#pragma unroll
    for (int u = 0; u < NAQ; ++u) ra_[u] = la(u, tid + u * kJT, k0, oa_[u]);
#pragma unroll
    for (int u = 0; u < NBQ; ++u)
      if (NBS % kJT == 0 || tid + u * kJT < NBS) rb_[u] = lb(u, tid + u * kJT, k0, ob_[u]);
  };
  auto stash = [&](int buf, const float4 (&ra_)[NAQ], const float4 (&rb_)[NBQ], const int (&oa_)[NAQ],
                   const int (&ob_)[NBQ]) {
    float* As = smem + buf * stage_floats<NB>();
    float* Bs = As + kAS;
#pragma unroll
    for (int u = 0; u < NAQ; ++u) *reinterpret_cast<float4*>(As + oa_[u]) = ra_[u];
#pragma unroll
    for (int u = 0; u < NBQ; ++u)
      if (NBS % kJT == 0 || tid + u * kJT < NBS) *reinterpret_cast<float4*>(Bs + ob_[u]) = rb_[u];
  };
  if (nt <= 0) return;
  const int m = 16 * wave + fr;
  auto multiply = [&](int buf) {
    const float* As = smem + buf * stage_floats<NB>();
    const float* Bs = As + kAS;
#pragma unroll
    for (int s = 0; s < kBK / 4; ++s) {
      const int k = 4 * s + fk;
      const float a = AKM ? As[k * kAML + m] : As[m * kALD + k];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[nb] = mfma4(a, Bs[k * b_ld(R) + 16 * nb + fr], acc[nb]);
    }
  };
  fetch(0, ra[0], rb[0], oa[0], ob[0]);
  if (nt > 1) fetch(1, ra[1], rb[1], oa[1], ob[1]);
  stash(0, ra[0], rb[0], oa[0], ob[0]);
  __syncthreads();
  // step t (parity P = t & 1): loads of t+2 into set P (stashed at step t-1),
  // multiply k-tile t from LDS buffer P, stash set 1-P (k-tile t+1) into
  // buffer 1-P.  Unrolled by two so that the register sets are static.
  auto step = [&](int t, float4 (&raP)[NAQ], float4 (&rbP)[NBQ], int (&oaP)[NAQ], int (&obP)[NBQ],
                  float4 (&raQ)[NAQ], float4 (&rbQ)[NBQ], int (&oaQ)[NAQ], int (&obQ)[NBQ], int bufP) {
    if (t + 2 < nt) fetch(t + 2, raP, rbP, oaP, obP);
    multiply(bufP);
    if (t + 1 < nt) stash(bufP ^ 1, raQ, rbQ, oaQ, obQ);
    __syncthreads();
  };
  for (int t = 0; t < nt; t += 2) {
    step(t, ra[0], rb[0], oa[0], ob[0], ra[1], rb[1], oa[1], ob[1], 0);
    if (t + 1 < nt) step(t + 1, ra[1], rb[1], oa[1], ob[1], ra[0], rb[0], oa[0], ob[0], 1);
  }
}

template <int NB>
__device__ __forceinline__ void zero_acc(f32x4 (&acc)[NB]) {
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// accumulators -> LDS rows [64][kEpLd]
template <int NB>
__device__ __forceinline__ void acc_to_lds(const f32x4 (&acc)[NB], float* dst) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int fr = lane & 15, fk = lane >> 4;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int v = 0; v < 4; ++v) dst[(16 * wave + 4 * fk + v) * kEpLd + 16 * nb + fr] = acc[nb][v];
}

// ------------------------------------------------------------ project kernels
// jd_pq_kernel: partial P or Q rows of a group of 64 / r_l LoRAs over one
// half of the reduction; jd_combine_kernel: sums the halves and forms the
// per-LoRA products of the requested mode.

struct PqArgs {
  const float* A; const float* B; const float* V; const float* U;
  const int32_t* lidx; int m;
  int r_l, d_in, d_out;
  float* part;                  // [split][2][m * r_l][r]
  int split;                    // pieces of the reduction (blockIdx.z)
  int zbase;                    // blockIdx.y + zbase: 0 = P, 1 = Q
};

template <int NB>
__global__ __launch_bounds__(kJT) void jd_pq_kernel(const PqArgs a) {
  __shared__ __attribute__((aligned(16))) float smem[2 * stage_floats<NB>()];
  constexpr int r = 16 * NB;
  const int lpw = kTM / a.r_l;
  const int q0 = blockIdx.x * lpw;
  const int nq = min(lpw, a.m - q0);
  if (nq <= 0) return;
  const bool isq = blockIdx.y + a.zbase == 1;
  const int ks = blockIdx.z;
  const int d = isq ? a.d_out : a.d_in;
  const int ntile = (d + kBK - 1) / kBK;
  const int k_lo = (ntile * ks / a.split) * kBK;
  const int k_hi = min(d, (ntile * (ks + 1) / a.split) * kBK);
  f32x4 acc[NB];
  zero_acc(acc);
  if (isq)
    tile_gemm<NB, true>(smem, k_lo, k_hi, LoadLoraBtP(a.B, a.lidx, q0, nq, a.r_l, a.d_out),
                        LoadRowsR{a.U, r, k_hi}, acc);
  else
    tile_gemm<NB, false>(smem, k_lo, k_hi, LoadLoraRowsP(a.A, a.lidx, q0, nq, a.r_l, a.d_in),
                         LoadRowsR{a.V, r, k_hi}, acc);
  const int64_t rows_all = static_cast<int64_t>(a.m) * a.r_l;
  float* out = a.part + ((static_cast<int64_t>(ks) * 2 + (isq ? 1 : 0)) * rows_all +
                         static_cast<int64_t>(q0) * a.r_l) * r;
  const int rows = nq * a.r_l;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int fr = lane & 15, fq = lane >> 4;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = 16 * wave + 4 * fq + v;
      if (row < rows) out[static_cast<int64_t>(row) * r + 16 * nb + fr] = acc[nb][v];
    }
}

struct ProjArgs {
  const int32_t* lidx; int m;
  int r_l;
  const float* part;            // from jd_pq_kernel
  int split;                    // its pieces of the reduction
  int mode;                     // 0: C, D   1: Sigma   2: score   3: C = P diag(s)
                                // 4: D = Q diag(s)   5: w = colsum(Q o P)
  const float* sdiag;           // modes 3, 4: [n][r] diagonals (by id)
  float* wout;                  // mode 5: [n][r] (by id)
  const float* w2;              // mode 0: per-LoRA weight of C, D (by id), or null
  const float* sscale;          // mode 1: per-LoRA scale of Sigma (by id), or null
  float* C; float* D;           // [m][r_l][r] by list position
  float* Sigma;                 // [n][r][r] by id
  float* score; int ld_score, score_col;
};

constexpr int kProjSmem = 2 * kTM * kEpLd + 2 * kTM * 64;

template <int NB>
__global__ __launch_bounds__(kJT) void jd_combine_kernel(const ProjArgs a) {
  __shared__ __attribute__((aligned(16))) float smem[kProjSmem];
  const int lpw = kTM / a.r_l;                       // LoRAs per workgroup
  const int q0 = blockIdx.x * lpw;
  const int nq = min(lpw, a.m - q0);
  if (nq <= 0) return;
  const int tid = threadIdx.x;
  constexpr int r = 16 * NB;
  const int r_l = a.r_l;
  const int rows = nq * r_l;
  float* Ps = smem;
  float* Qs = smem + kTM * kEpLd;
  {
    // the pieces summed in order; every load of a piece is issued before any
    // is used, and a half the mode does not read is not loaded
    const bool need_p = a.mode != 4, need_q = a.mode != 3;
    constexpr int EPT = kTM * r / kJT;                // elements per thread
    const int64_t rows_all = static_cast<int64_t>(a.m) * r_l;
    const float* base = a.part + static_cast<int64_t>(q0) * r_l * r;
    float pv[EPT], qv[EPT];
#pragma unroll
    for (int u = 0; u < EPT; ++u) pv[u] = qv[u] = 0.f;
    for (int ks = 0; ks < a.split; ++ks) {
      const float* bp = base + (static_cast<int64_t>(ks) * 2) * rows_all * r;
      const float* bq = bp + rows_all * r;
      float lp[EPT], lq[EPT];
#pragma unroll
      for (int u = 0; u < EPT; ++u) {
        const int e = tid + u * kJT;
        const bool in = e < rows * r;
        lp[u] = (in && need_p) ? bp[e] : 0.f;
        lq[u] = (in && need_q) ? bq[e] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < EPT; ++u) {
        pv[u] += lp[u];
        qv[u] += lq[u];
      }
    }
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
      const int e = tid + u * kJT;
      Ps[(e / r) * kEpLd + e % r] = pv[u];
      Qs[(e / r) * kEpLd + e % r] = qv[u];
    }
  }
  __syncthreads();

  if (a.mode == 3 || a.mode == 4) {
    // JD-Diag: C_q = P_q diag(s_q) (mode 3) or D_q = Q_q diag(s_q) (mode 4)
    const float* X = a.mode == 3 ? Ps : Qs;
    float* out = a.mode == 3 ? a.C : a.D;
    for (int e = tid; e < rows * r; e += kJT) {
      const int row = e / r, j = e - row * r;
      const int id = a.lidx[q0 + row / r_l];
      out[(static_cast<int64_t>(q0) * r_l + row) * r + j] = X[row * kEpLd + j] * a.sdiag[static_cast<int64_t>(id) * r + j];
    }
    return;
  }
  if (a.mode == 5) {
    // w_q[j] = sum_l Q_q[l][j] P_q[l][j] = (U^T B_q o V^T A_q^T) 1
    for (int e = tid; e < nq * r; e += kJT) {
      const int q = e / r, j = e - q * r;
      float w = 0.f;
      for (int l = 0; l < r_l; ++l) w = fmaf(Qs[(q * r_l + l) * kEpLd + j], Ps[(q * r_l + l) * kEpLd + j], w);
      a.wout[static_cast<int64_t>(a.lidx[q0 + q]) * r + j] = w;
    }
    return;
  }
  if (a.mode == 0) {
    // G_q = P_q P_q^T, H_q = Q_q Q_q^T (r_l x r_l per LoRA)
    float* Gs = Qs + kTM * kEpLd;
    float* Hs = Gs + kTM * 64;
    if (r_l <= 16) {
      // r_l divides 16, so every LoRA's rows sit inside one 16-row block:
      // G_q and H_q are the LoRA blocks on the diagonal of the 16 x 16
      // diagonal tiles of P P^T and Q Q^T (fp32 MFMA; wave w takes rows
      // 16 w .. 16 w + 15).  The tiles, zero off the LoRA blocks, then
      // multiply Q and P as block-diagonal matrices: C = w G Q, D = w H P.
      // Each tile is written and read by its own wave only.
      const int lane = tid & 63, wave = tid >> 6;
      const int fr = lane & 15, fk = lane >> 4;
      const int rb = 16 * wave;
      f32x4 g = {0.f, 0.f, 0.f, 0.f}, h = {0.f, 0.f, 0.f, 0.f};
      for (int k0 = 0; k0 < r; k0 += 4) {
        const float pv = Ps[(rb + fr) * kEpLd + k0 + fk];
        const float qv = Qs[(rb + fr) * kEpLd + k0 + fk];
        g = mfma4(pv, pv, g);
        h = mfma4(qv, qv, h);
      }
      float* Gt = Gs + wave * 16 * 17;
      float* Ht = Hs + wave * 16 * 17;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = 4 * fk + v;
        const bool same = i / r_l == fr / r_l;
        Gt[i * 17 + fr] = same ? g[v] : 0.f;
        Ht[i * 17 + fr] = same ? h[v] : 0.f;
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        f32x4 c = {0.f, 0.f, 0.f, 0.f}, d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const int k = 4 * ks + fk;
          c = mfma4(Gt[fr * 17 + k], Qs[(rb + k) * kEpLd + 16 * nb + fr], c);
          d = mfma4(Ht[fr * 17 + k], Ps[(rb + k) * kEpLd + 16 * nb + fr], d);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = rb + 4 * fk + v;
          if (row < rows) {
            const int q = row / r_l;
            const float w = a.w2 ? a.w2[a.lidx[q0 + q]] : 1.f;
            const int64_t f = static_cast<int64_t>(q0) * r_l + row;
            a.C[f * r + 16 * nb + fr] = c[v] * w;
            a.D[f * r + 16 * nb + fr] = d[v] * w;
          }
        }
      }
      return;
    }
    const int ng = rows * r_l;                        // entries of all G_q
    for (int e = tid; e < ng; e += kJT) {
      const int row = e / r_l, l2 = e - row * r_l;
      const int q = row / r_l;
      const float* p1 = Ps + row * kEpLd;
      const float* p2 = Ps + (q * r_l + l2) * kEpLd;
      const float* s1 = Qs + row * kEpLd;
      const float* s2 = Qs + (q * r_l + l2) * kEpLd;
      float g = 0.f, h = 0.f;
#pragma unroll 8
      for (int j = 0; j < r; ++j) {
        g = fmaf(p1[j], p2[j], g);
        h = fmaf(s1[j], s2[j], h);
      }
      Gs[e] = g;
      Hs[e] = h;
    }
    __syncthreads();
    // C_q = w G_q Q_q, D_q = w H_q P_q
    const int nc = rows * r;
    for (int e = tid; e < nc; e += kJT) {
      const int row = e / r, j = e - row * r;
      const int q = row / r_l;
      const float* g = Gs + row * r_l;
      const float* h = Hs + row * r_l;
      float c = 0.f, d = 0.f;
      for (int l2 = 0; l2 < r_l; ++l2) {
        c = fmaf(g[l2], Qs[(q * r_l + l2) * kEpLd + j], c);
        d = fmaf(h[l2], Ps[(q * r_l + l2) * kEpLd + j], d);
      }
      const float w = a.w2 ? a.w2[a.lidx[q0 + q]] : 1.f;
      const int64_t f = static_cast<int64_t>(q0) * r_l + row;
      a.C[f * r + j] = c * w;
      a.D[f * r + j] = d * w;
    }
    return;
  }
  // Sigma_q[x][y] = sum_l Q_q[l][x] P_q[l][y]
  constexpr int rr = r * r;
  if (a.mode == 1) {
    for (int e = tid; e < nq * rr; e += kJT) {
      const int q = e / rr, xy = e - q * rr, x = xy / r, y = xy - x * r;
      float s = 0.f;
      for (int l = 0; l < r_l; ++l) s = fmaf(Qs[(q * r_l + l) * kEpLd + x], Ps[(q * r_l + l) * kEpLd + y], s);
      const int id = a.lidx[q0 + q];
      if (a.sscale) s *= a.sscale[id];
      a.Sigma[static_cast<int64_t>(id) * rr + xy] = s;
    }
    return;
  }
  // mode 2: score_q = ||Sigma_q||_F^2 (sum per LoRA in a fixed order)
  float* red = Qs + kTM * kEpLd;                     // [lpw][kJT]
  for (int q = 0; q < nq; ++q) {
    float acc = 0.f;
    for (int xy = tid; xy < rr; xy += kJT) {
      const int x = xy / r, y = xy - x * r;
      float s = 0.f;
      for (int l = 0; l < r_l; ++l) s = fmaf(Qs[(q * r_l + l) * kEpLd + x], Ps[(q * r_l + l) * kEpLd + y], s);
      acc = fmaf(s, s, acc);
    }
    red[q * kJT + tid] = acc;
  }
  __syncthreads();
  if (tid < nq) {
    float s = 0.f;
    for (int t = 0; t < kJT; ++t) s += red[tid * kJT + t];
    a.score[static_cast<int64_t>(a.lidx[q0 + tid]) * a.ld_score + a.score_col] = s;
  }
}

// ------------------------------------------------------------- expand kernel
// blockIdx.z = 0: partU[s] rows of U' = sum B_i C_i; 1: partV[s] rows of
// V' = sum A_i^T D_i.  blockIdx.y = split s over the flat (LoRA, l) index.
struct ExpArgs {
  const float* A; const float* B; const int32_t* lidx; int m;
  int r_l, d_in, d_out;
  const float* C; const float* D;
  int split; float* partU; float* partV;
  int zbase;                    // blockIdx.z + zbase: 0 = U', 1 = V'
};

template <int NB>
__global__ __launch_bounds__(kJT) void jd_expand_kernel(const ExpArgs a) {
  __shared__ __attribute__((aligned(16))) float smem[2 * stage_floats<NB>()];
  constexpr int r = 16 * NB;
  const bool isv = blockIdx.z + a.zbase == 1;
  const int d = isv ? a.d_in : a.d_out;
  const int row0 = blockIdx.x * kTM;
  if (row0 >= d) return;
  const int fk_total = a.m * a.r_l;
  const int ntile = (fk_total + kBK - 1) / kBK;
  const int s = blockIdx.y;
  const int f_lo = static_cast<int>(static_cast<int64_t>(ntile) * s / a.split) * kBK;
  const int f_hi = min(fk_total, static_cast<int>(static_cast<int64_t>(ntile) * (s + 1) / a.split) * kBK);
  // the workgroup's slice of the LoRA list, staged in LDS when it fits (the
  // loads' addresses then wait on an LDS read, not on a global one)
  __shared__ int32_t s_ids[kExpIds];
  const int lg = __builtin_ctz(a.r_l);
  const int q_lo = f_lo >> lg, nids = ((f_hi + a.r_l - 1) >> lg) - q_lo;
  f32x4 acc[NB];
  zero_acc(acc);
  if (nids <= kExpIds) {
    for (int i = threadIdx.x; i < nids; i += kJT) s_ids[i] = a.lidx[q_lo + i];
    __syncthreads();
    if (isv)
      tile_gemm<NB, true>(smem, f_lo, f_hi, LoadExpandA<true>{a.A, s_ids, q_lo, lg, a.r_l, a.d_in, row0, f_hi},
                          LoadRowsR{a.D, r, f_hi}, acc);
    else
      tile_gemm<NB, false>(smem, f_lo, f_hi, LoadExpandB<true>{a.B, s_ids, q_lo, lg, a.r_l, a.d_out, row0, f_hi},
                           LoadRowsR{a.C, r, f_hi}, acc);
  } else if (isv) {
    tile_gemm<NB, true>(smem, f_lo, f_hi, LoadExpandA<false>{a.A, a.lidx, 0, lg, a.r_l, a.d_in, row0, f_hi},
                        LoadRowsR{a.D, r, f_hi}, acc);
  } else {
    tile_gemm<NB, false>(smem, f_lo, f_hi, LoadExpandB<false>{a.B, a.lidx, 0, lg, a.r_l, a.d_out, row0, f_hi},
                         LoadRowsR{a.C, r, f_hi}, acc);
  }
  float* part = (isv ? a.partV : a.partU) + static_cast<int64_t>(s) * d * r;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int fr = lane & 15, fq = lane >> 4;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = row0 + 16 * wave + 4 * fq + v;
      if (row < d) part[static_cast<int64_t>(row) * r + 16 * nb + fr] = acc[nb][v];
    }
}

// X[z][row][j] = sum_s part_z[s][row][j], z = 0 (U, d_out rows), 1 (V, d_in rows)
__global__ __launch_bounds__(kJT) void jd_reduce_kernel(const float* partU, const float* partV, int S,
                                                        int d_out, int d_in, int r, float* Uo, float* Vo,
                                                        int zbase) {
  const bool isv = blockIdx.y + zbase == 1;
  const int d = isv ? d_in : d_out;
  const int64_t n = static_cast<int64_t>(d) * r;
  const float* part = isv ? partV : partU;
  float* out = isv ? Vo : Uo;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(kJT) + threadIdx.x; e < n;
       e += static_cast<int64_t>(gridDim.x) * kJT) {
    float s = 0.f;
    for (int k = 0; k < S; ++k) s += part[k * n + e];
    out[e] = s;
  }
}

// ------------------------------------------------------ CholeskyQR pieces
// Rows of a basis X [d][r] as the A operand (m = row, k = column).
struct LoadBasisRows {
  const float* X; int r, row0, d;
  __device__ float4 operator()(int, int e, int k0, int& off) const {
    const int m = e >> 3, kq = e & 7;
    off = m * kALD + 4 * kq;
    const int row = row0 + m, k = k0 + 4 * kq;
    if (row >= d || k >= r) return float4{0.f, 0.f, 0.f, 0.f};
    return *reinterpret_cast<const float4*>(X + static_cast<int64_t>(row) * r + k);
  }
};

// X^T as the A operand (m = column a of X, k = row of X): k-major.
struct LoadBasisT {
  const float* X; int r, a0, k_end;
  __device__ float4 operator()(int, int e, int k0, int& off) const {
    const int kk = e >> 4, m4 = e & 15;
    off = kk * kAML + 4 * m4;
    const int row = k0 + kk, col = a0 + 4 * m4;
    if (row >= k_end || col >= r) return float4{0.f, 0.f, 0.f, 0.f};
    return *reinterpret_cast<const float4*>(X + static_cast<int64_t>(row) * r + col);
  }
};

// Partial Gram matrices: gp[z][b][x][y] = sum over rows of block b of
// X_z[row][x] Y_z[row][y] (Y = X when Y0/Y1 are null); grid (blocks, 2, r/64
// rounded up).
template <int NB>
__global__ __launch_bounds__(kJT) void jd_gram_kernel(const float* X0, const float* X1, const float* Y0,
                                                      const float* Y1, int d0, int d1, int nblk, float* gp) {
  __shared__ __attribute__((aligned(16))) float smem[2 * stage_floats<NB>()];
  constexpr int r = 16 * NB;
  const int z = blockIdx.y, b = blockIdx.x, a0 = blockIdx.z * kTM;
  const int d = z ? d1 : d0;
  const float* X = z ? X1 : X0;
  const float* Y = z ? (Y1 ? Y1 : X1) : (Y0 ? Y0 : X0);
  const int row_lo = b * kGramRows, row_hi = min(d, row_lo + kGramRows);
  f32x4 acc[NB];
  zero_acc(acc);
  if (row_lo < row_hi)
    tile_gemm<NB, true>(smem, row_lo, row_hi, LoadBasisT{X, r, a0, row_hi}, LoadRowsR{Y, r, row_hi}, acc);
  float* out = gp + (static_cast<int64_t>(z) * nblk + b) * r * r;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int fr = lane & 15, fq = lane >> 4;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int x = a0 + 16 * wave + 4 * fq + v;
      if (x < r) out[x * r + 16 * nb + fr] = acc[nb][v];
    }
}

// One workgroup per z: G = sum_b gp[z][b] (fixed order).  chol = 0: writes G
// to out[z].  chol = 1: G = R^T R (R upper, positive diagonal), writes R^-1.
// chol = 2 (G symmetric positive definite): writes G^-1 = R^-1 R^-T.
// chol = 3 (one workgroup): G = (sum_b gp[0][b]) o (sum_b gp[1][b]), the
// elementwise product of two Gram matrices (positive definite when both
// are), and writes G^-1 to out.
// The columns are equilibrated first (G' = E G E, E = diag(G)^(-1/2), R =
// R' E^-1): the columns of X = M U scale with M's eigenvalues, and without it
// the fp32 Cholesky of a nearly converged basis breaks down.  A pivot below
// 1e-12 (relative to the unit diagonal of G') is taken as 1e-12.
// Blocked in 16 x 16 tiles so that the workgroup meets few barriers.  Per
// block column J: wave 0 alone factors the diagonal tile in registers (lane c
// holds column c; the entries other lanes need are read with readlane, at
// constant lane indices) and inverts it the same way; then the waves form the
// block row R'_J,c = R'_JJ^-T G'_J,c as products with that inverse, and every
// thread updates the trailing triangle.  R'^-1 is built from the diagonal
// tiles' inverses outward, one block diagonal at a time, and G'^-1 = R'^-1
// R'^-T with an NB x NB register block of outputs per thread.
__device__ __forceinline__ float lane_val(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

template <int NB>
__global__ __launch_bounds__(kJT) void jd_chol_kernel(const float* gp, int nblk, int chol, float* out,
                                                      int nblk1) {
  constexpr int r = 16 * NB;
  constexpr int ld = r + 1;
  constexpr int rr = r * r;
  __shared__ float g[r * ld];
  __shared__ float inv[r * ld];
  __shared__ float esc[r];
  const int z = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  constexpr int NU = (rr + kJT - 1) / kJT;
  // partials summed in block order, four blocks' loads in flight
  auto sum_partials = [&](const float* src, int cnt, float (&acc)[NU]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < NU; ++u) acc[u] = 0.f;
    int b = 0;
    for (; b + 4 <= cnt; b += 4) {
      float v[4][NU];
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int u = 0; u < NU; ++u)
          v[q][u] = (tid + u * kJT < rr) ? src[static_cast<int64_t>(b + q) * rr + tid + u * kJT] : 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int u = 0; u < NU; ++u) acc[u] += v[q][u];
    }
    for (; b < cnt; ++b)
#pragma unroll
      for (int u = 0; u < NU; ++u)
        if (tid + u * kJT < rr) acc[u] += src[static_cast<int64_t>(b) * rr + tid + u * kJT];
  };
  float acc[NU];
  sum_partials(gp + static_cast<int64_t>(z) * nblk * rr, nblk, acc);
  if (chol == 3) {
    // the second set's partials are nblk apart too, but only its first
    // nblk1 blocks hold rows
    float acc1[NU];
    sum_partials(gp + static_cast<int64_t>(nblk) * rr, nblk1, acc1);
#pragma unroll
    for (int u = 0; u < NU; ++u) acc[u] *= acc1[u];
  }
  float* dst = out + static_cast<int64_t>(z) * rr;
  if (!chol) {
#pragma unroll
    for (int u = 0; u < NU; ++u)
      if (tid + u * kJT < rr) dst[tid + u * kJT] = acc[u];
    return;
  }
  // diagonal first (lane e % (r + 1) == 0 of the sums), then G' = E G E in place
#pragma unroll
  for (int u = 0; u < NU; ++u) {
    const int e = tid + u * kJT;
    if (e < rr && e % (r + 1) == 0) esc[e / (r + 1)] = acc[u] > 0.f ? 1.f / sqrtf(acc[u]) : 1.f;
  }
  for (int e = tid; e < r * ld; e += kJT) inv[e] = 0.f;
  __syncthreads();
#pragma unroll
  for (int u = 0; u < NU; ++u) {
    const int e = tid + u * kJT;
    if (e < rr) g[(e / r) * ld + e % r] = acc[u] * esc[e / r] * esc[e % r];
  }
  __syncthreads();

  // ---- blocked right-looking Cholesky of G' (R' in the upper triangle of g,
  // the diagonal tiles of R'^-1 in inv)
#pragma unroll
  for (int J = 0; J < NB; ++J) {
    const int o = 16 * J;
    if (wave == 0) {
      // Lanes 16..63 repeat lanes 0..15.  Entries below the diagonal (i > c)
      // are updated too, with values nothing reads: that saves the selects.
      const int c = lane & 15;
      float col[16], rdg[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) col[i] = g[(o + i) * ld + o + c];
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const float dk = fmaxf(lane_val(col[k], k), 1e-12f);
        const float rp = __builtin_amdgcn_rsqf(dk);      // 1 / R'[k][k]
        rdg[k] = rp;
        col[k] = (c == k) ? dk * rp : col[k] * rp;
#pragma unroll
        for (int i = k + 1; i < 16; ++i) col[i] = fmaf(-lane_val(col[k], i), col[k], col[i]);
      }
      // column c of R'_JJ^-1 by back substitution; R'[i][k] from lane k
      float x[16];
#pragma unroll
      for (int i = 15; i >= 0; --i) {
        float s = (i == c) ? 1.f : 0.f;
#pragma unroll
        for (int k = i + 1; k < 16; ++k) s = fmaf(-lane_val(col[i], k), x[k], s);
        x[i] = (i <= c) ? s * rdg[i] : 0.f;
      }
      if (lane < 16)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          if (i <= c) g[(o + i) * ld + o + c] = col[i];
          inv[(o + i) * ld + o + c] = x[i];
        }
    }
    if (J + 1 == NB) break;
    __syncthreads();
    // block row: R'[o+i][cc] = sum_{k <= i} (R'_JJ^-1)[k][i] G'[o+k][cc] for
    // cc >= o + 16.  Wave q takes columns o + 16 + 16 q + (lane % 16), lane / 16
    // picks four rows.  Each column belongs to one wave, and no lane of it
    // writes before every lane has read the whole column: each written value
    // depends on all sixteen reads, and a wave executes in lockstep.
    {
      const int w = r - o - 16;
      for (int cb = 16 * wave; cb < w; cb += 16 * (kJT / 64)) {
        const int cc = o + 16 + cb + (lane & 15);
        const int i0 = 4 * (lane >> 4);
        float gk[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) gk[k] = g[(o + k) * ld + cc];
        float y[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          y[q] = 0.f;
#pragma unroll
          for (int k = 0; k < 16; ++k) y[q] = fmaf(inv[(o + k) * ld + o + i0 + q], gk[k], y[q]);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) g[(o + i0 + q) * ld + cc] = y[q];
      }
    }
    __syncthreads();
    // trailing triangle: G'[i][c] -= sum_k R'[o+k][i] R'[o+k][c], o+16 <= i <= c
    {
      const int w = r - o - 16;
      for (int e = tid; e < w * w; e += kJT) {
        const int i = o + 16 + e / w, c = o + 16 + e % w;
        if (c >= i) {
          float s = g[i * ld + c];
#pragma unroll
          for (int k = 0; k < 16; ++k) s = fmaf(-g[(o + k) * ld + i], g[(o + k) * ld + c], s);
          g[i * ld + c] = s;
        }
      }
    }
    __syncthreads();
  }
  __syncthreads();

  // off-diagonal tiles of R'^-1 by distance d: X_IJ = -X_II sum_{K=I+1..J} R'_IK X_KJ.
  // T_IJ is kept transposed in tile JI of g's strict lower triangle, which
  // nothing reads after the factorization.
#pragma unroll
  for (int d = 1; d < NB; ++d) {
    for (int e = tid; e < (NB - d) * 256; e += kJT) {
      const int I = e / 256, a = (e % 256) / 16, bcol = e % 16;
      const int J = I + d;
      float s = 0.f;
      for (int K = I + 1; K <= J; ++K)
#pragma unroll
        for (int k = 0; k < 16; ++k)
          s = fmaf(g[(16 * I + a) * ld + 16 * K + k], inv[(16 * K + k) * ld + 16 * J + bcol], s);
      g[(16 * J + bcol) * ld + 16 * I + a] = s;
    }
    __syncthreads();
    for (int e = tid; e < (NB - d) * 256; e += kJT) {
      const int I = e / 256, a = (e % 256) / 16, bcol = e % 16;
      const int J = I + d;
      float s = 0.f;
#pragma unroll
      for (int k = 0; k < 16; ++k)
        s = fmaf(inv[(16 * I + a) * ld + 16 * I + k], g[(16 * J + bcol) * ld + 16 * I + k], s);
      inv[(16 * I + a) * ld + 16 * J + bcol] = -s;
    }
    __syncthreads();
  }
  if (chol == 1) {
    // R^-1 = E R'^-1
    for (int e = tid; e < rr; e += kJT) dst[e] = inv[(e / r) * ld + e % r] * esc[e / r];
    return;
  }
  // G^-1 = E R'^-1 R'^-T E; R'^-1 is upper triangular with explicit zeros
  // below the diagonal, so every product runs over all r terms.  Thread
  // (ti, tc) owns rows ti + 16 a and columns tc + 16 b (a, b < NB).
  {
    const int ti = tid >> 4, tc = tid & 15;
    float accm[NB][NB];
#pragma unroll
    for (int a = 0; a < NB; ++a)
#pragma unroll
      for (int bb = 0; bb < NB; ++bb) accm[a][bb] = 0.f;
    for (int k = 0; k < r; ++k) {
      float ra[NB], rb[NB];
#pragma unroll
      for (int a = 0; a < NB; ++a) ra[a] = inv[(ti + 16 * a) * ld + k];
#pragma unroll
      for (int bb = 0; bb < NB; ++bb) rb[bb] = inv[(tc + 16 * bb) * ld + k];
#pragma unroll
      for (int a = 0; a < NB; ++a)
#pragma unroll
        for (int bb = 0; bb < NB; ++bb) accm[a][bb] = fmaf(ra[a], rb[bb], accm[a][bb]);
    }
#pragma unroll
    for (int a = 0; a < NB; ++a)
#pragma unroll
      for (int bb = 0; bb < NB; ++bb) {
        const int i = ti + 16 * a, c = tc + 16 * bb;
        dst[i * r + c] = accm[a][bb] * esc[i] * esc[c];
      }
  }
}

// X_z[row][:] <- X_z[row][:] Rinv_z (64 rows per workgroup, in place: a
// workgroup reads only its own rows, and all of them before it writes)
template <int NB>
__global__ __launch_bounds__(kJT) void jd_apply_kernel(float* X0, float* X1, int d0, int d1,
                                                       const float* rinv, int zbase = 0) {
  __shared__ __attribute__((aligned(16))) float smem[2 * stage_floats<NB>()];
  constexpr int r = 16 * NB;
  const int z = blockIdx.y + zbase;
  const int d = z ? d1 : d0;
  float* X = z ? X1 : X0;
  const int row0 = blockIdx.x * kTM;
  if (row0 >= d) return;
  f32x4 acc[NB];
  zero_acc(acc);
  tile_gemm<NB, false>(smem, 0, r, LoadBasisRows{X, r, row0, d},
                       LoadRowsR{rinv + static_cast<int64_t>(z) * r * r, r, r}, acc);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int fr = lane & 15, fq = lane >> 4;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = row0 + 16 * wave + 4 * fq + v;
      if (row < d) X[static_cast<int64_t>(row) * r + 16 * nb + fr] = acc[nb][v];
    }
}

// Convergence measure, partial sums per 64-row block: E = Xn - Xo M_z,
// rp[z][b] = (||E||^2, ||Xn||^2) over the block.
template <int NB>
__global__ __launch_bounds__(kJT) void jd_resid_kernel(const float* Uo, const float* Un, const float* Vo,
                                                       const float* Vn, int d0, int d1, const float* M,
                                                       int nblk, float* rp) {
  __shared__ __attribute__((aligned(16))) float smem[2 * stage_floats<NB>()];
  __shared__ float red[2 * kJT];
  constexpr int r = 16 * NB;
  const int z = blockIdx.y, b = blockIdx.x;
  const int d = z ? d1 : d0;
  const float* Xo = z ? Vo : Uo;
  const float* Xn = z ? Vn : Un;
  const int row0 = b * kTM;
  float e2 = 0.f, x2 = 0.f;
  if (row0 < d) {
    f32x4 acc[NB];
    zero_acc(acc);
    tile_gemm<NB, false>(smem, 0, r, LoadBasisRows{Xo, r, row0, d},
                         LoadRowsR{M + static_cast<int64_t>(z) * r * r, r, r}, acc);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int fr = lane & 15, fq = lane >> 4;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = row0 + 16 * wave + 4 * fq + v;
        if (row < d) {
          const float xn = Xn[static_cast<int64_t>(row) * r + 16 * nb + fr];
          const float df = xn - acc[nb][v];
          e2 = fmaf(df, df, e2);
          x2 = fmaf(xn, xn, x2);
        }
      }
  }
  red[threadIdx.x] = e2;
  red[kJT + threadIdx.x] = x2;
  __syncthreads();
  if (threadIdx.x == 0) {
    float se = 0.f, sx = 0.f;
    for (int t = 0; t < kJT; ++t) { se += red[t]; sx += red[kJT + t]; }
    rp[(static_cast<int64_t>(z) * nblk + b) * 2] = se;
    rp[(static_cast<int64_t>(z) * nblk + b) * 2 + 1] = sx;
  }
}

// one wave: lane l sums blocks l, l + 64, ...; then lane 0 sums the lanes in order
__global__ void jd_crit_kernel(const float* rp, int nblk, float* crit) {
  __shared__ float part[4][64];
  const int l = threadIdx.x;
  for (int z = 0; z < 2; ++z) {
    float se = 0.f, sx = 0.f;
    for (int b = l; b < nblk; b += 64) {
      se += rp[(z * nblk + b) * 2];
      sx += rp[(z * nblk + b) * 2 + 1];
    }
    part[2 * z][l] = se;
    part[2 * z + 1][l] = sx;
  }
  __syncthreads();
  if (l != 0) return;
  float c = 0.f;
  for (int z = 0; z < 2; ++z) {
    float se = 0.f, sx = 0.f;
    for (int k = 0; k < 64; ++k) {
      se += part[2 * z][k];
      sx += part[2 * z + 1][k];
    }
    c = fmaxf(c, sqrtf(se / sx));
  }
  crit[0] = c;
}

// out[c][x] = in[x][c] for an [R][C] array (transposes a basis)
__global__ __launch_bounds__(kJT) void jd_transpose_kernel(const float* in, int R, int C, float* out) {
  __shared__ float tile[32][33];
  const int bx = blockIdx.x * 32, by = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;      // 32 x 8
  for (int k = ty; k < 32; k += 8) {
    const int rr = by + k, cc = bx + tx;
    tile[k][tx] = (rr < R && cc < C) ? in[static_cast<int64_t>(rr) * C + cc] : 0.f;
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) {
    const int cc = bx + k, rr = by + tx;
    if (cc < C && rr < R) out[static_cast<int64_t>(cc) * R + rr] = tile[tx][k];
  }
}

__global__ void jd_copy_kernel(const float* in, float* out, int64_t n) {
  for (int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; e < n;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x)
    out[e] = in[e];
}

// Bases of a cluster whose m members supply fewer than r directions (App. A.3
// Step 1 with m r_l < r; every pair holding the members' B_i and A_i^T
// columns reconstructs them exactly, Prop. 1), before orthonormalization:
//   Un [d_out][r] = [B_{memb[0]} ... B_{memb[m-1]} | Uc[:, :r - m r_l]]
//   Vn [d_in][r]  = [A_{memb[0]}^T ... A_{memb[m-1]}^T | Vtc[:r - m r_l]^T]
// grid (ceil(max(d_out, d_in) r / 256), 2): y = 0 fills Un, y = 1 Vn.
__global__ void jd_span_kernel(const float* A, const float* B, const int32_t* memb, int m, int r_l, int d_in,
                               int d_out, int r, const float* Uc, const float* Vtc, float* Un, float* Vn) {
  const bool u = blockIdx.y == 0;
  const int64_t rows = u ? d_out : d_in;
  const int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
  if (e >= rows * r) return;
  const int row = static_cast<int>(e / r), c = static_cast<int>(e % r);
  const int mc = m * r_l;
  float v;
  if (c < mc) {
    const int64_t i = memb[c / r_l], l = c % r_l;
    v = u ? B[(i * d_out + row) * r_l + l] : A[(i * r_l + l) * d_in + row];
  } else {
    v = u ? Uc[static_cast<int64_t>(row) * r + (c - mc)] : Vtc[static_cast<int64_t>(c - mc) * d_in + row];
  }
  (u ? Un : Vn)[e] = v;
}

__global__ void jd_iota_kernel(int32_t* out, int n) {
  for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < n; e += gridDim.x * blockDim.x) out[e] = e;
}

// ||B_i A_i||_F^2 = sum_{l,l'} (B_i^T B_i)[l][l'] (A_i A_i^T)[l][l'], one
// workgroup per LoRA; also w2[i] = 1 / norms2[i] and w[i] = 1 / ||B_i A_i||.
__global__ __launch_bounds__(kJT) void jd_norms_kernel(const float* A, const float* B, int r_l, int d_in,
                                                       int d_out, float* norms2, float* w2, float* w) {
  __shared__ float ga[64 * 64], gb[64 * 64];
  const int i = blockIdx.x;
  const float* Ai = A + static_cast<int64_t>(i) * r_l * d_in;
  const float* Bi = B + static_cast<int64_t>(i) * d_out * r_l;
  const int nn = r_l * r_l;
  for (int e = threadIdx.x; e < nn; e += kJT) {
    const int l = e / r_l, l2 = e - l * r_l;
    float sa = 0.f, sb = 0.f;
    for (int c = 0; c < d_in; ++c) sa = fmaf(Ai[static_cast<int64_t>(l) * d_in + c], Ai[static_cast<int64_t>(l2) * d_in + c], sa);
    for (int o = 0; o < d_out; ++o) sb = fmaf(Bi[static_cast<int64_t>(o) * r_l + l], Bi[static_cast<int64_t>(o) * r_l + l2], sb);
    ga[e] = sa;
    gb[e] = sb;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float s = 0.f;
    for (int e = 0; e < nn; ++e) s = fmaf(ga[e], gb[e], s);
    norms2[i] = s;
    if (w2) w2[i] = 1.f / s;
    if (w) w[i] = 1.f / sqrtf(s);
  }
}

// ------------------------------------------------------------ k-means pieces
// dist[i][j] = ||x_i - c_j||^2 (x = Sigma rows of dim r^2); one workgroup per i
__global__ __launch_bounds__(kJT) void km_dist_kernel(const float* X, const float* Cn, int dim, int K,
                                                      float* dist) {
  __shared__ float red[kJT];
  const int i = blockIdx.x;
  const float* x = X + static_cast<int64_t>(i) * dim;
  for (int j = 0; j < K; ++j) {
    const float* c = Cn + static_cast<int64_t>(j) * dim;
    float s = 0.f;
    for (int e = threadIdx.x; e < dim; e += kJT) {
      const float df = x[e] - c[e];
      s = fmaf(df, df, s);
    }
    red[threadIdx.x] = s;
    __syncthreads();
    for (int h = kJT / 2; h > 0; h >>= 1) {
      if (threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
      __syncthreads();
    }
    if (threadIdx.x == 0) dist[static_cast<int64_t>(i) * K + j] = red[0];
    __syncthreads();
  }
}

// labels[i] = arg min_j v[i][j] (sign = 1) or arg max (sign = -1), lowest j on
// ties; changed[0] = number of labels that differ from the previous ones
// (one workgroup, fixed order)
__global__ __launch_bounds__(kJT) void km_pick_kernel(const float* v, int n, int K, float sign,
                                                      int32_t* labels, int32_t* changed) {
  __shared__ int red[kJT];
  int cnt = 0;
  for (int i = threadIdx.x; i < n; i += kJT) {
    int best = 0;
    float bv = sign * v[static_cast<int64_t>(i) * K];
    for (int j = 1; j < K; ++j) {
      const float x = sign * v[static_cast<int64_t>(i) * K + j];
      if (x < bv) { bv = x; best = j; }
    }
    cnt += (labels[i] != best) ? 1 : 0;
    labels[i] = best;
  }
  red[threadIdx.x] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int t = 0; t < kJT; ++t) s += red[t];
    changed[0] = s;
  }
}

// centroid j = mean of the rows i with labels[i] == j (kept when empty);
// grid (ceil(dim / 256), K)
__global__ __launch_bounds__(kJT) void km_centroid_kernel(const float* X, const int32_t* labels, int n,
                                                          int dim, float* Cn) {
  const int j = blockIdx.y;
  const int e = blockIdx.x * kJT + threadIdx.x;
  if (e >= dim) return;
  float s = 0.f;
  int cnt = 0;
  for (int i = 0; i < n; ++i)
    if (labels[i] == j) {
      s += X[static_cast<int64_t>(i) * dim + e];
      ++cnt;
    }
  if (cnt > 0) Cn[static_cast<int64_t>(j) * dim + e] = s / static_cast<float>(cnt);
}

// centroids from rows init[j]
__global__ __launch_bounds__(kJT) void km_init_kernel(const float* X, const int32_t* init, int dim,
                                                      float* Cn) {
  const int j = blockIdx.y;
  const int e = blockIdx.x * kJT + threadIdx.x;
  if (e < dim) Cn[static_cast<int64_t>(j) * dim + e] = X[static_cast<int64_t>(init[j]) * dim + e];
}

// members of each cluster in increasing id order: memb[offs[j] ...], with
// offs[j] = number of LoRAs in clusters < j (one workgroup, fixed order)
__global__ __launch_bounds__(kJT) void km_members_kernel(const int32_t* labels, int n, int K,
                                                         int32_t* offs, int32_t* memb) {
  __shared__ int wcnt[kJT / 64];
  __shared__ int base;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  if (threadIdx.x == 0) base = 0;
  __syncthreads();
  for (int j = 0; j < K; ++j) {
    if (threadIdx.x == 0) offs[j] = base;
    for (int c0 = 0; c0 < n; c0 += kJT) {
      const int i = c0 + threadIdx.x;
      const bool in = i < n && labels[i] == j;
      const uint64_t bal = __ballot(in);
      if (lane == 0) wcnt[wave] = __popcll(bal);
      __syncthreads();
      int before = 0, total = 0;
      for (int w = 0; w < kJT / 64; ++w) {
        before += (w < wave) ? wcnt[w] : 0;
        total += wcnt[w];
      }
      if (in) memb[base + before + __popcll(bal & lt)] = i;
      __syncthreads();
      if (threadIdx.x == 0) base += total;
      __syncthreads();
    }
  }
  if (threadIdx.x == 0) offs[K] = base;
}

// ---------------------------------------------------------- JD-Diag pieces
// s_i = Ginv w_i for every LoRA (Ginv symmetric r x r): s[i][j] = sum_k Ginv[j][k] w[i][k]
template <int NB>
__global__ __launch_bounds__(kJT) void jd_diag_solve_kernel(const float* ginv, const float* w, int n, float* s) {
  constexpr int r = 16 * NB;
  __shared__ float sg[r * (r + 1)];                  // Ginv rows, padded against bank conflicts
  for (int e = threadIdx.x; e < r * r; e += kJT) sg[(e / r) * (r + 1) + e % r] = ginv[e];
  __syncthreads();
  const int64_t tot = static_cast<int64_t>(n) * r;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(kJT) + threadIdx.x; e < tot;
       e += static_cast<int64_t>(gridDim.x) * kJT) {
    const int64_t i = e / r;
    const int jj = static_cast<int>(e - i * r);
    const float* wr = w + i * r;                     // one row per r consecutive threads
    float acc = 0.f;
#pragma unroll 16
    for (int k = 0; k < r; ++k) acc = fmaf(sg[jj * (r + 1) + k], wr[k], acc);
    s[e] = acc;
  }
}

// nu[0] = sqrt(sum s^2) (one workgroup, fixed order)
__global__ __launch_bounds__(kJT) void jd_norm_kernel(const float* s, int64_t n, float* nu) {
  __shared__ float red[kJT];
  float acc = 0.f;
  for (int64_t e = threadIdx.x; e < n; e += kJT) acc = fmaf(s[e], s[e], acc);
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.f;
    for (int k = 0; k < kJT; ++k) t += red[k];
    nu[0] = sqrtf(t);
  }
}

// x[e] *= nu[0]^p (p = -1 or 1/2)
__global__ void jd_scale_kernel(float* x, int64_t n, const float* nu, int inverse) {
  const float f = inverse ? 1.f / nu[0] : sqrtf(nu[0]);
  for (int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; e < n;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x)
    x[e] *= f;
}

// ------------------------------------------------------------------ host side
// Calls f(std::integral_constant<int, NB>) for the compiled column-block
// counts NB = r / 16.
template <typename F>
hipError_t with_nb(int r, F f) {
  switch (r / 16) {
    case 1: return f(std::integral_constant<int, 1>{});
    case 2: return f(std::integral_constant<int, 2>{});
    case 3: return f(std::integral_constant<int, 3>{});
    case 4: return f(std::integral_constant<int, 4>{});
    case 6: return f(std::integral_constant<int, 6>{});
    case 8: return f(std::integral_constant<int, 8>{});
    default: return hipErrorInvalidValue;
  }
}

bool bad_ptr(const void* ptr, size_t align) {
  return ptr == nullptr || (reinterpret_cast<uintptr_t>(ptr) % align) != 0;
}

int validate(const cts_jd_problem* p) {
  if (!p) return CTS_ERR_INVALID_ARG;
  if (p->n <= 0 || p->d_out <= 0 || p->d_in <= 0 || p->r_lora <= 0 || p->r <= 0) return CTS_ERR_INVALID_ARG;
  const int rl = p->r_lora;
  if (!(rl == 4 || rl == 8 || rl == 16 || rl == 32 || rl == 64)) return CTS_ERR_UNSUPPORTED;
  if (!(p->r == 16 || p->r == 32 || p->r == 48 || p->r == 64 || p->r == 96 || p->r == 128))
    return CTS_ERR_UNSUPPORTED;
  if (p->n > 65536 || static_cast<int64_t>(p->n) * rl < p->r) return CTS_ERR_UNSUPPORTED;
  if (p->d_in % 4 || p->d_out % 4 || p->d_in < p->r || p->d_out < p->r || p->d_in > 65536 ||
      p->d_out > 65536)
    return CTS_ERR_UNSUPPORTED;
  const int64_t lim = int64_t(1) << 31;
  if (static_cast<int64_t>(p->n) * rl * p->d_in >= lim || static_cast<int64_t>(p->n) * rl * p->d_out >= lim ||
      static_cast<int64_t>(p->n) * p->r * p->r >= lim)
    return CTS_ERR_UNSUPPORTED;
  return CTS_OK;
}

// Workspace of one JD run (plus the clustering extras when K > 0).
struct JdPlan {
  int split, pq_split, nblk_out, nblk_in, nblk, nblk_n;
  size_t off_U, off_V, off_Uo, off_Vo, off_C, off_D, off_pq, off_pU, off_pV, off_gp, off_mat, off_rp, off_lidx,
      off_w2, off_w, off_n2, off_crit, total;
  // clustering
  size_t off_S, off_cent, off_dist, off_lab, off_chg, off_offs, off_memb, off_score;
  // JD-Diag
  size_t off_sd, off_wv, off_m, off_nu;
};

size_t align_up(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

// Workgroups of the projection and expansion kernels one compute unit holds
// at rank r (their LDS and registers, as compiled for gfx950), and the
// smallest split of a launch of `base` workgroups per piece that fills the
// resident slots of 256 compute units within 5% of the best such split.
int resident_wgs(int r) { return r <= 32 ? 4 : (r <= 64 ? 3 : 2); }

int pick_split(int64_t base, int occ, int smax) {
  const int64_t slots = 256LL * occ;
  int best = 1;
  double best_eff = 0.0;
  for (int s = 1; s <= smax; ++s) {
    const int64_t w = base * s, rounds = (w + slots - 1) / slots;
    const double eff = static_cast<double>(w) / static_cast<double>(rounds * slots);
    if (eff > best_eff + 0.05) {
      best = s;
      best_eff = eff;
    }
  }
  return best;
}

void plan_jd(const cts_jd_problem* p, int K, JdPlan* pl) {
  const int64_t n = p->n, rl = p->r_lora, r = p->r;
  const int64_t fk = n * rl;
  const int64_t ntile = (fk + kBK - 1) / kBK;
  // the expansion's pieces of the collection: at most kMaxExpSplit (chosen
  // per launch), at least 8 k-tiles each; the projection's pieces of d_in
  // and d_out: two (measured: more pieces were slower at 1000 LoRAs, 4096 x
  // 4096), one when a piece would have fewer than 8 k-tiles
  pl->split = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(kMaxExpSplit, ntile / 8)));
  pl->pq_split = (std::min(p->d_in, p->d_out) + kBK - 1) / kBK >= 16 ? 2 : 1;
  pl->nblk_out = (p->d_out + kGramRows - 1) / kGramRows;
  pl->nblk_in = (p->d_in + kGramRows - 1) / kGramRows;
  pl->nblk = std::max(pl->nblk_out, pl->nblk_in);
  pl->nblk_n = (p->n + kGramRows - 1) / kGramRows;
  const int nrb = (std::max(p->d_out, p->d_in) + 63) / 64;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes); return o; };
  pl->off_U = take(4ull * p->d_out * r);
  pl->off_V = take(4ull * p->d_in * r);
  pl->off_Uo = take(4ull * p->d_out * r);
  pl->off_Vo = take(4ull * p->d_in * r);
  pl->off_C = take(4ull * fk * r);
  pl->off_D = take(4ull * fk * r);
  pl->off_pq = take(4ull * pl->pq_split * 2 * fk * r);
  pl->off_pU = take(4ull * pl->split * p->d_out * r);
  pl->off_pV = take(4ull * pl->split * p->d_in * r);
  pl->off_gp = take(4ull * 2 * std::max(pl->nblk, pl->nblk_n) * r * r);
  pl->off_mat = take(4ull * 2 * r * r);
  pl->off_rp = take(4ull * 2 * nrb * 2);
  pl->off_lidx = take(4ull * n);
  pl->off_w2 = take(4ull * n);
  pl->off_w = take(4ull * n);
  pl->off_n2 = take(4ull * n);
  pl->off_crit = take(4ull * 4);
  pl->off_sd = take(4ull * n * r);
  pl->off_wv = take(4ull * n * r);
  pl->off_m = take(4ull * 8 * r * r);
  pl->off_nu = take(4ull * 4);
  pl->off_S = pl->off_cent = pl->off_dist = pl->off_lab = pl->off_chg = pl->off_offs = pl->off_memb =
      pl->off_score = 0;
  if (K > 0) {
    pl->off_S = take(4ull * n * r * r);
    pl->off_cent = take(4ull * K * r * r);
    pl->off_dist = take(4ull * n * K);
    pl->off_lab = take(4ull * n);
    pl->off_chg = take(4ull * 4);
    pl->off_offs = take(4ull * (K + 1));
    pl->off_memb = take(4ull * n);
    pl->off_score = take(4ull * n * K);
  }
  pl->total = off;
}

struct Jd {
  const cts_jd_problem* p;
  JdPlan pl;
  char* ws;
  hipStream_t st;
  template <typename T> T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }
};

// P = A_i V and/or Q = B_i^T U (zbase, zcount: halves 0 = P, 1 = Q; zcount
// 0: neither, the partials already hold them), then the per-LoRA products of
// `mode` (see jd_combine_kernel).
hipError_t launch_project(const Jd& j, const float* A, const float* B, const float* V, const float* U,
                          const int32_t* lidx, int m, int mode, const float* w2, const float* sscale,
                          float* Sigma, float* score, int ld_score, int score_col, int zbase = 0,
                          int zcount = 2, const float* sdiag = nullptr, float* wout = nullptr) {
  const cts_jd_problem* p = j.p;
  float* part = j.at<float>(j.pl.off_pq);
  PqArgs pa{A, B, V, U, lidx, m, p->r_lora, p->d_in, p->d_out, part, j.pl.pq_split, zbase};
  ProjArgs a{lidx, m, p->r_lora, part, j.pl.pq_split, mode, sdiag, wout, w2, sscale, j.at<float>(j.pl.off_C),
             j.at<float>(j.pl.off_D), Sigma, score, ld_score, score_col};
  const int lpw = kTM / p->r_lora;
  const unsigned groups = static_cast<unsigned>((m + lpw - 1) / lpw);
  return with_nb(p->r, [&](auto c) {
    if (zcount > 0) {
      hipLaunchKernelGGL(jd_pq_kernel<decltype(c)::value>, dim3(groups, zcount, j.pl.pq_split), dim3(kJT), 0, j.st,
                         pa);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(jd_combine_kernel<decltype(c)::value>, dim3(groups), dim3(kJT), 0, j.st, a);
    return hipGetLastError();
  });
}

// One eigenvalue-iteration step from (U, V) in the workspace to (Uo, Vo)
// (the new pair), then the measure into crit_out; swaps the buffers.
// Gram partials X0^T Y0 (d_out rows) and X1^T Y1 (d_in rows); Y null: X^T X.
hipError_t gram_pair(Jd& j, const float* X0, const float* X1, const float* Y0, const float* Y1) {
  const cts_jd_problem* p = j.p;
  const int r = p->r;
  const dim3 ggrid(j.pl.nblk, 2, (r + kTM - 1) / kTM);
  float* gp = j.at<float>(j.pl.off_gp);
  return with_nb(r, [&](auto c) {
    hipLaunchKernelGGL(jd_gram_kernel<decltype(c)::value>, ggrid, dim3(kJT), 0, j.st, X0, X1, Y0, Y1, p->d_out,
                       p->d_in, j.pl.nblk, gp);
    return hipGetLastError();
  });
}

// CholeskyQR2 on Un [d_out][r] and Vn [d_in][r] together, in place: the Q of
// the QR factorization with a positive diagonal of R.
hipError_t orthonormalize(Jd& j, float* Un, float* Vn) {
  const cts_jd_problem* p = j.p;
  const int r = p->r;
  float* gp = j.at<float>(j.pl.off_gp);
  float* mat = j.at<float>(j.pl.off_mat);
  const int nrb = (std::max(p->d_out, p->d_in) + 63) / 64;
  hipError_t e;
  for (int pass = 0; pass < 2; ++pass) {
    if ((e = gram_pair(j, Un, Vn, nullptr, nullptr)) != hipSuccess) return e;
    e = with_nb(r, [&](auto c) {
      hipLaunchKernelGGL(jd_chol_kernel<decltype(c)::value>, dim3(2), dim3(kJT), 0, j.st, gp, j.pl.nblk, 1, mat,
                         j.pl.nblk);
      return hipGetLastError();
    });
    if (e != hipSuccess) return e;
    e = with_nb(r, [&](auto c) {
      hipLaunchKernelGGL(jd_apply_kernel<decltype(c)::value>, dim3(nrb, 2), dim3(kJT), 0, j.st, Un, Vn, p->d_out,
                         p->d_in, mat);
      return hipGetLastError();
    });
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// App. A.3 Step 1 for a cluster of m members with m r_l < r (the members'
// ids at memb, device): the bases of jd_span_kernel, orthonormalized, in j's
// U / V buffers.
hipError_t span_bases(Jd& j, const float* A, const float* B, const int32_t* memb, int m, const float* Uc,
                      const float* Vtc) {
  const cts_jd_problem* p = j.p;
  const int64_t cells = static_cast<int64_t>(std::max(p->d_out, p->d_in)) * p->r;
  hipLaunchKernelGGL(jd_span_kernel, dim3(static_cast<unsigned>((cells + 255) / 256), 2), dim3(256), 0, j.st, A, B,
                     memb, m, p->r_lora, p->d_in, p->d_out, p->r, Uc, Vtc, j.at<float>(j.pl.off_U),
                     j.at<float>(j.pl.off_V));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return orthonormalize(j, j.at<float>(j.pl.off_U), j.at<float>(j.pl.off_V));
}

hipError_t jd_step(Jd& j, const float* A, const float* B, const int32_t* lidx, int m, const float* w2,
                   float* crit_out) {
  const cts_jd_problem* p = j.p;
  const int r = p->r;
  float* U = j.at<float>(j.pl.off_U);
  float* V = j.at<float>(j.pl.off_V);
  float* Un = j.at<float>(j.pl.off_Uo);
  float* Vn = j.at<float>(j.pl.off_Vo);
  hipError_t e = stage_mark(1, j.st);
  if (e != hipSuccess) return e;
  e = launch_project(j, A, B, V, U, lidx, m, 0, w2, nullptr, nullptr, nullptr, 0, 0);
  if (e != hipSuccess || (e = stage_mark(2, j.st)) != hipSuccess) return e;
  // expand, split so that the collection's share per workgroup is >= 8 k-tiles
  const int64_t ntile = (static_cast<int64_t>(m) * p->r_lora + kBK - 1) / kBK;
  const int rowt = (std::max(p->d_out, p->d_in) + kTM - 1) / kTM;
  const int split = pick_split(2LL * rowt, resident_wgs(r),
                               static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(j.pl.split, ntile / 8))));
  ExpArgs ea{A, B, lidx, m, p->r_lora, p->d_in, p->d_out, j.at<float>(j.pl.off_C),
             j.at<float>(j.pl.off_D), split, j.at<float>(j.pl.off_pU), j.at<float>(j.pl.off_pV), 0};
  e = with_nb(r, [&](auto c) {
    hipLaunchKernelGGL(jd_expand_kernel<decltype(c)::value>, dim3(rowt, split, 2), dim3(kJT), 0, j.st, ea);
    return hipGetLastError();
  });
  if (e != hipSuccess || (e = stage_mark(3, j.st)) != hipSuccess) return e;
  const int64_t nmax = static_cast<int64_t>(std::max(p->d_out, p->d_in)) * r;
  hipLaunchKernelGGL(jd_reduce_kernel, dim3(static_cast<unsigned>(std::min<int64_t>(1024, (nmax + kJT - 1) / kJT)), 2),
                     dim3(kJT), 0, j.st, j.at<float>(j.pl.off_pU), j.at<float>(j.pl.off_pV), split, p->d_out,
                     p->d_in, r, Un, Vn, 0);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = orthonormalize(j, Un, Vn)) != hipSuccess) return e;
  // measure: M = X_old^T X_new, E = X_new - X_old M
  float* gp = j.at<float>(j.pl.off_gp);
  float* mat = j.at<float>(j.pl.off_mat);
  const int nrb = (std::max(p->d_out, p->d_in) + 63) / 64;
  if ((e = gram_pair(j, U, V, Un, Vn)) != hipSuccess) return e;
  e = with_nb(r, [&](auto c) {
    hipLaunchKernelGGL(jd_chol_kernel<decltype(c)::value>, dim3(2), dim3(kJT), 0, j.st, gp, j.pl.nblk, 0, mat,
                       j.pl.nblk);
    return hipGetLastError();
  });
  if (e != hipSuccess) return e;
  float* rp = j.at<float>(j.pl.off_rp);
  e = with_nb(r, [&](auto c) {
    hipLaunchKernelGGL(jd_resid_kernel<decltype(c)::value>, dim3(nrb, 2), dim3(kJT), 0, j.st, U, Un, V, Vn,
                       p->d_out, p->d_in, mat, nrb, rp);
    return hipGetLastError();
  });
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(jd_crit_kernel, dim3(1), dim3(64), 0, j.st, rp, nrb, crit_out);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  std::swap(j.pl.off_U, j.pl.off_Uo);
  std::swap(j.pl.off_V, j.pl.off_Vo);
  return hipSuccess;
}

// basis in: U0 [d_out][r] -> U; Vt0 [r][d_in] -> V [d_in][r]
hipError_t load_bases(Jd& j, const float* U0, const float* Vt0) {
  const cts_jd_problem* p = j.p;
  const int64_t nu = static_cast<int64_t>(p->d_out) * p->r;
  hipLaunchKernelGGL(jd_copy_kernel, dim3(static_cast<unsigned>(std::min<int64_t>(1024, (nu + 255) / 256))),
                     dim3(256), 0, j.st, U0, j.at<float>(j.pl.off_U), nu);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(jd_transpose_kernel, dim3((p->d_in + 31) / 32, (p->r + 31) / 32), dim3(kJT), 0, j.st, Vt0,
                     p->r, p->d_in, j.at<float>(j.pl.off_V));
  return hipGetLastError();
}

hipError_t store_bases(Jd& j, float* U, float* Vt) {
  const cts_jd_problem* p = j.p;
  const int64_t nu = static_cast<int64_t>(p->d_out) * p->r;
  hipLaunchKernelGGL(jd_copy_kernel, dim3(static_cast<unsigned>(std::min<int64_t>(1024, (nu + 255) / 256))),
                     dim3(256), 0, j.st, j.at<float>(j.pl.off_U), U, nu);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(jd_transpose_kernel, dim3((p->r + 31) / 32, (p->d_in + 31) / 32), dim3(kJT), 0, j.st,
                     j.at<float>(j.pl.off_V), p->d_in, p->r, Vt);
  return hipGetLastError();
}

hipError_t norms(Jd& j, const float* A, const float* B) {
  const cts_jd_problem* p = j.p;
  hipLaunchKernelGGL(jd_norms_kernel, dim3(p->n), dim3(kJT), 0, j.st, A, B, p->r_lora, p->d_in, p->d_out,
                     j.at<float>(j.pl.off_n2), j.at<float>(j.pl.off_w2), j.at<float>(j.pl.off_w));
  return hipGetLastError();
}

// `iters` iterations (early stop below tau, waiting per iteration) on the
// LoRAs lidx[0..m); bases in j's U/V buffers.  crit: device array or null
// (then the workspace slot).
int run_jd(Jd& j, const float* A, const float* B, const int32_t* lidx, int m, const float* w2, int iters,
           float tau, float* crit, int* done) {
  float* cslot = j.at<float>(j.pl.off_crit);
  int t = 0;
  for (; t < iters; ++t) {
    float* c = crit ? crit + t : cslot;
    if (jd_step(j, A, B, lidx, m, w2, c) != hipSuccess) return CTS_ERR_HIP;
    if (tau > 0.f) {
      float h = 0.f;
      if (hipMemcpyAsync(&h, c, sizeof(float), hipMemcpyDeviceToHost, j.st) != hipSuccess ||
          hipStreamSynchronize(j.st) != hipSuccess)
        return CTS_ERR_HIP;
      if (h < tau) { ++t; break; }
    }
  }
  if (done) *done = t;
  return CTS_OK;
}

// ---- JD-Diag by alternating least squares (App. A.1 case 2)
// out = (X0^T X0 o X1^T X1)^-1 (X0: d0 rows, X1: d1 rows, r columns each);
// the elementwise product of the two Gram matrices is positive definite
// when both are
hipError_t gram_hadamard_inverse(Jd& j, const float* X0, int d0, const float* X1, int d1, float* out) {
  const int r = j.p->r;
  const int nb = (std::max(d0, d1) + kGramRows - 1) / kGramRows;
  float* gp = j.at<float>(j.pl.off_gp);
  return with_nb(r, [&](auto c) {
    hipLaunchKernelGGL(jd_gram_kernel<decltype(c)::value>, dim3(nb, 2, (r + kTM - 1) / kTM), dim3(kJT), 0, j.st,
                       X0, X1, nullptr, nullptr, d0, d1, nb, gp);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(jd_chol_kernel<decltype(c)::value>, dim3(1), dim3(kJT), 0, j.st, gp, nb, 3, out,
                       (d1 + kGramRows - 1) / kGramRows);
    return hipGetLastError();
  });
}

// X (d rows, z-th basis slot of the apply kernel) <- X M
hipError_t apply_one(Jd& j, float* X, int d, int z, const float* M2) {
  const int r = j.p->r;
  return with_nb(r, [&](auto c) {
    hipLaunchKernelGGL(jd_apply_kernel<decltype(c)::value>, dim3((d + kTM - 1) / kTM, 1), dim3(kJT), 0, j.st,
                       z == 0 ? X : nullptr, z == 1 ? X : nullptr, d, d, M2, z);
    return hipGetLastError();
  });
}

// one half of the expansion (z = 0: U' = sum B_i C_i into Uo; 1: V' = sum A_i^T D_i into Vo);
// mark > 0 records that profiling event between the expansion kernel and the
// sum of its pieces
hipError_t expand_one(Jd& j, const float* A, const float* B, const int32_t* lidx, int m, int z, float* out,
                      int mark = 0) {
  const cts_jd_problem* p = j.p;
  const int r = p->r;
  const int64_t ntile = (static_cast<int64_t>(m) * p->r_lora + kBK - 1) / kBK;
  const int d = z ? p->d_in : p->d_out;
  const int split = pick_split((d + kTM - 1) / kTM, resident_wgs(r),
                               static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(j.pl.split, ntile / 8))));
  ExpArgs ea{A, B, lidx, m, p->r_lora, p->d_in, p->d_out, j.at<float>(j.pl.off_C), j.at<float>(j.pl.off_D),
             split, j.at<float>(j.pl.off_pU), j.at<float>(j.pl.off_pV), z};
  hipError_t e = with_nb(r, [&](auto c) {
    hipLaunchKernelGGL(jd_expand_kernel<decltype(c)::value>, dim3((d + kTM - 1) / kTM, split, 1), dim3(kJT), 0, j.st,
                       ea);
    return hipGetLastError();
  });
  if (e != hipSuccess || (mark > 0 && (e = stage_mark(mark, j.st)) != hipSuccess)) return e;
  const int64_t nel = static_cast<int64_t>(d) * r;
  hipLaunchKernelGGL(jd_reduce_kernel, dim3(static_cast<unsigned>(std::min<int64_t>(1024, (nel + kJT - 1) / kJT)), 1),
                     dim3(kJT), 0, j.st, j.at<float>(j.pl.off_pU), j.at<float>(j.pl.off_pV), split, p->d_out, p->d_in,
                     r, z ? nullptr : out, z ? out : nullptr, z);
  return hipGetLastError();
}

// diagonals from the current pair: s_i = (U^T U o V^T V)^-1 (U^T B_i o V^T A_i^T) 1;
// P and Q must be current in the partial buffers unless `fresh` (then both
// are recomputed)
hipError_t als_sigma(Jd& j, const float* A, const float* B, const int32_t* lidx, bool fresh) {
  const cts_jd_problem* p = j.p;
  const int r = p->r;
  float* U = j.at<float>(j.pl.off_U);
  float* V = j.at<float>(j.pl.off_V);
  float* sd = j.at<float>(j.pl.off_sd);
  float* w = j.at<float>(j.pl.off_wv);
  float* m = j.at<float>(j.pl.off_m);            // [3]: (U^T U o V^T V)^-1
  hipError_t e = launch_project(j, A, B, V, U, lidx, p->n, 5, nullptr, nullptr, nullptr, nullptr, 0, 0,
                                fresh ? 0 : 0, fresh ? 2 : 1, nullptr, w);
  if (e != hipSuccess) return e;
  const int64_t rr = static_cast<int64_t>(r) * r;
  if ((e = gram_hadamard_inverse(j, U, p->d_out, V, p->d_in, m + 3 * rr)) != hipSuccess) return e;
  const int64_t tot = static_cast<int64_t>(p->n) * r;
  return with_nb(r, [&](auto c) {
    hipLaunchKernelGGL(jd_diag_solve_kernel<decltype(c)::value>,
                       dim3(static_cast<unsigned>(std::min<int64_t>(1024, (tot + kJT - 1) / kJT))), dim3(kJT), 0,
                       j.st, m + 3 * rr, w, p->n, sd);
    return hipGetLastError();
  });
}

// one sweep: U, then V (with the new U), then the diagonals, then the
// optional normalization.  p_current: the projection partials of P = A_i V
// are those of the current V (the diagonal step before this sweep computed
// them, and no normalization has rescaled V since); the U step then only
// forms C_i = P_i S_i from them.
hipError_t als_sweep(Jd& j, const float* A, const float* B, const int32_t* lidx, bool normalize, bool p_current) {
  const cts_jd_problem* p = j.p;
  const int r = p->r;
  const int64_t rr = static_cast<int64_t>(r) * r;
  float* sd = j.at<float>(j.pl.off_sd);
  float* m = j.at<float>(j.pl.off_m);
  hipError_t e;
  // U = (sum_i B_i A_i V S_i)(V^T V o S2)^-1, S2 = sum_i s_i s_i^T
  {
    float* U = j.at<float>(j.pl.off_U);
    float* V = j.at<float>(j.pl.off_V);
    float* Un = j.at<float>(j.pl.off_Uo);
    if ((e = stage_mark(1, j.st)) != hipSuccess) return e;
    if ((e = launch_project(j, A, B, V, U, lidx, p->n, 3, nullptr, nullptr, nullptr, nullptr, 0, 0, 0,
                            p_current ? 0 : 1, sd, nullptr)) != hipSuccess)
      return e;
    if ((e = stage_mark(2, j.st)) != hipSuccess) return e;
    if ((e = expand_one(j, A, B, lidx, p->n, 0, Un, 3)) != hipSuccess) return e;
    if ((e = gram_hadamard_inverse(j, V, p->d_in, sd, p->n, m + 4 * rr)) != hipSuccess) return e;
    if ((e = apply_one(j, Un, p->d_out, 0, m + 4 * rr)) != hipSuccess) return e;
    std::swap(j.pl.off_U, j.pl.off_Uo);
  }
  // V = (sum_i A_i^T B_i^T U S_i)(U^T U o S2)^-1
  {
    float* U = j.at<float>(j.pl.off_U);
    float* V = j.at<float>(j.pl.off_V);
    float* Vn = j.at<float>(j.pl.off_Vo);
    if ((e = launch_project(j, A, B, V, U, lidx, p->n, 4, nullptr, nullptr, nullptr, nullptr, 0, 0, 1, 1, sd,
                            nullptr)) != hipSuccess)
      return e;
    if ((e = expand_one(j, A, B, lidx, p->n, 1, Vn)) != hipSuccess) return e;
    if ((e = gram_hadamard_inverse(j, U, p->d_out, sd, p->n, m + 5 * rr)) != hipSuccess) return e;
    if ((e = apply_one(j, Vn, p->d_in, 1, m + 4 * rr)) != hipSuccess) return e;   // slot 1 = m + 5 rr
    std::swap(j.pl.off_V, j.pl.off_Vo);
  }
  // diagonals: Q = B^T U is current from the V step; P = A V is recomputed
  if ((e = als_sigma(j, A, B, lidx, false)) != hipSuccess) return e;
  if (normalize) {
    float* nu = j.at<float>(j.pl.off_nu);
    const int64_t ns = static_cast<int64_t>(p->n) * r;
    hipLaunchKernelGGL(jd_norm_kernel, dim3(1), dim3(kJT), 0, j.st, sd, ns, nu);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(jd_scale_kernel, dim3(256), dim3(256), 0, j.st, sd, ns, nu, 1);
    hipLaunchKernelGGL(jd_scale_kernel, dim3(256), dim3(256), 0, j.st, j.at<float>(j.pl.off_U),
                       static_cast<int64_t>(p->d_out) * r, nu, 0);
    hipLaunchKernelGGL(jd_scale_kernel, dim3(256), dim3(256), 0, j.st, j.at<float>(j.pl.off_V),
                       static_cast<int64_t>(p->d_in) * r, nu, 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace
}  // namespace cts

using cts::Jd;

extern "C" {

size_t cts_jd_workspace_size(const cts_jd_problem* p) {
  if (cts::validate(p) != CTS_OK) return 0;
  cts::JdPlan pl;
  cts::plan_jd(p, 0, &pl);
  return pl.total;
}

size_t cts_jd_cluster_workspace_size(const cts_jd_problem* p, int32_t K) {
  if (cts::validate(p) != CTS_OK || K < 1 || K > p->n) return 0;
  cts::JdPlan pl;
  cts::plan_jd(p, K, &pl);
  return pl.total;
}

int cts_lora_norms2(const cts_jd_problem* p, const float* A, const float* B, float* norms2, void* workspace,
                    size_t workspace_bytes, void* stream) {
  int st = cts::validate(p);
  if (st != CTS_OK) return st;
  if (cts::bad_ptr(A, 16) || cts::bad_ptr(B, 16) || cts::bad_ptr(norms2, 4) || cts::bad_ptr(workspace, 16))
    return CTS_ERR_INVALID_ARG;
  Jd j{p, {}, static_cast<char*>(workspace), static_cast<hipStream_t>(stream)};
  cts::plan_jd(p, 0, &j.pl);
  if (workspace_bytes < j.pl.total) return CTS_ERR_WORKSPACE;
  hipLaunchKernelGGL(cts::jd_norms_kernel, dim3(p->n), dim3(cts::kJT), 0, j.st, A, B, p->r_lora, p->d_in,
                     p->d_out, norms2, nullptr, nullptr);
  return hipGetLastError() == hipSuccess ? CTS_OK : CTS_ERR_HIP;
}

int cts_jd_full(const cts_jd_problem* p, const float* A, const float* B, const float* U0, const float* Vt0,
                int32_t iters, float tau, int32_t normalize, float* U, float* Vt, float* Sigma, float* crit,
                int32_t* iters_done, void* workspace, size_t workspace_bytes, void* stream) {
  int st = cts::validate(p);
  if (st != CTS_OK) return st;
  if (iters < 1 || cts::bad_ptr(A, 16) || cts::bad_ptr(B, 16) || cts::bad_ptr(U0, 16) || cts::bad_ptr(Vt0, 16) ||
      cts::bad_ptr(U, 16) || cts::bad_ptr(Vt, 16) || cts::bad_ptr(Sigma, 16) || cts::bad_ptr(crit, 4) ||
      cts::bad_ptr(workspace, 16))
    return CTS_ERR_INVALID_ARG;
  Jd j{p, {}, static_cast<char*>(workspace), static_cast<hipStream_t>(stream)};
  cts::plan_jd(p, 0, &j.pl);
  if (workspace_bytes < j.pl.total) return CTS_ERR_WORKSPACE;
  int32_t* lidx = j.at<int32_t>(j.pl.off_lidx);
  hipLaunchKernelGGL(cts::jd_iota_kernel, dim3((p->n + 255) / 256), dim3(256), 0, j.st, lidx, p->n);
  if (hipGetLastError() != hipSuccess) return CTS_ERR_HIP;
  if (normalize && cts::norms(j, A, B) != hipSuccess) return CTS_ERR_HIP;
  if (cts::load_bases(j, U0, Vt0) != hipSuccess) return CTS_ERR_HIP;
  int done = 0;
  st = cts::run_jd(j, A, B, lidx, p->n, normalize ? j.at<float>(j.pl.off_w2) : nullptr, iters, tau, crit, &done);
  if (st != CTS_OK) return st;
  if (cts::launch_project(j, A, B, j.at<float>(j.pl.off_V), j.at<float>(j.pl.off_U), lidx, p->n, 1, nullptr,
                          nullptr, Sigma, nullptr, 0, 0) != hipSuccess)
    return CTS_ERR_HIP;
  if (cts::store_bases(j, U, Vt) != hipSuccess) return CTS_ERR_HIP;
  if (iters_done) *iters_done = done;
  return CTS_OK;
}

int cts_jd_diag(const cts_jd_problem* p, const float* A, const float* B, const float* U0, const float* Vt0,
                int32_t sweeps, int32_t normalize, float* U, float* Vt, float* sigma, void* workspace,
                size_t workspace_bytes, void* stream) {
  int st = cts::validate(p);
  if (st != CTS_OK) return st;
  if (sweeps < 0 || cts::bad_ptr(A, 16) || cts::bad_ptr(B, 16) || cts::bad_ptr(U0, 16) || cts::bad_ptr(Vt0, 16) ||
      cts::bad_ptr(U, 16) || cts::bad_ptr(Vt, 16) || cts::bad_ptr(sigma, 16) || cts::bad_ptr(workspace, 16))
    return CTS_ERR_INVALID_ARG;
  Jd j{p, {}, static_cast<char*>(workspace), static_cast<hipStream_t>(stream)};
  cts::plan_jd(p, 0, &j.pl);
  if (workspace_bytes < j.pl.total) return CTS_ERR_WORKSPACE;
  int32_t* lidx = j.at<int32_t>(j.pl.off_lidx);
  hipLaunchKernelGGL(cts::jd_iota_kernel, dim3((p->n + 255) / 256), dim3(256), 0, j.st, lidx, p->n);
  if (hipGetLastError() != hipSuccess) return CTS_ERR_HIP;
  if (cts::load_bases(j, U0, Vt0) != hipSuccess) return CTS_ERR_HIP;
  if (cts::als_sigma(j, A, B, lidx, true) != hipSuccess) return CTS_ERR_HIP;
  // P = A_i V from the initial diagonals' step is current for the first U
  // step, and so is each sweep's diagonal step's P for the next one (V is
  // unchanged between them unless the normalization rescaled it)
  for (int t = 0; t < sweeps; ++t)
    if (cts::als_sweep(j, A, B, lidx, normalize != 0, t == 0 || normalize == 0) != hipSuccess) return CTS_ERR_HIP;
  if (cts::store_bases(j, U, Vt) != hipSuccess) return CTS_ERR_HIP;
  if (hipMemcpyAsync(sigma, j.at<float>(j.pl.off_sd), sizeof(float) * p->n * p->r, hipMemcpyDeviceToDevice,
                     j.st) != hipSuccess)
    return CTS_ERR_HIP;
  return CTS_OK;
}

int cts_jd_sigma(const cts_jd_problem* p, const float* A, const float* B, const float* U, const float* Vt,
                 float* Sigma, void* workspace, size_t workspace_bytes, void* stream) {
  int st = cts::validate(p);
  if (st != CTS_OK) return st;
  if (cts::bad_ptr(A, 16) || cts::bad_ptr(B, 16) || cts::bad_ptr(U, 16) || cts::bad_ptr(Vt, 16) ||
      cts::bad_ptr(Sigma, 16) || cts::bad_ptr(workspace, 16))
    return CTS_ERR_INVALID_ARG;
  Jd j{p, {}, static_cast<char*>(workspace), static_cast<hipStream_t>(stream)};
  cts::plan_jd(p, 0, &j.pl);
  if (workspace_bytes < j.pl.total) return CTS_ERR_WORKSPACE;
  int32_t* lidx = j.at<int32_t>(j.pl.off_lidx);
  hipLaunchKernelGGL(cts::jd_iota_kernel, dim3((p->n + 255) / 256), dim3(256), 0, j.st, lidx, p->n);
  if (hipGetLastError() != hipSuccess) return CTS_ERR_HIP;
  if (cts::load_bases(j, U, Vt) != hipSuccess) return CTS_ERR_HIP;
  if (cts::launch_project(j, A, B, j.at<float>(j.pl.off_V), j.at<float>(j.pl.off_U), lidx, p->n, 1, nullptr,
                          nullptr, Sigma, nullptr, 0, 0) != hipSuccess)
    return CTS_ERR_HIP;
  return CTS_OK;
}

int cts_jd_cluster(const cts_jd_problem* p, int32_t K, const float* A, const float* B, const float* U0,
                   const float* Vt0, const float* Uc0, const float* Vtc0, const int32_t* init_idx,
                   int32_t jd_iters, int32_t max_rounds, int32_t normalize, int32_t* cluster_of, float* U,
                   float* Vt, float* Sigma, int32_t* rounds, void* workspace, size_t workspace_bytes,
                   void* stream) {
  int st = cts::validate(p);
  if (st != CTS_OK) return st;
  if (K < 1 || K > p->n || jd_iters < 1 || max_rounds < 1 || !init_idx) return CTS_ERR_INVALID_ARG;
  for (int k = 0; k < K; ++k)
    if (init_idx[k] < 0 || init_idx[k] >= p->n) return CTS_ERR_INVALID_ARG;
  if (cts::bad_ptr(A, 16) || cts::bad_ptr(B, 16) || cts::bad_ptr(U0, 16) || cts::bad_ptr(Vt0, 16) ||
      cts::bad_ptr(Uc0, 16) || cts::bad_ptr(Vtc0, 16) || cts::bad_ptr(cluster_of, 4) || cts::bad_ptr(U, 16) ||
      cts::bad_ptr(Vt, 16) || cts::bad_ptr(Sigma, 16) || cts::bad_ptr(workspace, 16))
    return CTS_ERR_INVALID_ARG;
  if (static_cast<int64_t>(K) * p->d_out * p->r >= (int64_t(1) << 31) ||
      static_cast<int64_t>(K) * p->r * p->r * p->n >= (int64_t(1) << 40))
    return CTS_ERR_UNSUPPORTED;
  Jd j{p, {}, static_cast<char*>(workspace), static_cast<hipStream_t>(stream)};
  cts::plan_jd(p, K, &j.pl);
  if (workspace_bytes < j.pl.total) return CTS_ERR_WORKSPACE;
  const int n = p->n, r = p->r, rr = r * r;
  const int64_t usz = static_cast<int64_t>(p->d_out) * r, vsz = static_cast<int64_t>(r) * p->d_in;
  int32_t* lidx = j.at<int32_t>(j.pl.off_lidx);
  int32_t* lab = j.at<int32_t>(j.pl.off_lab);
  int32_t* chg = j.at<int32_t>(j.pl.off_chg);
  int32_t* offs = j.at<int32_t>(j.pl.off_offs);
  int32_t* memb = j.at<int32_t>(j.pl.off_memb);
  float* S = j.at<float>(j.pl.off_S);
  float* cent = j.at<float>(j.pl.off_cent);
  float* dist = j.at<float>(j.pl.off_dist);
  float* score = j.at<float>(j.pl.off_score);
  const float* w2 = normalize ? j.at<float>(j.pl.off_w2) : nullptr;
  const float* w = normalize ? j.at<float>(j.pl.off_w) : nullptr;
  hipStream_t s = j.st;
  auto ok = [](hipError_t e) { return e == hipSuccess; };
  auto last = []() { return hipGetLastError() == hipSuccess; };

  hipLaunchKernelGGL(cts::jd_iota_kernel, dim3((n + 255) / 256), dim3(256), 0, s, lidx, n);
  if (!last()) return CTS_ERR_HIP;
  if (normalize && !ok(cts::norms(j, A, B))) return CTS_ERR_HIP;
  // single-basis JD and its cores (normalized LoRAs when asked)
  if (!ok(cts::load_bases(j, U0, Vt0))) return CTS_ERR_HIP;
  st = cts::run_jd(j, A, B, lidx, n, w2, jd_iters, 0.f, nullptr, nullptr);
  if (st != CTS_OK) return st;
  if (!ok(cts::launch_project(j, A, B, j.at<float>(j.pl.off_V), j.at<float>(j.pl.off_U), lidx, n, 1, nullptr, w, S,
                              nullptr, 0, 0)))
    return CTS_ERR_HIP;
  // k-means on vec(Sigma_i)
  std::vector<int32_t> init(init_idx, init_idx + K);
  int32_t* init_dev = memb;                         // staging for the K indices
  if (!ok(hipMemcpyAsync(init_dev, init.data(), sizeof(int32_t) * K, hipMemcpyHostToDevice, s)))
    return CTS_ERR_HIP;
  hipLaunchKernelGGL(cts::km_init_kernel, dim3((rr + 255) / 256, K), dim3(cts::kJT), 0, s, S, init_dev, rr, cent);
  if (!last()) return CTS_ERR_HIP;
  int32_t h_chg = 0;
  for (int it = 0; it < cts::kMaxKm; ++it) {
    hipLaunchKernelGGL(cts::km_dist_kernel, dim3(n), dim3(cts::kJT), 0, s, S, cent, rr, K, dist);
    if (!last()) return CTS_ERR_HIP;
    hipLaunchKernelGGL(cts::km_pick_kernel, dim3(1), dim3(cts::kJT), 0, s, dist, n, K, 1.f, lab, chg);
    if (!last()) return CTS_ERR_HIP;
    if (!ok(hipMemcpyAsync(&h_chg, chg, sizeof(int32_t), hipMemcpyDeviceToHost, s)) || !ok(hipStreamSynchronize(s)))
      return CTS_ERR_HIP;
    if (it > 0 && h_chg == 0) break;   // (the first assignment's count is not used)
    hipLaunchKernelGGL(cts::km_centroid_kernel, dim3((rr + 255) / 256, K), dim3(cts::kJT), 0, s, S, lab, n, rr,
                       cent);
    if (!last()) return CTS_ERR_HIP;
  }
  // rounds of per-cluster JD-Full and reassignment
  std::vector<int32_t> h_offs(K + 1);
  int rd = 0;
  for (rd = 1; rd <= max_rounds; ++rd) {
    hipLaunchKernelGGL(cts::km_members_kernel, dim3(1), dim3(cts::kJT), 0, s, lab, n, K, offs, memb);
    if (!last()) return CTS_ERR_HIP;
    if (!ok(hipMemcpyAsync(h_offs.data(), offs, sizeof(int32_t) * (K + 1), hipMemcpyDeviceToHost, s)) ||
        !ok(hipStreamSynchronize(s)))
      return CTS_ERR_HIP;
    for (int k = 0; k < K; ++k) {
      const int cnt = h_offs[k + 1] - h_offs[k];
      if (static_cast<int64_t>(cnt) * p->r_lora >= r) {
        if (!ok(cts::load_bases(j, Uc0 + k * usz, Vtc0 + k * vsz))) return CTS_ERR_HIP;
        st = cts::run_jd(j, A, B, memb + h_offs[k], cnt, w2, jd_iters, 0.f, nullptr, nullptr);
        if (st != CTS_OK) return st;
        if (!ok(cts::store_bases(j, U + k * usz, Vt + k * vsz))) return CTS_ERR_HIP;
      } else if (cnt > 0) {
        // fewer than r directions: the members' columns completed by the
        // given bases (a Step 1 minimizer, exact for every member)
        if (!ok(cts::span_bases(j, A, B, memb + h_offs[k], cnt, Uc0 + k * usz, Vtc0 + k * vsz)) ||
            !ok(cts::store_bases(j, U + k * usz, Vt + k * vsz)))
          return CTS_ERR_HIP;
      } else if (rd == 1) {
        // empty: keeps the given bases
        if (!ok(cts::load_bases(j, Uc0 + k * usz, Vtc0 + k * vsz)) || !ok(cts::store_bases(j, U + k * usz, Vt + k * vsz)))
          return CTS_ERR_HIP;
      }
    }
    // scores of every LoRA against every cluster's bases
    for (int k = 0; k < K; ++k) {
      if (!ok(cts::load_bases(j, U + k * usz, Vt + k * vsz))) return CTS_ERR_HIP;
      if (!ok(cts::launch_project(j, A, B, j.at<float>(j.pl.off_V), j.at<float>(j.pl.off_U), lidx, n, 2, nullptr,
                                  nullptr, nullptr, score, K, k)))
        return CTS_ERR_HIP;
    }
    hipLaunchKernelGGL(cts::km_pick_kernel, dim3(1), dim3(cts::kJT), 0, s, score, n, K, -1.f, lab, chg);
    if (!last()) return CTS_ERR_HIP;
    if (!ok(hipMemcpyAsync(&h_chg, chg, sizeof(int32_t), hipMemcpyDeviceToHost, s)) || !ok(hipStreamSynchronize(s)))
      return CTS_ERR_HIP;
    if (h_chg == 0) break;
  }
  if (rd > max_rounds) rd = max_rounds;
  // cores in each LoRA's own cluster bases (restored norms)
  hipLaunchKernelGGL(cts::km_members_kernel, dim3(1), dim3(cts::kJT), 0, s, lab, n, K, offs, memb);
  if (!last()) return CTS_ERR_HIP;
  if (!ok(hipMemcpyAsync(h_offs.data(), offs, sizeof(int32_t) * (K + 1), hipMemcpyDeviceToHost, s)) ||
      !ok(hipStreamSynchronize(s)))
    return CTS_ERR_HIP;
  for (int k = 0; k < K; ++k) {
    const int cnt = h_offs[k + 1] - h_offs[k];
    if (cnt == 0) continue;
    if (!ok(cts::load_bases(j, U + k * usz, Vt + k * vsz))) return CTS_ERR_HIP;
    if (!ok(cts::launch_project(j, A, B, j.at<float>(j.pl.off_V), j.at<float>(j.pl.off_U), memb + h_offs[k], cnt, 1,
                                nullptr, nullptr, Sigma, nullptr, 0, 0)))
      return CTS_ERR_HIP;
  }
  if (!ok(hipMemcpyAsync(cluster_of, lab, sizeof(int32_t) * n, hipMemcpyDeviceToDevice, s))) return CTS_ERR_HIP;
  if (rounds) *rounds = rd;
  return CTS_OK;
}

}  // extern "C"
