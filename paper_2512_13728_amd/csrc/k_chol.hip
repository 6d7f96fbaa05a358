// Orthogonalize (the paper leaves the method open; here: the thin-QR factor
// with positive-diagonal R, by CholQR): given the Gram matrix W = P~^T P~,
// factor W = T^T T (T upper triangular) and form P = P~ T^{-1}.
//
// Blocked in CB = 64 columns, fp64 throughout, every launch batched over all
// layers of the group (they share r):
//   chol_diag  (one wave per layer)  T_kk = chol(W_kk) in registers and its
//              inverse D_k = T_kk^{-1}; the first block also sets the pivot
//              floor max(1e-13 * max_i W_ii, 1e-60) (smaller or NaN pivots are raised to
//              it, the rest of their row of T is zero, and the layer is flagged
//              rank deficient; the absolute floor keeps T^{-1} finite in fp32
//              when P~ is numerically zero)
//   chol_panel X = D_k^T W[k, k+1:]: the k-th block row of T, zero in the
//              rows of floored pivots                              (fp64 MFMA)
//   chol_trail W[k+1:, k+1:] -= X^T X, upper tiles only            (fp64 MFMA)
// and the triangular solve, one launch per block column c:
//   P[:, c] = (P~[:, c] - P[:, :c] T[:c, c]) D_c                   (fp64 MFMA)
#include "chol_wave.hpp"
#include "common.hpp"
#include "mfma_tile.hpp"

namespace cd {
namespace {

constexpr int CB = CHOL_BLOCK;
using Wave64 = WaveChol<CB>;

// Orders the LDS accesses of the workgroup's waves across a barrier without
// waiting for their global stores (a plain __syncthreads would also wait for
// every store of T and D in flight, once per pivot).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Two waves per layer: the factorisation of the diagonal block and its
// inverse D_k in one pivot loop.  Wave 0 holds the block, one column per lane
// (rows shifted by one per pivot, as in chol_wave.hpp), and stores each row
// of T_kk over W_kk as soon as it is known; wave 1 holds the identity's
// columns and applies the same row operations, which turn I into
// E = T_kk^{-T} (the two-wave form of factor_inv, whose one-wave form carries
// both halves for blocks of up to 32 columns): row p of E is final once
// scaled by 1 / T[p][p], zero for a floored pivot, and D_k[c][p] = E[p][c].
// Per pivot, wave 0 publishes row p of T and the pivot's reciprocal in LDS
// (double-buffered by pivot parity), one barrier, then both waves update
// their rows below p.  Where the one-wave kernel ran the 64-step back
// substitution after the factorisation, wave 1 works beside wave 0.
__global__ __launch_bounds__(128) void k_chol_diag(const CholTab* __restrict__ tab, int r, int kb,
                                                   int pass, const int* run_if, int gated) {
  constexpr int ELD = CB + 1;
  constexpr int SEG = Wave64::SEG;
  __shared__ __attribute__((aligned(16))) double rowb[2][2 * CB];   // row p of T, then zeros
  __shared__ double pinv[2];                                         // 1 / T[p][p]; 0: floored
  __shared__ double Es[CB * ELD];                                    // E[p][c] at p * ELD + c
  __shared__ int okb[CB];
  if (skip_launch(run_if)) return;
  const CholTab t = tab[blockIdx.x];
  if (gated && *global_view(t.nid_ok)) return;
  double* const W = global_view(t.W);
  double* const floor_ = global_view(t.floor_);
  int* const rankdef = global_view(t.rankdef);
  const int tid = threadIdx.x, j = tid & 63;
  const bool ewave = tid >= 64;                 // uniform per wave
  const long long ld = r;
  const int k0 = kb * CB, nb = min(CB, r - k0);
  double fl = 0.0;
  if (!ewave) {
    if (kb == 0) {
      double md = 0.0;
      for (int k = j; k < r; k += 64) md = fmax(md, W[k * ld + k]);
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) md = fmax(md, __shfl_xor(md, o, 64));
      fl = fmax(1e-13 * md, 1e-60);
      if (j == 0) {
        *floor_ = fl;
        if (pass == 0) {
          *rankdef = 0;
          if (t.rankdef_host) *t.rankdef_host = 0;
        }
      }
    } else {
      fl = *floor_;
    }
  }
  double a[CB];   // a[i] = row p + i of this lane's column at pivot p
#pragma unroll
  for (int i = 0; i < CB; ++i) {
    if (ewave) a[i] = (i == j && j < nb) ? 1.0 : 0.0;
    else if (i < nb && j < nb) a[i] = i <= j ? W[(k0 + i) * ld + k0 + j] : 0.0;
    else a[i] = i == j ? 1.0 : 0.0;
  }
  if (!ewave) {
    rowb[0][CB + j] = 0.0;
    rowb[1][CB + j] = 0.0;
  }
  bool def = false;                             // wave 0: a pivot was floored
  auto pivot = [&](auto na, int p) {
    constexpr int NA = decltype(na)::value;
    const int b = p & 1;
    double tp;
    if (!ewave) {
      const double a0 = a[0];
      double d = __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(a0), p),
                                  __builtin_amdgcn_readlane(__double2loint(a0), p));
      const bool floored = !(d > fl);
      if (floored) { d = fl; def = true; }
      double inv = __builtin_amdgcn_rsq(d);
#pragma unroll
      for (int it = 0; it < 2; ++it) inv = fma(inv, fma(-0.5 * d * inv, inv, 0.5), inv);
      const double piv = d * inv;
      tp = j == p ? piv : (j > p && !floored ? a0 * inv : 0.0);
      if (j >= p && j < nb) W[(k0 + p) * ld + k0 + j] = tp;
      rowb[b][j] = tp;
      if (j == p) {
        pinv[b] = floored ? 0.0 : inv;
        okb[p] = floored ? 0 : 1;
      }
    }
    lds_barrier();
    if (ewave) {
      tp = a[0] * pinv[b];
      Es[p * ELD + j] = tp;
    }
    chunked<NA - 1>([&](int i) { return rowb[b][p + 1 + i]; },
                    [&](int i, double v) { a[i] = fma(-v, tp, a[i + 1]); });
    a[NA - 1] = 0.0;
  };
  // segment g: pivots [g SEG, (g + 1) SEG) with CB - g SEG live rows (both
  // waves run the same pivots, hence the same barriers)
  static_for<CB / SEG>([&](auto gc) {
    constexpr int G = decltype(gc)::value;
#pragma unroll 1
    for (int p = G * SEG; p < min(nb, (G + 1) * SEG); ++p) pivot(std::integral_constant<int, CB - G * SEG>{}, p);
  });
  __syncthreads();
  if (!ewave && j < nb) global_view(t.rowok)[k0 + j] = okb[j];
  double* const D = global_view(t.Dinv) + static_cast<long long>(kb) * CB * CB;
  for (int idx = tid; idx < CB * CB; idx += 128) {
    const int p = idx / CB, q = idx % CB;
    D[idx] = (p < nb && q < nb) ? Es[q * ELD + p] : 0.0;   // (T^{-1})[p][q] = E[q][p]
  }
  if (tid == 0 && def) {
    *rankdef = 1;
    if (t.rankdef_host) *t.rankdef_host = 1;
  }
}

__global__ __launch_bounds__(256) void k_chol_panel(const CholTab* __restrict__ tab, int r, int kb,
                                                    const int* run_if, int gated) {
  __shared__ __attribute__((aligned(16))) double As[tile_elems<CB>()];
  __shared__ __attribute__((aligned(16))) double Bs[tile_elems<CB>()];
  if (skip_launch(run_if)) return;
  const CholTab t = tab[blockIdx.y];
  if (gated && *global_view(t.nid_ok)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 32, wn0 = (wave & 1) * 32;
  const int k0 = kb * CB, nb = min(CB, r - k0), k1 = k0 + nb;
  const int j0 = k1 + blockIdx.x * CB;
  const double* D = global_view(t.Dinv) + static_cast<long long>(kb) * CB * CB;
  double* const W = global_view(t.W);
  const int* const rowok = global_view(t.rowok);
  const double* Wp = W + static_cast<long long>(k0) * r;  // block row k
  Tile64 T;
  T.zero();
  for (int kk0 = 0; kk0 < nb; kk0 += GBK) {
    // A(i, k) = D[k][i];  B(k, j) = W[k0 + k][j0 + j]
    stage_tile<double, double, CB, 256, false>(As, D, CB, 0, nb, kk0, nb, tid);
    stage_tile<double, double, CB, 256, false>(Bs, Wp + j0, r, 0, r - j0, kk0, nb, tid);
    __syncthreads();
    T.mma_stage<false>(As, Bs, wm0, wn0, lane);
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = wm0 + i * 16 + Mfma<double>::out_row(lane, v);
        const int col = j0 + wn0 + j * 16 + (lane & 15);
        if (row < nb && col < r)
          W[static_cast<long long>(k0 + row) * r + col] = rowok[k0 + row] ? T.acc[i][j][v] : 0.0;
      }
}

__global__ __launch_bounds__(256) void k_chol_trail(const CholTab* __restrict__ tab, int r, int kb,
                                                    const int* run_if, int gated) {
  __shared__ __attribute__((aligned(16))) double As[tile_elems<CB>()];
  __shared__ __attribute__((aligned(16))) double Bs[tile_elems<CB>()];
  if (skip_launch(run_if)) return;
  const CholTab t = tab[blockIdx.y];
  if (gated && *global_view(t.nid_ok)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 32, wn0 = (wave & 1) * 32;
  const int k0 = kb * CB, nb = min(CB, r - k0), k1 = k0 + nb;
  const int nt = (r - k1 + CB - 1) / CB;
  int u = blockIdx.x, ti = 0;
  while (u >= nt - ti) { u -= nt - ti; ++ti; }
  const int tj = ti + u;
  const int i0 = k1 + ti * CB, j0 = k1 + tj * CB;
  double* const W = global_view(t.W);
  const double* X = W + static_cast<long long>(k0) * r;   // rows k0..k1 of T
  Tile64 T;
  T.zero();
  for (int kk0 = 0; kk0 < nb; kk0 += GBK) {
    // A(i, p) = X[p][i0 + i];  B(p, j) = X[p][j0 + j]
    stage_tile<double, double, CB, 256, false>(As, X + i0, r, 0, r - i0, kk0, nb, tid);
    stage_tile<double, double, CB, 256, false>(Bs, X + j0, r, 0, r - j0, kk0, nb, tid);
    __syncthreads();
    T.mma_stage<false>(As, Bs, wm0, wn0, lane);
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = i0 + wm0 + i * 16 + Mfma<double>::out_row(lane, v);
        const int col = j0 + wn0 + j * 16 + (lane & 15);
        if (row < r && col < r) W[static_cast<long long>(row) * r + col] -= T.acc[i][j][v];
      }
}

// Completion of the basis past the numerical rank, between the two CholQR
// passes: a column of P1 = P~ T^{-1} whose pivot was floored is zero; it is
// replaced by a fixed pseudo-random vector of unit expected norm, which the
// second pass orthonormalises against the other columns.  P then has
// orthonormal columns, as a Householder QR factor of a rank-deficient P~
// does, and the columns of Q that belong to them are not lost for the later
// steps.  Workgroups of layers whose factorisation floored no pivot return
// at once.
constexpr int FILL_ROWS = 64;

template <typename T>
__global__ __launch_bounds__(256) void k_fill_dead(const CholTab* __restrict__ ct,
                                                   const TrsmTab* __restrict__ tt, int r, const int* run_if) {
  if (skip_launch(run_if)) return;
  const CholTab c = ct[blockIdx.y];
  if (*global_view(c.rankdef) == 0) return;
  const int* const rowok = global_view(c.rowok);
  const TrsmTab t = tt[blockIdx.y];
  T* P1 = global_view(static_cast<T*>(t.Pout));
  const int i0 = blockIdx.x * FILL_ROWS;
  const int rows = min(FILL_ROWS, t.m - i0);
  if (rows <= 0) return;
  const float scale = sqrtf(3.0f / static_cast<float>(t.m));
  for (int e = threadIdx.x; e < rows * r; e += 256) {
    const int i = i0 + e / r, j = e % r;
    if (!rowok[j]) P1[static_cast<long long>(i) * r + j] = static_cast<T>(fill_value(i, j, scale));
  }
}

// Block column c of P = P~ T^{-1}; one 64-row tile of one layer per workgroup.
// IDENT: P~ is the identity (P = T^{-1}, upper triangular, exact zeros below).
// mlimit > 0 caps the row count (the identity has r rows).
template <typename TIn, typename TOut, bool IDENT>
__global__ __launch_bounds__(256) void k_trsm(const TrsmTab* __restrict__ tab, const int2* __restrict__ tiles,
                                              int r, int cb, int mlimit, const int* run_if) {
  constexpr int YLD = CB + 4;
  // Y takes the A tile's place once the first product is done (52 KB in all
  // instead of 70: the workgroup then fits where one workgroup of the
  // concurrently running update or product kernels left)
  constexpr int AY = tile_elems<CB>() > CB * YLD ? tile_elems<CB>() : CB * YLD;
  __shared__ __attribute__((aligned(16))) double AYs[AY];
  __shared__ __attribute__((aligned(16))) double Bs[tile_elems<CB>()];
  double* const As = AYs;
  double* const Ys = AYs;
  if (skip_launch(run_if)) return;
  const int2 lt = tiles[blockIdx.x];
  const TrsmTab t = tab[lt.x];
  const int m = mlimit > 0 ? min(t.m, mlimit) : t.m;
  const int i0 = lt.y * CB;
  if (i0 >= m) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 32, wn0 = (wave & 1) * 32;
  const int c0 = cb * CB, nbc = min(CB, r - c0);
  const TIn* Pin = global_view(static_cast<const TIn*>(t.Pin));
  TOut* Pout = global_view(static_cast<TOut*>(t.Pout));
  const double* const W = global_view(t.W);
  if constexpr (IDENT) {
    // T^{-1} is upper triangular: a row tile below the diagonal block is zero
    if (lt.y > cb) {
      for (int idx = tid; idx < CB * CB; idx += 256) {
        const int row = idx / CB, col = idx % CB;
        if (i0 + row < m && col < nbc) Pout[static_cast<long long>(i0 + row) * r + c0 + col] = TOut(0);
      }
      return;
    }
  }
  Tile64 T;
  T.zero();
  // acc = P[:, :c0] T[:c0, c0:c0+64]   (P is the output: earlier block columns;
  // for T^{-1} its rows i0.. are zero left of column i0)
  // (the next stage's loads are in flight while this one is multiplied)
  const int kbeg = IDENT ? i0 : 0;
  const TOut* Prow = Pout + static_cast<long long>(i0) * r;
  Prefetch<TOut, CB, 256, true> pa;
  Prefetch<double, CB, 256, false> pb;
  if (kbeg < c0) {
    pa.load(Prow, r, 0, m - i0, kbeg, c0, tid);
    pb.load(W + c0, r, 0, nbc, kbeg, c0, tid);
  }
  for (int k0 = kbeg; k0 < c0; k0 += GBK) {
    pa.template store<double>(As, tid);
    pb.template store<double>(Bs, tid);
    __syncthreads();
    if (k0 + GBK < c0) {
      pa.load(Prow, r, 0, m - i0, k0 + GBK, c0, tid);
      pb.load(W + c0, r, 0, nbc, k0 + GBK, c0, tid);
    }
    T.mma_stage<true>(As, Bs, wm0, wn0, lane);
    __syncthreads();
  }
  // Y = P~[:, c-block] - acc, into LDS as the next A operand ([row][k], k = column)
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = wm0 + i * 16 + Mfma<double>::out_row(lane, v);
        const int col = wn0 + j * 16 + (lane & 15);
        double y = 0.0;
        if (i0 + row < m && col < nbc) {
          double pin;
          if constexpr (IDENT) pin = (i0 + row == c0 + col) ? 1.0 : 0.0;
          else pin = static_cast<double>(Pin[static_cast<long long>(i0 + row) * r + c0 + col]);
          y = pin - T.acc[i][j][v];
        }
        Ys[row * YLD + col] = y;
      }
  const double* D = global_view(t.Dinv) + static_cast<long long>(cb) * CB * CB;
  T.zero();
  for (int k0 = 0; k0 < nbc; k0 += GBK) {
    stage_tile<double, double, CB, 256, false>(Bs, D, CB, 0, nbc, k0, nbc, tid);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GBK; kk += 16) {
      f64x4 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const f64x4*>(Ys + (wm0 + i * 16 + (lane & 15)) * YLD + k0 + kk +
                                               4 * (lane >> 4));
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = frag<double, CB, false>(Bs, wn0 + j * 16, kk, lane);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            T.acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i][q], b[j][q], T.acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = wm0 + i * 16 + Mfma<double>::out_row(lane, v);
        const int col = wn0 + j * 16 + (lane & 15);
        if (i0 + row < m && col < nbc)
          Pout[static_cast<long long>(i0 + row) * r + c0 + col] = static_cast<TOut>(T.acc[i][j][v]);
      }
}

// The same solve for fp64 panels in place (fp32-gradient layers), right-
// looking: launch c (-1 <= c <= nblk - 2) reads the finished block column c
// and takes every block column j > c of one 64-row tile per workgroup,
//   j = c + 1:  P[:, j] = (P~[:, j] - P[:, c] T[c, j]) D_j   (c = -1: P~[:, 0] D_0)
//   j > c + 1:  P~[:, j] -= P[:, c] T[c, j]
// Every block of the panel is written by one workgroup and column c by none,
// so a launch has no races.  It spans nblk - c - 1 column blocks of each row
// tile, each with one or two 64 x 64 x 64 products, where the left-looking
// form keeps m / 64 workgroups busy for the whole K = 64 c of every column.
__global__ __launch_bounds__(256) void k_trsm_rl(const TrsmTab* __restrict__ tab, const int2* __restrict__ tiles,
                                                 int r, int c, const int* run_if) {
  constexpr int YLD = CB + 4;
  constexpr int AY = tile_elems<CB>() > CB * YLD ? tile_elems<CB>() : CB * YLD;
  __shared__ __attribute__((aligned(16))) double AYs[AY];
  __shared__ __attribute__((aligned(16))) double Bs[tile_elems<CB>()];
  double* const As = AYs;
  double* const Ys = AYs;
  if (skip_launch(run_if)) return;
  const int2 lt = tiles[blockIdx.x];
  const TrsmTab t = tab[lt.x];
  const int m = t.m, i0 = lt.y * CB;
  if (i0 >= m) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 32, wn0 = (wave & 1) * 32;
  const int j = c + 1 + blockIdx.y, j0 = j * CB, nbj = min(CB, r - j0);
  double* const P = global_view(static_cast<double*>(t.Pout));
  const double* const W = global_view(t.W);
  Tile64 T;
  T.zero();
  if (c >= 0) {
    // acc = P[i-tile, c-block] T[c-block, j-block]; block c is whole (c < nblk - 1)
    const int c0 = c * CB;
    for (int k0 = 0; k0 < CB; k0 += GBK) {
      stage_tile<double, double, CB, 256, true>(As, P + static_cast<long long>(i0) * r + c0, r, 0, m - i0, k0, CB,
                                                tid);
      stage_tile<double, double, CB, 256, false>(Bs, W + static_cast<long long>(c0) * r + j0, r, 0, nbj, k0, CB,
                                                 tid);
      __syncthreads();
      T.mma_stage<true>(As, Bs, wm0, wn0, lane);
      __syncthreads();
    }
  }
  if (j > c + 1) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = wm0 + i * 16 + Mfma<double>::out_row(lane, v);
          const int col = wn0 + jj * 16 + (lane & 15);
          if (i0 + row < m && col < nbj) P[static_cast<long long>(i0 + row) * r + j0 + col] -= T.acc[i][jj][v];
        }
    return;
  }
  // Y = P~[:, j] - acc, into LDS as the A operand of Y D_j ([row][k], k = column)
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = wm0 + i * 16 + Mfma<double>::out_row(lane, v);
        const int col = wn0 + jj * 16 + (lane & 15);
        double y = 0.0;
        if (i0 + row < m && col < nbj) y = P[static_cast<long long>(i0 + row) * r + j0 + col] - T.acc[i][jj][v];
        Ys[row * YLD + col] = y;
      }
  const double* D = global_view(t.Dinv) + static_cast<long long>(j) * CB * CB;
  T.zero();
  for (int k0 = 0; k0 < nbj; k0 += GBK) {
    stage_tile<double, double, CB, 256, false>(Bs, D, CB, 0, nbj, k0, nbj, tid);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GBK; kk += 16) {
      f64x4 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const f64x4*>(Ys + (wm0 + i * 16 + (lane & 15)) * YLD + k0 + kk +
                                               4 * (lane >> 4));
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) b[jj] = frag<double, CB, false>(Bs, wn0 + jj * 16, kk, lane);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int jj = 0; jj < 2; ++jj)
            T.acc[i][jj] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i][q], b[jj][q], T.acc[i][jj], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = wm0 + i * 16 + Mfma<double>::out_row(lane, v);
        const int col = wn0 + jj * 16 + (lane & 15);
        if (i0 + row < m && col < nbj) P[static_cast<long long>(i0 + row) * r + j0 + col] = T.acc[i][jj][v];
      }
}

}  // namespace

hipError_t launch_cholesky(const CholTab* tab, int nlayers, int r, int pass, hipStream_t s, const int* run_if,
                           bool gated) {
  if (nlayers <= 0) return hipSuccess;
  if (r < 1) return hipErrorInvalidValue;
  const int nblk = (r + CB - 1) / CB, g = gated ? 1 : 0;
  for (int kb = 0; kb < nblk; ++kb) {
    hipLaunchKernelGGL(k_chol_diag, dim3(nlayers), dim3(128), 0, s, tab, r, kb, pass, run_if, g);
    const int k1 = min(r, (kb + 1) * CB);
    if (k1 >= r) break;
    const int nt = (r - k1 + CB - 1) / CB;
    hipLaunchKernelGGL(k_chol_panel, dim3(nt, nlayers), dim3(256), 0, s, tab, r, kb, run_if, g);
    hipLaunchKernelGGL(k_chol_trail, dim3(nt * (nt + 1) / 2, nlayers), dim3(256), 0, s, tab, r, kb, run_if, g);
  }
  return hipGetLastError();
}

hipError_t launch_fill_dead(const CholTab* ct, const TrsmTab* tt, int nlayers, int mmax, int r, bool p64,
                            hipStream_t s, const int* run_if) {
  if (nlayers <= 0 || mmax <= 0) return hipSuccess;
  const dim3 grid((mmax + FILL_ROWS - 1) / FILL_ROWS, nlayers);
  if (p64) hipLaunchKernelGGL(k_fill_dead<double>, grid, dim3(256), 0, s, ct, tt, r, run_if);
  else hipLaunchKernelGGL(k_fill_dead<float>, grid, dim3(256), 0, s, ct, tt, r, run_if);
  return hipGetLastError();
}

hipError_t launch_trsm_rl(const TrsmTab* tab, const int2* tiles, int ntiles, int r, hipStream_t s,
                          const int* run_if) {
  if (ntiles <= 0) return hipSuccess;
  if (r < 1) return hipErrorInvalidValue;
  const int nblk = (r + CB - 1) / CB;
  // c = -1 only finishes block column 0 (there is nothing to subtract yet)
  for (int c = -1; c <= nblk - 2; ++c)
    hipLaunchKernelGGL(k_trsm_rl, dim3(ntiles, c < 0 ? 1 : nblk - c - 1), dim3(256), 0, s, tab, tiles, r, c,
                       run_if);
  return hipGetLastError();
}

hipError_t launch_trsm(const TrsmTab* tab, const int2* tiles, int ntiles, int r, bool in64, bool out64,
                       hipStream_t s, bool ident, int mlimit, const int* run_if) {
  if (ntiles <= 0) return hipSuccess;
  const int nblk = (r + CB - 1) / CB;
  const dim3 grid(ntiles), block(256);
  for (int cb = 0; cb < nblk; ++cb) {
    if (ident) {
      if (out64) hipLaunchKernelGGL((k_trsm<double, double, true>), grid, block, 0, s, tab, tiles, r, cb, mlimit, run_if);
      else hipLaunchKernelGGL((k_trsm<double, float, true>), grid, block, 0, s, tab, tiles, r, cb, mlimit, run_if);
    } else if (in64 && out64) {
      hipLaunchKernelGGL((k_trsm<double, double, false>), grid, block, 0, s, tab, tiles, r, cb, mlimit, run_if);
    } else if (in64) {
      hipLaunchKernelGGL((k_trsm<double, float, false>), grid, block, 0, s, tab, tiles, r, cb, mlimit, run_if);
    } else if (out64) {
      hipLaunchKernelGGL((k_trsm<float, double, false>), grid, block, 0, s, tab, tiles, r, cb, mlimit, run_if);
    } else {
      hipLaunchKernelGGL((k_trsm<float, float, false>), grid, block, 0, s, tab, tiles, r, cb, mlimit, run_if);
    }
  }
  return hipGetLastError();
}

}  // namespace cd
