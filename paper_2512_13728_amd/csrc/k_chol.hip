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
#include <type_traits>
#include <utility>

#include "common.hpp"
#include "mfma_tile.hpp"

namespace cd {
namespace {

constexpr int CB = CHOL_BLOCK;

// One wave per layer: lane j holds column j of the 64 x 64 diagonal block
// (upper triangle; rows past the matrix padded with the identity) in
// registers.  Right-looking Cholesky: at pivot p the lanes publish row p of
// the updated block in LDS and every lane reads it back with uniform-address
// loads (a broadcast), then updates its own column.  The register array is
// shifted by one row per pivot inside the update (a[i] holds row p + i), so
// the pivot row is always a[0] and every index is a constant while the pivot
// loop itself stays rolled: the kernel is a few KB of code instead of a
// fully unrolled 100 KB that the instruction cache cannot hold.
//
// A pivot at or below the floor is raised to it and the rest of its row of T
// is set to zero (as is the row of the block row that k_chol_panel forms,
// through rowok): the numerically dependent direction then adds nothing to
// the trailing matrix.  Dividing its rounding-level residuals by the floor's
// square root instead would subtract their squares from the next pivots,
// which fall under the floor in turn, and the entries grow without bound.
//
// D = T^{-1} follows by back substitution, lane c solving T d = e_c from the
// last row up, with T read from LDS and the unknowns shifted the same way;
// the columns of floored pivots are stored as zero, so that P~ T^{-1} is
// zero in those columns (k_fill_dead then gives them new directions).
constexpr int TLD = CB + 1;   // padded row of T in LDS (column stores hit distinct banks)
constexpr int TPAD = CB;      // leading doubles: back-substitution reads above row 0 stay in the array
constexpr int SEG = 8;        // pivots per segment of the diagonal-block loops

// f(integral_constant<int, 0>) ... f(integral_constant<int, N - 1>), in order
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_chol_diag(const CholTab* __restrict__ tab, int r, int kb,
                                                  int pass, const int* run_if) {
  __shared__ __attribute__((aligned(16))) double rowb[2 * CB];   // row p, then zeros
  __shared__ double Tsb[TPAD + CB * TLD];
  __shared__ double pinv[CB];                                     // 1 / T[p][p]
  __shared__ int okb[CB];                                         // pivot p not floored
  double* const Ts = Tsb + TPAD;   // Ts[j * TLD + i] = T[i][j]
  if (skip_launch(run_if)) return;
  const CholTab t = tab[blockIdx.x];
  const int j = threadIdx.x;
  const long long ld = r;
  const int k0 = kb * CB, nb = min(CB, r - k0);
  double fl;
  if (kb == 0) {
    double md = 0.0;
    for (int k = j; k < r; k += 64) md = fmax(md, t.W[k * ld + k]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) md = fmax(md, __shfl_xor(md, o, 64));
    fl = fmax(1e-13 * md, 1e-60);
    if (j == 0) {
      *t.floor_ = fl;
      if (pass == 0) {
        *t.rankdef = 0;
        if (t.rankdef_host) *t.rankdef_host = 0;
      }
    }
  } else {
    fl = *t.floor_;
  }
  double a[CB];   // a[i] = A[p + i][j] at pivot p
#pragma unroll
  for (int i = 0; i < CB; ++i) {
    if (i < nb && j < nb) a[i] = i <= j ? t.W[(k0 + i) * ld + k0 + j] : 0.0;
    else a[i] = i == j ? 1.0 : 0.0;
  }
  rowb[CB + j] = 0.0;
  Tsb[j] = 0.0;
  bool def = false;
  // Only the block's nb pivots run: the identity padding of a last, partial
  // block would factor to itself, and its rows are never stored.  At pivot p
  // only rows p .. 63 remain, so the pivots run in segments of SEG whose
  // register arrays carry 64, 64 - SEG, ... rows (rows past the live range
  // stay untouched and unused).
  auto pivot = [&](auto na, int p) {
    constexpr int NA = decltype(na)::value;
    // the pivot A[p][p] is lane p's a[0]: read across the wave (no LDS trip)
    const double a0 = a[0];
    double d = __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(a0), p),
                                __builtin_amdgcn_readlane(__double2loint(a0), p));
    const bool floored = !(d > fl);   // uniform over the wave
    if (floored) { d = fl; def = true; }
    // 1/sqrt(d): the hardware estimate refined by two Newton steps (error
    // squared each step), then sqrt(d) = d / sqrt(d); both within about an
    // ulp, with no divide in the pivot's dependency chain
    double inv = __builtin_amdgcn_rsq(d);
#pragma unroll
    for (int it = 0; it < 2; ++it) inv = fma(inv, fma(-0.5 * d * inv, inv, 0.5), inv);
    const double piv = d * inv;
    // row p of T (zero left of the diagonal, and right of a floored pivot)
    const double tp = j == p ? piv : (j > p && !floored ? a[0] * inv : 0.0);
    Ts[j * TLD + p] = tp;
    if (j == p) {
      pinv[p] = inv;
      okb[p] = floored ? 0 : 1;
      t.rowok[k0 + p] = floored ? 0 : 1;
    }
    __syncthreads();
    rowb[j] = tp;
    __syncthreads();
    // rows below p: A[p + i][j] -= T[p][p + i] T[p][j], shifted up one row;
    // lanes j < p + i only touch the (unused) lower triangle.  The row is read
    // whole before the update (one LDS round trip, not one per pair).
    double rv[NA];
#pragma unroll
    for (int i = 1; i < NA; ++i) rv[i] = rowb[p + i];
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 1; i < NA; ++i) a[i - 1] = fma(-rv[i], tp, a[i]);
    a[NA - 1] = 0.0;
    __syncthreads();
  };
  // segment s: pivots [s SEG, (s + 1) SEG) with CB - s SEG live rows
  static_for<CB / SEG>([&](auto sc) {
    constexpr int S = decltype(sc)::value;
#pragma unroll 1
    for (int p = S * SEG; p < min(nb, (S + 1) * SEG); ++p) pivot(std::integral_constant<int, CB - S * SEG>{}, p);
  });

  // f[k] = d[p - k] at step p, from p = nb - 1 down; entries with k > p lie
  // above row 0 and are never stored, so the steps of pivots below
  // 64 - SEG s carry only 64 - SEG s entries
  double f[CB];
#pragma unroll
  for (int k = 0; k < CB; ++k) f[k] = k == nb - 1 - j ? 1.0 : 0.0;
  double* D = t.Dinv + static_cast<long long>(kb) * CB * CB;
  // the column of a floored pivot is stored as zero: P~ T^{-1} then has a
  // zero column there and the other columns are unchanged (with row p of T
  // zero right of the diagonal, column j != p of T^{-1} is zero in row p)
  const bool cin = j < nb && okb[j];
  for (int p = nb; p < CB; ++p) D[p * CB + j] = 0.0;   // rows past a partial block
  auto back = [&](auto nf, int p) {
    constexpr int NF = decltype(nf)::value;
    const double x = f[0] * pinv[p];
    D[p * CB + j] = cin ? x : 0.0;
    const double* col = Ts + p * TLD + p;   // col[-k] = T[p - k][p]
    double cv[NF];
#pragma unroll
    for (int k = 1; k < NF; ++k) cv[k] = col[-k];
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int k = 1; k < NF; ++k) f[k - 1] = fma(-cv[k], x, f[k]);
    f[NF - 1] = 0.0;
  };
  // segments from the last down: segment s carries (s + 1) SEG entries
  static_for<CB / SEG>([&](auto ic) {
    constexpr int S = CB / SEG - 1 - decltype(ic)::value;
#pragma unroll 1
    for (int p = min(nb, (S + 1) * SEG) - 1; p >= S * SEG; --p) back(std::integral_constant<int, (S + 1) * SEG>{}, p);
  });
#pragma unroll 4
  for (int i = 0; i < nb; ++i)
    if (j < nb && i <= j) t.W[(k0 + i) * ld + k0 + j] = Ts[j * TLD + i];
  if (j == 0 && def) {
    *t.rankdef = 1;
    if (t.rankdef_host) *t.rankdef_host = 1;
  }
}

// 64 x 64 fp64 MFMA tile: acc += A(64 x K) B(K x 64) with both operands staged
// through LDS.  4 waves as 2 x 2, each 32 x 32.
struct Tile64 {
  f64x4 acc[2][2];
  __device__ void zero() {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = f64x4{};
  }
  // B is always staged k-major; A as A_KC says
  template <bool A_KC>
  __device__ void mma_stage(const double* As, const double* Bs, int wm0, int wn0, int lane) {
#pragma unroll
    for (int kk = 0; kk < GBK; kk += 16) {
      f64x4 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = frag<double, CB, A_KC>(As, wm0 + i * 16, kk, lane);
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = frag<double, CB, false>(Bs, wn0 + j * 16, kk, lane);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i][q], b[j][q], acc[i][j], 0, 0, 0);
    }
  }
};

__global__ __launch_bounds__(256) void k_chol_panel(const CholTab* __restrict__ tab, int r, int kb,
                                                    const int* run_if) {
  __shared__ __attribute__((aligned(16))) double As[tile_elems<CB>()];
  __shared__ __attribute__((aligned(16))) double Bs[tile_elems<CB>()];
  if (skip_launch(run_if)) return;
  const CholTab t = tab[blockIdx.y];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 32, wn0 = (wave & 1) * 32;
  const int k0 = kb * CB, nb = min(CB, r - k0), k1 = k0 + nb;
  const int j0 = k1 + blockIdx.x * CB;
  const double* D = t.Dinv + static_cast<long long>(kb) * CB * CB;
  const double* Wp = t.W + static_cast<long long>(k0) * r;  // block row k
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
          t.W[static_cast<long long>(k0 + row) * r + col] = t.rowok[k0 + row] ? T.acc[i][j][v] : 0.0;
      }
}

__global__ __launch_bounds__(256) void k_chol_trail(const CholTab* __restrict__ tab, int r, int kb,
                                                    const int* run_if) {
  __shared__ __attribute__((aligned(16))) double As[tile_elems<CB>()];
  __shared__ __attribute__((aligned(16))) double Bs[tile_elems<CB>()];
  if (skip_launch(run_if)) return;
  const CholTab t = tab[blockIdx.y];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 32, wn0 = (wave & 1) * 32;
  const int k0 = kb * CB, nb = min(CB, r - k0), k1 = k0 + nb;
  const int nt = (r - k1 + CB - 1) / CB;
  int u = blockIdx.x, ti = 0;
  while (u >= nt - ti) { u -= nt - ti; ++ti; }
  const int tj = ti + u;
  const int i0 = k1 + ti * CB, j0 = k1 + tj * CB;
  const double* X = t.W + static_cast<long long>(k0) * r;   // rows k0..k1 of T
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
        if (row < r && col < r) t.W[static_cast<long long>(row) * r + col] -= T.acc[i][j][v];
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

__device__ __forceinline__ float fill_value(unsigned i, unsigned j, float scale) {
  // integer hash of (row, column): xorshift-multiply rounds
  unsigned h = i * 0x9E3779B1u + j * 0x85EBCA77u + 0x27D4EB2Fu;
  h ^= h >> 16; h *= 0x7FEB352Du;
  h ^= h >> 15; h *= 0x846CA68Bu;
  h ^= h >> 16;
  return scale * (static_cast<float>(h >> 8) * (2.0f / 16777216.0f) - 1.0f);   // uniform in [-1, 1)
}

template <typename T>
__global__ __launch_bounds__(256) void k_fill_dead(const CholTab* __restrict__ ct,
                                                   const TrsmTab* __restrict__ tt, int r, const int* run_if) {
  if (skip_launch(run_if)) return;
  const CholTab c = ct[blockIdx.y];
  if (*c.rankdef == 0) return;
  const TrsmTab t = tt[blockIdx.y];
  T* P1 = static_cast<T*>(t.Pout);
  const int i0 = blockIdx.x * FILL_ROWS;
  const int rows = min(FILL_ROWS, t.m - i0);
  if (rows <= 0) return;
  const float scale = sqrtf(3.0f / static_cast<float>(t.m));
  for (int e = threadIdx.x; e < rows * r; e += 256) {
    const int i = i0 + e / r, j = e % r;
    if (!c.rowok[j]) P1[static_cast<long long>(i) * r + j] = static_cast<T>(fill_value(i, j, scale));
  }
}

// Block column c of P = P~ T^{-1}; one 64-row tile of one layer per workgroup.
// IDENT: P~ is the identity (P = T^{-1}, upper triangular, exact zeros below).
// mlimit > 0 caps the row count (the identity has r rows).
template <typename TIn, typename TOut, bool IDENT>
__global__ __launch_bounds__(256) void k_trsm(const TrsmTab* __restrict__ tab, const int2* __restrict__ tiles,
                                              int r, int cb, int mlimit, const int* run_if) {
  constexpr int YLD = CB + 4;
  __shared__ __attribute__((aligned(16))) double As[tile_elems<CB>()];
  __shared__ __attribute__((aligned(16))) double Bs[tile_elems<CB>()];
  __shared__ __attribute__((aligned(16))) double Ys[CB * YLD];
  if (skip_launch(run_if)) return;
  const int2 lt = tiles[blockIdx.x];
  const TrsmTab t = tab[lt.x];
  const int m = mlimit > 0 ? min(t.m, mlimit) : t.m;
  const int i0 = lt.y * CB;
  if (i0 >= m) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 32, wn0 = (wave & 1) * 32;
  const int c0 = cb * CB, nbc = min(CB, r - c0);
  const TIn* Pin = static_cast<const TIn*>(t.Pin);
  TOut* Pout = static_cast<TOut*>(t.Pout);
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
    pb.load(t.W + c0, r, 0, nbc, kbeg, c0, tid);
  }
  for (int k0 = kbeg; k0 < c0; k0 += GBK) {
    pa.template store<double>(As, tid);
    pb.template store<double>(Bs, tid);
    __syncthreads();
    if (k0 + GBK < c0) {
      pa.load(Prow, r, 0, m - i0, k0 + GBK, c0, tid);
      pb.load(t.W + c0, r, 0, nbc, k0 + GBK, c0, tid);
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
  const double* D = t.Dinv + static_cast<long long>(cb) * CB * CB;
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

}  // namespace

hipError_t launch_cholesky(const CholTab* tab, int nlayers, int r, int pass, hipStream_t s, const int* run_if) {
  if (nlayers <= 0) return hipSuccess;
  if (r < 1) return hipErrorInvalidValue;
  const int nblk = (r + CB - 1) / CB;
  for (int kb = 0; kb < nblk; ++kb) {
    hipLaunchKernelGGL(k_chol_diag, dim3(nlayers), dim3(64), 0, s, tab, r, kb, pass, run_if);
    const int k1 = min(r, (kb + 1) * CB);
    if (k1 >= r) break;
    const int nt = (r - k1 + CB - 1) / CB;
    hipLaunchKernelGGL(k_chol_panel, dim3(nt, nlayers), dim3(256), 0, s, tab, r, kb, run_if);
    hipLaunchKernelGGL(k_chol_trail, dim3(nt * (nt + 1) / 2, nlayers), dim3(256), 0, s, tab, r, kb, run_if);
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
