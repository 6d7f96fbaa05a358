// The second CholQR pass (Orthogonalize of Algorithm 1 / 2) of fp32-gradient
// layers without a pivot chain.  After the first pass P1 = P~ T0^{-1} is
// orthonormal to about kappa^2 u_fp64, so its Gram matrix is W1 = I + E with
// E tiny (||E||_F about 1e-4 at kappa = 1e6, r = 1024).  Its Cholesky factor
// is T1 = I + U with U upper triangular and U + U^T + U^T U = E, that is the
// fixed point of
//     U = Phi(E - U^T U),   Phi(S) = strict upper triangle of S + diag(S) / 2,
// which the iteration U_0 = Phi(E), U_{k+1} = Phi(E - U_k^T U_k) reaches:
// ||Phi(S)||_F <= ||S||_F / sqrt(2) for symmetric S, so ||U||_F <=
// ||E||_F / sqrt(2), the error of U_0 is at most ||E||_F^2 / (2 sqrt(2)) and
// every further step multiplies it by at most about ||E||_F; whenever
// ||E||_F <= 2^-10, NID_ITERS = 4 products leave it below 1e-18.  The
// inverses of the diagonal 64 x 64 blocks, which the triangular solve needs,
// follow from the series (I + U_kk)^{-1} = sum_j (-U_kk)^j, cut after the
// fifth power (remainder below ||U_kk||^6, about 1e-19).  Every product
// runs in parallel over 32 x 32 quadrants of the upper 64 x 64 tiles on the
// fp64 MFMA, where the blocked factorisation makes r / 64 dependent steps of
// a few microseconds each.
//
// Layers whose ||E||_F exceeds the bound (a floored first-pass pivot, whose
// column was replaced by a pseudo-random direction, or kappa past about
// 3e6) take the blocked factorisation instead: the last kernel here sets the
// layer's flag, and the factorisation kernels of that pass run only where it
// is 0.  The decision sums fixed per-tile partial sums in index order, so it
// is the same in every kernel and on every run.
#include "common.hpp"
#include "mfma_tile.hpp"

namespace cd {
namespace {

constexpr int NB = CHOL_BLOCK;
constexpr int NID_ITERS = 4;
constexpr int NID_SERIES = 5;
constexpr double NID_BOUND2 = 1.0 / 1048576.0;   // (2^-10)^2, bound on ||E||_F^2

// upper tile t of an nblk x nblk block grid -> (ti, tj), ti <= tj, row-major
__device__ __forceinline__ void upper_tile(int t, int nblk, int& ti, int& tj) {
  int u = t;
  ti = 0;
  while (u >= nblk - ti) { u -= nblk - ti; ++ti; }
  tj = ti + u;
}

// ||E||_F^2 of layer tab from its per-tile partial sums (index order); every
// thread of the block gets it
__device__ double e_norm2(const CholTab& t, int r, int ntiles, double* sh) {
  const double* part = global_view(t.nid) + 2LL * r * r;
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int i = 0; i < ntiles; ++i) s += part[i];
    *sh = s;
  }
  __syncthreads();
  return *sh;
}

// U_0 = Phi(W - I) on upper tile blockIdx.x, and the tile's share of
// ||E||_F^2 (diagonal entries once, the others twice: E is symmetric).
__global__ __launch_bounds__(256) void k_nid_start(const CholTab* __restrict__ tab, int r, const int* run_if) {
  __shared__ double red[4];
  if (skip_launch(run_if)) return;
  const CholTab t = tab[blockIdx.y];
  const int nblk = (r + NB - 1) / NB;
  int ti, tj;
  upper_tile(blockIdx.x, nblk, ti, tj);
  const double* const W = global_view(t.W);
  double* const U = global_view(t.nid);
  const int tid = threadIdx.x, col = tj * NB + (tid & 63);
  double ss = 0.0;
#pragma unroll 4
  for (int q = 0; q < NB / 4; ++q) {
    const int row = ti * NB + (tid >> 6) + 4 * q;
    if (row < r && col < r) {
      double u = 0.0;
      if (row <= col) {
        const double e = W[static_cast<long long>(row) * r + col] - (row == col ? 1.0 : 0.0);
        u = row == col ? 0.5 * e : e;
        ss += (row == col ? 1.0 : 2.0) * e * e;
      }
      U[static_cast<long long>(row) * r + col] = u;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  if (tid == 0) global_view(t.nid)[2LL * r * r + blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// U_dst = Phi(E - U_src^T U_src) on one 32 x 32 quadrant of an upper 64 x 64
// tile (src, dst: 0 or 1, the two r x r buffers; dst < 0: the last step,
// T1 = I + U goes over W).  Four workgroups per tile, so that the tiles of
// the last block rows, whose K runs to r, take a quarter of the time one
// workgroup would; the four waves take every fourth 32-wide k slice and their
// partial products are added in wave order.
constexpr int NQ = 32;
__global__ __launch_bounds__(256) void k_nid_iter(const CholTab* __restrict__ tab, int r, int src, int dst,
                                                  const int* run_if) {
  constexpr int SL = GBK * (NQ + KPAD);   // one staged k slice of 32 columns
  constexpr int RLD = NQ + 1;
  static_assert(4 * NQ * RLD <= 4 * SL, "the wave partials fit in the A staging");
  __shared__ __attribute__((aligned(16))) double As[4 * SL];
  __shared__ __attribute__((aligned(16))) double Bs[4 * SL];
  __shared__ double sh;
  if (skip_launch(run_if)) return;
  const CholTab t = tab[blockIdx.y];
  const int nblk = (r + NB - 1) / NB;
  if (!(e_norm2(t, r, nblk * (nblk + 1) / 2, &sh) <= NID_BOUND2)) return;
  int ti, tj;
  upper_tile(blockIdx.x >> 2, nblk, ti, tj);
  const int qi = (blockIdx.x >> 1) & 1, qj = blockIdx.x & 1;
  const int i0 = ti * NB + qi * NQ, j0 = tj * NB + qj * NQ;
  if (i0 >= r || j0 >= r) return;         // a quadrant past a partial last block
  double* const W = global_view(t.W);
  double* const Ud = dst >= 0 ? global_view(t.nid) + static_cast<long long>(dst) * r * r : nullptr;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (ti == tj && qi > qj) {              // below the diagonal: U is zero there
    if (Ud)
      for (int e = tid; e < NQ * NQ; e += 256) {
        const int row = i0 + e / NQ, col = j0 + e % NQ;
        if (row < r && col < r) Ud[static_cast<long long>(row) * r + col] = 0.0;
      }
    return;
  }
  const double* const Us = global_view(t.nid) + static_cast<long long>(src) * r * r;
  // (U^T U)[i][j] = sum_k U[k][i] U[k][j]; U is upper triangular, so k < i0 + 32
  const int kend = min(i0 + NQ, r);
  f64x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f64x4{};
  for (int k0 = 0; k0 < kend; k0 += 4 * GBK) {
    // slice w: A(i, k) = U[k][i0 + i], B(k, j) = U[k][j0 + j], k in k0 + 32 w ..
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      stage_tile<double, double, NQ, 256, false>(As + w * SL, Us + i0, r, 0, r - i0, k0 + w * GBK, kend, tid);
      stage_tile<double, double, NQ, 256, false>(Bs + w * SL, Us + j0, r, 0, r - j0, k0 + w * GBK, kend, tid);
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GBK; kk += 16) {
      f64x4 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = frag<double, NQ, false>(As + wave * SL, i * 16, kk, lane);
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = frag<double, NQ, false>(Bs + wave * SL, j * 16, kk, lane);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i][q], b[j][q], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  double* const red = As;                 // [wave][row][RLD]
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        red[(wave * NQ + i * 16 + Mfma<double>::out_row(lane, v)) * RLD + j * 16 + (lane & 15)] = acc[i][j][v];
  __syncthreads();
  for (int e = tid; e < NQ * NQ; e += 256) {
    const int lr = e / NQ, lc = e % NQ, row = i0 + lr, col = j0 + lc;
    if (row >= r || col >= r) continue;
    const long long o = static_cast<long long>(row) * r + col;
    if (row > col) {                      // below the diagonal of a diagonal tile
      if (Ud) Ud[o] = 0.0;
      continue;
    }
    const double* const p = red + lr * RLD + lc;
    const double sum = ((p[0] + p[NQ * RLD]) + p[2 * NQ * RLD]) + p[3 * NQ * RLD];
    const double sv = (W[o] - (row == col ? 1.0 : 0.0)) - sum;
    const double u = row == col ? 0.5 * sv : sv;
    if (Ud) Ud[o] = u;
    else W[o] = row == col ? 1.0 + u : u;
  }
}

// D_k = (T1_kk)^{-1} = sum_{j <= NID_SERIES} (-U_kk)^j by Horner's rule
// (V <- I - U V), zero outside the block's nb x nb; and the layer's flag:
// 1 when this iteration formed T1, 0 when the blocked factorisation must.
__global__ __launch_bounds__(256) void k_nid_dinv(const CholTab* __restrict__ tab, int r, const int* run_if) {
  constexpr int LD = NB + 1;
  __shared__ double Ul[NB * LD];
  __shared__ double Vl[NB * LD];
  __shared__ double sh;
  if (skip_launch(run_if)) return;
  const CholTab t = tab[blockIdx.y];
  const int nblk = (r + NB - 1) / NB;
  const bool ok = e_norm2(t, r, nblk * (nblk + 1) / 2, &sh) <= NID_BOUND2;
  const int tid = threadIdx.x;
  if (blockIdx.x == 0 && tid == 0) *global_view(t.nid_ok) = ok ? 1 : 0;
  if (!ok) return;
  const int k0 = blockIdx.x * NB, nb = min(NB, r - k0);
  const double* const W = global_view(t.W);
  const int j = tid & 63, w = tid >> 6;
  // U_kk (upper triangle of T1_kk minus I) and V = I
  for (int q = 0; q < NB / 4; ++q) {
    const int i = w + 4 * q;
    const bool in = i < nb && j < nb && i <= j;
    Ul[i * LD + j] = in ? W[static_cast<long long>(k0 + i) * r + k0 + j] - (i == j ? 1.0 : 0.0) : 0.0;
    Vl[i * LD + j] = i == j ? 1.0 : 0.0;
  }
  __syncthreads();
  for (int it = 0; it < NID_SERIES; ++it) {
    // V'[i][j] = delta_ij - sum_k U[i][k] V[k][j]; thread: column j, rows w + 4q
    // (all reads of V before the barrier, the new V after it)
    double acc[NB / 4];
#pragma unroll
    for (int q = 0; q < NB / 4; ++q) acc[q] = 0.0;
    for (int k = 0; k < NB; ++k) {
      const double vk = Vl[k * LD + j];
#pragma unroll
      for (int q = 0; q < NB / 4; ++q) acc[q] = fma(Ul[(w + 4 * q) * LD + k], vk, acc[q]);
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < NB / 4; ++q) {
      const int i = w + 4 * q;
      Vl[i * LD + j] = (i == j ? 1.0 : 0.0) - acc[q];
    }
    __syncthreads();
  }
  double* const D = global_view(t.Dinv) + static_cast<long long>(blockIdx.x) * NB * NB;
  for (int q = 0; q < NB / 4; ++q) {
    const int i = w + 4 * q;
    D[i * NB + j] = (i < nb && j < nb) ? Vl[i * LD + j] : 0.0;
  }
}

}  // namespace

int nearid_parts(int r) {
  const int nblk = (r + NB - 1) / NB;
  return nblk * (nblk + 1) / 2;
}

hipError_t launch_nearid(const CholTab* tab, int nlayers, int r, hipStream_t s, const int* run_if) {
  if (nlayers <= 0) return hipSuccess;
  if (r < 1) return hipErrorInvalidValue;
  const int nblk = (r + NB - 1) / NB, nt = nearid_parts(r);
  hipLaunchKernelGGL(k_nid_start, dim3(nt, nlayers), dim3(256), 0, s, tab, r, run_if);
  for (int it = 0; it < NID_ITERS; ++it) {
    const int src = it & 1, dst = it + 1 < NID_ITERS ? (src ^ 1) : -1;
    hipLaunchKernelGGL(k_nid_iter, dim3(4 * nt, nlayers), dim3(256), 0, s, tab, r, src, dst, run_if);
  }
  hipLaunchKernelGGL(k_nid_dinv, dim3(nblk, nlayers), dim3(256), 0, s, tab, r, run_if);
  return hipGetLastError();
}

}  // namespace cd
