// Cholesky factor of the Gram matrix and its inverse, for the CholQR
// orthonormalisation of P~ (the paper's Orthogonalize step is unspecified; the
// thin-QR factor with positive-diagonal R is what it computes here).
//
// W = P~^T P~ = T^T T with T upper triangular, then U = T^{-1}; P~ U has
// orthonormal columns and P~ = (P~ U) T is the thin QR factorisation.
// One 1024-thread workgroup factors one layer's r x r matrix (r <= 1024) in
// fp64: right-looking blocked Cholesky with 16-row panels staged in LDS, then
// a blocked back-substitution for the inverse, bottom row-block first.  A
// pivot that is not above floor = 1e-13 * max_k W_kk (or is NaN) is raised to
// the floor and the layer is flagged rank deficient.
#include "common.hpp"

namespace cd {
namespace {

constexpr int CNB = 16;
constexpr int CT = 1024;
constexpr int NW = CT / 64;

__global__ __launch_bounds__(CT) void k_chol_inv(CholArgs a) {
  extern __shared__ double Pn[];              // CNB x r panel
  __shared__ double D[CNB][CNB + 1];
  __shared__ double E[CNB][CNB + 1];
  __shared__ double red[NW];
  __shared__ double s_floor;
  __shared__ int s_rankdef;
  const int l = blockIdx.x, r = a.r, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  double* __restrict__ W = a.W[l];
  double* __restrict__ U = a.U[l];
  const long long ld = r;

  double md = 0.0;
  for (int k = tid; k < r; k += CT) {
    const double d = W[k * ld + k];
    if (d > md) md = d;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) md = fmax(md, __shfl_xor(md, o, 64));
  if (lane == 0) red[wave] = md;
  __syncthreads();
  if (tid == 0) {
    double m = 0.0;
    for (int i = 0; i < NW; ++i) m = fmax(m, red[i]);
    s_floor = fmax(1e-13 * m, 1e-300);
    s_rankdef = 0;
  }
  __syncthreads();
  const double floor_ = s_floor;

  // ---- Cholesky: T overwrites the upper triangle of W --------------------
  for (int k0 = 0; k0 < r; k0 += CNB) {
    const int nb = min(CNB, r - k0), k1 = k0 + nb;
    if (tid < CNB * CNB) {
      const int i = tid / CNB, j = tid % CNB;
      D[i][j] = (i < nb && j < nb && j >= i) ? W[(k0 + i) * ld + k0 + j] : 0.0;
    }
    __syncthreads();
    for (int p = 0; p < nb; ++p) {
      if (tid == 0) {
        double d = D[p][p];
        if (!(d > floor_)) { d = floor_; s_rankdef = 1; }
        D[p][p] = sqrt(d);
      }
      __syncthreads();
      if (tid > p && tid < nb) D[p][tid] /= D[p][p];
      __syncthreads();
      if (tid < CNB * CNB) {
        const int i = tid / CNB, j = tid % CNB;
        if (i > p && i < nb && j >= i && j < nb) D[i][j] -= D[p][i] * D[p][j];
      }
      __syncthreads();
    }
    if (tid < CNB * CNB) {
      const int i = tid / CNB, j = tid % CNB;
      if (i < nb && j < nb && j >= i) W[(k0 + i) * ld + k0 + j] = D[i][j];
    }
    // panel row block: T_kk^T X = W[k0:k1, k1:r].  The empty asm with a memory
    // clobber keeps the compiler from hoisting all of D into registers.
#pragma unroll 1
    for (int c = k1 + tid; c < r; c += CT) {
      __asm__ volatile("" ::: "memory");
      double x[CNB];
#pragma unroll
      for (int p = 0; p < CNB; ++p) {
        x[p] = 0.0;
        if (p < nb) {
          double v = W[(k0 + p) * ld + c];
#pragma unroll
          for (int q = 0; q < p; ++q) v -= D[q][p] * x[q];
          x[p] = v / D[p][p];
        }
      }
#pragma unroll
      for (int p = 0; p < CNB; ++p)
        if (p < nb) {
          W[(k0 + p) * ld + c] = x[p];
          Pn[p * r + c] = x[p];
        }
    }
    __syncthreads();
    // trailing update of the upper triangle: W[i][j] -= sum_p X[p][i] X[p][j]
    for (int i = k1 + wave; i < r; i += NW) {
      double pi[CNB];
#pragma unroll
      for (int p = 0; p < CNB; ++p) pi[p] = (p < nb) ? Pn[p * r + i] : 0.0;
#pragma unroll 1
      for (int j = i + lane; j < r; j += 64) {
        double s = 0.0;
#pragma unroll
        for (int p = 0; p < CNB; ++p)
          if (p < nb) s += pi[p] * Pn[p * r + j];
        W[i * ld + j] -= s;
      }
    }
    __syncthreads();
  }

  // ---- U = T^{-1}, row blocks from the bottom ------------------------------
  const int nblk = (r + CNB - 1) / CNB;
  for (int bi = nblk - 1; bi >= 0; --bi) {
    const int k0 = bi * CNB, nb = min(CNB, r - k0), k1 = k0 + nb;
    if (tid < CNB * CNB) {
      const int i = tid / CNB, j = tid % CNB;
      D[i][j] = (i < nb && j < nb && j >= i) ? W[(k0 + i) * ld + k0 + j] : 0.0;
    }
    __syncthreads();
    if (tid < nb) {
      const int c = tid;
      E[c][c] = 1.0 / D[c][c];
      for (int i = c - 1; i >= 0; --i) {
        double s = 0.0;
        for (int p = i + 1; p <= c; ++p) s += D[i][p] * E[p][c];
        E[i][c] = -s / D[i][i];
      }
      for (int i = c + 1; i < CNB; ++i) E[i][c] = 0.0;
    }
    const int w = r - k1;
    for (int idx = tid; idx < nb * w; idx += CT) {
      const int p = idx / w, c = k1 + idx % w;
      Pn[p * r + c] = W[(k0 + p) * ld + c];
    }
    __syncthreads();
    // U[k0+i][c] = -sum_p E[i][p] * sum_{q=k1..c} T[k0+p][q] U[q][c]
#pragma unroll 1
    for (int c = k1 + tid; c < r; c += CT) {
      double S[CNB];
#pragma unroll
      for (int p = 0; p < CNB; ++p) S[p] = 0.0;
#pragma unroll 2
      for (int q = k1; q <= c; ++q) {
        const double u = U[q * ld + c];
#pragma unroll
        for (int p = 0; p < CNB; ++p)
          if (p < nb) S[p] += Pn[p * r + q] * u;
      }
      __asm__ volatile("" ::: "memory");
#pragma unroll
      for (int i = 0; i < CNB; ++i)
        if (i < nb) {
          double v = 0.0;
#pragma unroll
          for (int p = 0; p < CNB; ++p)
            if (p >= i && p < nb) v += E[i][p] * S[p];
          U[(k0 + i) * ld + c] = -v;
        }
    }
    if (tid < CNB * CNB) {
      const int i = tid / CNB, j = tid % CNB;
      if (i < nb && j < nb) U[(k0 + i) * ld + k0 + j] = (j >= i) ? E[i][j] : 0.0;
    }
    __syncthreads();
  }

  // zero the strictly lower triangle so U can be used as a full r x r operand
  for (long long idx = tid; idx < ld * ld; idx += CT) {
    const long long i = idx / ld, j = idx - i * ld;
    if (j < i) U[idx] = 0.0;
  }
  if (tid == 0) {
    if (a.accumulate) {
      if (s_rankdef) *a.rankdef[l] = 1;
    } else {
      *a.rankdef[l] = s_rankdef;
    }
  }
}

}  // namespace

hipError_t launch_chol_inv(const CholArgs& a, int nl, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  if (a.r < 1 || a.r > 1024) return hipErrorInvalidValue;
  const size_t lds = static_cast<size_t>(CNB) * a.r * sizeof(double);
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_chol_inv),
                            hipFuncAttributeMaxDynamicSharedMemorySize, CNB * 1024 * 8);
  hipLaunchKernelGGL(k_chol_inv, dim3(nl), dim3(CT), lds, s, a);
  return hipGetLastError();
}

}  // namespace cd
