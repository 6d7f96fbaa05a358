// ColumnNormalize and the fused rank-r update of the Dion sync branch
// (Algorithm 1 / Algorithm 2):
//   Q_j = R_j / max(‖R_j‖, 1e-30)                 (column 2-norms in fp64)
//   M   = B - (1 - mu) P R^T                      (error feedback; B is in M)
//   X   = X - eta sqrt(m/n) P Q^T                 (weight update)
// The update reads each B and X tile once and forms both rank-r products on
// fp32 MFMA from one staged P tile.
#include "common.hpp"
#include "mfma_tile.hpp"

namespace cd {
namespace {

// Partial column sums of squares over COLNORM_ROWS rows, in row order.
__global__ __launch_bounds__(256) void k_colsq(ColnormArgs a) {
  const int l = blockIdx.z, chunk = blockIdx.x;
  const float* R = a.R[l];
  const int i0 = chunk * COLNORM_ROWS, i1 = min(a.n, i0 + COLNORM_ROWS);
  for (int j = threadIdx.x; j < a.r; j += 256) {
    double s = 0.0;
    for (int i = i0; i < i1; ++i) {
      const double v = R[static_cast<long long>(i) * a.r + j];
      s += v * v;
    }
    a.part[l][static_cast<long long>(chunk) * a.r + j] = s;
  }
}

__global__ __launch_bounds__(256) void k_colnorm_final(ColnormArgs a) {
  const int l = blockIdx.z;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= a.r) return;
  double s = 0.0;
  for (int c = 0; c < a.nchunks; ++c) s += a.part[l][static_cast<long long>(c) * a.r + j];
  a.nrm[l][j] = static_cast<float>(fmax(sqrt(s), 1e-30));
}

__global__ __launch_bounds__(256) void k_colscale(ColnormArgs a) {
  const int l = blockIdx.z;
  const long long total = static_cast<long long>(a.n) * a.r;
  const float* R = a.R[l];
  const float* nrm = a.nrm[l];
  float* Q = a.Q[l];
  for (long long i = blockIdx.x * 256LL + threadIdx.x; i < total; i += 256LL * gridDim.x) {
    Q[i] = R[i] / nrm[i % a.r];
  }
}

// 64 x 64 output tile, 4 waves as 2 x 2, each 32 x 32 with two accumulator sets.
constexpr int UBM = 64, UBN = 64;

__global__ __launch_bounds__(256) void k_update(UpdateArgs u) {
  __shared__ __attribute__((aligned(16))) float Ps[UBM * GLDK];
  __shared__ __attribute__((aligned(16))) float Rs[UBN * GLDK];
  __shared__ __attribute__((aligned(16))) float Qs[UBN * GLDK];
  const int l = blockIdx.z;
  const int tiles_n = (u.n + UBN - 1) / UBN;
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x - tm * tiles_n;
  const int m0 = tm * UBM, n0 = tn * UBN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 32, wn0 = (wave & 1) * 32;
  const float* P = u.P[l];
  const float* R = u.R[l];
  const float* Q = u.Q[l];

  f32x4 am[2][2], ax[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) { am[i][j] = f32x4{}; ax[i][j] = f32x4{}; }

  for (int k0 = 0; k0 < u.r; k0 += GBK) {
    stage_tile<float, float, UBM, 256>(Ps, P, u.r, true, m0, u.m, k0, u.r, tid);
    stage_tile<float, float, UBN, 256>(Rs, R, u.r, true, n0, u.n, k0, u.r, tid);
    stage_tile<float, float, UBN, 256>(Qs, Q, u.r, true, n0, u.n, k0, u.r, tid);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GBK; kk += 16) {
      f32x4 pa[2], rb[2], qb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) pa[i] = frag<float>(Ps, wm0 + i * 16, kk, lane);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        rb[j] = frag<float>(Rs, wn0 + j * 16, kk, lane);
        qb[j] = frag<float>(Qs, wn0 + j * 16, kk, lane);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            am[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(pa[i][q], rb[j][q], am[i][j], 0, 0, 0);
            ax[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(pa[i][q], qb[j][q], ax[i][j], 0, 0, 0);
          }
    }
    __syncthreads();
  }

  float* M = u.M[l];
  float* X = u.X[l];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = m0 + wm0 + i * 16 + 4 * (lane >> 4) + v;
        const int col = n0 + wn0 + j * 16 + (lane & 15);
        if (row < u.m && col < u.n) {
          const long long o = static_cast<long long>(row) * u.n + col;
          M[o] = fmaf(-u.one_minus_mu, am[i][j][v], M[o]);
          X[o] = fmaf(-u.c, ax[i][j][v], X[o]);
        }
      }
}

}  // namespace

hipError_t launch_colnorm(const ColnormArgs& a, int nl, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_colsq, dim3(a.nchunks, 1, nl), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_colnorm_final, dim3((a.r + 255) / 256, 1, nl), dim3(256), 0, s, a);
  long long total = static_cast<long long>(a.n) * a.r;
  long long blocks = (total + 255) / 256;
  if (blocks > 2048) blocks = 2048;
  hipLaunchKernelGGL(k_colscale, dim3(static_cast<unsigned>(blocks), 1, nl), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_update(const UpdateArgs& u, int nl, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  const int tiles = ((u.m + UBM - 1) / UBM) * ((u.n + UBN - 1) / UBN);
  hipLaunchKernelGGL(k_update, dim3(tiles, 1, nl), dim3(256), 0, s, u);
  return hipGetLastError();
}

}  // namespace cd
