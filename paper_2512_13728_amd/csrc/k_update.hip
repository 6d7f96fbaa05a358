// ColumnNormalize of the Dion sync branch (Algorithm 1 / Algorithm 2):
//   Q_j = R_j / max(‖R_j‖, 1e-30)        (column 2-norms accumulated in fp64,
//                                          partials in a fixed row order)
#include "common.hpp"

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

}  // namespace cd
