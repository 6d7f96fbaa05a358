// ColumnNormalize of the Dion sync branch (Algorithm 1 / Algorithm 2):
//   Q_j = R_j / max(‖R_j‖, 1e-30)        (column 2-norms accumulated in fp64,
//                                          partials in a fixed row order)
// fused with the bf16 split planes of R and Q that the update streams.
#include "common.hpp"

namespace cd {
namespace {

// Partial column sums of squares over COLNORM_ROWS rows: thread j owns
// column j; four interleaved accumulators (row i goes to i % 4) keep 16 loads
// in flight and are combined in a fixed order.
__global__ __launch_bounds__(256) void k_colsq(ColnormArgs a) {
  if (skip_launch(a.run_if)) return;
  const int l = blockIdx.z, chunk = blockIdx.x;
  const int j = blockIdx.y * 256 + threadIdx.x;
  if (j >= a.r) return;
  const float* R = a.R[l];
  const int i0 = chunk * COLNORM_ROWS, i1 = min(a.n, i0 + COLNORM_ROWS);
  double s[4] = {0.0, 0.0, 0.0, 0.0};
  int i = i0;
  for (; i + 16 <= i1; i += 16) {
    float v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = R[static_cast<long long>(i + u) * a.r + j];
#pragma unroll
    for (int u = 0; u < 16; ++u) s[u & 3] += static_cast<double>(v[u]) * v[u];
  }
  for (; i < i1; ++i) {
    const double v = R[static_cast<long long>(i) * a.r + j];
    s[(i - i0) & 3] += v * v;
  }
  a.part[l][static_cast<long long>(chunk) * a.r + j] = (s[0] + s[1]) + (s[2] + s[3]);
}

// Column norms from the partials: 16 columns per block and 16 threads per
// column, thread c summing partials c, c + 16, c + 32, ... (four interleaved
// accumulators, so four loads are in flight), then a fixed-order tree over
// the 16 sums.  The order depends only on n, not on scheduling.
constexpr int CN_COLS = 16, CN_LANES = 16;
__global__ __launch_bounds__(256) void k_colnorm_final(ColnormArgs a) {
  __shared__ double sh[CN_LANES][CN_COLS + 1];
  if (skip_launch(a.run_if)) return;
  const int l = blockIdx.z;
  const int jj = threadIdx.x % CN_COLS, cl = threadIdx.x / CN_COLS;
  const int j = blockIdx.x * CN_COLS + jj;
  double s[4] = {0.0, 0.0, 0.0, 0.0};
  if (j < a.r) {
    const double* p = a.part[l] + j;
    const long long step = static_cast<long long>(a.r) * CN_LANES;
    int c = cl;
    for (; c + 3 * CN_LANES < a.nchunks; c += 4 * CN_LANES) {
      const double* q = p + static_cast<long long>(c) * a.r;
      const double v0 = q[0], v1 = q[step], v2 = q[2 * step], v3 = q[3 * step];
      s[0] += v0; s[1] += v1; s[2] += v2; s[3] += v3;
    }
    // at most three left: c, c + 16, c + 32
    const double* q = p + static_cast<long long>(c) * a.r;
    if (c < a.nchunks) s[0] += q[0];
    if (c + CN_LANES < a.nchunks) s[1] += q[step];
    if (c + 2 * CN_LANES < a.nchunks) s[2] += q[2 * step];
  }
  sh[cl][jj] = (s[0] + s[1]) + (s[2] + s[3]);
  __syncthreads();
#pragma unroll
  for (int w = CN_LANES / 2; w >= 1; w >>= 1) {
    if (cl < w) sh[cl][jj] += sh[cl + w][jj];
    __syncthreads();
  }
  if (cl == 0 && j < a.r) a.nrm[l][j] = static_cast<float>(fmax(sqrt(sh[0][jj]), 1e-30));
}

// Q = R / norms, and the bf16 planes of R and Q (piece s of a value is
// bf16(value - pieces < s), as for every split operand): one pass over R.
// Four consecutive columns per thread; columns r..rp-1 of the planes are zero.
__global__ __launch_bounds__(256) void k_colscale_planes(ColnormArgs a) {
  if (skip_launch(a.run_if)) return;
  const int l = blockIdx.z;
  const int qpr = a.rp / 4;   // quads per row
  const long long quads = static_cast<long long>(a.n) * qpr;
  const long long plane = static_cast<long long>(a.n) * a.rp;
  const float* R = a.R[l];
  const float* nrm = a.nrm[l];
  float* Q = a.Q[l];
  __bf16* Rp = a.Rpl[l];
  __bf16* Qp = a.Qpl[l];
  const bool vec = (a.r & 3) == 0;   // 16-byte rows segments of R and Q (and of the norms)
  for (long long q = blockIdx.x * 256LL + threadIdx.x; q < quads; q += 256LL * gridDim.x) {
    const long long row = q / qpr;
    const int k = static_cast<int>(q - row * qpr) * 4;
    float rv[4], qv[4];
    if (vec && k + 3 < a.r) {
      const float4 x = *reinterpret_cast<const float4*>(R + row * a.r + k);
      const float4 d = *reinterpret_cast<const float4*>(nrm + k);
      rv[0] = x.x; rv[1] = x.y; rv[2] = x.z; rv[3] = x.w;
      qv[0] = x.x / d.x; qv[1] = x.y / d.y; qv[2] = x.z / d.z; qv[3] = x.w / d.w;
      *reinterpret_cast<float4*>(Q + row * a.r + k) = make_float4(qv[0], qv[1], qv[2], qv[3]);
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const bool in = k + c < a.r;
        rv[c] = in ? R[row * a.r + k + c] : 0.0f;
        qv[c] = in ? rv[c] / nrm[k + c] : 0.0f;
        if (in) Q[row * a.r + k + c] = qv[c];
      }
    }
    float rr[4] = {rv[0], rv[1], rv[2], rv[3]}, qr[4] = {qv[0], qv[1], qv[2], qv[3]};
    for (int s = 0; s < a.S; ++s) {
      __bf16 pr[4], pq[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        pr[c] = static_cast<__bf16>(rr[c]);
        rr[c] -= static_cast<float>(pr[c]);
        pq[c] = static_cast<__bf16>(qr[c]);
        qr[c] -= static_cast<float>(pq[c]);
      }
      typedef __bf16 b4 __attribute__((ext_vector_type(4)));
      const b4 wr = {pr[0], pr[1], pr[2], pr[3]}, wq = {pq[0], pq[1], pq[2], pq[3]};
      *reinterpret_cast<b4*>(Rp + s * plane + row * a.rp + k) = wr;
      *reinterpret_cast<b4*>(Qp + s * plane + row * a.rp + k) = wq;
    }
  }
}

}  // namespace

hipError_t launch_colnorm(const ColnormArgs& a, int nl, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  // S = 0: no planes (the fp32 vector update reads R and Q themselves)
  if (a.rp % 32 != 0 || a.rp < a.r || a.S < 0 || a.S > 3) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_colsq, dim3(a.nchunks, (a.r + 255) / 256, nl), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_colnorm_final, dim3((a.r + CN_COLS - 1) / CN_COLS, 1, nl), dim3(256), 0, s, a);
  long long quads = static_cast<long long>(a.n) * (a.rp / 4);
  long long blocks = (quads + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_colscale_planes, dim3(static_cast<unsigned>(blocks), 1, nl), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace cd
