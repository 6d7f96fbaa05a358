// The M / X update of the Dion sync branch (Algorithm 1 / Algorithm 2) for
// fp32-gradient layers at small rank (r <= 32), on the fp32 vector units:
//   M = B - (1 - mu) P R^T,    X -= eta sqrt(m/n) P Q^T
// At r <= 32 the correction costs at most 4r = 128 flops per element, well
// under what the vector units give per streamed byte, so the kernel only has to stream M
// and X at the HBM rate.  Each lane holds its column's rows of R and Q in
// registers for the whole launch; the row of P is the same for a whole wave
// (broadcast across the lanes); M and X move with non-temporal accesses.
// The products accumulate in fp32 over k in order.
#include <algorithm>

#include "common.hpp"

namespace cd {
namespace {

__device__ __forceinline__ float load_g(const void* G, bool bf, long long i) {
  if (bf) return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(G)[i]) << 16);
  return static_cast<const float*>(G)[i];
}

// One wave per (column strip of 64, row band): lane l owns column
// strip0 + l, the wave walks rows i, i + 4, ... of the block's band (the
// block's four waves interleave), U rows at a time: the M and X elements of
// the U rows are all requested before any arithmetic.  2 RMAX registers hold
// the lane's row of R and of Q (zero past r and past n).  Row t's P[row, :]
// arrives as one vector load (lane k holds P[row, k], k < r) in flight with
// the M and X elements, and each P[row, k] reaches the FMAs by readlane (a
// wave-uniform operand).
template <int RMAX, int U>
__global__ __launch_bounds__(256) void k_update_vec(UpdateVecArgs u) {
  static_assert(RMAX <= 64, "P's row is spread over the lanes of one wave");
  if (u.ctl != nullptr && u.ctl->flag == 0) return;   // not a sync step
  const int l = blockIdx.z;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int lane = threadIdx.x & 63;
  const int j = blockIdx.x * 64 + lane;
  const int n = u.n, m = u.m, r = u.r;
  const bool in = j < n;
  const float* __restrict__ P = u.P[l];

  float rr[RMAX], qq[RMAX];
  {
    const float* __restrict__ R = u.R[l] + static_cast<long long>(in ? j : 0) * r;
    const float* __restrict__ Q = u.Q[l] + static_cast<long long>(in ? j : 0) * r;
#pragma unroll
    for (int k = 0; k < RMAX; ++k) {
      rr[k] = (in && k < r) ? R[k] : 0.0f;
      qq[k] = (in && k < r) ? Q[k] : 0.0f;
    }
  }

  float* const Mo = u.M[l];
  float* const Xo = u.X[l];
  const void* const G = u.G[l];
  const bool gbf = u.g_bf16 != 0;
  const bool spec = (u.spec == 2 ? u.ctl->spec_cur : u.spec) != 0;
  const float gc = spec ? u.gc[l] : 0.0f, xd = spec ? 1.0f : u.xdecay[l];
  const float cm = -u.one_minus_mu, cx = -u.c;
  const int i_end = min(m, (blockIdx.y + 1) * u.band);
  for (int i = blockIdx.y * u.band + wave; i < i_end; i += 4 * U) {
    float w[U], x[U], pv[U];
#pragma unroll
    for (int t = 0; t < U; ++t) {
      const int row = i + 4 * t;
      const long long off = static_cast<long long>(row) * n + j;
      const bool live = row < i_end;   // uniform over the wave
      pv[t] = (live && lane < r) ? P[static_cast<long long>(row) * r + lane] : 0.0f;
      w[t] = (live && in) ? __builtin_nontemporal_load(Mo + off) : 0.0f;
      x[t] = (live && in) ? __builtin_nontemporal_load(Xo + off) : 0.0f;
    }
#pragma unroll
    for (int t = 0; t < U; ++t) {
      const int row = i + 4 * t;
      if (row >= i_end) break;   // uniform over the wave
      float sm = 0.0f, sx = 0.0f;
#pragma unroll
      for (int k = 0; k < RMAX; ++k) {
        const float pk = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, pv[t]), k));
        sm = fmaf(pk, rr[k], sm);
        sx = fmaf(pk, qq[k], sx);
      }
      if (!in) continue;
      const long long off = static_cast<long long>(row) * n + j;
      // undo a speculative skip-branch update (it already applied the weight
      // decay), else apply the decay (xd = 1 after a speculative update)
      const float xv = gc != 0.0f ? fmaf(gc, load_g(G, gbf, off), x[t]) : x[t] * xd;
      __builtin_nontemporal_store(fmaf(cm, sm, w[t]), Mo + off);
      __builtin_nontemporal_store(fmaf(cx, sx, xv), Xo + off);
    }
  }
}

}  // namespace

// up to r = 32: at r = 48 and 64 this form took 0.49-0.50 ms on 4096 x 16384
// (189 VGPRs, two waves per SIMD) against 0.36 ms for the bf16-split MFMA update
bool update_vec_fits(int r) { return r >= 1 && r <= 32; }

hipError_t launch_update_vec(UpdateVecArgs u, int nl, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  if (!update_vec_fits(u.r) || u.m < 1 || u.n < 1) return hipErrorInvalidValue;
  // one column per lane and eight rows per batch: measured best on
  // 4096 x 16384 against two or four columns per lane (fewer resident waves)
  // and 1-16 rows
  constexpr int U = 8;
  const int strips = (u.n + 63) / 64;
  // about 16 waves per CU over the whole launch, at least one row per wave
  const long long target = 4096;
  const long long waves_per_strip = std::max(1LL, target / (static_cast<long long>(strips) * nl));
  const long long rows_per_wave = std::max(1LL, (u.m + waves_per_strip - 1) / waves_per_strip);
  u.band = static_cast<int>(std::min<long long>(4 * rows_per_wave, u.m));
  const int bands = (u.m + u.band - 1) / u.band;
  const dim3 grid(strips, bands, nl);
  if (u.r <= 16) hipLaunchKernelGGL((k_update_vec<16, U>), grid, dim3(256), 0, s, u);
  else hipLaunchKernelGGL((k_update_vec<32, U>), grid, dim3(256), 0, s, u);
  return hipGetLastError();
}

}  // namespace cd
