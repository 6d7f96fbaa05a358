// The M / X update of the Dion sync branch (Algorithm 1 / Algorithm 2) for
// fp32-gradient layers at small rank (r <= 32), on the fp32 vector units:
//   M = B - (1 - mu) P R^T,    X -= eta sqrt(m/n) P Q^T
// At r <= 32 the correction costs 4r flops per element, far under what the
// vector units give per streamed byte, so the kernel only has to stream M
// and X at the HBM rate.  Each lane holds its CPT columns of R and Q in
// registers for the whole launch; the row of P is the same for a whole wave
// (wave-uniform loads); M and X move as non-temporal CPT-element segments.
// The products accumulate in fp32 over k in order.
#include <algorithm>

#include "common.hpp"

namespace cd {
namespace {

typedef float nt4 __attribute__((ext_vector_type(4)));
typedef float nt2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float load_g(const void* G, bool bf, long long i) {
  if (bf) return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(G)[i]) << 16);
  return static_cast<const float*>(G)[i];
}

// One wave per (column strip, row band): lane l owns columns
// strip0 + CPT l .. + CPT - 1, the wave walks rows i, i + 4, ... of the
// block's band (the block's four waves interleave), U rows at a time: the M
// and X segments of the U rows are all requested before any arithmetic.
// RMAX * CPT * 2 registers hold R and Q (zero past r and past n).  Row t's
// P[row, :] arrives as one vector load (lane k holds P[row, k], k < r) in
// flight with the M and X segments, and each P[row, k] reaches the FMAs by
// readlane (a wave-uniform operand).
template <int RMAX, int CPT, int U>
__global__ __launch_bounds__(256) void k_update_vec(UpdateVecArgs u) {
  static_assert(RMAX <= 64, "P's row is spread over the lanes of one wave");
  const int l = blockIdx.z;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int lane = threadIdx.x & 63;
  const int j0 = blockIdx.x * (64 * CPT) + lane * CPT;
  const int n = u.n, m = u.m, r = u.r;
  const float* __restrict__ P = u.P[l];
  const float* __restrict__ R = u.R[l];
  const float* __restrict__ Q = u.Q[l];

  float rr[CPT][RMAX], qq[CPT][RMAX];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const bool in = j0 + c < n;
    const long long base = static_cast<long long>(in ? j0 + c : 0) * r;
#pragma unroll
    for (int k = 0; k < RMAX; ++k) {
      rr[c][k] = (in && k < r) ? R[base + k] : 0.0f;
      qq[c][k] = (in && k < r) ? Q[base + k] : 0.0f;
    }
  }

  float* const Mo = u.M[l];
  float* const Xo = u.X[l];
  const void* const G = u.G[l];
  const bool gbf = u.g_bf16 != 0;
  const float gc = u.gc[l], xd = u.xdecay[l];
  const float cm = -u.one_minus_mu, cx = -u.c;
  const bool vec = (n % CPT) == 0 && j0 + CPT <= n;
  const int i_end = min(m, (blockIdx.y + 1) * u.band);
  for (int i = blockIdx.y * u.band + wave; i < i_end; i += 4 * U) {
    float w[U][CPT], x[U][CPT], pv[U];
#pragma unroll
    for (int t = 0; t < U; ++t) {
      const int row = i + 4 * t;
      const long long off = static_cast<long long>(row) * n + j0;
      pv[t] = (row < i_end && lane < r) ? P[static_cast<long long>(row) * r + lane] : 0.0f;
      if (row < i_end && vec) {
        if constexpr (CPT == 4) {
          const nt4 a = __builtin_nontemporal_load(reinterpret_cast<const nt4*>(Mo + off));
          const nt4 b = __builtin_nontemporal_load(reinterpret_cast<const nt4*>(Xo + off));
          w[t][0] = a.x; w[t][1] = a.y; w[t][2] = a.z; w[t][3] = a.w;
          x[t][0] = b.x; x[t][1] = b.y; x[t][2] = b.z; x[t][3] = b.w;
        } else if constexpr (CPT == 2) {
          const nt2 a = __builtin_nontemporal_load(reinterpret_cast<const nt2*>(Mo + off));
          const nt2 b = __builtin_nontemporal_load(reinterpret_cast<const nt2*>(Xo + off));
          w[t][0] = a.x; w[t][1] = a.y;
          x[t][0] = b.x; x[t][1] = b.y;
        } else {
          w[t][0] = __builtin_nontemporal_load(Mo + off);
          x[t][0] = __builtin_nontemporal_load(Xo + off);
        }
      } else {
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
          const bool in = row < i_end && j0 + c < n;
          w[t][c] = in ? Mo[off + c] : 0.0f;
          x[t][c] = in ? Xo[off + c] : 0.0f;
        }
      }
    }
#pragma unroll
    for (int t = 0; t < U; ++t) {
      const int row = i + 4 * t;
      if (row >= i_end) break;   // uniform over the wave
      const long long off = static_cast<long long>(row) * n + j0;
      float sm[CPT], sx[CPT];
#pragma unroll
      for (int c = 0; c < CPT; ++c) { sm[c] = 0.0f; sx[c] = 0.0f; }
#pragma unroll
      for (int k = 0; k < RMAX; ++k) {
        const float pk = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, pv[t]), k));
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
          sm[c] = fmaf(pk, rr[c][k], sm[c]);
          sx[c] = fmaf(pk, qq[c][k], sx[c]);
        }
      }
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        w[t][c] = fmaf(cm, sm[c], w[t][c]);
        // undo a speculative skip-branch update (it already applied the
        // weight decay), else apply the decay
        const float xv = gc != 0.0f ? fmaf(gc, load_g(G, gbf, off + c), x[t][c]) : x[t][c] * xd;
        x[t][c] = fmaf(cx, sx[c], xv);
      }
      if (vec) {
        if constexpr (CPT == 4) {
          __builtin_nontemporal_store(nt4{w[t][0], w[t][1], w[t][2], w[t][3]}, reinterpret_cast<nt4*>(Mo + off));
          __builtin_nontemporal_store(nt4{x[t][0], x[t][1], x[t][2], x[t][3]}, reinterpret_cast<nt4*>(Xo + off));
        } else if constexpr (CPT == 2) {
          __builtin_nontemporal_store(nt2{w[t][0], w[t][1]}, reinterpret_cast<nt2*>(Mo + off));
          __builtin_nontemporal_store(nt2{x[t][0], x[t][1]}, reinterpret_cast<nt2*>(Xo + off));
        } else {
          __builtin_nontemporal_store(w[t][0], Mo + off);
          __builtin_nontemporal_store(x[t][0], Xo + off);
        }
      } else {
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
          if (j0 + c >= n) continue;
          Mo[off + c] = w[t][c];
          Xo[off + c] = x[t][c];
        }
      }
    }
  }
}

}  // namespace

bool update_vec_fits(int r) { return r >= 1 && r <= 32; }

hipError_t launch_update_vec(UpdateVecArgs u, int nl, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  if (!update_vec_fits(u.r) || u.m < 1 || u.n < 1) return hipErrorInvalidValue;
  // one column per lane, eight rows per batch (measured best on 4096 x 16384
  // against two or four columns per lane and 1-16 rows)
  constexpr int CPT = 1, U = 8;
  const int strips = (u.n + 64 * CPT - 1) / (64 * CPT);
  // about 16 waves per CU over the whole launch, at least one row per wave
  const long long target = 4096;
  const long long waves_per_strip = std::max(1LL, target / (static_cast<long long>(strips) * nl));
  const long long rows_per_wave = std::max(1LL, (u.m + waves_per_strip - 1) / waves_per_strip);
  u.band = static_cast<int>(std::min<long long>(4 * rows_per_wave, u.m));
  const int bands = (u.m + u.band - 1) / u.band;
  const dim3 grid(strips, bands, nl);
  if (u.r <= 16) hipLaunchKernelGGL((k_update_vec<16, CPT, U>), grid, dim3(256), 0, s, u);
  else hipLaunchKernelGGL((k_update_vec<32, CPT, U>), grid, dim3(256), 0, s, u);
  return hipGetLastError();
}

}  // namespace cd
