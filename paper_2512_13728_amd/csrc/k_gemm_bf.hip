// Skinny GEMMs and the fused M/X update on the bf16 MFMA with split fp32
// operands (see bf16_split.hpp):
//   R  = B^T P            (A = B^T, not k-contiguous; B operand = P)
//   P~ = B Q              (A = B row-major; B operand = Q)
//   M  = B - (1 - mu) P R^T,  X -= c P Q^T   (both products from one P tile)
// 128-row tiles, 4 waves as 2 x 2, next stage prefetched into registers while
// the current one is multiplied.  Block index -> tile is XCD-aware.
#include "bf16_split.hpp"
#include "common.hpp"

namespace cd {
namespace {

template <int S, int BM, int BN, bool A_KC, bool B_KC>
__global__ __launch_bounds__(256) void k_gemm_bf(GemmArgs g) {
  constexpr int WN_WAVES = (BN >= 64) ? 2 : 1;
  constexpr int WM_WAVES = 4 / WN_WAVES;
  constexpr int WM = BM / WM_WAVES, WN = BN / WN_WAVES;
  constexpr int TM = WM / 16, TN = WN / 16;
  static_assert(TM >= 1 && TN >= 1, "tile too small");
  __shared__ __attribute__((aligned(16))) __bf16 As[S * BM * BLD];
  __shared__ __attribute__((aligned(16))) __bf16 Bs[S * BN * BLD];

  const int layer = blockIdx.z;
  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  const int t = xcd_tile(blockIdx.x, tiles_m * tiles_n);
  if (t >= tiles_m * tiles_n) return;
  const int tm = t / tiles_n, tn = t - tm * tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kb = blockIdx.y * g.kchunk;
  const int ke = min(g.K, kb + g.kchunk);
  const float* A = static_cast<const float*>(g.A[layer]);
  const float* Bm = static_cast<const float*>(g.B[layer]);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / WN_WAVES) * WM, wn0 = (wave % WN_WAVES) * WN;

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{};

  Stage<BM, 256> sa;
  Stage<BN, 256> sb;
  if (kb < ke) {
    sa.load(A, g.lda, A_KC, m0, g.M, kb, ke, tid);
    sb.load(Bm, g.ldb, B_KC, n0, g.N, kb, ke, tid);
  }
  for (int k0 = kb; k0 < ke; k0 += BK16) {
    sa.template store<S>(As, A_KC, tid);
    sb.template store<S>(Bs, B_KC, tid);
    __syncthreads();
    if (k0 + BK16 < ke) {
      sa.load(A, g.lda, A_KC, m0, g.M, k0 + BK16, ke, tid);
      sb.load(Bm, g.ldb, B_KC, n0, g.N, k0 + BK16, ke, tid);
    }
    bf16x8 a[TM][S], b[TN][S];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int s = 0; s < S; ++s) a[i][s] = bfrag(As + s * BM * BLD, wm0 + i * 16, lane);
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int s = 0; s < S; ++s) b[j][s] = bfrag(Bs + s * BN * BLD, wn0 + j * 16, lane);
    // piece products p + q <= S - 1 (0-based), smallest first
#pragma unroll
    for (int sum = S - 1; sum >= 0; --sum)
#pragma unroll
      for (int p = 0; p <= sum; ++p)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) acc[i][j] = mfma_bf16(a[i][p], b[j][sum - p], acc[i][j]);
    __syncthreads();
  }

  float* C = static_cast<float*>(g.C[layer]) + static_cast<long long>(blockIdx.y) * g.split_stride;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = m0 + wm0 + i * 16 + 4 * (lane >> 4) + v;
        const int col = n0 + wn0 + j * 16 + (lane & 15);
        if (row < g.M && col < g.N) C[static_cast<long long>(row) * g.ldc + col] = acc[i][j][v];
      }
}

// M = B - (1 - mu) P R^T and X -= c P Q^T on a 128 x 64 tile of the m x n
// matrices; K = r.  P (m x r), R and Q (n x r) are all k-contiguous.
constexpr int UBM = 128, UBN = 64;

template <int S>
__global__ __launch_bounds__(256) void k_update_bf(UpdateArgs u) {
  constexpr int TM = 4, TN = 2;   // wave tile 64 x 32
  __shared__ __attribute__((aligned(16))) __bf16 Ps[S * UBM * BLD];
  __shared__ __attribute__((aligned(16))) __bf16 Rs[S * UBN * BLD];
  __shared__ __attribute__((aligned(16))) __bf16 Qs[S * UBN * BLD];
  const int l = blockIdx.z;
  const int tiles_n = (u.n + UBN - 1) / UBN;
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x - tm * tiles_n;
  const int m0 = tm * UBM, n0 = tn * UBN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 64, wn0 = (wave & 1) * 32;
  const float* P = u.P[l];
  const float* R = u.R[l];
  const float* Q = u.Q[l];

  f32x4 am[TM][TN], ax[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) { am[i][j] = f32x4{}; ax[i][j] = f32x4{}; }

  Stage<UBM, 256> sp;
  Stage<UBN, 256> sr, sq;
  sp.load(P, u.r, true, m0, u.m, 0, u.r, tid);
  sr.load(R, u.r, true, n0, u.n, 0, u.r, tid);
  sq.load(Q, u.r, true, n0, u.n, 0, u.r, tid);
  for (int k0 = 0; k0 < u.r; k0 += BK16) {
    sp.template store<S>(Ps, true, tid);
    sr.template store<S>(Rs, true, tid);
    sq.template store<S>(Qs, true, tid);
    __syncthreads();
    if (k0 + BK16 < u.r) {
      sp.load(P, u.r, true, m0, u.m, k0 + BK16, u.r, tid);
      sr.load(R, u.r, true, n0, u.n, k0 + BK16, u.r, tid);
      sq.load(Q, u.r, true, n0, u.n, k0 + BK16, u.r, tid);
    }
    bf16x8 a[TM][S], rb[TN][S], qb[TN][S];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int s = 0; s < S; ++s) a[i][s] = bfrag(Ps + s * UBM * BLD, wm0 + i * 16, lane);
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int s = 0; s < S; ++s) {
        rb[j][s] = bfrag(Rs + s * UBN * BLD, wn0 + j * 16, lane);
        qb[j][s] = bfrag(Qs + s * UBN * BLD, wn0 + j * 16, lane);
      }
#pragma unroll
    for (int sum = S - 1; sum >= 0; --sum)
#pragma unroll
      for (int p = 0; p <= sum; ++p)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            am[i][j] = mfma_bf16(a[i][p], rb[j][sum - p], am[i][j]);
            ax[i][j] = mfma_bf16(a[i][p], qb[j][sum - p], ax[i][j]);
          }
    __syncthreads();
  }

  float* M = u.M[l];
  float* X = u.X[l];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
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

template <int S, int BM, int BN>
hipError_t launch_bm(const GemmArgs& g, int nl, hipStream_t s) {
  const int tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  const dim3 grid(xcd_grid(tiles), g.splits, nl);
  if (g.a_kc && !g.b_kc) hipLaunchKernelGGL((k_gemm_bf<S, BM, BN, true, false>), grid, dim3(256), 0, s, g);
  else if (!g.a_kc && !g.b_kc) hipLaunchKernelGGL((k_gemm_bf<S, BM, BN, false, false>), grid, dim3(256), 0, s, g);
  else if (g.a_kc && g.b_kc) hipLaunchKernelGGL((k_gemm_bf<S, BM, BN, true, true>), grid, dim3(256), 0, s, g);
  else hipLaunchKernelGGL((k_gemm_bf<S, BM, BN, false, true>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

template <int S>
hipError_t launch_s(const GemmArgs& g, int nl, hipStream_t s) {
  if (g.N > 64) return launch_bm<S, 128, 128>(g, nl, s);
  if (g.N > 32) return launch_bm<S, 128, 64>(g, nl, s);
  return launch_bm<S, 128, 32>(g, nl, s);
}

}  // namespace

int gemm_bf_bm(int N) { (void)N; return 128; }
int gemm_bf_bn(int N) { return N > 64 ? 128 : (N > 32 ? 64 : 32); }

hipError_t launch_gemm_bf(const GemmArgs& g, int nl, int pieces, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  if (pieces == 3) return launch_s<3>(g, nl, s);
  if (pieces == 2) return launch_s<2>(g, nl, s);
  return launch_s<1>(g, nl, s);
}

hipError_t launch_update_bf(const UpdateArgs& u, int nl, int pieces, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  const int tiles = ((u.m + UBM - 1) / UBM) * ((u.n + UBN - 1) / UBN);
  const dim3 grid(tiles, 1, nl);
  if (pieces == 3) hipLaunchKernelGGL(k_update_bf<3>, grid, dim3(256), 0, s, u);
  else if (pieces == 2) hipLaunchKernelGGL(k_update_bf<2>, grid, dim3(256), 0, s, u);
  else hipLaunchKernelGGL(k_update_bf<1>, grid, dim3(256), 0, s, u);
  return hipGetLastError();
}

}  // namespace cd
