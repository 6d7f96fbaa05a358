// The sync branch of small layers (r <= SMALL_R, m r and n r <= SMALL_MR) in
// four launches instead of the blocked pipeline's seventeen or so: the power
// products P~ = B Q and R = B^T P run on the fp64 GEMM kernels (no split-K),
// and the two kernels here do the rest.
//
//   k_small_cholqr   Orthogonalize (Algorithm 1 / 2): the thin-QR factor of
//                    P~ with positive diagonal by CholQR twice, one workgroup
//                    per layer with the whole m x r panel in LDS, fp64
//                    throughout (Gram matrix on the fp64 MFMA, the one-wave
//                    Cholesky factorisation and inverse of the blocked
//                    kernels' diagonal blocks, P T^-1), the same pivot floor
//                    and completion past the numerical rank as the blocked
//                    kernels.  Writes P in fp64 (for R = B^T P) and fp32.
//   k_small_update   ColumnNormalize and the error-feedback / weight updates:
//                    every workgroup forms the column norms of R (fixed order,
//                    fp64), Q = R / norm (the first workgroup stores Q), and
//                    updates its rows of M = B - (1 - mu) P R^T and
//                    X -= eta sqrt(m/n) P Q^T with fp32 products, k in order.
//
// At these sizes every launch is a few microseconds of latency and the work a
// fraction of it, so fewer launches is what the step needs.
#include "chol_wave.hpp"
#include "common.hpp"
#include "mfma_tile.hpp"

namespace cd {
namespace {

constexpr int SQR_THREADS = 256;
constexpr int BATCH = 8;   // global loads issued before their LDS stores

// dst[e] = f(src[e]) for e < count, BATCH loads per thread in flight (a copy
// loop that stores each value before loading the next would wait out the
// memory latency once per element)
template <int NT, typename TD, typename TS, typename F>
__device__ __forceinline__ void copy_batched(TD* dst, const TS* src, int count, int tid, F&& f) {
  for (int e0 = 0; e0 < count; e0 += NT * BATCH) {
    TS v[BATCH];
#pragma unroll
    for (int u = 0; u < BATCH; ++u) {
      const int e = e0 + u * NT + tid;
      v[u] = e < count ? src[e] : TS(0);
    }
#pragma unroll
    for (int u = 0; u < BATCH; ++u) {
      const int e = e0 + u * NT + tid;
      if (e < count) f(dst, e, v[u]);
    }
  }
}

// One workgroup per layer, the whole m x r panel in LDS (fp64, row-major).
// Each CholQR pass:
//   W = P^T P        fp64 MFMA, 16 x 16 upper tiles; wave w takes the 16-row
//                    groups w, w + 4, ..., and the four partial sums are added
//                    into W in wave order
//   W = T^T T, T^-1  wave 0 (chol_wave.hpp), the same pivot floor as the
//                    blocked kernels; T^-1 is written over W
//   P <- P T^-1      fp64 MFMA, 16 x 16 tiles (the columns of floored pivots
//                    come out zero)
// then, after pass 0, the completion past the numerical rank.
// LDS at NB = 64: panel 64 KB, W 32 KB, factorisation 35 KB.
template <int NB>
__global__ __launch_bounds__(SQR_THREADS) void k_small_cholqr(SmallQrArgs a) {
  using WC = WaveChol<NB>;
  constexpr int NT = NB / 16;                  // 16-column blocks
  constexpr int NTILE = NT * (NT + 1) / 2;     // upper 16 x 16 tiles of W
  __shared__ double Pl[SMALL_MR];
  __shared__ double Wl[NB * NB];               // W (upper triangle), then T^-1; row stride NB
  __shared__ __attribute__((aligned(16))) typename WC::Lds wc;
  __shared__ int floored;
  if (skip_launch(a.run_if)) return;
  const int l = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m = a.m, r = a.r, mr = m * r;
  copy_batched<SQR_THREADS>(Pl, a.Pt[l], mr, tid, [](double* d, int e, double v) { d[e] = v; });
  __syncthreads();
  // MFMA operands: lane owns column (lane % 16) of a 16-column block and rows
  // (k indices) 4 (lane / 16) + q of a group of 16, q = 0..3 (one per MFMA)
  const int col = lane & 15, kq = 4 * (lane >> 4);
  bool any_dead = false;   // uniform: every thread reads the same flags
  for (int pass = 0; pass < 2; ++pass) {
    {
      f64x4 acc[NTILE];
#pragma unroll
      for (int t = 0; t < NTILE; ++t) acc[t] = f64x4{};
      for (int k0 = wave * 16; k0 < m; k0 += 4 * 16) {
        double x[NT][4];
#pragma unroll
        for (int b = 0; b < NT; ++b)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int row = k0 + kq + q, c = b * 16 + col;
            x[b][q] = (row < m && c < r) ? Pl[row * r + c] : 0.0;
          }
        int t = 0;
#pragma unroll
        for (int bi = 0; bi < NT; ++bi)
#pragma unroll
          for (int bj = bi; bj < NT; ++bj, ++t)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              acc[t] = __builtin_amdgcn_mfma_f64_16x16x4f64(x[bi][q], x[bj][q], acc[t], 0, 0, 0);
      }
#pragma unroll 1
      for (int w = 0; w < 4; ++w) {
        if (wave == w) {
          int t = 0;
#pragma unroll
          for (int bi = 0; bi < NT; ++bi)
#pragma unroll
            for (int bj = bi; bj < NT; ++bj, ++t)
#pragma unroll
              for (int v = 0; v < 4; ++v) {
                const int row = bi * 16 + Mfma<double>::out_row(lane, v), c = bj * 16 + col;
                if (row < r && c < r) {
                  double* const wp = Wl + row * NB + c;
                  *wp = (w == 0 ? 0.0 : *wp) + acc[t][v];
                }
              }
        }
        __syncthreads();
      }
    }
    if (wave == 0) {
      // j made opaque here: otherwise the compiler keeps the register
      // arrays' initial values (functions of j and r only) live across the
      // pass loop, and spills
      int j = lane;
      __asm__ volatile("" : "+v"(j));
      // pivot floor: 1e-13 of the largest diagonal (at least 1e-60)
      double md = j < r ? Wl[j * NB + j] : 0.0;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) md = fmax(md, __shfl_xor(md, o, 64));
      const double fl = fmax(1e-13 * md, 1e-60);
      // the factorisation holds W in registers once it starts, so T^-1 may
      // go over it (NB <= 32: formed in the factorisation's own pivot loop)
      bool def;
      if constexpr (NB <= 32) {
        def = WC::factor_inv(wc, j, r, fl, [&](int i) { return Wl[i * NB + j]; },
                             [&](int c, int p, double x) { Wl[c * NB + p] = x; });
      } else {
        def = WC::factor(wc, j, r, fl, [&](int i) { return Wl[i * NB + j]; });
        WC::inverse(wc, j, r, [&](int p, double x) {
          if (j < r) Wl[p * NB + j] = x;
        });
      }
      if (j == 0) floored = def ? 1 : 0;
    }
    __syncthreads();
    const bool dead = floored != 0;
    any_dead = any_dead || dead;
    // P T^-1 on the fp64 MFMA in 16 x 16 output tiles (row block ib, column
    // block jb), K over the column blocks kb <= jb (T^-1 is upper
    // triangular).  A tile reads only its own row block of P, so the tiles go
    // in rounds of whole row blocks: every wave forms its tiles of the round
    // (at most 4), then, after a barrier, the pass-0 result goes over the
    // panel (pass 1: straight to P64 / P32).
    {
      const int nbk = (r + 15) / 16, mb = (m + 15) / 16;
      const int rows_per_round = 16 / nbk;   // nbk <= 4
      const float scale = sqrtf(3.0f / static_cast<float>(m));
      double* __restrict__ P64 = a.P64[l];
      float* __restrict__ P32 = a.P32[l];
      for (int ib0 = 0; ib0 < mb; ib0 += rows_per_round) {
        const int ntile = min(rows_per_round, mb - ib0) * nbk;
        f64x4 o[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          o[u] = f64x4{};
          const int t = wave + 4 * u;
          if (t < ntile) {
            const int ib = ib0 + t / nbk, jb = t - (t / nbk) * nbk;
            const int row = ib * 16 + col, cj = jb * 16 + col;
            for (int kb = 0; kb <= jb; ++kb)
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const int k = kb * 16 + kq + q;
                const double x = (row < m && k < r) ? Pl[row * r + k] : 0.0;
                const double y = (k < r && cj < r) ? Wl[k * NB + cj] : 0.0;
                o[u] = __builtin_amdgcn_mfma_f64_16x16x4f64(x, y, o[u], 0, 0, 0);
              }
          }
        }
        if (pass == 0) __syncthreads();
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int t = wave + 4 * u;
          if (t < ntile) {
            const int ib = ib0 + t / nbk, jb = t - (t / nbk) * nbk;
            const int j = jb * 16 + col;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int i = ib * 16 + Mfma<double>::out_row(lane, v);
              if (i < m && j < r) {
                const int e = i * r + j;
                if (pass == 0) {
                  // completion past the numerical rank: the fixed pseudo-random
                  // direction of each column whose pass-0 pivot was floored,
                  // orthonormalised by the second pass
                  Pl[e] = (dead && !wc.okb[j]) ? static_cast<double>(fill_value(i, j, scale)) : o[u][v];
                } else {
                  P64[e] = o[u][v];
                  P32[e] = static_cast<float>(o[u][v]);
                }
              }
            }
          }
        }
      }
      __syncthreads();
    }
  }
  if (tid == 0) {
    *a.rankdef[l] = any_dead ? 1 : 0;
    if (a.rankdef_host[l]) *a.rankdef_host[l] = any_dead ? 1 : 0;
  }
}

// P~ = B Q of small layers (N = r <= 64, K = n <= 1024; A = B fp32
// row-major, B = Q fp32, C fp64) on the fp64 MFMA: one workgroup per 16 rows
// of C, the four waves taking a quarter of K each, every operand loaded
// straight into registers (a wave's whole K range in at most two rounds of
// loads, the second requested before the first is used), and the four
// partial tiles added in wave order through LDS.  At these sizes the blocked
// kernel's K loop is a chain of memory latencies, one per stage: 256 x 256,
// r = 16 took 10.2 us there and takes 7.6 here.  (For R = B^T P, whose A
// operand is not k-contiguous, the same scheme measured 10.6 us against the
// blocked kernel's 9.3, which therefore stays.)
constexpr int SG_KMAX = 1024;
template <typename TB, typename TC, bool A_KC, int NT>
__global__ __launch_bounds__(256) void k_small_gemm(GemmArgs g) {
  constexpr int D = 4 / NT;              // 16-k chunks per round of loads
  constexpr int NC = NT * 16;
  __shared__ double red[4][16][NC + 1];
  if (skip_launch(g.run_if)) return;
  const int l = blockIdx.y, row0 = blockIdx.x * 16;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* __restrict__ A = static_cast<const float*>(g.A[l]);
  const TB* __restrict__ B = static_cast<const TB*>(g.B[l]);
  // the wave's K range: a quarter of K, rounded up to 16
  const int kw = (g.K + 63) / 64 * 16;
  const int kw0 = wave * kw, kw1 = min(g.K, kw0 + kw);
  // MFMA operand of lane l for the q-th product of a 16-k chunk at k0: row
  // (or column) l % 16, k = k0 + 4 (l / 16) + q
  const int ri = lane & 15, kl = 4 * (lane >> 4);
  const int row = row0 + ri;
  f64x4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = f64x4{};
  double a[2][D][4], b[2][D][NT][4];
  auto load = [&](int buf, int kb) {
#pragma unroll
    for (int d = 0; d < D; ++d)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = kb + 16 * d + kl + q;
        const bool kin = k < kw1;
        a[buf][d][q] = (kin && row < g.M)
                           ? static_cast<double>(A_KC ? A[static_cast<long long>(row) * g.lda + k]
                                                      : A[static_cast<long long>(k) * g.lda + row])
                           : 0.0;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const int c = t * 16 + ri;
          b[buf][d][t][q] = (kin && c < g.N) ? static_cast<double>(B[static_cast<long long>(k) * g.ldb + c]) : 0.0;
        }
      }
  };
  auto mult = [&](int buf) {
#pragma unroll
    for (int d = 0; d < D; ++d)
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int t = 0; t < NT; ++t)
          acc[t] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[buf][d][q], b[buf][d][t][q], acc[t], 0, 0, 0);
  };
  constexpr int KR = 16 * D;             // k per round
  if (kw0 < kw1) load(0, kw0);
  if (kw0 + KR < kw1) load(1, kw0 + KR);
  for (int kb = kw0; kb < kw1; kb += 2 * KR) {
    mult(0);
    if (kb + 2 * KR < kw1) load(0, kb + 2 * KR);
    if (kb + KR < kw1) {
      mult(1);
      if (kb + 3 * KR < kw1) load(1, kb + 3 * KR);
    }
  }
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int v = 0; v < 4; ++v) red[wave][Mfma<double>::out_row(lane, v)][t * 16 + ri] = acc[t][v];
  __syncthreads();
  TC* __restrict__ C = static_cast<TC*>(g.C[l]);
  for (int e = tid; e < 16 * NC; e += 256) {
    const int i = e / NC, c = e - i * NC;
    if (row0 + i < g.M && c < g.N)
      C[static_cast<long long>(row0 + i) * g.ldc + c] =
          static_cast<TC>(((red[0][i][c] + red[1][i][c]) + red[2][i][c]) + red[3][i][c]);
  }
}

constexpr int SUP_THREADS = 256;

// One workgroup per (row band, layer).  Every global read is requested at
// the start, so that their latencies overlap: this thread's column of the
// band's M, X (and G) rows, the band's rows of P, and R.  R and Q are held
// transposed in LDS (k-major, row stride n + 1), so that the lanes of a wave,
// which own consecutive columns c, read consecutive words, and the
// transposing stores of consecutive k fall into different banks.  The
// products: a thread takes its column of R and Q into registers once, then
// forms the band's rows together (k outer, rows inner, each sum in k order),
// reading P as broadcasts from LDS.
template <int NR>
__global__ __launch_bounds__(SUP_THREADS) void k_small_update(SmallUpdArgs a) {
  __shared__ float Rt[SMALL_MR + SMALL_R];
  __shared__ float Qt[SMALL_MR + SMALL_R];
  __shared__ float Pb[SMALL_ROWS * SMALL_R];
  __shared__ double part[SUP_THREADS];
  __shared__ float nrm[SMALL_R];
  if (a.ctl != nullptr && a.ctl->flag == 0) return;   // not a sync step
  const int l = blockIdx.y, tid = threadIdx.x;
  const int m = a.m, n = a.n, r = a.r, ldt = n + 1;
  const int i0 = blockIdx.x * SMALL_ROWS, rows = min(SMALL_ROWS, m - i0);
  float* __restrict__ Mo = a.M[l];
  float* __restrict__ Xo = a.X[l];
  const void* G = a.G[l];
  const bool spec = (a.spec == 2 ? a.ctl->spec_cur : a.spec) != 0;
  const float gc = spec ? a.gc[l] : 0.0f, xd = spec ? 1.0f : a.xdecay[l];
  const float cm = -a.one_minus_mu, cx = -a.c;
  // each thread owns one column c of every row of the band
  float mv[SMALL_ROWS], xv[SMALL_ROWS], gv[SMALL_ROWS];
  auto load_column = [&](int c) {
#pragma unroll
    for (int t = 0; t < SMALL_ROWS; ++t) {
      if (t < rows) {
        const long long off = static_cast<long long>(i0 + t) * n + c;
        mv[t] = Mo[off];
        xv[t] = Xo[off];
        gv[t] = gc == 0.0f ? 0.0f
                           : (a.g_bf16 ? __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(G)[off]) << 16)
                                       : static_cast<const float*>(G)[off]);
      }
    }
  };
  if (tid < n) load_column(tid);
  // this band's rows of P, and R (n x r, row-major) into Rt (k-major); the
  // loads in batches, row-major order, then the stores
  // P's band in rows of NR values (zero past r and past the band), so the
  // products below need no bounds: a zero adds nothing to a sum
  {
    const float* __restrict__ Pg = a.P[l] + static_cast<long long>(i0) * r;
    constexpr int PE = SMALL_ROWS * NR, PPER = (PE + SUP_THREADS - 1) / SUP_THREADS;
    float v[PPER];
#pragma unroll
    for (int u = 0; u < PPER; ++u) {
      const int e = u * SUP_THREADS + tid, t = e / NR, k = e - t * NR;
      v[u] = (e < PE && t < rows && k < r) ? Pg[t * r + k] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < PPER; ++u) {
      const int e = u * SUP_THREADS + tid;
      if (e < PE) Pb[e] = v[u];
    }
  }
  copy_batched<SUP_THREADS>(Rt, a.R[l], n * r, tid, [ldt, r](float* d, int e, float v) {
    const int c = e / r, k = e - c * r;
    d[k * ldt + c] = v;
  });
  __syncthreads();
  // column norms: tpc consecutive threads per column k, thread q summing
  // rows q, q + tpc, ... in order, then the tpc partial sums in order (the
  // order depends on n and r only)
  const int tpc = SUP_THREADS / r;
  {
    double s = 0.0;
    const int k = tid / tpc, q = tid - k * tpc;
    if (k < r)
      for (int c = q; c < n; c += tpc) {
        const double v = Rt[k * ldt + c];
        s = fma(v, v, s);
      }
    part[tid] = s;
  }
  __syncthreads();
  if (tid < r) {
    double s = 0.0;
    for (int q = 0; q < tpc; ++q) s += part[tid * tpc + q];
    nrm[tid] = static_cast<float>(fmax(sqrt(s), 1e-30));
  }
  __syncthreads();
  float* __restrict__ Qo = a.Q[l];
  for (int e = tid; e < n * r; e += SUP_THREADS) {
    const int k = e / n, c = e - k * n;
    const float q = Rt[k * ldt + c] / nrm[k];
    Qt[k * ldt + c] = q;
    if (blockIdx.x == 0) Qo[c * r + k] = q;
  }
  __syncthreads();
  for (int c = tid; c < n; c += SUP_THREADS) {
    if (c != tid) load_column(c);
    constexpr int KB = NR < 32 ? NR : 32;   // k values of R and Q held at a time
    float sm[SMALL_ROWS], sx[SMALL_ROWS];
#pragma unroll
    for (int t = 0; t < SMALL_ROWS; ++t) { sm[t] = 0.0f; sx[t] = 0.0f; }
    // (no early exits, so that the loops unroll: past r the R and Q values
    // and P's entries are zero, and a sum that starts at +0 is unchanged by
    // adding 0 x 0).  P is read through an offset the compiler cannot see
    // through, so that it does not hoist the whole band into registers
    // across the column loop.
    int pofs = 0;
    __asm__ volatile("" : "+v"(pofs));
    const float* const Pr = Pb + pofs;
#pragma unroll
    for (int k0 = 0; k0 < NR; k0 += KB) {
      if (k0 < r) {
        float rc[KB], qc[KB];
#pragma unroll
        for (int k = 0; k < KB; ++k) {
          rc[k] = k0 + k < r ? Rt[(k0 + k) * ldt + c] : 0.0f;
          qc[k] = k0 + k < r ? Qt[(k0 + k) * ldt + c] : 0.0f;
        }
#pragma unroll
        for (int k = 0; k < KB; ++k)
#pragma unroll
          for (int t = 0; t < SMALL_ROWS; ++t) {
            const float pk = Pr[t * NR + k0 + k];
            sm[t] = fmaf(pk, rc[k], sm[t]);
            sx[t] = fmaf(pk, qc[k], sx[t]);
          }
      }
    }
#pragma unroll
    for (int t = 0; t < SMALL_ROWS; ++t) {
      if (t < rows) {
        const long long off = static_cast<long long>(i0 + t) * n + c;
        const float x = gc != 0.0f ? fmaf(gc, gv[t], xv[t]) : xv[t] * xd;
        Mo[off] = fmaf(cm, sm[t], mv[t]);
        Xo[off] = fmaf(cx, sx[t], x);
      }
    }
  }
}

}  // namespace

bool small_sync_fits(int m, int n, int r) {
  return r >= 1 && r <= SMALL_R && 1LL * m * r <= SMALL_MR && 1LL * n * r <= SMALL_MR;
}

template <typename TB, typename TC, bool A_KC>
hipError_t launch_sg(const GemmArgs& g, int nl, hipStream_t s) {
  const dim3 grid((g.M + 15) / 16, nl);
  if (g.N <= 16) hipLaunchKernelGGL((k_small_gemm<TB, TC, A_KC, 1>), grid, dim3(256), 0, s, g);
  else if (g.N <= 32) hipLaunchKernelGGL((k_small_gemm<TB, TC, A_KC, 2>), grid, dim3(256), 0, s, g);
  else hipLaunchKernelGGL((k_small_gemm<TB, TC, A_KC, 4>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

bool small_gemm_fits(int N, int K) { return N >= 1 && N <= SMALL_R && K >= 1 && K <= SG_KMAX; }

hipError_t launch_small_gemm(const GemmArgs& g, int nl, GemmKind kind, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  if (!small_gemm_fits(g.N, g.K) || g.splits != 1 || g.b_kc) return hipErrorInvalidValue;
  if (kind == GemmKind::F64_FROM_F32 && g.a_kc) return launch_sg<float, double, true>(g, nl, s);
  return hipErrorInvalidValue;
}

hipError_t launch_small_cholqr(const SmallQrArgs& a, int nl, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  if (!small_sync_fits(a.m, 1, a.r)) return hipErrorInvalidValue;
  if (a.r <= 16) hipLaunchKernelGGL(k_small_cholqr<16>, dim3(nl), dim3(SQR_THREADS), 0, s, a);
  else if (a.r <= 32) hipLaunchKernelGGL(k_small_cholqr<32>, dim3(nl), dim3(SQR_THREADS), 0, s, a);
  else hipLaunchKernelGGL(k_small_cholqr<64>, dim3(nl), dim3(SQR_THREADS), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_small_update(const SmallUpdArgs& a, int nl, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  if (!small_sync_fits(a.m, a.n, a.r) || (a.spec == 2 && !a.ctl)) return hipErrorInvalidValue;
  const dim3 grid((a.m + SMALL_ROWS - 1) / SMALL_ROWS, nl);
  // the products run over NR k values whatever r is (zeros past r): NR the
  // smallest of 4, 8, 16, 32, 64 that holds r
  if (a.r <= 4) hipLaunchKernelGGL(k_small_update<4>, grid, dim3(SUP_THREADS), 0, s, a);
  else if (a.r <= 8) hipLaunchKernelGGL(k_small_update<8>, grid, dim3(SUP_THREADS), 0, s, a);
  else if (a.r <= 16) hipLaunchKernelGGL(k_small_update<16>, grid, dim3(SUP_THREADS), 0, s, a);
  else if (a.r <= 32) hipLaunchKernelGGL(k_small_update<32>, grid, dim3(SUP_THREADS), 0, s, a);
  else hipLaunchKernelGGL(k_small_update<64>, grid, dim3(SUP_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace cd
