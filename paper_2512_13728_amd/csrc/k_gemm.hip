// Skinny GEMMs of the Dion power iteration (Algorithm 1 / Algorithm 2, sync
// branch) on MFMA:
//   P~ = B Q            (m x n . n x r; A = B row-major, k contiguous)
//   W  = P~^T P~        (Gram matrix, upper tiles only)
//   R  = B^T P          (fp32-gradient layers: B fp32, P fp64, R rounded to fp32)
// These run in fp64 (v_mfma_f64_16x16x4_f64 on fp32 or fp64 operands): P~
// is the ill-conditioned panel, and keeping it, its Gram matrix and the CholQR
// passes in fp64 makes the orthonormal P accurate to fp32 rounding whatever
// kappa(P~) is.  (R = B^T P and the fp32-accurate variants run on the
// bf16-split kernels.)
// K can be split over blockIdx.y into partial products that
// launch_reduce_splits adds in a fixed order (deterministic).
#include "common.hpp"
#include "mfma_tile.hpp"

namespace cd {
namespace {

// TIn: element type of the A operand; TInB: of the B operand.
template <typename T, typename TIn, typename TOut, int BM, int BN, bool A_KC, bool B_KC, typename TInB = TIn>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs g) {
  constexpr int WN_WAVES = (BN >= 64) ? 2 : 1;
  constexpr int WM_WAVES = 4 / WN_WAVES;
  constexpr int WM = BM / WM_WAVES, WN = BN / WN_WAVES;
  constexpr int TM = WM / 16, TN = WN / 16;
  static_assert(TM >= 1 && TN >= 1, "tile too small");
  __shared__ __attribute__((aligned(16))) T As[tile_elems<BM>()];
  __shared__ __attribute__((aligned(16))) T Bs[tile_elems<BN>()];
  if (skip_launch(g.run_if)) return;

  const int layer = blockIdx.z;
  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  const int t = xcd_tile(blockIdx.x, tiles_m * tiles_n);
  if (t >= tiles_m * tiles_n) return;
  const int tm = t / tiles_n, tn = t - tm * tiles_n;
  if (g.upper_only && tm > tn) return;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kb = blockIdx.y * g.kchunk;
  const int ke = min(g.K, kb + g.kchunk);
  const TIn* A = static_cast<const TIn*>(g.A[layer]);
  const TInB* Bm = static_cast<const TInB*>(g.B[layer]);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / WN_WAVES) * WM, wn0 = (wave % WN_WAVES) * WN;

  typename Mfma<T>::acc_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = typename Mfma<T>::acc_t{};

  Prefetch<TIn, BM, 256, A_KC> pa;
  Prefetch<TInB, BN, 256, B_KC> pb;
  if (kb < ke) {
    pa.load(A, g.lda, m0, g.M, kb, ke, tid);
    pb.load(Bm, g.ldb, n0, g.N, kb, ke, tid);
  }
  for (int k0 = kb; k0 < ke; k0 += GBK) {
    pa.template store<T>(As, tid);
    pb.template store<T>(Bs, tid);
    __syncthreads();
    if (k0 + GBK < ke) {
      pa.load(A, g.lda, m0, g.M, k0 + GBK, ke, tid);
      pb.load(Bm, g.ldb, n0, g.N, k0 + GBK, ke, tid);
    }
#pragma unroll
    for (int kk = 0; kk < GBK; kk += 16) {
      typename Mfma<T>::vec4_t a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) a[i] = frag<T, BM, A_KC>(As, wm0 + i * 16, kk, lane);
#pragma unroll
      for (int j = 0; j < TN; ++j) b[j] = frag<T, BN, B_KC>(Bs, wn0 + j * 16, kk, lane);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) acc[i][j] = Mfma<T>::mma(a[i][q], b[j][q], acc[i][j]);
    }
    __syncthreads();
  }

  // split partials keep the accumulation type; a single slice writes TOut
  const bool partial = g.splits > 1;
  T* Cp = static_cast<T*>(g.C[layer]) + static_cast<long long>(blockIdx.y) * g.split_stride;
  TOut* Co = static_cast<TOut*>(g.C[layer]);
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = m0 + wm0 + i * 16 + Mfma<T>::out_row(lane, v);
        const int col = n0 + wn0 + j * 16 + (lane & 15);
        if (row < g.M && col < g.N) {
          const long long o = static_cast<long long>(row) * g.ldc + col;
          if (partial) Cp[o] = acc[i][j][v];
          else Co[o] = static_cast<TOut>(acc[i][j][v]);
        }
      }
}

// Sum of the split-K partials in split order.  16-byte vectors of V
// elements when the sizes and bases allow (count and stride multiples of V),
// so that every thread has `splits` vector loads in flight.
template <typename TP, typename TO>
__global__ __launch_bounds__(256) void k_reduce(ReduceArgs a) {
  if (skip_launch(a.run_if)) return;
  constexpr int V = 16 / sizeof(TP);
  typedef TP vec_t __attribute__((ext_vector_type(V)));
  const int l = blockIdx.y;
  const TP* p = static_cast<const TP*>(a.part[l]);
  TO* o = static_cast<TO*>(a.out[l]);
  const bool vec = a.count % V == 0 && a.stride % V == 0 &&
                   (reinterpret_cast<unsigned long long>(p) & 15) == 0 &&
                   (reinterpret_cast<unsigned long long>(o) & (sizeof(TO) * V - 1)) == 0;
  if (vec) {
    const long long nv = a.count / V;
    for (long long i = blockIdx.x * 256LL + threadIdx.x; i < nv; i += 256LL * gridDim.x) {
      vec_t s = *reinterpret_cast<const vec_t*>(p + i * V);
      for (int k = 1; k < a.splits; ++k) s += *reinterpret_cast<const vec_t*>(p + k * a.stride + i * V);
#pragma unroll
      for (int c = 0; c < V; ++c) o[i * V + c] = static_cast<TO>(s[c]);
    }
    return;
  }
  for (long long i = blockIdx.x * 256LL + threadIdx.x; i < a.count; i += 256LL * gridDim.x) {
    TP s = p[i];
    for (int k = 1; k < a.splits; ++k) s += p[k * a.stride + i];
    o[i] = static_cast<TO>(s);
  }
}

template <typename T, typename TIn, typename TOut, int BM, int BN, typename TInB = TIn>
hipError_t launch_t(const GemmArgs& g, int nl, hipStream_t s) {
  const int tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  const dim3 grid(xcd_grid(tiles), g.splits, nl);
  if (g.a_kc && !g.b_kc)
    hipLaunchKernelGGL((k_gemm<T, TIn, TOut, BM, BN, true, false, TInB>), grid, dim3(256), 0, s, g);
  else if (!g.a_kc && !g.b_kc)
    hipLaunchKernelGGL((k_gemm<T, TIn, TOut, BM, BN, false, false, TInB>), grid, dim3(256), 0, s, g);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// Narrow products (r <= 32) take 64 x 16 or 64 x 32 tiles (one wave column,
// four waves down): a 64-wide tile would spend most of its MFMAs on padding.
int tile_n(int N) { return N <= 16 ? 16 : (N <= 32 ? 32 : 64); }

template <typename T, typename TIn, typename TOut, typename TInB = TIn>
hipError_t launch_n(const GemmArgs& g, int nl, hipStream_t s) {
  switch (tile_n(g.N)) {
    case 16: return launch_t<T, TIn, TOut, 64, 16, TInB>(g, nl, s);
    case 32: return launch_t<T, TIn, TOut, 64, 32, TInB>(g, nl, s);
    default: return launch_t<T, TIn, TOut, 64, 64, TInB>(g, nl, s);
  }
}

}  // namespace

// Tile shape of the fp64 kernels: 64 rows, 16 / 32 / 64 columns by N.
int gemm_bm(int N, bool fp64) { (void)N; (void)fp64; return 64; }
int gemm_bn(int N, bool fp64) { (void)fp64; return tile_n(N); }

hipError_t launch_gemm(const GemmArgs& g, int nl, GemmKind kind, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  switch (kind) {
    case GemmKind::F64_FROM_F32: return launch_n<double, float, double>(g, nl, s);
    case GemmKind::F64: return launch_n<double, double, double>(g, nl, s);
    case GemmKind::F64_TO_F32: return launch_n<double, double, float>(g, nl, s);
    case GemmKind::F32_F64_TO_F32: return launch_n<double, float, float, double>(g, nl, s);
    case GemmKind::F32: break;  // fp32 contractions run on the bf16-split kernels
  }
  return hipErrorInvalidValue;
}

hipError_t launch_reduce_splits(const ReduceArgs& a, int nl, bool part64, bool out64, hipStream_t s) {
  if (nl <= 0 || a.count <= 0) return hipSuccess;
  long long blocks = (a.count / 2 + 255) / 256;   // two or four elements per thread
  if (blocks > 4096) blocks = 4096;
  const dim3 grid(static_cast<unsigned>(blocks), nl);
  if (part64 && out64) hipLaunchKernelGGL((k_reduce<double, double>), grid, dim3(256), 0, s, a);
  else if (part64) hipLaunchKernelGGL((k_reduce<double, float>), grid, dim3(256), 0, s, a);
  else if (out64) hipLaunchKernelGGL((k_reduce<float, double>), grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL((k_reduce<float, float>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace cd
