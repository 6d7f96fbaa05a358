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

// W64: the result is written as fp64 (one split only); a separate
// instantiation, so the common fp32 kernel carries no second store path.
template <int S, int BM, int BN, bool A_KC, bool B_KC, bool W64>
__global__ __launch_bounds__(256, 2) void k_gemm_bf(GemmArgs g) {
  constexpr int WN_WAVES = (BN >= 64) ? 2 : 1;
  constexpr int WM_WAVES = 4 / WN_WAVES;
  constexpr int WM = BM / WM_WAVES, WN = BN / WN_WAVES;
  constexpr int TM = WM / 16, TN = WN / 16;
  static_assert(TM >= 1 && TN >= 1, "tile too small");
  __shared__ __attribute__((aligned(16))) __bf16 As[S * BM * BLD];
  __shared__ __attribute__((aligned(16))) __bf16 Bs[S * BN * BLD];
  if (skip_launch(g.run_if)) return;

  const int layer = blockIdx.z;
  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  const int t = xcd_tile(blockIdx.x, tiles_m * tiles_n);
  if (t >= tiles_m * tiles_n) return;
  const int tm = t / tiles_n, tn = t - tm * tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kb = blockIdx.y * g.kchunk;
  // an upper-triangular B contributes nothing past the tile's last column; a
  // split left with an empty range still writes its (zero) partial
  const int ke = g.b_upper ? min(min(g.K, kb + g.kchunk), n0 + BN) : min(g.K, kb + g.kchunk);
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
    // The multiply phase runs at raised priority: the co-resident
    // workgroup's staging work then fills the issue slots between the MFMAs.
    // A fragments stay in registers for the whole stage; B fragments are
    // fetched one 16-column block at a time (wide wave tiles would not hold
    // them all).
    __builtin_amdgcn_s_setprio(1);
    bf16x8 a[TM][S];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int s = 0; s < S; ++s) a[i][s] = bfrag(As + s * BM * BLD, wm0 + i * 16, lane);
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      bf16x8 b[S];
#pragma unroll
      for (int s = 0; s < S; ++s) b[s] = bfrag(Bs + s * BN * BLD, wn0 + j * 16, lane);
      // piece products p + q <= S - 1 (0-based), smallest first
#pragma unroll
      for (int sum = S - 1; sum >= 0; --sum)
#pragma unroll
        for (int p = 0; p <= sum; ++p)
#pragma unroll
          for (int i = 0; i < TM; ++i) acc[i][j] = mfma_bf16(a[i][p], b[sum - p], acc[i][j]);
    }
    __builtin_amdgcn_s_setprio(0);
    __syncthreads();
  }

  // fp32 split partials, or the result (fp32, or fp64 for W64).  The
  // whole-tile test is uniform over the block, so the interior store loop is
  // free of per-element branches.
  auto put = [&](auto* C) {
    const int rb = m0 + wm0 + 4 * (lane >> 4), cb = n0 + wn0 + (lane & 15);
    if (m0 + BM <= g.M && n0 + BN <= g.N) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            C[static_cast<long long>(rb + i * 16 + v) * g.ldc + cb + j * 16] = acc[i][j][v];
    } else {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int row = rb + i * 16 + v, col = cb + j * 16;
            if (row < g.M && col < g.N) C[static_cast<long long>(row) * g.ldc + col] = acc[i][j][v];
          }
    }
  };
  if constexpr (W64) put(static_cast<double*>(g.C[layer]));
  else put(static_cast<float*>(g.C[layer]) + static_cast<long long>(blockIdx.y) * g.split_stride);
}

// bf16 planes of an fp32 matrix (rows x r): plane s holds the s-th split piece,
// row stride rp (r rounded up to 32, padding zero-filled).
__global__ __launch_bounds__(256) void k_split_planes(PlaneArgs a) {
  if (skip_launch(a.run_if)) return;
  const int l = blockIdx.y;
  const long long quads = static_cast<long long>(a.rows) * (a.rp / 4);
  const long long plane = static_cast<long long>(a.rows) * a.rp;
  const float* src = a.src[l];
  __bf16* dst = a.dst[l];
  for (long long q = blockIdx.x * 256LL + threadIdx.x; q < quads; q += 256LL * gridDim.x) {
    const long long row = q / (a.rp / 4);
    const int k = static_cast<int>(q - row * (a.rp / 4)) * 4;
    float v[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) v[c] = (k + c < a.r) ? src[row * a.r + k + c] : 0.0f;
    __bf16 pc[4][3];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      float rest = v[c];
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        pc[c][s] = static_cast<__bf16>(rest);
        rest -= static_cast<float>(pc[c][s]);
      }
    }
    for (int s = 0; s < a.S; ++s) {
      bf16x4 w = {pc[0][s], pc[1][s], pc[2][s], pc[3][s]};
      *reinterpret_cast<bf16x4*>(dst + s * plane + row * a.rp + k) = w;
    }
  }
}

// M = B - (1 - mu) P R^T and X -= c P Q^T on a 128 x BN tile of the m x n
// matrices; K = r.  P, R, Q come as bf16 planes (k_split_planes), so a stage
// is plain 16-byte loads into LDS; the XCD-aware grouped tile order keeps the
// P, R and Q slices of the tiles in flight on one XCD inside its L2.
constexpr int UBM = 128;
typedef float nt4 __attribute__((ext_vector_type(4)));

// G elements for the reversal of a speculative skip update: fp32, or bf16
// widened exactly.
__device__ __forceinline__ float4 load_g4(const void* G, bool bf, long long i) {
  if (bf) {
    const uint2 v = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(G) + i);
    return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                       __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
  }
  return *reinterpret_cast<const float4*>(static_cast<const float*>(G) + i);
}

__device__ __forceinline__ float load_g1(const void* G, bool bf, long long i) {
  if (bf) return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(G)[i]) << 16);
  return static_cast<const float*>(G)[i];
}

template <int S, int BN>
__global__ __launch_bounds__(256, 4) void k_update_pl(UpdatePlArgs u) {
  constexpr int TM = 4, TN = BN / 32;   // wave tile 64 x BN/2
  constexpr int PLANE_BYTES = S * (UBM + 2 * BN) * BLD64 * 2;
  constexpr int SLD = BN + 4;           // padded row of the fp32 accumulator staging tile
  constexpr int STAGE_BYTES = UBM * SLD * 4;
  constexpr int SMEM = PLANE_BYTES > STAGE_BYTES ? PLANE_BYTES : STAGE_BYTES;
  constexpr int ROWS = UBM + 2 * BN;    // LDS rows per plane: P, then R, then Q
  // the R and Q regions start at multiples of 4 rows, so the swizzle of
  // lds_off64 agrees between plane rows (stores) and region rows (bfrag64)
  static_assert(UBM % 4 == 0 && BN % 4 == 0, "region offsets must be multiples of 4 rows");
  constexpr int CHUNKS = S * ROWS * (BK16 / 8);   // 16-byte chunks per stage
  constexpr int CPT = CHUNKS / 256;
  static_assert(CHUNKS % 256 == 0, "whole chunks per thread");
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  if (u.ctl != nullptr && u.ctl->flag == 0) return;   // not a sync step
  __bf16* Ls = reinterpret_cast<__bf16*>(smem);   // [S][ROWS][BLD64]
  const int l = blockIdx.z;
  const int tiles_n = (u.n + BN - 1) / BN;
  const int tiles_m = (u.m + UBM - 1) / UBM;
  const int ntiles = tiles_m * tiles_n;
  const int t = xcd_tile(blockIdx.x, ntiles);
  if (t >= ntiles) return;
  // bands of 16 tile rows, columns advancing inside a band: the tiles one XCD
  // holds at a time share 16 P slices and a few R/Q slices, which stay in its
  // L2 (half the fetched bytes of row-major order, and 6% less time)
  int tm, tn;
  grouped_tile(t, tiles_m, tiles_n, 16, tm, tn);
  const int m0 = tm * UBM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 64, wn0 = (wave & 1) * (BN / 2);
  const long long pP = static_cast<long long>(u.m) * u.rp, pN = static_cast<long long>(u.n) * u.rp;

  // The thread's chunks: chunk i is row (tid / 4) + 64 (i % 4) of the stage's
  // rows [P | R | Q] in plane i / 4, 8 k values from 8 (tid % 4).  Its source
  // is a base that is uniform over the workgroup plus a 32-bit byte offset
  // (rows past m (P) or n (R, Q) read the last row instead: they only reach
  // outputs past the matrix, which are not written); its LDS slot is one
  // per-thread offset plus a constant.
  static_assert(ROWS == 256, "four 64-row groups per plane");
  const int crow = tid >> 2, kg = (tid & 3) * 8;
  const char* bp[CPT];
  unsigned off[CPT];
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int s = i / 4, row = crow + 64 * (i % 4);
    const __bf16* base;
    int grow;
    if (row < UBM) { base = u.P[l] + s * pP; grow = min(m0 + row, u.m - 1); }
    else if (row < UBM + BN) { base = u.R[l] + s * pN; grow = min(n0 + row - UBM, u.n - 1); }
    else { base = u.Q[l] + s * pN; grow = min(n0 + row - UBM - BN, u.n - 1); }
    bp[i] = reinterpret_cast<const char*>(base);
    off[i] = static_cast<unsigned>((grow * u.rp + kg) * 2);
  }
  const int slot0 = lds_off64(crow, kg);   // + (s * ROWS + 64 (i % 4)) * BLD64 for chunk i
  // native vectors (the HIP uint4 struct would keep the array in scratch memory)
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  u32x4 pre[CPT];
  f32x4 am[TM][TN], ax[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) { am[i][j] = f32x4{}; ax[i][j] = f32x4{}; }

#pragma unroll
  for (int i = 0; i < CPT; ++i) pre[i] = *reinterpret_cast<const u32x4*>(bp[i] + off[i]);
  for (int k0 = 0; k0 < u.rp; k0 += BK16) {
#pragma unroll
    for (int i = 0; i < CPT; ++i)
      *reinterpret_cast<u32x4*>(Ls + slot0 + ((i / 4) * ROWS + 64 * (i % 4)) * BLD64) = pre[i];
    __syncthreads();
    if (k0 + BK16 < u.rp) {
      const unsigned kb = static_cast<unsigned>((k0 + BK16) * 2);
#pragma unroll
      for (int i = 0; i < CPT; ++i) pre[i] = *reinterpret_cast<const u32x4*>(bp[i] + off[i] + kb);
    }
#pragma unroll
    for (int sum = S - 1; sum >= 0; --sum)
#pragma unroll
      for (int p = 0; p <= sum; ++p) {
        const __bf16* Pp = Ls + p * ROWS * BLD64;
        const __bf16* Rq = Ls + ((sum - p) * ROWS + UBM) * BLD64;
        const __bf16* Qq = Rq + BN * BLD64;
        bf16x8 a[TM];
#pragma unroll
        for (int i = 0; i < TM; ++i) a[i] = bfrag64(Pp, wm0 + i * 16, lane);
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const bf16x8 rb = bfrag64(Rq, wn0 + j * 16, lane);
          const bf16x8 qb = bfrag64(Qq, wn0 + j * 16, lane);
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            am[i][j] = mfma_bf16(a[i], rb, am[i][j]);
            ax[i][j] = mfma_bf16(a[i], qb, ax[i][j]);
          }
        }
      }
    __syncthreads();
  }

  // Epilogue through LDS so that M and X are read and written as contiguous
  // 16-byte row segments: M += -(1 - mu) (P R^T), then X += -c (P Q^T).
  float* st = reinterpret_cast<float*>(smem);
  const bool vec = (u.n & 3) == 0;
  auto dump = [&](const f32x4 (&acc)[TM][TN]) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          st[(wm0 + i * 16 + 4 * (lane >> 4) + v) * SLD + wn0 + j * 16 + (lane & 15)] = acc[i][j][v];
  };
  if (vec && m0 + UBM <= u.m && n0 + BN <= u.n && u.n < (1 << 23)) {
    // Interior tile.  Every load a thread makes (its 8 row segments of M, then
    // of X) is issued before the first store: a store to M may alias a later
    // load as far as the compiler knows, so a load-modify-store loop would
    // keep one 16-byte request per thread in flight and leave the epilogue
    // bound by memory latency.
    constexpr int SEGS = BN / 4;                  // 16-byte segments per tile row
    constexpr int PER = UBM * SEGS / 256;         // per thread and matrix
    constexpr int RSTEP = 256 / SEGS;             // tile rows between a thread's segments
    const int row0 = tid / SEGS, c4 = (tid % SEGS) * 4;
    // tile base (uniform) plus a 32-bit element offset per segment: 128 rows
    // of any layer this library accepts stay far below 2^31 elements
    const long long tile0 = static_cast<long long>(__builtin_amdgcn_readfirstlane(m0)) * u.n +
                            __builtin_amdgcn_readfirstlane(n0);
    char* const Mt = reinterpret_cast<char*>(u.M[l] + tile0);
    char* const Xt = reinterpret_cast<char*>(u.X[l] + tile0);
    unsigned o[PER];   // byte offsets (under 2^32: 128 rows of at most 2^23 columns)
#pragma unroll
    for (int i = 0; i < PER; ++i) o[i] = static_cast<unsigned>((row0 + i * RSTEP) * u.n + c4) * 4u;
    const float* const sr = st + row0 * SLD + c4;
    nt4 w[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) w[i] = __builtin_nontemporal_load(reinterpret_cast<const nt4*>(Mt + o[i]));
    dump(am);
    __syncthreads();
    nt4 x[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) x[i] = __builtin_nontemporal_load(reinterpret_cast<const nt4*>(Xt + o[i]));
    const float cm = -u.one_minus_mu;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const float4 a = *reinterpret_cast<const float4*>(sr + i * RSTEP * SLD);
      nt4 v = w[i];
      v.x = fmaf(cm, a.x, v.x); v.y = fmaf(cm, a.y, v.y);
      v.z = fmaf(cm, a.z, v.z); v.w = fmaf(cm, a.w, v.w);
      __builtin_nontemporal_store(v, reinterpret_cast<nt4*>(Mt + o[i]));
    }
    // X: first undo a speculative skip-branch update (X += gc G; that update
    // already applied the weight decay), else apply the decay
    const bool spec = (u.spec == 2 ? u.ctl->spec_cur : u.spec) != 0;
    const float gc = spec ? u.gc[l] : 0.f;
    if (gc != 0.f) {
      const void* const G = u.G[l];
      const bool gbf = u.g_bf16 != 0;
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const float4 g = load_g4(G, gbf, tile0 + o[i] / 4);
        x[i].x = fmaf(gc, g.x, x[i].x); x[i].y = fmaf(gc, g.y, x[i].y);
        x[i].z = fmaf(gc, g.z, x[i].z); x[i].w = fmaf(gc, g.w, x[i].w);
      }
    } else if (!spec) {
      const float xd = u.xdecay[l];
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        x[i].x *= xd; x[i].y *= xd; x[i].z *= xd; x[i].w *= xd;
      }
    }
    __syncthreads();
    dump(ax);
    __syncthreads();
    const float cx = -u.c;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const float4 a = *reinterpret_cast<const float4*>(sr + i * RSTEP * SLD);
      nt4 v = x[i];
      v.x = fmaf(cx, a.x, v.x); v.y = fmaf(cx, a.y, v.y);
      v.z = fmaf(cx, a.z, v.z); v.w = fmaf(cx, a.w, v.w);
      __builtin_nontemporal_store(v, reinterpret_cast<nt4*>(Xt + o[i]));
    }
    return;
  }
#pragma unroll
  for (int which = 0; which < 2; ++which) {
    dump(which == 0 ? am : ax);
    __syncthreads();
    float* Y = which == 0 ? u.M[l] : u.X[l];
    const float coef = which == 0 ? -u.one_minus_mu : -u.c;
    // X only: first undo a speculative skip-branch update (X += gc G; that
    // update already applied the weight decay), else apply the decay
    const bool spec = which == 1 && (u.spec == 2 ? u.ctl->spec_cur : u.spec) != 0;
    const float gc = spec ? u.gc[l] : 0.f;
    const float xd = (which == 0 || spec) ? 1.f : u.xdecay[l];
    const void* const G = u.G[l];
    const bool gbf = u.g_bf16 != 0;
#pragma unroll 4
    for (int e = tid; e < UBM * (BN / 4); e += 256) {
      const int row = e / (BN / 4), c4 = (e % (BN / 4)) * 4;
      const int grow = m0 + row, gcol = n0 + c4;
      if (grow >= u.m) continue;
      const float4 a = *reinterpret_cast<const float4*>(st + row * SLD + c4);
      const long long off = static_cast<long long>(grow) * u.n + gcol;
      float* y = Y + off;
      if (vec && gcol + 3 < u.n) {
        // non-temporal: M and X are touched once; the P/R/Q slices should keep L2
        const nt4 wv = __builtin_nontemporal_load(reinterpret_cast<const nt4*>(y));
        float4 w = make_float4(wv.x, wv.y, wv.z, wv.w);
        if (gc != 0.f) {
          const float4 g = load_g4(G, gbf, off);
          w.x = fmaf(gc, g.x, w.x); w.y = fmaf(gc, g.y, w.y);
          w.z = fmaf(gc, g.z, w.z); w.w = fmaf(gc, g.w, w.w);
        } else if (!spec) {
          w.x *= xd; w.y *= xd; w.z *= xd; w.w *= xd;
        }
        w.x = fmaf(coef, a.x, w.x); w.y = fmaf(coef, a.y, w.y);
        w.z = fmaf(coef, a.z, w.z); w.w = fmaf(coef, a.w, w.w);
        const nt4 ov = {w.x, w.y, w.z, w.w};
        __builtin_nontemporal_store(ov, reinterpret_cast<nt4*>(y));
      } else {
        const float av[4] = {a.x, a.y, a.z, a.w};
        for (int c = 0; c < 4; ++c) {
          if (gcol + c >= u.n) continue;
          float w = y[c];
          if (gc != 0.f) w = fmaf(gc, load_g1(G, gbf, off + c), w);
          else if (!spec) w *= xd;
          y[c] = fmaf(coef, av[c], w);
        }
      }
    }
    __syncthreads();
  }
}

template <int S, int BM, int BN>
hipError_t launch_bm(const GemmArgs& g, int nl, hipStream_t s) {
  const int tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  const dim3 grid(xcd_grid(tiles), g.splits, nl);
  if (g.out64 && g.splits == 1) {
    // fp64 results are only asked of the three-piece Gram (both operands
    // transposed); other combinations are refused
    if constexpr (S == 3) {
      if (!g.a_kc && !g.b_kc) {
        hipLaunchKernelGGL((k_gemm_bf<S, BM, BN, false, false, true>), grid, dim3(256), 0, s, g);
        return hipGetLastError();
      }
    }
    return hipErrorInvalidValue;
  }
  if (g.a_kc && !g.b_kc) hipLaunchKernelGGL((k_gemm_bf<S, BM, BN, true, false, false>), grid, dim3(256), 0, s, g);
  else if (!g.a_kc && !g.b_kc) hipLaunchKernelGGL((k_gemm_bf<S, BM, BN, false, false, false>), grid, dim3(256), 0, s, g);
  else if (g.a_kc && g.b_kc) hipLaunchKernelGGL((k_gemm_bf<S, BM, BN, true, true, false>), grid, dim3(256), 0, s, g);
  else hipLaunchKernelGGL((k_gemm_bf<S, BM, BN, false, true, false>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

template <int S>
hipError_t launch_s(const GemmArgs& g, int nl, hipStream_t s) {
  // 128 x 256 tiles (64 x 128 per wave) read a quarter less LDS per MFMA and
  // half as many copies of the A operand; three-piece splits keep 128 x 128
  if constexpr (S <= 2) {
    if (g.N >= 256) return launch_bm<S, 128, 256>(g, nl, s);
  }
  if (g.N > 64) return launch_bm<S, 128, 128>(g, nl, s);
  if (g.N > 32) return launch_bm<S, 128, 64>(g, nl, s);
  return launch_bm<S, 128, 32>(g, nl, s);
}

}  // namespace

int gemm_bf_bm(int N) { (void)N; return 128; }
int gemm_bf_bn(int N, int pieces) {
  if (pieces <= 2 && N >= 256) return 256;
  return N > 64 ? 128 : (N > 32 ? 64 : 32);
}

hipError_t launch_gemm_bf(const GemmArgs& g, int nl, int pieces, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  if (pieces == 3) return launch_s<3>(g, nl, s);
  if (pieces == 2) return launch_s<2>(g, nl, s);
  return launch_s<1>(g, nl, s);
}

hipError_t launch_split_planes(const PlaneArgs& a, int nl, hipStream_t s) {
  if (nl <= 0 || a.rows <= 0) return hipSuccess;
  long long quads = static_cast<long long>(a.rows) * (a.rp / 4);
  long long blocks = (quads + 255) / 256;
  if (blocks > 2048) blocks = 2048;
  hipLaunchKernelGGL(k_split_planes, dim3(static_cast<unsigned>(blocks), nl), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_update_planes(const UpdatePlArgs& u, int nl, int pieces, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  if (pieces == 3) {
    const int tiles = ((u.m + UBM - 1) / UBM) * ((u.n + 63) / 64);
    hipLaunchKernelGGL((k_update_pl<3, 64>), dim3(xcd_grid(tiles), 1, nl), dim3(256), 0, s, u);
  } else {
    // 128 x 64 tiles: the LDS staging of the epilogue (35 KB) leaves room for
    // more resident workgroups than 128 x 128 tiles
    const int tiles = ((u.m + UBM - 1) / UBM) * ((u.n + 63) / 64);
    hipLaunchKernelGGL((k_update_pl<1, 64>), dim3(xcd_grid(tiles), 1, nl), dim3(256), 0, s, u);
  }
  return hipGetLastError();
}

}  // namespace cd
