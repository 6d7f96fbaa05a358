// B = M + G fused into P~ = B Q (see form_bq.hpp), bf16 gradients, r in
// (256, 512]: a workgroup of eight waves owns a 128-row band of B and every
// column of P~ within one K slice, so each element of B is formed, written
// over M and squared by exactly one workgroup (no other one reads that M
// element).  The product itself is the two-piece split of k_gemm_bf (three
// bf16 MFMA products, fp32 accumulation): waves as 2 x 4, 64 x 128 each;
// the next stage's operands prefetched into registers while the current one
// is multiplied.  The block's sum of B^2 (fp64, each thread's elements in
// stage order, then a fixed-order tree) goes to part[tile row * splits +
// split], which the gate adds in index order.
#include "bf16_split.hpp"
#include "common.hpp"
#include "form_bq.hpp"

namespace cd {
namespace {

constexpr int FB_NT = 512;
constexpr int FB_BN = FBQ_RMAX;

typedef unsigned fb_u2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float4 widen4(fb_u2 u) {
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
}
__device__ __forceinline__ float bf1(const __bf16* g, long long i) {
  return __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(g)[i]) << 16);
}

template <int S>
__global__ __launch_bounds__(FB_NT, 1) void k_form_bq(FormBqArgs g) {
  constexpr int WN_WAVES = 4, WM_WAVES = 2;
  constexpr int WM = FBQ_BM / WM_WAVES, WN = FB_BN / WN_WAVES;   // 64 x 128
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int A_PER = FBQ_BM * (BK16 / 4) / FB_NT;            // float4 slots of A per thread
  static_assert(A_PER * FB_NT == FBQ_BM * (BK16 / 4), "A slots must divide evenly");
  __shared__ __attribute__((aligned(16))) __bf16 As[S * FBQ_BM * BLD];
  __shared__ __attribute__((aligned(16))) __bf16 Bs[S * FB_BN * BLD];
  __shared__ double wsum[FB_NT / 64];

  const int layer = blockIdx.z;
  const int tiles_m = (g.m + FBQ_BM - 1) / FBQ_BM;
  const int tm = xcd_tile(blockIdx.x, tiles_m);
  if (tm >= tiles_m) return;
  const int m0 = tm * FBQ_BM;
  const int kb = blockIdx.y * g.kchunk;
  const int ke = min(g.n, kb + g.kchunk);
  float* const M = g.M[layer];
  const __bf16* const G = g.G[layer];
  const float* const Q = g.Q[layer];
  const int n = g.n;
  const bool vec = (n & 3) == 0;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / WN_WAVES) * WM, wn0 = (wave % WN_WAVES) * WN;

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{};

  // A operand: B = M + G, formed at load time; slot (row, 4 k) per float4
  float4 bv[A_PER];
  double ss = 0.0;
  auto slot_rk = [&](int i, int& row, int& kq) {
    const int slot = tid + i * FB_NT;
    row = slot / (BK16 / 4);
    kq = (slot % (BK16 / 4)) * 4;
  };
  auto load_a = [&](int k0) {
    const bool interior = vec && m0 + FBQ_BM <= g.m && k0 + BK16 <= ke;
#pragma unroll
    for (int i = 0; i < A_PER; ++i) {
      int row, kq;
      slot_rk(i, row, kq);
      const long long o = static_cast<long long>(m0 + row) * n + k0 + kq;
      if (interior) {
        const float4 mv = *reinterpret_cast<const float4*>(M + o);
        const float4 gv = widen4(*reinterpret_cast<const fb_u2*>(G + o));
        bv[i] = make_float4(mv.x + gv.x, mv.y + gv.y, mv.z + gv.z, mv.w + gv.w);
      } else {
        float e[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const bool in = m0 + row < g.m && k0 + kq + c < ke;
          e[c] = in ? M[o + c] + bf1(G, o + c) : 0.0f;
        }
        bv[i] = make_float4(e[0], e[1], e[2], e[3]);
      }
    }
  };
  // B back over M, its squares, and its split pieces into LDS
  auto store_a = [&](int k0) {
    const bool interior = vec && m0 + FBQ_BM <= g.m && k0 + BK16 <= ke;
#pragma unroll
    for (int i = 0; i < A_PER; ++i) {
      int row, kq;
      slot_rk(i, row, kq);
      const long long o = static_cast<long long>(m0 + row) * n + k0 + kq;
      const float4 b = bv[i];
      if (interior) {
        *reinterpret_cast<float4*>(M + o) = b;
      } else {
        const float e[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
        for (int c = 0; c < 4; ++c)
          if (m0 + row < g.m && k0 + kq + c < ke) M[o + c] = e[c];
      }
      // elements outside the matrix are zero and add nothing
      ss += static_cast<double>(b.x) * b.x;
      ss += static_cast<double>(b.y) * b.y;
      ss += static_cast<double>(b.z) * b.z;
      ss += static_cast<double>(b.w) * b.w;
      put4<S, FBQ_BM>(As, row, kq, b.x, b.y, b.z, b.w);
    }
  };

  Stage<FB_BN, FB_NT> sb;
  if (kb < ke) {
    load_a(kb);
    sb.load(Q, g.r, false, 0, g.r, kb, ke, tid);
  }
  for (int k0 = kb; k0 < ke; k0 += BK16) {
    store_a(k0);
    sb.template store<S>(Bs, false, tid);
    __syncthreads();
    if (k0 + BK16 < ke) {
      load_a(k0 + BK16);
      sb.load(Q, g.r, false, 0, g.r, k0 + BK16, ke, tid);
    }
    bf16x8 a[TM][S];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int s = 0; s < S; ++s) a[i][s] = bfrag(As + s * FBQ_BM * BLD, wm0 + i * 16, lane);
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      bf16x8 b[S];
#pragma unroll
      for (int s = 0; s < S; ++s) b[s] = bfrag(Bs + s * FB_BN * BLD, wn0 + j * 16, lane);
      // piece products p + q <= S - 1 (0-based), smallest first
#pragma unroll
      for (int sum = S - 1; sum >= 0; --sum)
#pragma unroll
        for (int p = 0; p <= sum; ++p)
#pragma unroll
          for (int i = 0; i < TM; ++i) acc[i][j] = mfma_bf16(a[i][p], b[sum - p], acc[i][j]);
    }
    __syncthreads();
  }

  // P~ (one slice) or this slice's fp32 partial
  float* const C = g.C[layer] + static_cast<long long>(blockIdx.y) * g.split_stride;
  const int rb = m0 + wm0 + 4 * (lane >> 4), cb = wn0 + (lane & 15);
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = rb + i * 16 + v, col = cb + j * 16;
        if (row < g.m && col < g.r) C[static_cast<long long>(row) * g.r + col] = acc[i][j][v];
      }

  // the block's sum of B^2 in a fixed order
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  if (lane == 0) wsum[wave] = ss;
  __syncthreads();
  if (tid == 0) {
    double t = 0.0;
#pragma unroll
    for (int w = 0; w < FB_NT / 64; ++w) t += wsum[w];
    g.part[layer][tm * g.splits + blockIdx.y] = t;
  }
}

}  // namespace

hipError_t launch_form_bq(const FormBqArgs& a, int nl, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  if (nl > MAXB || a.r < FBQ_RMIN || a.r > FBQ_RMAX || a.m < 1 || a.n < 1 || a.splits < 1 ||
      a.kchunk % BK16 != 0 || static_cast<long long>(a.splits) * a.kchunk < a.n ||
      static_cast<long long>(a.splits - 1) * a.kchunk >= a.n)
    return hipErrorInvalidValue;
  const int tiles_m = (a.m + FBQ_BM - 1) / FBQ_BM;
  const dim3 grid(xcd_grid(tiles_m), a.splits, nl);
  hipLaunchKernelGGL(k_form_bq<2>, grid, dim3(FB_NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace cd
