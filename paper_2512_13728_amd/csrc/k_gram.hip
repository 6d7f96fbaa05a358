// The pass-0 Gram matrix W = P~^T P~ of CholQR (Orthogonalize of Algorithm 1 /
// Algorithm 2) for an fp32 panel P~ (m x r), on the bf16 MFMA, exact up to a
// truncation of P~ at 2^-25 of the largest entry of each column in each
// 128-row chunk, and the final fp64 additions.
//
// Why: P~ = B Q is ill-conditioned (kappa up to ~1e6 in these workloads), so
// W must be the Gram matrix of (a matrix within fp32 rounding of) P~ to about
// fp64 accuracy, or the Cholesky factor breaks down.  A product of two bf16
// values is exact in fp32, and a sum of such products is exact as long as
// every term lies on one grid and the total stays below 2^24 grid units.  So
// in every chunk c of GX_CHUNK rows each column j of P~ is scaled by
// 2^-e (e = e_cj: the chunk's largest magnitude in the column is below 2^e)
// and cut into three fixed-point slices,
//     x 2^-e = a1 + a2 + a3 (+ a remainder below 2^-25),
//     a_s an integer multiple of 2^-8s with |a_s / 2^-8s| <= 256,
// each exactly a bf16 value (k_slice, once per element, into bf16 planes with
// the rows of a column contiguous).  The product of slices s and t lies on the
// grid 2^-8(s+t); k_gram_x accumulates the nine slice products of a chunk in
// five fp32 groups by s + t (one grid per group), which keeps every group's
// sum below 2^24 of its grid units, hence exact, and then adds the groups,
// scaled by 2^(e_ci + e_cj), to an fp64 accumulator.  The result is the fp64
// Gram matrix of P~' = P~ + E with |E_kj| <= 2^-25 max over the chunk of
// |P~_.j|: positive semidefinite by construction, so the Cholesky factor T
// exists; CholQR then forms P1 = P~ T^-1 from P~ itself, which keeps
// span(P1) = span(P~) exactly and only moves P1 away from orthonormal by
// about |E| / sigma_min(P~), which the second pass removes.
//
// Tiles of 64 x 64 (upper tiles only), four waves of 32 x 32 on
// v_mfma_f32_32x32x16_bf16; K (the rows of P~) split over blockIdx.y in
// multiples of GX_CHUNK into fp64 partials that launch_reduce_splits adds in
// a fixed order.
#include "bf16_split.hpp"
#include "common.hpp"

namespace cd {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

// e with mx < 2^e (0 for a zero or non-finite maximum: no scaling).
__device__ __forceinline__ int col_exponent(float mx) {
  if (!(mx > 0.f) || !(mx < INFINITY)) return 0;
  int e;
  (void)frexpf(mx, &e);   // mx = f 2^e, f in [0.5, 1)
  return e;
}

// Slices of x (|x| < 1 after scaling; NaN and Inf propagate as NaN).
__device__ __forceinline__ void slice3(float x, __bf16& p1, __bf16& p2, __bf16& p3) {
  const float a1 = rintf(x * 256.0f) * (1.0f / 256.0f);
  const float r1 = x - a1;
  const float a2 = rintf(r1 * 65536.0f) * (1.0f / 65536.0f);
  const float r2 = r1 - a2;
  const float a3 = rintf(r2 * 16777216.0f) * (1.0f / 16777216.0f);
  p1 = static_cast<__bf16>(a1);
  p2 = static_cast<__bf16>(a2);
  p3 = static_cast<__bf16>(a3);
}

// One workgroup per (64 columns, GX_CHUNK rows) of one layer: the chunk's
// column exponents and the three slice planes, written column-major (rows
// of a column contiguous), rows past m as zeros.  A thread holds eight
// consecutive rows of four columns, so each of its slice runs is one
// 16-byte store.
__global__ __launch_bounds__(256) void k_slice(GramXArgs a) {
  __shared__ float red[GX_CHUNK / 8][64];
  __shared__ int es[64];
  if (skip_launch(a.run_if)) return;
  const int l = blockIdx.z, chunk = blockIdx.y;
  const int j0 = blockIdx.x * 64, k0 = chunk * GX_CHUNK;
  const float* P = a.P[l];
  const int tid = threadIdx.x;
  const int cq = (tid & 15) * 4, rb = (tid >> 4) * 8;   // columns cq.., rows rb .. rb + 7
  const bool vec = (a.r & 3) == 0 && j0 + cq + 3 < a.r;
  float v[8][4];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int k = k0 + rb + u;
    if (k < a.m && vec) {
      const float4 f = *reinterpret_cast<const float4*>(P + static_cast<long long>(k) * a.r + j0 + cq);
      v[u][0] = f.x; v[u][1] = f.y; v[u][2] = f.z; v[u][3] = f.w;
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c)
        v[u][c] = (k < a.m && j0 + cq + c < a.r) ? P[static_cast<long long>(k) * a.r + j0 + cq + c] : 0.0f;
    }
  }
  // column maxima over the chunk: per thread, then over the 16 row blocks
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    float mx = 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) mx = fmaxf(mx, fabsf(v[u][c]));
    red[rb / 8][cq + c] = mx;
  }
  __syncthreads();
  if (tid < 64) {
    float mx = 0.f;
#pragma unroll
    for (int g = 0; g < GX_CHUNK / 8; ++g) mx = fmaxf(mx, red[g][tid]);
    const int e = col_exponent(mx);
    es[tid] = e;
    if (j0 + tid < a.r) a.E[l][static_cast<long long>(chunk) * a.r + j0 + tid] = e;
  }
  __syncthreads();
  const long long plane = static_cast<long long>(a.r) * a.mp;
  __bf16* S = a.S[l];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    if (j0 + cq + c >= a.r) break;
    const float sc = ldexpf(1.0f, -es[cq + c]);
    bf16x8 w1, w2, w3;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      __bf16 x1, x2, x3;
      slice3(v[u][c] * sc, x1, x2, x3);
      w1[u] = x1; w2[u] = x2; w3[u] = x3;
    }
    __bf16* d = S + static_cast<long long>(j0 + cq + c) * a.mp + k0 + rb;
    *reinterpret_cast<bf16x8*>(d) = w1;
    *reinterpret_cast<bf16x8*>(d + plane) = w2;
    *reinterpret_cast<bf16x8*>(d + 2 * plane) = w3;
  }
}

// 32-row fragment of a 32x32x16 MFMA: lane l owns row (l % 32) and
// k = 16 h + 8 (l / 32) .. + 7.
__device__ __forceinline__ bf16x8 frag32(const __bf16* plane, int row0, int h, int lane) {
  return *reinterpret_cast<const bf16x8*>(plane + lds_off64(row0 + (lane & 31), 16 * h + 8 * (lane >> 5)));
}

__global__ __launch_bounds__(256, 2) void k_gram_x(GramXArgs a) {
  // LDS: [operand A|B][slice][64 rows][32 k], rows as lds_off64 lays them out
  // (a staging store and a fragment read each cover the 64 banks once)
  __shared__ __attribute__((aligned(16))) __bf16 Ls[2 * 3 * 64 * BK16];
  __shared__ int es[2][64];
  if (skip_launch(a.run_if)) return;
  const int l = blockIdx.z;
  const int tiles = (a.r + 63) / 64;
  const int t = xcd_tile(blockIdx.x, tiles * tiles);
  if (t >= tiles * tiles) return;
  const int ti = t / tiles, tj = t - ti * tiles;
  if (ti > tj) return;   // upper tiles only
  const int i0 = ti * 64, j0 = tj * 64;
  const int kb = blockIdx.y * a.kchunk, ke = min(a.mp, kb + a.kchunk);
  const int* E = a.E[l];
  const long long plane = static_cast<long long>(a.r) * a.mp;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 32, wn0 = (wave & 1) * 32;

  // Staging: 2 operands x 3 slices x 64 columns x 4 pieces of 8 rows = 1536
  // 16-byte pieces per stage, six per thread.  Piece u of a thread belongs
  // to operand u / 3 and slice u % 3 (uniform over the workgroup), column
  // c = tid / 4 and rows 8 (tid % 4) ..; its source is a uniform base plus a
  // 32-bit byte offset that advances by one stage per step.  Columns past r
  // read column r - 1 instead: they only reach outputs past r, which are
  // not written.
  const int c = tid >> 2, pc = tid & 3;
  const char* base[6];
  unsigned off[2];
#pragma unroll
  for (int o = 0; o < 2; ++o) {
    const int col = min((o == 0 ? i0 : j0) + c, a.r - 1);
    off[o] = static_cast<unsigned>((static_cast<long long>(col) * a.mp + kb + pc * 8) * 2);
  }
#pragma unroll
  for (int u = 0; u < 6; ++u) base[u] = reinterpret_cast<const char*>(a.S[l] + (u % 3) * plane);
  const int soff = lds_off64(c, pc * 8);
  uint4 p0, p1, p2, p3, p4, p5;   // the next stage's pieces
#define GX_LOAD(step)                                                                                     \
  do {                                                                                                    \
    const unsigned so = static_cast<unsigned>((step) * (BK16 * 2));                                       \
    p0 = *reinterpret_cast<const uint4*>(base[0] + off[0] + so);                                          \
    p1 = *reinterpret_cast<const uint4*>(base[1] + off[0] + so);                                          \
    p2 = *reinterpret_cast<const uint4*>(base[2] + off[0] + so);                                          \
    p3 = *reinterpret_cast<const uint4*>(base[3] + off[1] + so);                                          \
    p4 = *reinterpret_cast<const uint4*>(base[4] + off[1] + so);                                          \
    p5 = *reinterpret_cast<const uint4*>(base[5] + off[1] + so);                                          \
  } while (0)
  f32x16 acc[5];
  double acc64[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) acc64[e] = 0.0;
  // lane l, element e: row 8 (e / 4) + 4 (l / 32) + e % 4, column l % 32
  const int col = wn0 + (lane & 31);
  const __bf16* As = Ls;
  const __bf16* Bs = Ls + 3 * 64 * BK16;
  const int nst = (ke - kb) / BK16;   // stages; a multiple of GX_CHUNK / BK16
  if (nst > 0) GX_LOAD(0);
  for (int st = 0; st < nst; ++st) {
    const int sub = st % (GX_CHUNK / BK16);
    if (sub == 0 && tid < 128) {
      // the chunk's exponents (every wave has flushed the previous chunk)
      const int o = tid >> 6, cc = (o == 0 ? i0 : j0) + (tid & 63);
      es[o][tid & 63] = cc < a.r ? E[static_cast<long long>((kb / BK16 + st) / (GX_CHUNK / BK16)) * a.r + cc] : 0;
    }
    *reinterpret_cast<uint4*>(Ls + 0 * 64 * BK16 + soff) = p0;
    *reinterpret_cast<uint4*>(Ls + 1 * 64 * BK16 + soff) = p1;
    *reinterpret_cast<uint4*>(Ls + 2 * 64 * BK16 + soff) = p2;
    *reinterpret_cast<uint4*>(Ls + 3 * 64 * BK16 + soff) = p3;
    *reinterpret_cast<uint4*>(Ls + 4 * 64 * BK16 + soff) = p4;
    *reinterpret_cast<uint4*>(Ls + 5 * 64 * BK16 + soff) = p5;
    __syncthreads();
    if (st + 1 < nst) GX_LOAD(st + 1);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      bf16x8 fa[3], fb[3];
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        fa[s] = frag32(As + s * 64 * BK16, wm0, h, lane);
        fb[s] = frag32(Bs + s * 64 * BK16, wn0, h, lane);
      }
      // products grouped by s + u; a chunk's first product of each group
      // starts from zero, the three of group 2 are spread out
      if (sub == 0 && h == 0) {
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0], fb[0], f32x16{}, 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0], fb[1], f32x16{}, 0, 0, 0);
        acc[2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0], fb[2], f32x16{}, 0, 0, 0);
        acc[3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1], fb[2], f32x16{}, 0, 0, 0);
        acc[4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[2], fb[2], f32x16{}, 0, 0, 0);
      } else {
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0], fb[0], acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0], fb[1], acc[1], 0, 0, 0);
        acc[2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0], fb[2], acc[2], 0, 0, 0);
        acc[3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1], fb[2], acc[3], 0, 0, 0);
        acc[4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[2], fb[2], acc[4], 0, 0, 0);
      }
      acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1], fb[0], acc[1], 0, 0, 0);
      acc[2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1], fb[1], acc[2], 0, 0, 0);
      acc[3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[2], fb[1], acc[3], 0, 0, 0);
      acc[2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[2], fb[0], acc[2], 0, 0, 0);
    }
    if (sub == GX_CHUNK / BK16 - 1) {
      // the chunk's exact group sums, scaled, into fp64
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = wm0 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        double s = static_cast<double>(acc[4][e]);
#pragma unroll
        for (int d = 3; d >= 0; --d) s += static_cast<double>(acc[d][e]);
        acc64[e] += ldexp(s, es[0][row] + es[1][col]);
      }
    }
    __syncthreads();
  }

#undef GX_LOAD
  const bool partial = a.splits > 1;
  double* C = static_cast<double*>(a.C[l]) + (partial ? static_cast<long long>(blockIdx.y) * a.split_stride : 0);
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int row = wm0 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
    if (i0 + row < a.r && j0 + col < a.r) C[static_cast<long long>(i0 + row) * a.r + j0 + col] = acc64[e];
  }
}

}  // namespace

hipError_t launch_gram_x(const GramXArgs& a, int nl, hipStream_t s) {
  if (nl <= 0) return hipSuccess;
  if (a.kchunk % GX_CHUNK != 0 || a.mp % GX_CHUNK != 0 || a.mp < a.m) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_slice, dim3((a.r + 63) / 64, a.mp / GX_CHUNK, nl), dim3(256), 0, s, a);
  const int tiles = (a.r + 63) / 64;
  hipLaunchKernelGGL(k_gram_x, dim3(xcd_grid(tiles * tiles), a.splits, nl), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace cd
