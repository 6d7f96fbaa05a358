// Building blocks for the MFMA GEMM kernels (gfx950, wave64).
//
// Tiles are staged in LDS as [rows][LDK] with k contiguous, whatever the
// layout in global memory, so that every lane reads its MFMA operands with
// one 16-byte LDS load: for a 16-wide k slice, lane l of a 16x16x4 MFMA group
// owns row (l % 16) and k = 4 * (l / 16) + q for the q-th of four MFMAs.  A
// and B operands use the same k permutation, so the contraction is unchanged.
// With LDK = 36 (BK = 32 plus 4 pad) the 16 rows read by one b128 load fall on
// distinct bank groups.
#pragma once

#include <hip/hip_runtime.h>

#include "common.hpp"

namespace cd {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef double f64x4 __attribute__((ext_vector_type(4)));

constexpr int GLDK = GBK + 4;    // padded LDS row

template <typename T> struct Mfma;
// Output layout: lane l, accumulator register v holds D[out_row(l, v)][l % 16].
// (Measured on gfx950: fp32 16x16x4 packs four consecutive rows per lane
// group, fp64 16x16x4 interleaves them with stride 4.)
template <> struct Mfma<float> {
  typedef f32x4 acc_t;
  typedef f32x4 vec4_t;
  static __device__ __forceinline__ int out_row(int lane, int v) { return 4 * (lane >> 4) + v; }
  static __device__ __forceinline__ acc_t mma(float a, float b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};
template <> struct Mfma<double> {
  typedef f64x4 acc_t;
  typedef f64x4 vec4_t;
  static __device__ __forceinline__ int out_row(int lane, int v) { return (lane >> 4) + 4 * v; }
  static __device__ __forceinline__ acc_t mma(double a, double b, acc_t c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
  }
};

// Four consecutive elements of an fp32 or fp64 operand (16- or 32-byte load).
__device__ __forceinline__ void load4(const float* p, float& a, float& b, float& c, float& d) {
  const float4 f = *reinterpret_cast<const float4*>(p);
  a = f.x; b = f.y; c = f.z; d = f.w;
}
__device__ __forceinline__ void load4(const double* p, double& a, double& b, double& c, double& d) {
  const double2 f = *reinterpret_cast<const double2*>(p);
  const double2 g = *reinterpret_cast<const double2*>(p + 2);
  a = f.x; b = f.y; c = g.x; d = g.y;
}

// LDS tiles.  A k-contiguous operand (element (row, k) at src[row * ld + k]) is
// staged row-major, S[row][GLDK], and an operand of the other layout
// (element (row, k) at src[k * ld + row]) is staged k-major, S[k][ROWS + KPAD];
// either way the global loads and the LDS stores are 4-element vectors.
constexpr int KPAD = 4;
template <int ROWS>
constexpr int tile_elems() { return ROWS * GLDK > GBK * (ROWS + KPAD) ? ROWS * GLDK : GBK * (ROWS + KPAD); }

template <typename T>
__device__ __forceinline__ void store4(T* d, T a, T b, T c, T e) {
  d[0] = a; d[1] = b; d[2] = c; d[3] = e;
}

// Stage rows [r0, r0 + ROWS) x k in [k0, k0 + GBK) of an operand of element
// type TIn into S (type T), zero-filling rows >= nrows and k >= kend.  Vector
// loads need ld % 4 == 0 (and an aligned base).
template <typename T, typename TIn, int ROWS, int NT, bool KC>
__device__ __forceinline__ void stage_tile(T* __restrict__ S, const TIn* __restrict__ src, int ld,
                                           int r0, int nrows, int k0, int kend, int tid) {
  const bool vec = (ld & 3) == 0;
  if constexpr (KC) {
    constexpr int SLOTS = ROWS * (GBK / 4);
#pragma unroll
    for (int slot = tid; slot < SLOTS; slot += NT) {
      const int row = slot / (GBK / 4);
      const int kq = (slot % (GBK / 4)) * 4;
      const int gr = r0 + row, gk = k0 + kq;
      TIn v0 = 0, v1 = 0, v2 = 0, v3 = 0;
      if (gr < nrows) {
        const TIn* p = src + static_cast<long long>(gr) * ld + gk;
        if (vec && gk + 3 < kend) {
          load4(p, v0, v1, v2, v3);
        } else {
          if (gk + 0 < kend) v0 = p[0];
          if (gk + 1 < kend) v1 = p[1];
          if (gk + 2 < kend) v2 = p[2];
          if (gk + 3 < kend) v3 = p[3];
        }
      }
      store4<T>(S + row * GLDK + kq, v0, v1, v2, v3);
    }
  } else {
    constexpr int SLOTS = GBK * (ROWS / 4);
#pragma unroll
    for (int slot = tid; slot < SLOTS; slot += NT) {
      const int kk = slot / (ROWS / 4);
      const int rq = (slot % (ROWS / 4)) * 4;
      const int gr = r0 + rq, gk = k0 + kk;
      TIn v0 = 0, v1 = 0, v2 = 0, v3 = 0;
      if (gk < kend) {
        const TIn* p = src + static_cast<long long>(gk) * ld + gr;
        if (vec && gr + 3 < nrows) {
          load4(p, v0, v1, v2, v3);
        } else {
          if (gr + 0 < nrows) v0 = p[0];
          if (gr + 1 < nrows) v1 = p[1];
          if (gr + 2 < nrows) v2 = p[2];
          if (gr + 3 < nrows) v3 = p[3];
        }
      }
      store4<T>(S + kk * (ROWS + KPAD) + rq, v0, v1, v2, v3);
    }
  }
}

// The same staging split in two halves, so that the next stage's global loads
// are in flight while the current stage is multiplied: load() fills registers
// (same slot -> element mapping as stage_tile), store() writes them to LDS.
template <typename TIn, int ROWS, int NT, bool KC>
struct Prefetch {
  static constexpr int SLOTS = KC ? ROWS * (GBK / 4) : GBK * (ROWS / 4);
  static constexpr int PER = (SLOTS + NT - 1) / NT;
  TIn v[PER][4];

  __device__ __forceinline__ void load(const TIn* __restrict__ src, int ld, int r0, int nrows, int k0,
                                       int kend, int tid) {
    const bool vec = (ld & 3) == 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int slot = tid + i * NT;
      TIn v0 = 0, v1 = 0, v2 = 0, v3 = 0;
      if (slot < SLOTS) {
        if constexpr (KC) {
          const int row = slot / (GBK / 4), kq = (slot % (GBK / 4)) * 4;
          const int gr = r0 + row, gk = k0 + kq;
          if (gr < nrows) {
            const TIn* p = src + static_cast<long long>(gr) * ld + gk;
            if (vec && gk + 3 < kend) {
              load4(p, v0, v1, v2, v3);
            } else {
              if (gk + 0 < kend) v0 = p[0];
              if (gk + 1 < kend) v1 = p[1];
              if (gk + 2 < kend) v2 = p[2];
              if (gk + 3 < kend) v3 = p[3];
            }
          }
        } else {
          const int kk = slot / (ROWS / 4), rq = (slot % (ROWS / 4)) * 4;
          const int gr = r0 + rq, gk = k0 + kk;
          if (gk < kend) {
            const TIn* p = src + static_cast<long long>(gk) * ld + gr;
            if (vec && gr + 3 < nrows) {
              load4(p, v0, v1, v2, v3);
            } else {
              if (gr + 0 < nrows) v0 = p[0];
              if (gr + 1 < nrows) v1 = p[1];
              if (gr + 2 < nrows) v2 = p[2];
              if (gr + 3 < nrows) v3 = p[3];
            }
          }
        }
      }
      v[i][0] = v0; v[i][1] = v1; v[i][2] = v2; v[i][3] = v3;
    }
  }

  template <typename T>
  __device__ __forceinline__ void store(T* __restrict__ S, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int slot = tid + i * NT;
      if (slot < SLOTS) {
        T* d;
        if constexpr (KC) d = S + (slot / (GBK / 4)) * GLDK + (slot % (GBK / 4)) * 4;
        else d = S + (slot / (ROWS / 4)) * (ROWS + KPAD) + (slot % (ROWS / 4)) * 4;
        store4<T>(d, static_cast<T>(v[i][0]), static_cast<T>(v[i][1]), static_cast<T>(v[i][2]),
                  static_cast<T>(v[i][3]));
      }
    }
  }
};

// Operand fragment of a 16x16x4 MFMA for the 16 rows starting at row0 and the
// k slice kk: lane l owns row (l % 16) and k = 4 (l / 16) + q, q = 0..3.
template <typename T, int ROWS, bool KC>
__device__ __forceinline__ typename Mfma<T>::vec4_t frag(const T* S, int row0, int kk, int lane) {
  if constexpr (KC) {
    return *reinterpret_cast<const typename Mfma<T>::vec4_t*>(S + (row0 + (lane & 15)) * GLDK + kk +
                                                              4 * (lane >> 4));
  } else {
    const T* p = S + (kk + 4 * (lane >> 4)) * (ROWS + KPAD) + row0 + (lane & 15);
    typename Mfma<T>::vec4_t v;
    v[0] = p[0];
    v[1] = p[ROWS + KPAD];
    v[2] = p[2 * (ROWS + KPAD)];
    v[3] = p[3 * (ROWS + KPAD)];
    return v;
  }
}

// 64 x 64 fp64 MFMA tile: acc += A(64 x K) B(K x 64) with both operands staged
// through LDS.  4 waves as 2 x 2, each 32 x 32.
struct Tile64 {
  f64x4 acc[2][2];
  __device__ void zero() {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = f64x4{};
  }
  // B is always staged k-major; A as A_KC says
  template <bool A_KC>
  __device__ void mma_stage(const double* As, const double* Bs, int wm0, int wn0, int lane) {
#pragma unroll
    for (int kk = 0; kk < GBK; kk += 16) {
      f64x4 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = frag<double, 64, A_KC>(As, wm0 + i * 16, kk, lane);
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = frag<double, 64, false>(Bs, wn0 + j * 16, kk, lane);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i][q], b[j][q], acc[i][j], 0, 0, 0);
    }
  }
};

// Block index -> tile index so that consecutive tiles land on the same XCD
// (workgroups are dispatched round-robin over the 8 XCDs).  The grid must be
// padded to 8 * per; indices >= ntiles are idle.
__device__ __forceinline__ int xcd_tile(int b, int ntiles) {
  const int per = (ntiles + 7) >> 3;
  return (b & 7) * per + (b >> 3);
}
__host__ __device__ inline int xcd_grid(int ntiles) { return ((ntiles + 7) >> 3) * 8; }

// Tile (tm, tn) of a tiles_m x tiles_n grid for linear index t, in bands of
// G tile rows: inside a band the column advances only after all of its rows,
// so consecutive tiles (one XCD's share under xcd_tile) touch at most G row
// slices and a few column slices of the operands, which then stay in that
// XCD's L2.  A bijection of [0, tiles_m * tiles_n).
__device__ __forceinline__ void grouped_tile(int t, int tiles_m, int tiles_n, int G, int& tm, int& tn) {
  const int span = G * tiles_n;
  const int band = t / span, rem = t - band * span;
  const int rows = min(G, tiles_m - band * G);
  tn = rem / rows;
  tm = band * G + (rem - tn * rows);
}

}  // namespace cd
