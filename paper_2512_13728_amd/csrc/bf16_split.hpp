// fp32 contractions on the bf16 MFMA (v_mfma_f32_16x16x32_bf16, gfx950).
//
// Each fp32 operand value v is split into S bf16 pieces, v = p1 + p2 + p3
// (p1 = bf16(v), p2 = bf16(v - p1), p3 = bf16(v - p1 - p2); each difference is
// exact in fp32), and a product a*b is formed from the piece products p_i q_j
// with i + j <= S + 1.  S = 3 (six products) reproduces the fp32 product to
// about 2^-24; S = 1 is a plain bf16 product.  Accumulation is fp32.
//
// Tiles are staged in LDS as bf16 planes [piece][row][k] (k contiguous, rows
// padded to 40 elements so the sixteen 16-byte fragment reads of a quarter-wave
// hit distinct banks).  Operands whose global layout is not k-contiguous are
// transposed in registers in 4 x 4 blocks before the LDS store, so every LDS
// store is 8 contiguous bytes.  The four 16-byte k-granules of a row are
// XOR-permuted by bits 4-5 of the row (lds_off): the transposed stores, where
// the 16 lanes of a quarter-wave write rows 4 apart, then fall on distinct
// banks too, and a fragment (16 consecutive rows from a multiple of 16) sees
// one permutation for all its rows.
#pragma once

#include <hip/hip_runtime.h>

#include "common.hpp"
#include "mfma_tile.hpp"

namespace cd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr int BK16 = 32;          // k per stage (one MFMA depth)
constexpr int BLD = BK16 + 8;     // padded LDS row (bf16 elements)

// Element offset of (row, k), k < BK16, inside one LDS plane.
__device__ __forceinline__ int lds_off(int row, int k) {
  return row * BLD + ((((k >> 3) ^ (row >> 4)) & 3) << 3) + (k & 7);
}

template <int S>
__device__ __forceinline__ void split_bf16(float v, __bf16 (&p)[S]) {
  float rest = v;
#pragma unroll
  for (int i = 0; i < S; ++i) {
    p[i] = static_cast<__bf16>(rest);
    rest -= static_cast<float>(p[i]);
  }
}

// A second layout for tiles staged only as whole 16-byte k granules (a
// quarter-wave storing four consecutive rows): rows of 64 bytes, the four
// granules XOR-permuted by bits 2-3 of the row.  Such a store, and a fragment
// read (16 consecutive rows, one granule), each cover all 64 banks once.
constexpr int BLD64 = BK16;
__device__ __forceinline__ int lds_off64(int row, int k) {
  return row * BLD64 + ((((k >> 3) ^ (row >> 2)) & 3) << 3) + (k & 7);
}

// Store 4 consecutive-k values of one row into the S planes.
template <int S, int ROWS>
__device__ __forceinline__ void put4(__bf16* planes, int row, int kq, float v0, float v1, float v2,
                                     float v3) {
  __bf16 a[S], b[S], c[S], d[S];
  split_bf16<S>(v0, a);
  split_bf16<S>(v1, b);
  split_bf16<S>(v2, c);
  split_bf16<S>(v3, d);
#pragma unroll
  for (int s = 0; s < S; ++s) {
    bf16x4 w = {a[s], b[s], c[s], d[s]};
    *reinterpret_cast<bf16x4*>(planes + s * ROWS * BLD + lds_off(row, kq)) = w;
  }
}

// Global -> registers for one stage of a ROWS x BK16 tile (rows r0.., k k0..),
// and registers -> LDS planes.  kc: element (row, k) at src[row * ld + k];
// otherwise at src[k * ld + row].  Out-of-range elements read as zero.
template <int ROWS, int NT>
struct Stage {
  // kc: ROWS * BK16 / 4 float4 slots; non-kc: (ROWS / 4) * (BK16 / 4) 4x4 blocks
  static constexpr int KC_SLOTS = ROWS * (BK16 / 4);
  static constexpr int KC_PER = (KC_SLOTS + NT - 1) / NT;
  static constexpr int T_SLOTS = (ROWS / 4) * (BK16 / 4);
  static constexpr int T_PER = (T_SLOTS + NT - 1) / NT;
  static constexpr int NREG = KC_PER * 4 > T_PER * 16 ? KC_PER * 4 : T_PER * 16;
  float v[NREG];

  __device__ __forceinline__ void load(const float* __restrict__ src, int ld, bool kc, int r0, int nrows,
                                       int k0, int kend, int tid) {
    const bool vec = (ld & 3) == 0;
    // interior stage (every row and k in range, 16-byte rows): no per-element
    // checks; the condition is uniform over the workgroup
    if (vec && r0 + ROWS <= nrows && k0 + BK16 <= kend) {
      if (kc) {
#pragma unroll
        for (int i = 0; i < KC_PER; ++i) {
          const int slot = tid + i * NT;
          if (KC_SLOTS % NT == 0 || slot < KC_SLOTS) {
            const int row = slot / (BK16 / 4), kq = (slot % (BK16 / 4)) * 4;
            const float4 f =
                *reinterpret_cast<const float4*>(src + static_cast<long long>(r0 + row) * ld + k0 + kq);
            v[4 * i] = f.x; v[4 * i + 1] = f.y; v[4 * i + 2] = f.z; v[4 * i + 3] = f.w;
          }
        }
      } else {
#pragma unroll
        for (int i = 0; i < T_PER; ++i) {
          const int slot = tid + i * NT;
          if (T_SLOTS % NT == 0 || slot < T_SLOTS) {
            const int rq = (slot % (ROWS / 4)) * 4, kq = (slot / (ROWS / 4)) * 4;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
              const float4 f = *reinterpret_cast<const float4*>(
                  src + static_cast<long long>(k0 + kq + kk) * ld + r0 + rq);
              v[16 * i + 4 * kk + 0] = f.x; v[16 * i + 4 * kk + 1] = f.y;
              v[16 * i + 4 * kk + 2] = f.z; v[16 * i + 4 * kk + 3] = f.w;
            }
          }
        }
      }
      return;
    }
    if (kc) {
#pragma unroll
      for (int i = 0; i < KC_PER; ++i) {
        const int slot = tid + i * NT;
        const int row = slot / (BK16 / 4), kq = (slot % (BK16 / 4)) * 4;
        const int gr = r0 + row, gk = k0 + kq;
        float a = 0.f, b = 0.f, c = 0.f, d = 0.f;
        if (slot < KC_SLOTS && gr < nrows) {
          const float* p = src + static_cast<long long>(gr) * ld + gk;
          if (vec && gk + 3 < kend) {
            const float4 f = *reinterpret_cast<const float4*>(p);
            a = f.x; b = f.y; c = f.z; d = f.w;
          } else {
            if (gk + 0 < kend) a = p[0];
            if (gk + 1 < kend) b = p[1];
            if (gk + 2 < kend) c = p[2];
            if (gk + 3 < kend) d = p[3];
          }
        }
        v[4 * i + 0] = a; v[4 * i + 1] = b; v[4 * i + 2] = c; v[4 * i + 3] = d;
      }
    } else {
#pragma unroll
      for (int i = 0; i < T_PER; ++i) {
        const int slot = tid + i * NT;
        const int rq = (slot % (ROWS / 4)) * 4, kq = (slot / (ROWS / 4)) * 4;
        const int gr = r0 + rq;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int gk = k0 + kq + kk;
          float a = 0.f, b = 0.f, c = 0.f, d = 0.f;
          if (slot < T_SLOTS && gk < kend) {
            const float* p = src + static_cast<long long>(gk) * ld + gr;
            if (vec && gr + 3 < nrows) {
              const float4 f = *reinterpret_cast<const float4*>(p);
              a = f.x; b = f.y; c = f.z; d = f.w;
            } else {
              if (gr + 0 < nrows) a = p[0];
              if (gr + 1 < nrows) b = p[1];
              if (gr + 2 < nrows) c = p[2];
              if (gr + 3 < nrows) d = p[3];
            }
          }
          // v[16 i + 4 kk + c]: element (row rq + c, k kq + kk)
          v[16 * i + 4 * kk + 0] = a; v[16 * i + 4 * kk + 1] = b;
          v[16 * i + 4 * kk + 2] = c; v[16 * i + 4 * kk + 3] = d;
        }
      }
    }
  }

  template <int S>
  __device__ __forceinline__ void store(__bf16* planes, bool kc, int tid) const {
    if (kc) {
#pragma unroll
      for (int i = 0; i < KC_PER; ++i) {
        const int slot = tid + i * NT;
        if (slot < KC_SLOTS) {
          const int row = slot / (BK16 / 4), kq = (slot % (BK16 / 4)) * 4;
          put4<S, ROWS>(planes, row, kq, v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < T_PER; ++i) {
        const int slot = tid + i * NT;
        if (slot < T_SLOTS) {
          const int rq = (slot % (ROWS / 4)) * 4, kq = (slot / (ROWS / 4)) * 4;
#pragma unroll
          for (int c = 0; c < 4; ++c)
            put4<S, ROWS>(planes, rq + c, kq, v[16 * i + c], v[16 * i + 4 + c], v[16 * i + 8 + c],
                          v[16 * i + 12 + c]);
        }
      }
    }
  }
};

// bf16 fragment: lane l owns row (l % 16) and k = 8 (l / 16) .. + 7.
__device__ __forceinline__ bf16x8 bfrag(const __bf16* plane, int row0, int lane) {
  return *reinterpret_cast<const bf16x8*>(plane + lds_off(row0 + (lane & 15), 8 * (lane >> 4)));
}
__device__ __forceinline__ bf16x8 bfrag64(const __bf16* plane, int row0, int lane) {
  return *reinterpret_cast<const bf16x8*>(plane + lds_off64(row0 + (lane & 15), 8 * (lane >> 4)));
}

__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

}  // namespace cd
