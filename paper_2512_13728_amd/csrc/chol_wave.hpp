// One wave's Cholesky factorisation W = T^T T of an nb x nb block (nb <= NB,
// NB = 16, 32 or 64) and the inverse T^{-1}, for the diagonal blocks of the
// blocked factorisation and for whole small Gram matrices.
//
// Lane j holds column j of the block (upper triangle; rows past the block
// padded with the identity) in registers.  Right-looking: at pivot p the
// lanes publish row p of the updated block in LDS and every lane reads it
// back with uniform-address loads (a broadcast), then updates its own column.
// The register array is shifted by one row per pivot inside the update (a[i]
// holds row p + i), so the pivot row is always a[0] and every index is a
// constant while the pivot loop itself stays rolled (a few KB of code instead
// of a fully unrolled loop the instruction cache cannot hold).
//
// A pivot at or below the floor fl is raised to it and the rest of its row of
// T is set to zero: the numerically dependent direction then adds nothing to
// the trailing matrix.  Dividing its rounding-level residuals by the floor's
// square root instead would subtract their squares from the next pivots,
// which fall under the floor in turn, and the entries grow without bound.
//
// T^{-1} follows by back substitution, lane c solving T d = e_c from the last
// row up, with T read from LDS and the unknowns shifted the same way; the
// columns of floored pivots are returned as zero, so that P~ T^{-1} is zero
// in those columns.
//
// Only the lanes of one wave take part.  They exchange values through LDS in
// program order: the LDS executes the accesses of one wave in order, so a
// wave-level barrier (which keeps the compiler from moving accesses across
// it) orders them; no workgroup barrier is involved.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>
#include <utility>

namespace cd {

// f(integral_constant<int, 0>) ... f(integral_constant<int, N - 1>), in order
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// orders the LDS accesses of the lanes of one wave (see above)
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// use(i, load(i)) for i = 0 .. N - 1, the loads in chunks of up to CHUNK:
// chunk c + 1 is requested before chunk c is used (the compiler may not move
// loads or uses across the scheduling barriers), so the values in flight
// never exceed two chunks' registers.
template <int N, int CHUNK = 16, class Load, class Use>
__device__ __forceinline__ void chunked(Load&& load, Use&& use) {
  constexpr int NC = (N + CHUNK - 1) / CHUNK;
  if constexpr (N > 0) {
    double buf[2][CHUNK];
    static_for<NC + 1>([&](auto cc) {
      constexpr int C = decltype(cc)::value;
      if constexpr (C < NC) {
#pragma unroll
        for (int i = 0; i < CHUNK && C * CHUNK + i < N; ++i) buf[C & 1][i] = load(C * CHUNK + i);
      }
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (C > 0) {
#pragma unroll
        for (int i = 0; i < CHUNK && (C - 1) * CHUNK + i < N; ++i) use((C - 1) * CHUNK + i, buf[(C - 1) & 1][i]);
      }
      __builtin_amdgcn_sched_barrier(0);
    });
  }
}

template <int NB>
struct WaveChol {
  static_assert(NB == 16 || NB == 32 || NB == 64, "block of 16, 32 or 64 columns");
  static constexpr int SEG = 8;         // pivots per segment of the register loops
  static constexpr int TLD = NB + 1;    // padded row of T in LDS (column stores hit distinct banks)
  static constexpr int TPAD = NB;       // leading doubles: back-substitution reads above row 0 stay in the array
  // LDS of one factorisation
  struct Lds {
    double rowb[2 * NB];                // row p, then zeros
    double Tsb[TPAD + NB * TLD];        // Ts[j * TLD + i] = T[i][j]
    double pinv[NB];                    // 1 / T[p][p]
    int okb[NB];                        // pivot p not floored
  };
  __device__ static double* Ts(Lds& s) { return s.Tsb + TPAD; }

  // The factorisation of the nb x nb block whose entries load(i) (row i of
  // lane j's column; i <= j < nb) gives; returns whether a pivot was floored
  // (uniform over the wave).  Leaves T (transposed) in Ts, 1 / T[p][p] in
  // pinv and the pivot flags in okb.
  template <class Load>
  __device__ static bool factor(Lds& s, int j, int nb, double fl, Load&& load) {
    const bool lane_in = j < NB;
    double* const T = Ts(s);
    double a[NB];   // a[i] = A[p + i][j] at pivot p
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if (i < nb && j < nb) a[i] = i <= j ? load(i) : 0.0;
      else a[i] = i == j ? 1.0 : 0.0;
    }
    if (lane_in) {
      s.rowb[NB + j] = 0.0;
      s.Tsb[j] = 0.0;
    }
    bool def = false;
    // Only the block's nb pivots run: the identity padding of a partial block
    // would factor to itself, and its rows are never used.  At pivot p only
    // rows p .. NB - 1 remain, so the pivots run in segments of SEG whose
    // register arrays carry NB, NB - SEG, ... rows (rows past the live range
    // stay untouched and unused).
    auto pivot = [&](auto na, int p) {
      constexpr int NA = decltype(na)::value;
      // the pivot A[p][p] is lane p's a[0]: read across the wave (no LDS trip)
      const double a0 = a[0];
      double d = __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(a0), p),
                                  __builtin_amdgcn_readlane(__double2loint(a0), p));
      const bool floored = !(d > fl);   // uniform over the wave
      if (floored) { d = fl; def = true; }
      // 1/sqrt(d): the hardware estimate refined by two Newton steps (error
      // squared each step), then sqrt(d) = d / sqrt(d); both within about an
      // ulp, with no divide in the pivot's dependency chain
      double inv = __builtin_amdgcn_rsq(d);
#pragma unroll
      for (int it = 0; it < 2; ++it) inv = fma(inv, fma(-0.5 * d * inv, inv, 0.5), inv);
      const double piv = d * inv;
      // row p of T (zero left of the diagonal, and right of a floored pivot)
      const double tp = j == p ? piv : (j > p && !floored ? a[0] * inv : 0.0);
      if (lane_in) T[j * TLD + p] = tp;
      if (j == p) {
        s.pinv[p] = inv;
        s.okb[p] = floored ? 0 : 1;
      }
      wave_sync();
      if (lane_in) s.rowb[j] = tp;
      wave_sync();
      // rows below p: A[p + i][j] -= T[p][p + i] T[p][j], shifted up one row;
      // lanes j < p + i only touch the (unused) lower triangle.  The row is
      // read in chunks, each requested before the previous one is used, so
      // that one LDS round trip is exposed per pivot and at most two chunks
      // are held.
      chunked<NA - 1>([&](int i) { return s.rowb[p + 1 + i]; },
                      [&](int i, double v) { a[i] = fma(-v, tp, a[i + 1]); });
      a[NA - 1] = 0.0;
      wave_sync();
    };
    // segment g: pivots [g SEG, (g + 1) SEG) with NB - g SEG live rows
    static_for<NB / SEG>([&](auto gc) {
      constexpr int G = decltype(gc)::value;
#pragma unroll 1
      for (int p = G * SEG; p < min(nb, (G + 1) * SEG); ++p) pivot(std::integral_constant<int, NB - G * SEG>{}, p);
    });
    return def;
  }

  // factor() with T^{-1} formed in the same pivot loop (NB <= 32): lanes NB ..
  // 2 NB - 1 hold the columns of the identity and undergo the same row
  // operations.  With W = T^T T, the elimination that turns W into T turns I
  // into E = T^{-T}: at pivot p, row p of E is final once scaled by
  // 1 / sqrt(d), and every row i > p takes E[i][c] -= T[p][i] E[p][c] /
  // sqrt(d), the update the W columns take.  Row p of E, i.e. column p of
  // T^{-1}, is zero for a floored pivot, as inverse() returns it.
  // put_inv(c, p, x): x = (T^{-1})[c][p] for c < NB, p < nb.  Replaces
  // inverse() and its nb back-substitution steps.
  template <class Load, class PutInv>
  __device__ static bool factor_inv(Lds& s, int j, int nb, double fl, Load&& load, PutInv&& put_inv) {
    static_assert(NB <= 32, "two columns per lane pair: the block and the identity");
    const bool lane_in = j < NB;
    const bool lane_e = j >= NB && j < 2 * NB;
    const int c = j - NB;                 // identity column of an E lane
    double* const T = Ts(s);
    double a[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if (lane_in) {
        if (i < nb && j < nb) a[i] = i <= j ? load(i) : 0.0;
        else a[i] = i == j ? 1.0 : 0.0;
      } else {
        a[i] = (lane_e && i == c && c < nb) ? 1.0 : 0.0;
      }
    }
    if (lane_in) {
      s.rowb[NB + j] = 0.0;
      s.Tsb[j] = 0.0;
    }
    bool def = false;
    auto pivot = [&](auto na, int p) {
      constexpr int NA = decltype(na)::value;
      const double a0 = a[0];
      double d = __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(a0), p),
                                  __builtin_amdgcn_readlane(__double2loint(a0), p));
      const bool floored = !(d > fl);
      if (floored) { d = fl; def = true; }
      double inv = __builtin_amdgcn_rsq(d);
#pragma unroll
      for (int it = 0; it < 2; ++it) inv = fma(inv, fma(-0.5 * d * inv, inv, 0.5), inv);
      const double piv = d * inv;
      // row p of T (block lanes) or of E (identity lanes)
      const double tp = lane_in ? (j == p ? piv : (j > p && !floored ? a[0] * inv : 0.0))
                                : (floored ? 0.0 : a[0] * inv);
      if (lane_in) T[j * TLD + p] = tp;
      if (lane_e) put_inv(c, p, tp);
      if (j == p) {
        s.pinv[p] = inv;
        s.okb[p] = floored ? 0 : 1;
      }
      wave_sync();
      if (lane_in) s.rowb[j] = tp;
      wave_sync();
      chunked<NA - 1>([&](int i) { return s.rowb[p + 1 + i]; },
                      [&](int i, double v) { a[i] = fma(-v, tp, a[i + 1]); });
      a[NA - 1] = 0.0;
      wave_sync();
    };
    static_for<NB / SEG>([&](auto gc) {
      constexpr int G = decltype(gc)::value;
#pragma unroll 1
      for (int p = G * SEG; p < min(nb, (G + 1) * SEG); ++p) pivot(std::integral_constant<int, NB - G * SEG>{}, p);
    });
    return def;
  }

  // Lane j (< nb) computes column j of T^{-1} after factor(): put(p, x) with
  // x = (T^{-1})[p][j] for p = nb - 1 down to 0, x = 0 in the column of a
  // floored pivot (with row p of T zero right of the diagonal, column j != p
  // of T^{-1} is zero in row p).  Lanes j >= nb call put with x = 0.
  template <class Put>
  __device__ static void inverse(Lds& s, int j, int nb, Put&& put) {
    double* const T = Ts(s);
    // f[k] = d[p - k] at step p, from p = nb - 1 down; entries with k > p lie
    // above row 0 and are never used, so the steps of pivots below
    // NB - SEG g carry only NB - SEG g entries
    double f[NB];
#pragma unroll
    for (int k = 0; k < NB; ++k) f[k] = k == nb - 1 - j ? 1.0 : 0.0;
    const bool cin = j < nb && s.okb[j];
    auto back = [&](auto nf, int p) {
      constexpr int NF = decltype(nf)::value;
      const double x = f[0] * s.pinv[p];
      put(p, cin ? x : 0.0);
      const double* col = T + p * TLD + p;   // col[-k] = T[p - k][p]
      chunked<NF - 1>([&](int k) { return col[-1 - k]; },
                      [&](int k, double v) { f[k] = fma(-v, x, f[k + 1]); });
      f[NF - 1] = 0.0;
    };
    // segments from the last down: segment g carries (g + 1) SEG entries
    static_for<NB / SEG>([&](auto ic) {
      constexpr int G = NB / SEG - 1 - decltype(ic)::value;
#pragma unroll 1
      for (int p = min(nb, (G + 1) * SEG) - 1; p >= G * SEG; --p) back(std::integral_constant<int, (G + 1) * SEG>{}, p);
    });
  }
};

}  // namespace cd
