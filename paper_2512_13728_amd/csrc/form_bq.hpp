// The buffer pass fused into the first power-iteration product, for steps of
// bf16-gradient layers that are predicted (or fixed) to sync: B = M + G is
// formed in the operand staging of P~ = B Q (Algorithm 2 buffer update and
// power iteration), written over M, and summed in squares for the RMMC
// statistic (Eq. 1), so such a step streams M and G once instead of a
// buffer pass followed by a second read of B.
#pragma once

#include "common.hpp"

namespace cd {

constexpr int FBQ_BM = 128;         // rows of B per workgroup
constexpr int FBQ_RMAX = 512;       // every column of P~ in one workgroup: r <= 512
constexpr int FBQ_RMIN = 257;       // the 512-wide tile would mostly multiply padding below

struct FormBqArgs {
  int m, n, r;                     // B is m x n, Q n x r
  int splits, kchunk;              // K (= n) in `splits` slices of kchunk (multiple of 32)
  long long split_stride;          // elements between the fp32 partials of P~ (m * r)
  float* M[MAXB];                  // in: M_{t-1}; out: B_t
  const __bf16* G[MAXB];           // bf16 gradient
  const float* Q[MAXB];            // n x r
  float* C[MAXB];                  // P~ (splits == 1) or its split partials
  double* part[MAXB];              // out: partial sums of B^2, tiles_m x splits per layer
};
// Partial sums of B^2 this launch writes per layer (tile-row major, then split).
inline int form_bq_nparts(int m, int splits) { return (m + FBQ_BM - 1) / FBQ_BM * splits; }
hipError_t launch_form_bq(const FormBqArgs& a, int nl, hipStream_t s);

}  // namespace cd
