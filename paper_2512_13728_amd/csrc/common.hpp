// Shared declarations of the CurvaDion HIP kernels (gfx950, wave64).
//
// Kernels take small by-value argument structs that carry one pointer per
// layer for up to CD_MAXB layers of identical shape ("batch"); blockIdx.z (or
// .y) selects the layer.  Host launchers live next to their kernels and are
// declared here for the C-ABI layer in api.cpp.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.hpp"

namespace cd {

constexpr int GBK = 32;           // GEMM k per LDS stage; split-K slices are multiples

// ---- the step's device-resident control word ---------------------------------
// Written by the gate kernel of every step, read by the kernels that follow
// it on the device, so that a step can be enqueued whole without the host
// reading the decision first (the asynchronous step): each kernel of either
// branch then checks the decision and returns at once when its branch was not
// taken.
struct StepCtl {
  int flag;        // the branch of the last gated step: 1 = sync
  int spec_next;   // prediction for the next step: 1 = local (fuse the skip update)
  int spec_cur;    // 1 when this step's buffer pass applied the skip update
  int pad;
};
// Where a kernel may return at once: run_if NULL = always run; else run only
// when *run_if != 0 (the sync branch's kernels take &ctl->flag).
__device__ __forceinline__ bool skip_launch(const int* run_if) { return run_if != nullptr && *run_if == 0; }

// A pointer that a kernel reads from a device-side table is generic to the
// compiler, which then accesses it with flat instructions; a flat access also
// counts against the LDS wait counter, so every wait for an LDS result waits
// for the outstanding global loads and stores as well (a prefetch no longer
// overlaps, a store costs its full latency).  global_view marks such a pointer
// as global memory (the round trip through an integer keeps the compiler from
// folding the cast away) and its accesses become global loads and stores.
template <typename T>
__device__ __forceinline__ T* global_view(T* p) {
  return (T*)(__attribute__((address_space(1))) T*)(reinterpret_cast<unsigned long long>(p));
}

// ---- a1: B = M + G and per-block sum of B^2 -------------------------------
// Every block covers FORM_CHUNK consecutive elements of one layer; one launch
// covers up to MAXS layers of any shapes (the passes are elementwise), layer
// j owning blocks [block0[j], block0[j + 1]).
struct FormArgs {
  int nl;                          // layers in this launch
  long long numel[MAXS];           // elements of each layer (m*n)
  int block0[MAXS + 1];            // first block of each layer; block0[nl] = blocks of the launch
  float* M[MAXS];                  // in: M_{t-1}; out: B_t
  const void* G[MAXS];             // fp32 or bf16
  double* part[MAXS];              // out: ceil(numel / FORM_CHUNK) partial sums of B^2 per layer
  float* X[MAXS];                  // with_x: the skip-branch update X = xdecay X - coef G, fused
  float coef[MAXS];                // eta_local per layer (with_x only)
  float xdecay[MAXS];              // 1 - eta * weight_decay per layer (with_x only)
  const StepCtl* ctl;              // spec_mode 2: with_x = ctl->spec_next
};
// spec_mode: 0 = buffer only, 1 = with the skip update, 2 = as ctl->spec_next says
hipError_t launch_form_buffer(const FormArgs& a, bool g_bf16, int spec_mode, hipStream_t s);

// ---- local branch: X = X - eta_local G --------------------------------------
struct LocalArgs {                 // launch layout as FormArgs
  int nl;
  long long numel[MAXS];
  int block0[MAXS + 1];
  float* X[MAXS];
  const void* G[MAXS];
  float coef[MAXS];                // eta_local per layer
  float xdecay[MAXS];              // 1 - eta * weight_decay per layer
  const StepCtl* ctl;              // NULL: run; else only when the step took the local
                                   // branch and its buffer pass did not apply the update
};
hipError_t launch_local_update(const LocalArgs& a, bool g_bf16, hipStream_t s);

// ---- gate: fixed-order reduction of the partials, RMMC, prev update, max ----
struct GateOut {                   // result of the gate (device and host copies)
  double g;                        // max over layers of RMMC (NaN if any is NaN)
  int flag;                        // the branch: g > tau, or the fixed policy's
  int nonfinite;                   // some ‖B‖ was NaN/Inf
  int spec;                        // the step's buffer pass applied the skip update
  int pad;
  // followed by L doubles: RMMC per layer
};
struct GateArgs {
  int L;                           // layers in the group
  int nparts_stride;               // leading dimension of parts (per layer)
  const double* parts;             // [L][nparts_stride]
  const int* nparts;               // [L] partials per layer
  double* const* prev;             // [L] pointers to each layer's prev_norm
  double eps;
  double tau;
  GateOut* out;                    // + L doubles after the header
  double* norms;                   // [L] workspace: ‖B‖ per layer
  unsigned* counter;               // zero between launches (the last block resets it)
  // the same result in pinned, coherent host memory (device view): header and
  // L doubles, then `seq` at host_seq, stored after everything else is
  // visible (host_out NULL: device copy only)
  GateOut* host_out;
  unsigned long long* host_seq;
  unsigned long long seq;
  StepCtl* ctl;                    // the decision for the kernels that follow
  int spec_mode;                   // as the step's buffer pass (0, 1, or 2 = ctl->spec_next)
  int fixed_flag;                  // -1: flag = g > tau; else the fixed policy's branch
};
hipError_t launch_gate(const GateArgs& a, hipStream_t s);

// ---- skinny GEMM on MFMA ----------------------------------------------------
// C[M x N] = A[M x K] * B[K x N] for a batch of layers with identical sizes.
// A(i,k) is at A[i*lda + k] when a_kc (k contiguous) else A[k*lda + i];
// B(k,j) is at B[j*ldb + k] when b_kc else B[k*ldb + j].  With splits > 1 the
// K range is cut in `splits` slices and slice s writes its partial product (in
// the accumulation type) to part + s*split_stride; launch_reduce_splits adds
// them in order s = 0, 1, ... into C.
enum class GemmKind {
  F32,          // fp32 operands, fp32 MFMA, fp32 result
  F64_FROM_F32, // fp32 operands, fp64 MFMA, fp64 result
  F64,          // fp64 operands, fp64 MFMA, fp64 result
  F64_TO_F32,   // fp64 operands, fp64 MFMA, result rounded to fp32
  F32_F64_TO_F32  // fp32 A, fp64 B, fp64 MFMA, result rounded to fp32
};
struct GemmArgs {
  int M, N, K;
  int lda, ldb, ldc;
  int splits;
  int kchunk;                      // K per split (multiple of GBK)
  long long split_stride;          // elements between split partials
  bool a_kc, b_kc;
  bool upper_only;                 // fp32/fp64 kernels: skip tiles strictly below the diagonal
  bool out64;                      // bf16-split kernels: write the result as fp64
  bool b_upper;                    // bf16-split kernels: B is upper triangular (K x N),
                                   // so output column j needs k <= j only
  const void* A[MAXB];
  const void* B[MAXB];
  void* C[MAXB];                   // result (splits == 1) or partials (splits > 1)
  const int* run_if;               // see skip_launch
};
hipError_t launch_gemm(const GemmArgs& a, int nl, GemmKind kind, hipStream_t s);
int gemm_bm(int N, bool fp64);     // tile rows the launcher uses for this N
int gemm_bn(int N, bool fp64);     // tile columns
inline bool gemm_acc64(GemmKind k) { return k != GemmKind::F32; }

// The same contraction for fp32 operands on the bf16 MFMA with each operand
// split into `pieces` bf16 terms (3: about fp32 accuracy; 1: plain bf16).
// fp32 result (or fp32 split partials).
hipError_t launch_gemm_bf(const GemmArgs& a, int nl, int pieces, hipStream_t s);
int gemm_bf_bm(int N);
int gemm_bf_bn(int N, int pieces);

// out[i] = sum_{s < splits} part[s*stride + i] in order s = 0, 1, ...
// Partials are fp64 when part64, and the output is fp64 when out64.
struct ReduceArgs {
  long long count;
  long long stride;
  int splits;
  const void* part[MAXB];
  void* out[MAXB];
  const int* run_if;
};
hipError_t launch_reduce_splits(const ReduceArgs& a, int nl, bool part64, bool out64, hipStream_t s);

// ---- exact Gram matrix of an fp32 panel on the bf16 MFMA (k_gram.hip) -------
// W = P^T P (r x r, upper 64 x 64 tiles) of P (m x r, row-major): per chunk
// of GX_CHUNK rows, column exponents E and three bf16 slice planes S
// (column-major, mp = m rounded up to GX_CHUNK rows per column), then the
// product, split over K like the GEMMs (fp64 partials, or W itself when
// splits == 1).
constexpr int GX_CHUNK = 128;
struct GramXArgs {
  int m, mp, r;
  int splits, kchunk;              // K split (kchunk a multiple of GX_CHUNK)
  long long split_stride;          // doubles between partials (r * r)
  const float* P[MAXB];
  __bf16* S[MAXB];                 // 3 planes of r x mp
  int* E[MAXB];                    // (mp / GX_CHUNK) x r exponents
  void* C[MAXB];                   // fp64 W (splits == 1) or partials
  const int* run_if;
};
// bytes of the slice planes and exponents for m x r (16-byte aligned pieces)
inline size_t gram_x_bytes(long long m, long long r) {
  const long long mp = (m + GX_CHUNK - 1) / GX_CHUNK * GX_CHUNK;
  return static_cast<size_t>(6 * r * mp + (4 * r * (mp / GX_CHUNK) + 15) / 16 * 16 + 16);
}
hipError_t launch_gram_x(const GramXArgs& a, int nl, hipStream_t s);

// ---- Cholesky of the Gram matrix and triangular solve ------------------------
// Per-layer workspace pointers (static for the life of a group) for the
// blocked fp64 Cholesky W = T^T T (T overwrites the upper triangle of W, r x r,
// ld = r) and the inverses D_k of its CHOL_BLOCK x CHOL_BLOCK diagonal blocks.
constexpr int CHOL_BLOCK = 64;
struct CholTab {
  double* W;
  double* Dinv;                    // ceil(r / CHOL_BLOCK) blocks of 64 x 64
  double* floor_;                  // pivot floor of the current factorisation
  int* rankdef;                    // set to 1 when a pivot was raised to the floor
  int* rowok;                      // r: 0 for the rows of floored pivots, else 1
  int* rankdef_host;               // NULL, or a mirror of rankdef in pinned host memory
  double* nid;                     // second pass without pivots: two r x r buffers, then
                                   // nearid_parts(r) partial sums
  int* nid_ok;                     // 1: the second pass's factor came from launch_nearid
};
// All CHOL_BLOCK steps for `nlayers` layers of rank r; `pass` 0 clears rankdef.
// gated: layers whose nid_ok is set are skipped (their factor is formed).
hipError_t launch_cholesky(const CholTab* tab, int nlayers, int r, int pass, hipStream_t s,
                           const int* run_if = nullptr, bool gated = false);
// The factor T1 of a Gram matrix W1 = I + E with ||E||_F <= 2^-10 and the
// inverses of its diagonal blocks, by a fixed-point iteration (k_nearid.hip);
// sets nid_ok per layer.  W1 in, T1 out over its upper triangle.
hipError_t launch_nearid(const CholTab* tab, int nlayers, int r, hipStream_t s, const int* run_if = nullptr);
int nearid_parts(int r);           // partial sums launch_nearid keeps per layer

// The fixed pseudo-random direction that completes column j of P1 past the
// numerical rank (row i; scale sqrt(3/m) gives unit expected norm): an
// integer hash of (row, column), uniform in [-scale, scale).
__device__ __forceinline__ float fill_value(unsigned i, unsigned j, float scale) {
  // integer hash of (row, column): xorshift-multiply rounds
  unsigned h = i * 0x9E3779B1u + j * 0x85EBCA77u + 0x27D4EB2Fu;
  h ^= h >> 16; h *= 0x7FEB352Du;
  h ^= h >> 15; h *= 0x846CA68Bu;
  h ^= h >> 16;
  return scale * (static_cast<float>(h >> 8) * (2.0f / 16777216.0f) - 1.0f);   // uniform in [-1, 1)
}


// P = P~ T^{-1} by block columns.  In place (Pin == Pout, same type) is
// allowed: the workgroup of a row tile reads its block column of P~ before it
// writes that block column of P, and reads only finished columns of P
// besides.
struct TrsmTab {
  const void* Pin;                 // m x r, fp64 or fp32
  void* Pout;                      // m x r, fp64 or fp32
  const double* W;                 // T in the upper triangle
  const double* Dinv;
  int m;
};
// tiles: one (layer, 64-row tile) pair per workgroup.  ident: Pin is the
// identity (the result is T^{-1}); mlimit > 0 caps every layer's row count.
// Between the CholQR passes: columns of P1 (TrsmTab::Pout, fp32 m x r) whose
// pivot was floored get fixed pseudo-random directions (layers with
// rankdef == 0 are left alone).  mmax: the largest m of the layers.
// p64: P1 is fp64 (fp32-gradient layers), else fp32.
hipError_t launch_fill_dead(const CholTab* ct, const TrsmTab* tt, int nlayers, int mmax, int r, bool p64,
                            hipStream_t s, const int* run_if = nullptr);
hipError_t launch_trsm(const TrsmTab* tab, const int2* tiles, int ntiles, int r, bool in64, bool out64,
                       hipStream_t s, bool ident = false, int mlimit = 0, const int* run_if = nullptr);
// The same solve, right-looking, for fp64 panels in place (Pin == Pout).
hipError_t launch_trsm_rl(const TrsmTab* tab, const int2* tiles, int ntiles, int r, hipStream_t s,
                          const int* run_if = nullptr);

// ---- ColumnNormalize --------------------------------------------------------
constexpr int COLNORM_ROWS = 64;   // rows per partial
struct ColnormArgs {
  int n, r;
  int nchunks;                     // ceil(n / COLNORM_ROWS)
  const float* R[MAXB];
  double* part[MAXB];              // [nchunks][r]
  float* nrm[MAXB];                // [r] max(‖R_j‖, floor) as fp32
  float* Q[MAXB];                  // out: n x r
  // bf16 planes (pieces S, row stride rp) of R and of Q for the update
  int S, rp;
  __bf16* Rpl[MAXB];
  __bf16* Qpl[MAXB];
  const int* run_if;
};
hipError_t launch_colnorm(const ColnormArgs& a, int nl, hipStream_t s);

// ---- the sync branch of small layers (k_small.hip) ----------------------------
// Layers with r <= SMALL_R and m r, n r <= SMALL_MR: P~ = B Q and R = B^T P
// on the fp64 GEMM kernels, then the two kernels below.
constexpr int SMALL_R = 64;
constexpr int SMALL_MR = 8192;
constexpr int SMALL_ROWS = 16;    // rows of M and X per workgroup of the update
bool small_sync_fits(int m, int n, int r);
struct SmallQrArgs {               // CholQR twice, one workgroup per layer
  int m, r;
  const double* Pt[MAXB];          // P~ (m x r fp64)
  double* P64[MAXB];               // out: P in fp64 (may be Pt)
  float* P32[MAXB];                // out: P in fp32
  int* rankdef[MAXB];              // out: 1 if a pivot was floored
  int* rankdef_host[MAXB];         // NULL, or its mirror in pinned host memory
  const int* run_if;
};
hipError_t launch_small_cholqr(const SmallQrArgs& a, int nl, hipStream_t s);
// C = A B for P~ = B Q of small layers (no split-K): kind F64_FROM_F32, A
// k-contiguous, B row-major (b_kc false), N <= SMALL_R, K <= 1024.
bool small_gemm_fits(int N, int K);
hipError_t launch_small_gemm(const GemmArgs& g, int nl, GemmKind kind, hipStream_t s);
struct SmallUpdArgs {              // column norms, Q and the M / X update
  int m, n, r;
  float one_minus_mu;
  float c;                         // eta sqrt(m / n)
  float* M[MAXB];
  float* X[MAXB];
  const float* P[MAXB];            // m x r fp32
  const float* R[MAXB];            // n x r fp32
  float* Q[MAXB];                  // out: n x r
  const void* G[MAXB];             // reversal of a speculative skip update, as UpdateVecArgs
  float gc[MAXB];
  int g_bf16;
  int spec;                        // 0, 1, or 2 = ctl->spec_cur
  float xdecay[MAXB];
  const StepCtl* ctl;              // NULL: run; else only on a sync step
};
hipError_t launch_small_update(const SmallUpdArgs& a, int nl, hipStream_t s);

// ---- error-feedback momentum and weight update ------------------------------
// M = M - (1-mu) P R^T (M holds B on entry); X = X - c P Q^T, c = eta sqrt(m/n)
// fp32 operands on the vector units, for r <= 32 (k_update_vec): P m x r,
// R and Q n x r, all fp32 row-major; band = rows per block (set by the
// launcher)
struct UpdateVecArgs {
  int m, n, r, band;
  float one_minus_mu;
  float c;
  float* M[MAXB];
  float* X[MAXB];
  const float* P[MAXB];
  const float* R[MAXB];
  const float* Q[MAXB];
  // spec = 1: the buffer pass already applied the skip branch's
  // X = xdecay X - eta_local G (the decay included); the update first adds
  // gc G back (gc = eta_local; no read of G when it is 0).  spec = 0: X
  // still needs the decay, X = xdecay X, before the rank-r correction.
  const void* G[MAXB];
  float gc[MAXB];
  int g_bf16;
  int spec;              // 0, 1, or 2 = ctl->spec_cur
  float xdecay[MAXB];
  const StepCtl* ctl;    // NULL: run; else only on a sync step
};
bool update_vec_fits(int r);
hipError_t launch_update_vec(UpdateVecArgs a, int nl, hipStream_t s);
// bf16 planes of fp32 matrices (rows x r): plane s (s < S <= 3) holds the
// s-th bf16 piece of each value, rows padded to rp (multiple of 32) with zeros.
struct PlaneArgs {
  int rows, r, rp, S;
  const float* src[MAXB];
  __bf16* dst[MAXB];               // S * rows * rp elements
  const int* run_if;
};
hipError_t launch_split_planes(const PlaneArgs& a, int nl, hipStream_t s);

// The update from bf16 planes of P (m x rp), R and Q (n x rp) on the bf16
// MFMA; pieces = 3 forms fp32-accurate products, pieces = 1 plain bf16 ones.
struct UpdatePlArgs {
  int m, n, r, rp;
  float one_minus_mu;
  float c;
  float* M[MAXB];
  float* X[MAXB];
  const __bf16* P[MAXB];
  const __bf16* R[MAXB];
  const __bf16* Q[MAXB];
  // spec = 1: the buffer pass already applied the skip branch's
  // X = xdecay X - eta_local G (the decay included); the update first adds
  // gc G back (gc = eta_local; no read of G when it is 0).  spec = 0: the
  // decoupled weight decay X = xdecay X comes first.
  const void* G[MAXB];
  float gc[MAXB];
  int g_bf16;
  int spec;              // 0, 1, or 2 = ctl->spec_cur
  float xdecay[MAXB];
  const StepCtl* ctl;    // NULL: run; else only on a sync step
};
hipError_t launch_update_planes(const UpdatePlArgs& a, int nl, int pieces, hipStream_t s);

}  // namespace cd
