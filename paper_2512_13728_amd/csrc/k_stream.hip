// Streaming kernels of the CurvaDion step: buffer formation with the fused
// sum of squares (B = M + G; Algorithm 2, local buffer update, feeding the
// norm of Eq. 1), optionally with the skip branch's weight update fused into
// the same pass, the stand-alone skip-branch update (X -= eta_local G), and
// the gate (fixed-order reduction, RMMC, prev_norm update, max over layers).
//
// These passes are HBM-bound: blocks own fixed 4096-element chunks of one
// layer (four 16-byte segments per thread and stream), every operand is read
// and written once with non-temporal hints (nothing is reused, so nothing
// should displace other lines), and every reduction runs in a fixed order so
// that the statistic is bit-reproducible run to run.
#include "common.hpp"

namespace cd {
namespace {

typedef float nt_f4 __attribute__((ext_vector_type(4)));
typedef unsigned nt_u2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float4 ld_nt(const float* p) {
  const nt_f4 v = __builtin_nontemporal_load(reinterpret_cast<const nt_f4*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ void st_nt(float* p, float4 v) {
  const nt_f4 w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, reinterpret_cast<nt_f4*>(p));
}

// G element loads: fp32, or bf16 widened exactly (bf16 bits are the top half
// of the fp32 bit pattern).
template <bool BF16>
__device__ __forceinline__ float4 load_g4(const void* G, long long i) {
  if constexpr (BF16) {
    const nt_u2 u = __builtin_nontemporal_load(
        reinterpret_cast<const nt_u2*>(static_cast<const uint16_t*>(G) + i));
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
  } else {
    return ld_nt(static_cast<const float*>(G) + i);
  }
}

template <bool BF16>
__device__ __forceinline__ float load_g1(const void* G, long long i) {
  if constexpr (BF16) {
    return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(G)[i]) << 16);
  } else {
    return static_cast<const float*>(G)[i];
  }
}

__device__ __forceinline__ double sq(float x) { return static_cast<double>(x) * static_cast<double>(x); }

// Sum over the block in a fixed order; the result is valid in thread 0.
__device__ double block_sum(double v) {
  __shared__ double ws[NTHREADS / 64];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) ws[w] = v;
  __syncthreads();
  double s = 0.0;
  if (threadIdx.x == 0) {
#pragma unroll
    for (int i = 0; i < NTHREADS / 64; ++i) s += ws[i];
  }
  return s;
}

constexpr int VPT = FORM_CHUNK / (NTHREADS * 4);   // float4 groups per thread (4)

// The layer that block b of a launch belongs to: block0 increases, so a
// binary search (uniform over the block, kernel arguments only) finds the
// last j with block0[j] <= b.
__device__ __forceinline__ int layer_of(const int* block0, int nl, int b) {
  int lo = 0, hi = nl - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (b >= block0[mid]) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// B = M + G in place, the block's partial sum of B^2, and (wx) the skip
// branch's X = xdecay X - coef G in the same pass over G (xdecay = 1 - eta
// weight_decay; 1 without weight decay, where the product is exact).  WXM:
// 0 = no X update, 1 = with it, 2 = as the control word predicts (uniform
// over the launch).
template <bool BF16, int WXM>
__global__ __launch_bounds__(NTHREADS) void k_form_buffer(FormArgs a) {
  const bool wx = WXM == 1 || (WXM == 2 && a.ctl->spec_next != 0);
  const int l = layer_of(a.block0, a.nl, blockIdx.x);
  const int lb = blockIdx.x - a.block0[l];   // block within the layer
  float* __restrict__ M = a.M[l];
  const void* __restrict__ G = a.G[l];
  float* __restrict__ X = a.X[l];
  const float c = a.coef[l];
  const float d = a.xdecay[l];
  const long long base = static_cast<long long>(lb) * FORM_CHUNK;
  const long long end = min(base + FORM_CHUNK, a.numel[l]);
  double acc = 0.0;
  if (end - base == FORM_CHUNK) {
    float4 m[VPT], g[VPT], x[VPT];
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const long long i = base + 4LL * (threadIdx.x + v * NTHREADS);
      m[v] = ld_nt(M + i);
      g[v] = load_g4<BF16>(G, i);
      if (wx) x[v] = ld_nt(X + i);
    }
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const long long i = base + 4LL * (threadIdx.x + v * NTHREADS);
      float4 b;
      b.x = m[v].x + g[v].x; b.y = m[v].y + g[v].y;
      b.z = m[v].z + g[v].z; b.w = m[v].w + g[v].w;
      st_nt(M + i, b);
      acc += sq(b.x); acc += sq(b.y); acc += sq(b.z); acc += sq(b.w);
      if (wx) {
        float4 y;
        y.x = fmaf(-c, g[v].x, d * x[v].x); y.y = fmaf(-c, g[v].y, d * x[v].y);
        y.z = fmaf(-c, g[v].z, d * x[v].z); y.w = fmaf(-c, g[v].w, d * x[v].w);
        st_nt(X + i, y);
      }
    }
  } else {
    for (long long i = base + 4LL * threadIdx.x; i < end; i += 4LL * NTHREADS) {
      if (i + 3 < end) {
        const float4 mv = *reinterpret_cast<const float4*>(M + i);
        const float4 gv = load_g4<BF16>(G, i);
        float4 b;
        b.x = mv.x + gv.x; b.y = mv.y + gv.y; b.z = mv.z + gv.z; b.w = mv.w + gv.w;
        *reinterpret_cast<float4*>(M + i) = b;
        acc += sq(b.x); acc += sq(b.y); acc += sq(b.z); acc += sq(b.w);
        if (wx) {
          const float4 xv = *reinterpret_cast<const float4*>(X + i);
          float4 y;
          y.x = fmaf(-c, gv.x, d * xv.x); y.y = fmaf(-c, gv.y, d * xv.y);
          y.z = fmaf(-c, gv.z, d * xv.z); y.w = fmaf(-c, gv.w, d * xv.w);
          *reinterpret_cast<float4*>(X + i) = y;
        }
      } else {
        for (long long j = i; j < end; ++j) {
          const float gj = load_g1<BF16>(G, j);
          const float b = M[j] + gj;
          M[j] = b;
          acc += sq(b);
          if (wx) X[j] = fmaf(-c, gj, d * X[j]);
        }
      }
    }
  }
  const double s = block_sum(acc);
  if (threadIdx.x == 0) a.part[l][lb] = s;
}

template <bool BF16>
__global__ __launch_bounds__(NTHREADS) void k_local_update(LocalArgs a) {
  if (a.ctl != nullptr && (a.ctl->flag != 0 || a.ctl->spec_cur != 0)) return;
  const int l = layer_of(a.block0, a.nl, blockIdx.x);
  float* __restrict__ X = a.X[l];
  const void* __restrict__ G = a.G[l];
  const float c = a.coef[l];
  const float d = a.xdecay[l];
  const long long base = static_cast<long long>(blockIdx.x - a.block0[l]) * FORM_CHUNK;
  const long long end = min(base + FORM_CHUNK, a.numel[l]);
  if (end - base == FORM_CHUNK) {
    float4 x[VPT], g[VPT];
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const long long i = base + 4LL * (threadIdx.x + v * NTHREADS);
      x[v] = ld_nt(X + i);
      g[v] = load_g4<BF16>(G, i);
    }
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const long long i = base + 4LL * (threadIdx.x + v * NTHREADS);
      float4 y;
      y.x = fmaf(-c, g[v].x, d * x[v].x); y.y = fmaf(-c, g[v].y, d * x[v].y);
      y.z = fmaf(-c, g[v].z, d * x[v].z); y.w = fmaf(-c, g[v].w, d * x[v].w);
      st_nt(X + i, y);
    }
  } else {
    for (long long i = base + 4LL * threadIdx.x; i < end; i += 4LL * NTHREADS) {
      if (i + 3 < end) {
        const float4 xv = *reinterpret_cast<const float4*>(X + i);
        const float4 gv = load_g4<BF16>(G, i);
        float4 y;
        y.x = fmaf(-c, gv.x, d * xv.x); y.y = fmaf(-c, gv.y, d * xv.y);
        y.z = fmaf(-c, gv.z, d * xv.z); y.w = fmaf(-c, gv.w, d * xv.w);
        *reinterpret_cast<float4*>(X + i) = y;
      } else {
        for (long long j = i; j < end; ++j) X[j] = fmaf(-c, load_g1<BF16>(G, j), d * X[j]);
      }
    }
  }
}

// One block per layer reduces that layer's partials in a fixed order (strided
// per thread, then the block tree), forms RMMC and replaces prev_norm.  The
// last block to finish (device-scope counter, which wraps back to zero) takes
// the max over layers; max is order-free, and any NaN makes the max NaN (and
// NaN > tau is false).
constexpr int GATE_THREADS = 256;

__device__ __forceinline__ double load_coherent(const double* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(GATE_THREADS) void k_gate(GateArgs a) {
  __shared__ int last;
  __shared__ double wmax[GATE_THREADS / 64];
  __shared__ int wflags[GATE_THREADS / 64];
  const int l = blockIdx.x;
  const double* p = a.parts + static_cast<long long>(l) * a.nparts_stride;
  const int np = a.nparts[l];
  double s = 0.0;
  for (int i = threadIdx.x; i < np; i += GATE_THREADS) s += p[i];
  s = block_sum(s);
  double* out_rm = reinterpret_cast<double*>(a.out + 1);
  if (threadIdx.x == 0) {
    const double nb = sqrt(s);
    double* prev = a.prev[l];
    const double pv = *prev;
    out_rm[l] = fabs(nb - pv) / (pv + a.eps);
    a.norms[l] = nb;
    *prev = nb;
    __threadfence();
    last = atomicInc(a.counter, static_cast<unsigned>(a.L - 1)) == static_cast<unsigned>(a.L - 1);
  }
  __syncthreads();
  if (!last) return;
  __threadfence();
  double g = -INFINITY;
  int flags = 0;   // bit 0: a NaN RMMC; bit 1: a non-finite norm
  for (int i = threadIdx.x; i < a.L; i += GATE_THREADS) {
    const double v = load_coherent(out_rm + i);
    if (isnan(v)) flags |= 1;
    else g = fmax(g, v);
    if (!isfinite(load_coherent(a.norms + i))) flags |= 2;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    g = fmax(g, __shfl_xor(g, o, 64));
    flags |= __shfl_xor(flags, o, 64);
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { wmax[w] = g; wflags[w] = flags; }
  __syncthreads();
  if (threadIdx.x == 0) {
#pragma unroll
    for (int i = 0; i < GATE_THREADS / 64; ++i) { g = fmax(g, wmax[i]); flags |= wflags[i]; }
    if (flags & 1) g = NAN;
    // the branch and the speculation this step used, for the kernels after
    // the gate, and the prediction for the next step (its previous branch)
    const int flag = a.fixed_flag >= 0 ? a.fixed_flag : ((g > a.tau) ? 1 : 0);
    const int spec = a.spec_mode == 2 ? a.ctl->spec_next : a.spec_mode;
    a.ctl->flag = flag;
    a.ctl->spec_cur = spec;
    a.ctl->spec_next = flag ? 0 : 1;
    a.out->g = g;
    a.out->flag = flag;
    a.out->nonfinite = (flags & 2) ? 1 : 0;
    a.out->spec = spec;
    if (a.host_out) {
      a.host_out->g = g;
      a.host_out->flag = flag;
      a.host_out->nonfinite = (flags & 2) ? 1 : 0;
      a.host_out->spec = spec;
    }
  }
  if (!a.host_out) return;
  // the host copy: every value first, then (once all of them are visible at
  // system scope) the step's sequence number, which the host polls
  double* host_rm = reinterpret_cast<double*>(a.host_out + 1);
  for (int i = threadIdx.x; i < a.L; i += GATE_THREADS) host_rm[i] = load_coherent(out_rm + i);
  __threadfence_system();
  __syncthreads();
  if (threadIdx.x == 0) *reinterpret_cast<volatile unsigned long long*>(a.host_seq) = a.seq;
}

}  // namespace

hipError_t launch_form_buffer(const FormArgs& a, bool g_bf16, int spec_mode, hipStream_t s) {
  if (a.nl <= 0 || a.nl > MAXS || a.block0[a.nl] <= 0) return a.nl == 0 ? hipSuccess : hipErrorInvalidValue;
  if (spec_mode < 0 || spec_mode > 2 || (spec_mode == 2 && !a.ctl)) return hipErrorInvalidValue;
  const dim3 grid(a.block0[a.nl]), block(NTHREADS);
  if (g_bf16) {
    if (spec_mode == 1) hipLaunchKernelGGL((k_form_buffer<true, 1>), grid, block, 0, s, a);
    else if (spec_mode == 2) hipLaunchKernelGGL((k_form_buffer<true, 2>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((k_form_buffer<true, 0>), grid, block, 0, s, a);
  } else {
    if (spec_mode == 1) hipLaunchKernelGGL((k_form_buffer<false, 1>), grid, block, 0, s, a);
    else if (spec_mode == 2) hipLaunchKernelGGL((k_form_buffer<false, 2>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((k_form_buffer<false, 0>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_local_update(const LocalArgs& a, bool g_bf16, hipStream_t s) {
  if (a.nl <= 0 || a.nl > MAXS || a.block0[a.nl] <= 0) return a.nl == 0 ? hipSuccess : hipErrorInvalidValue;
  const dim3 grid(a.block0[a.nl]), block(NTHREADS);
  if (g_bf16) hipLaunchKernelGGL(k_local_update<true>, grid, block, 0, s, a);
  else hipLaunchKernelGGL(k_local_update<false>, grid, block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gate(const GateArgs& a, hipStream_t s) {
  if (a.L <= 0 || !a.counter || !a.norms || !a.out || !a.ctl || (a.host_out && !a.host_seq) ||
      a.spec_mode < 0 || a.spec_mode > 2)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_gate, dim3(a.L), dim3(GATE_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace cd
