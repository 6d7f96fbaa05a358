// Streaming kernels of the CurvaDion step: buffer formation with the fused
// sum of squares (B = M + G; Algorithm 2, local buffer update, feeding the
// norm of Eq. 1), the local-branch weight update (X -= eta_local G), and the
// gate (fixed-order reduction, RMMC, prev_norm update, max over layers).
//
// These passes are HBM-bound: each thread keeps eight 16-byte loads in flight,
// blocks own fixed 8192-element chunks of one layer, and every reduction runs
// in a fixed order so that the statistic is bit-reproducible run to run.
#include "common.hpp"

namespace cd {
namespace {

// G element loads: fp32, or bf16 widened exactly (bf16 bits are the top half
// of the fp32 bit pattern).
template <bool BF16>
__device__ __forceinline__ float4 load_g4(const void* G, long long i) {
  if constexpr (BF16) {
    const uint2 u = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(G) + i);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
  } else {
    return *reinterpret_cast<const float4*>(static_cast<const float*>(G) + i);
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

constexpr int VPT = FORM_CHUNK / (NTHREADS * 4);   // float4 groups per thread (8)

template <bool BF16>
__global__ __launch_bounds__(NTHREADS) void k_form_buffer(FormArgs a) {
  const int l = blockIdx.y;
  float* __restrict__ M = a.M[l];
  const void* __restrict__ G = a.G[l];
  const long long base = static_cast<long long>(blockIdx.x) * FORM_CHUNK;
  const long long end = min(base + FORM_CHUNK, a.numel);
  double acc = 0.0;
  if (end - base == FORM_CHUNK) {
    float4 m[VPT], g[VPT];
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const long long i = base + 4LL * (threadIdx.x + v * NTHREADS);
      m[v] = *reinterpret_cast<const float4*>(M + i);
      g[v] = load_g4<BF16>(G, i);
    }
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const long long i = base + 4LL * (threadIdx.x + v * NTHREADS);
      float4 b;
      b.x = m[v].x + g[v].x; b.y = m[v].y + g[v].y;
      b.z = m[v].z + g[v].z; b.w = m[v].w + g[v].w;
      *reinterpret_cast<float4*>(M + i) = b;
      acc += sq(b.x); acc += sq(b.y); acc += sq(b.z); acc += sq(b.w);
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
      } else {
        for (long long j = i; j < end; ++j) {
          const float b = M[j] + load_g1<BF16>(G, j);
          M[j] = b;
          acc += sq(b);
        }
      }
    }
  }
  const double s = block_sum(acc);
  if (threadIdx.x == 0) a.part[l][blockIdx.x] = s;
}

template <bool BF16>
__global__ __launch_bounds__(NTHREADS) void k_local_update(LocalArgs a) {
  const int l = blockIdx.y;
  float* __restrict__ X = a.X[l];
  const void* __restrict__ G = a.G[l];
  const float c = a.coef[l];
  const long long base = static_cast<long long>(blockIdx.x) * FORM_CHUNK;
  const long long end = min(base + FORM_CHUNK, a.numel);
  if (end - base == FORM_CHUNK) {
    float4 x[VPT], g[VPT];
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const long long i = base + 4LL * (threadIdx.x + v * NTHREADS);
      x[v] = *reinterpret_cast<const float4*>(X + i);
      g[v] = load_g4<BF16>(G, i);
    }
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const long long i = base + 4LL * (threadIdx.x + v * NTHREADS);
      float4 y;
      y.x = fmaf(-c, g[v].x, x[v].x); y.y = fmaf(-c, g[v].y, x[v].y);
      y.z = fmaf(-c, g[v].z, x[v].z); y.w = fmaf(-c, g[v].w, x[v].w);
      *reinterpret_cast<float4*>(X + i) = y;
    }
  } else {
    for (long long i = base + 4LL * threadIdx.x; i < end; i += 4LL * NTHREADS) {
      if (i + 3 < end) {
        const float4 xv = *reinterpret_cast<const float4*>(X + i);
        const float4 gv = load_g4<BF16>(G, i);
        float4 y;
        y.x = fmaf(-c, gv.x, xv.x); y.y = fmaf(-c, gv.y, xv.y);
        y.z = fmaf(-c, gv.z, xv.z); y.w = fmaf(-c, gv.w, xv.w);
        *reinterpret_cast<float4*>(X + i) = y;
      } else {
        for (long long j = i; j < end; ++j) X[j] = fmaf(-c, load_g1<BF16>(G, j), X[j]);
      }
    }
  }
}

// One block of 16 waves; wave w reduces layers w, w+16, ... with lane-strided
// partial sums and a fixed xor tree, then thread 0 takes the max in layer
// order.  NaN propagates into the max (and NaN > tau is false).
constexpr int GATE_THREADS = 1024;
constexpr int GATE_MAX_LAYERS = 4096;

__global__ __launch_bounds__(GATE_THREADS) void k_gate(GateArgs a) {
  __shared__ double rm[GATE_MAX_LAYERS];
  __shared__ int nonfinite;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (threadIdx.x == 0) nonfinite = 0;
  __syncthreads();
  for (int l = w; l < a.L; l += GATE_THREADS / 64) {
    const double* p = a.parts + static_cast<long long>(l) * a.nparts_stride;
    const int np = a.nparts[l];
    double s = 0.0;
    for (int i = lane; i < np; i += 64) s += p[i];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    if (lane == 0) {
      const double nb = sqrt(s);
      const double prev = *a.prev[l];
      const double v = fabs(nb - prev) / (prev + a.eps);
      *a.prev[l] = nb;
      rm[l] = v;
      if (!isfinite(nb)) atomicOr(&nonfinite, 1);
    }
  }
  __syncthreads();
  double* out_rm = reinterpret_cast<double*>(a.out + 1);
  for (int l = threadIdx.x; l < a.L; l += GATE_THREADS) out_rm[l] = rm[l];
  if (threadIdx.x == 0) {
    double g = -INFINITY;
    bool has_nan = false;
    for (int l = 0; l < a.L; ++l) {
      const double v = rm[l];
      if (isnan(v)) has_nan = true;
      else if (v > g) g = v;
    }
    if (has_nan) g = NAN;
    a.out->g = g;
    a.out->flag = (g > a.tau) ? 1 : 0;
    a.out->nonfinite = nonfinite;
  }
}

}  // namespace

hipError_t launch_form_buffer(const FormArgs& a, int nl, bool g_bf16, hipStream_t s) {
  if (nl <= 0 || a.blocks_per_layer <= 0) return hipSuccess;
  const dim3 grid(a.blocks_per_layer, nl), block(NTHREADS);
  if (g_bf16) hipLaunchKernelGGL(k_form_buffer<true>, grid, block, 0, s, a);
  else hipLaunchKernelGGL(k_form_buffer<false>, grid, block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_local_update(const LocalArgs& a, int nl, bool g_bf16, hipStream_t s) {
  if (nl <= 0 || a.blocks_per_layer <= 0) return hipSuccess;
  const dim3 grid(a.blocks_per_layer, nl), block(NTHREADS);
  if (g_bf16) hipLaunchKernelGGL(k_local_update<true>, grid, block, 0, s, a);
  else hipLaunchKernelGGL(k_local_update<false>, grid, block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gate(const GateArgs& a, hipStream_t s) {
  if (a.L <= 0 || a.L > GATE_MAX_LAYERS) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_gate, dim3(1), dim3(GATE_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace cd
