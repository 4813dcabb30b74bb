// Calibration probes: the sustained bf16 MFMA rate and the HBM stream rates of
// the device, measured with the instructions the hot path uses (MFMA
// 32x32x16 bf16; 16-byte vector loads and stores).  They are not part of the
// optimizer step; bench.py reports the optimizer's rates against these
// measured ceilings beside the spec figures.
#include "prm_internal.h"

namespace prm {

typedef __bf16 pbf16x8 __attribute__((ext_vector_type(8)));
typedef float pfloatx16 __attribute__((ext_vector_type(16)));

// Every wave runs 8 independent accumulator chains, so the MFMA pipe never
// waits on a result; operands stay in registers (no memory traffic).  The
// operands are 4 sets of pseudo-random values in [-1, 1) and consecutive MFMAs
// take different ones, as in a GEMM: the power drawn, and with it the clock
// the power limit allows, depends on how much the operand bits toggle (fixed
// operands run about 10% faster, an optimistic ceiling).
__global__ __launch_bounds__(256) void probe_mfma_kernel(float* sink, unsigned long long* clk, int iters) {
  const int lane = threadIdx.x & 63;
  pbf16x8 a[4], b[4];
  unsigned h = 2654435761u * (unsigned)(lane + 1) + 97u * blockIdx.x;
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      h = h * 1664525u + 1013904223u;
      a[s][e] = (__bf16)((float)((int)(h >> 8) - (1 << 23)) * (1.0f / (1 << 23)));
      h = h * 1664525u + 1013904223u;
      b[s][e] = (__bf16)((float)((int)(h >> 8) - (1 << 23)) * (1.0f / (1 << 23)));
    }
  pfloatx16 c[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int v = 0; v < 16; ++v) c[j][v] = 0.f;
  const unsigned long long t0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(j >> 1) & 3], b[j & 3], c[j], 0, 0, 0);
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += c[j][v];
  sink[blockIdx.x * 256 + threadIdx.x] = s;
  if (threadIdx.x == 0) {
    clk[2 * blockIdx.x] = t1 - t0;      // shader clock cycles
    clk[2 * blockIdx.x + 1] = r1 - r0;  // 100 MHz reference ticks
  }
}

typedef unsigned int pu32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void probe_read_kernel(const pu32x4* __restrict__ x, int64_t n, unsigned* sink) {
  pu32x4 acc = {0u, 0u, 0u, 0u};
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    acc ^= __builtin_nontemporal_load(x + i);
  if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9e3779b9u) sink[0] = 1u;  // keeps the loads
}

__global__ __launch_bounds__(256) void probe_write_kernel(pu32x4* __restrict__ y, int64_t n) {
  const pu32x4 v = {1u, 2u, 3u, 4u};
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    __builtin_nontemporal_store(v, y + i);
}

__global__ __launch_bounds__(256) void probe_copy_kernel(const pu32x4* __restrict__ x, pu32x4* __restrict__ y,
                                                         int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    __builtin_nontemporal_store(__builtin_nontemporal_load(x + i), y + i);
}

// The row-wise step's element traffic: per element a bf16 gradient, an fp32
// momentum and a bf16 weight are read, the momentum and the weight written
// back (8 + 6 bytes).  Pieces of 4 elements: the momentum lives in x (16 bytes
// a piece), gradient and weight share y (8 + 8).  Each thread takes pieces
// p and p + 256 of its block's 512, so every access instruction covers one
// contiguous span per wave; a thread that instead owns 32 contiguous momentum
// bytes, written by two stores issued far apart, leaves half-written lines in
// L2 and runs at about 60% of this rate.
typedef unsigned int pu32x2 __attribute__((ext_vector_type(2)));
__global__ __launch_bounds__(256) void probe_rowwise_kernel(pu32x4* __restrict__ x, pu32x4* __restrict__ y,
                                                            int64_t npieces) {
  pu32x2* G = reinterpret_cast<pu32x2*>(y);
  pu32x2* W = G + npieces;
  const int64_t p0 = (int64_t)blockIdx.x * 512 + threadIdx.x;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int64_t p = p0 + 256 * h;
    if (p < npieces) {
      const pu32x2 g = __builtin_nontemporal_load(G + p);
      pu32x4 m = __builtin_nontemporal_load(x + p);
      pu32x2 w = __builtin_nontemporal_load(W + p);
      m.xy += g;
      m.zw ^= g;
      w += m.xy ^ m.zw;
      __builtin_nontemporal_store(m, x + p);
      __builtin_nontemporal_store(w, W + p);
    }
  }
}

hipError_t launch_probe_mfma(int blocks, float* sink, unsigned long long* clk, int iters, hipStream_t s) {
  probe_mfma_kernel<<<dim3(blocks), dim3(256), 0, s>>>(sink, clk, iters);
  return hipGetLastError();
}

hipError_t launch_probe_stream(int kind, int blocks, const void* x, void* y, int64_t n16, unsigned* sink,
                               hipStream_t s) {
  switch (kind) {
    case 0: probe_read_kernel<<<dim3(blocks), dim3(256), 0, s>>>((const pu32x4*)x, n16, sink); break;
    case 1: probe_write_kernel<<<dim3(blocks), dim3(256), 0, s>>>((pu32x4*)y, n16); break;
    case 2: probe_copy_kernel<<<dim3(blocks), dim3(256), 0, s>>>((const pu32x4*)x, (pu32x4*)y, n16); break;
    default: probe_rowwise_kernel<<<dim3(blocks), dim3(256), 0, s>>>((pu32x4*)x, (pu32x4*)y, n16); break;
  }
  return hipGetLastError();
}

}  // namespace prm
