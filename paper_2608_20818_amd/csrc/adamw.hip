// Fused AdamW over the auxiliary (non-matrix) parameter group: biases, norm
// scales and shifts, embedders.  The paper keeps these on AdamW with
// decoupled weight decay (Sec. 2, Muon setup; App. "Optimizer and Training
// Hyperparameters": LR 1e-4, betas (0.9, 0.95), eps 1e-8, weight decay 0.01).
//
// Per element, in fp32:
//   m <- beta1 m + (1 - beta1) g,  v <- beta2 v + (1 - beta2) g^2
//   p <- (1 - lr wd) p - (lr / (1 - beta1^t)) m / (sqrt(v) / sqrt(1 - beta2^t) + eps)
// which is p - lr (m^ / (sqrt(v^) + eps) + wd p) with the bias-corrected m^, v^.
//
// HBM-bound: 2 x param + grad + 16 bytes per element (22 with bf16 p and g).
// One block per chunk of 2048 elements of one tensor (a one-shot grid over all
// tensors of the group); each thread takes pieces of 4 elements at offsets
// 4x and 1024 + 4x of its chunk, so every load and store instruction covers
// one contiguous span per wave and lines are written whole.
#include "prm_device.h"
#include "prm_internal.h"

namespace prm {

template <DType D> struct AuxStore;
template <> struct AuxStore<F32> { using T = float; };
template <> struct AuxStore<BF16> { using T = uint16_t; };

__device__ __forceinline__ void adamw_update(float& p, float g, float& m, float& v, const AdamwParams& a) {
  m = a.beta1 * m + a.omb1 * g;
  v = a.beta2 * v + a.omb2 * (g * g);
  const float denom = sqrtf(v) * a.inv_sqrt_bc2 + a.eps;
  p = p * a.decay - a.step_size * (m / denom);
}

template <DType PD, DType GD>
__global__ __launch_bounds__(256) void adamw_kernel(const AuxDesc* __restrict__ desc,
                                                    const AuxChunk* __restrict__ chunks, AdamwParams a) {
  using PT = typename AuxStore<PD>::T;
  using GT = typename AuxStore<GD>::T;
  const AuxChunk ch = chunks[blockIdx.x];
  const AuxDesc d = desc[ch.t];
  PT* P = reinterpret_cast<PT*>(d.P);
  const GT* G = reinterpret_cast<const GT*>(d.G);
  float p[2][4], g[2][4], m[2][4], v[2][4];
  bool full[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int64_t e = ch.start + 4 * (threadIdx.x + 256 * h);
    full[h] = e + 4 <= d.n;
    if (full[h]) {
      VecNT<PT>::load4(P + e, p[h]);
      VecNT<GT>::load4(G + e, g[h]);
      VecNT<float>::load4(d.M + e, m[h]);
      VecNT<float>::load4(d.V + e, v[h]);
    }
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int64_t e = ch.start + 4 * (threadIdx.x + 256 * h);
    if (full[h]) {
#pragma unroll
      for (int k = 0; k < 4; ++k) adamw_update(p[h][k], g[h][k], m[h][k], v[h][k], a);
      VecNT<PT>::store4(P + e, p[h]);
      VecNT<float>::store4(d.M + e, m[h]);
      VecNT<float>::store4(d.V + e, v[h]);
    } else {
      // ragged tail of a tensor: at most 3 elements
      for (int64_t i = e; i < d.n; ++i) {
        float pi = VecNT<PT>::load1(P + i), mi = VecNT<float>::load1(d.M + i), vi = VecNT<float>::load1(d.V + i);
        adamw_update(pi, VecNT<GT>::load1(G + i), mi, vi, a);
        VecNT<PT>::store1(P + i, pi);
        VecNT<float>::store1(d.M + i, mi);
        VecNT<float>::store1(d.V + i, vi);
      }
    }
  }
}

hipError_t launch_adamw(DType pt, DType gt, const AuxDesc* desc, const AuxChunk* chunks, int32_t nchunks,
                        const AdamwParams& p, hipStream_t s) {
  if (nchunks <= 0) return hipSuccess;
  const dim3 grid(nchunks), block(256);
  if (pt == BF16 && gt == BF16) adamw_kernel<BF16, BF16><<<grid, block, 0, s>>>(desc, chunks, p);
  else if (pt == BF16) adamw_kernel<BF16, F32><<<grid, block, 0, s>>>(desc, chunks, p);
  else if (gt == BF16) adamw_kernel<F32, BF16><<<grid, block, 0, s>>>(desc, chunks, p);
  else adamw_kernel<F32, F32><<<grid, block, 0, s>>>(desc, chunks, p);
  return hipGetLastError();
}

}  // namespace prm
