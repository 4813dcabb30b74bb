// Row-wise (off-refresh) step of Periodic Row-wise Muon on gfx950.
//
// For every matrix: momentum update, RowNorm of the oriented momentum scaled
// by gamma, shape scale, decoupled weight decay and parameter write -- eq.
// (periodic-direction) with rho_t = 0, eq. (rownorm), Alg. 1 -- fused so that
// every element of G, M and W crosses HBM once (14 bytes per element for bf16
// W and G with fp32 M).
//
// Wide and square matrices (m <= n): an oriented row is a stored row.  One row
// is owned by TPR threads that keep its elements in registers across the
// sum-of-squares reduction (wave64 shuffles, then LDS across waves), so M is
// read once and written once.
//
// Tall matrices (m > n): an oriented row is a stored column, whose norm needs
// every stored row.  As in the sharded RowNorm of the paper's distributed
// execution (eq. sharded-tall-rownorm, App. "Correctness of sharded RowNorm"),
// row blocks play the role of the shards: pass 1 updates M and writes per-
// block column sums of squares, a finalize step reduces them in a fixed order
// and clamps after the square root, pass 2 writes W.
//
// All reductions have a fixed order, so results are bitwise reproducible.
#include "prm_device.h"

namespace prm {

template <DType D> struct Store;
template <> struct Store<F32> { using T = float; };
template <> struct Store<BF16> { using T = uint16_t; };

// Sum over the TPR threads that own one row.  All NT threads must call it.
template <int NT, int TPR>
__device__ __forceinline__ float row_sum(float v, float* red) {
  v = wave_sum(v);
  if constexpr (TPR == 64) {
    return v;
  } else {
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[w] = v;
    __syncthreads();
    constexpr int WPR = TPR / 64;
    const int first = (threadIdx.x / TPR) * WPR;
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < WPR; ++i) t += red[first + i];
    return t;
  }
}

// ---------------------------------------------------------------------------
// Wide rows in registers: NT threads per block, TPR threads per row, each
// thread owning NCH chunks of 8 consecutive elements.  Requires n % 8 == 0
// and 16-byte aligned rows.
// ---------------------------------------------------------------------------
template <int NT, int TPR, int NCH, DType WD, DType GD>
__global__ __launch_bounds__(NT) void rw_wide_kernel(const MatDesc* __restrict__ md,
                                                     const int32_t* __restrict__ seg_mat,
                                                     const int32_t* __restrict__ seg_start,
                                                     int32_t nseg, RwParams p) {
  using WT = typename Store<WD>::T;
  using GT = typename Store<GD>::T;
  constexpr int RPB = NT / TPR;
  __shared__ float red[NT / 64];

  const int b = blockIdx.x;
  const int seg = find_segment(seg_start, nseg, b);
  const MatDesc& d = md[seg_mat[seg]];
  const int64_t n = d.n;
  const int lt = threadIdx.x % TPR;
  const int64_t row = (int64_t)(b - seg_start[seg]) * RPB + threadIdx.x / TPR;
  const bool row_ok = row < d.m;

  const GT* G = reinterpret_cast<const GT*>(d.G) + row * n;
  float* M = d.M + row * n;
  WT* W = reinterpret_cast<WT*>(d.W) + row * n;

  float g[NCH][8], u[NCH][8], w[NCH][8];
  bool ok[NCH];
#pragma unroll
  for (int it = 0; it < NCH; ++it) {
    const int64_t e = (int64_t)(it * TPR + lt) * 8;
    ok[it] = row_ok && e < n;
    if (ok[it]) {
      VecNT<GT>::load8(G + e, g[it]);
      VecNT<float>::load8(M + e, u[it]);
      VecNT<WT>::load8(W + e, w[it]);
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int it = 0; it < NCH; ++it) {
    if (ok[it]) {
      const int64_t e = (int64_t)(it * TPR + lt) * 8;
#pragma unroll
      for (int k = 0; k < 8; ++k) u[it][k] = p.beta * u[it][k] + p.gcoef * g[it][k];
      VecNT<float>::store8(M + e, u[it]);
      if (p.nesterov) {
#pragma unroll
        for (int k = 0; k < 8; ++k) u[it][k] = g[it][k] + p.beta * u[it][k];
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) ss += u[it][k] * u[it][k];
    }
  }
  ss = row_sum<NT, TPR>(ss, red);
  const float nu = fmaxf(sqrtf(ss), p.eps);
  const float kcoef = p.gamma * d.s * (1.0f / nu);
  float* const Dp = (p.write_d && d.D) ? d.D + row * n : nullptr;
#pragma unroll
  for (int it = 0; it < NCH; ++it) {
    if (ok[it]) {
      const int64_t e = (int64_t)(it * TPR + lt) * 8;
      float dv[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        dv[k] = u[it][k] * kcoef;
        w[it][k] = w[it][k] * p.decay - p.lr * dv[k];
      }
      VecNT<WT>::store8(W + e, w[it]);
      if (Dp) VecNT<float>::store8(Dp + e, dv);
    }
  }
}

// ---------------------------------------------------------------------------
// Any wide row (any length, any alignment): one row per block, two sweeps; the
// second sweep re-reads the momentum this thread has just written.
// ---------------------------------------------------------------------------
template <DType WD, DType GD>
__global__ __launch_bounds__(256) void rw_generic_kernel(const MatDesc* __restrict__ md,
                                                         const int32_t* __restrict__ seg_mat,
                                                         const int32_t* __restrict__ seg_start,
                                                         int32_t nseg, RwParams p) {
  using WT = typename Store<WD>::T;
  using GT = typename Store<GD>::T;
  __shared__ float red[4];
  const int b = blockIdx.x;
  const int seg = find_segment(seg_start, nseg, b);
  const MatDesc& d = md[seg_mat[seg]];
  const int64_t n = d.n;
  const int64_t row = b - seg_start[seg];
  const GT* G = reinterpret_cast<const GT*>(d.G) + row * n;
  float* M = d.M + row * n;
  WT* W = reinterpret_cast<WT*>(d.W) + row * n;
  // a thread sums up to n / 256 squares (2^16 for the longest rows): with
  // compensation (Kahan) the sum stays within a few ulps
  float ss = 0.f, comp = 0.f;
  for (int64_t e = threadIdx.x; e < n; e += 256) {
    const float g = VecNT<GT>::load1(G + e);
    float m = p.beta * Vec<float>::load1(M + e) + p.gcoef * g;
    Vec<float>::store1(M + e, m);
    const float u = p.nesterov ? g + p.beta * m : m;
    const float y = u * u - comp;
    const float t = ss + y;
    comp = (t - ss) - y;
    ss = t;
  }
  ss = block_sum<256>(ss, red);
  const float nu = fmaxf(sqrtf(ss), p.eps);
  const float kcoef = p.gamma * d.s * (1.0f / nu);
  float* const Dp = (p.write_d && d.D) ? d.D + row * n : nullptr;
  for (int64_t e = threadIdx.x; e < n; e += 256) {
    const float m = Vec<float>::load1(M + e);
    const float u = p.nesterov ? VecNT<GT>::load1(G + e) + p.beta * m : m;
    const float dv = u * kcoef;
    VecNT<WT>::store1(W + e, VecNT<WT>::load1(W + e) * p.decay - p.lr * dv);
    if (Dp) Vec<float>::store1(Dp + e, dv);
  }
}

// ---------------------------------------------------------------------------
// Tall pass 1: momentum update and partial column sums of squares.
//
// n % 4 == 0: one block per tile of kTallRows (32) rows x 256 columns, and
// every thread loads its whole share once: wave w takes rows 8w .. 8w+7 of the
// tile, lane l the 4 columns 4l .. 4l+3, so each load or store instruction
// covers one contiguous 1 KB (fp32) or 512 B (bf16) span of a row.  Grids of
// such one-shot blocks stream HBM ~13% faster than blocks that loop over
// rows.  The four waves' column sums meet in LDS and wave 0 writes the
// tile's partial (fixed order).
// ---------------------------------------------------------------------------
constexpr int kTallRowsPerWave = kTallRows / 4;
static_assert(kTallRows % 4 == 0, "four waves share a tile's rows");

template <DType GD>
__global__ __launch_bounds__(256) void rw_tall_stats_kernel(const MatDesc* __restrict__ md,
                                                            const Item* __restrict__ items,
                                                            RwParams p) {
  using GT = typename Store<GD>::T;
  constexpr int U = kTallRowsPerWave;
  __shared__ float red[4][64][4];
  const Item it = items[blockIdx.x];
  const MatDesc& d = md[it.mat];
  const int64_t n = d.n;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t col = (int64_t)it.tn * 256 + 4 * lane;
  const int64_t r0 = (int64_t)it.tm * kTallRows + w * U;
  const bool ok = col < n;
  const GT* G = reinterpret_cast<const GT*>(d.G);
  float* M = d.M;
  float g[U][4], m[U][4];
#pragma unroll
  for (int q = 0; q < U; ++q) {
    if (ok && r0 + q < d.m) {
      const int64_t off = (r0 + q) * n + col;
      VecNT<GT>::load4(G + off, g[q]);
      VecNT<float>::load4(M + off, m[q]);
    }
  }
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int q = 0; q < U; ++q) {
    if (ok && r0 + q < d.m) {
      const int64_t off = (r0 + q) * n + col;
#pragma unroll
      for (int k = 0; k < 4; ++k) m[q][k] = p.beta * m[q][k] + p.gcoef * g[q][k];
      VecNT<float>::store4(M + off, m[q]);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float u = p.nesterov ? g[q][k] + p.beta * m[q][k] : m[q][k];
        acc[k] += u * u;
      }
    }
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) red[w][lane][k] = acc[k];
  __syncthreads();
  if (w == 0 && ok) {
    float s[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) s[k] = ((red[0][lane][k] + red[1][lane][k]) + red[2][lane][k]) + red[3][lane][k];
    VecNT<float>::store4(d.colpart + (int64_t)it.tm * n + col, s);
  }
}

// n % 4 != 0: one column per thread, 256 columns and kTallRows rows per block.
template <DType GD>
__global__ __launch_bounds__(256) void rw_tall_stats_scalar_kernel(const MatDesc* __restrict__ md,
                                                                   const Item* __restrict__ items,
                                                                   RwParams p) {
  using GT = typename Store<GD>::T;
  const Item it = items[blockIdx.x];
  const MatDesc& d = md[it.mat];
  const int64_t n = d.n;
  const int64_t col = (int64_t)it.tn * 256 + threadIdx.x;
  if (col >= n) return;
  const int64_t r0 = (int64_t)it.tm * kTallRows;
  const int64_t r1 = min(d.m, r0 + kTallRows);
  const GT* G = reinterpret_cast<const GT*>(d.G);
  float* M = d.M;
  float acc = 0.f;
  for (int64_t r = r0; r < r1; ++r) {
    const int64_t off = r * n + col;
    const float g = VecNT<GT>::load1(G + off);
    const float m = p.beta * Vec<float>::load1(M + off) + p.gcoef * g;
    Vec<float>::store1(M + off, m);
    const float u = p.nesterov ? g + p.beta * m : m;
    acc += u * u;
  }
  Vec<float>::store1(d.colpart + (int64_t)it.tm * n + col, acc);
}

// Column norms of a tall matrix: fixed-order sum over row blocks, square root,
// then the clamp at eps (Alg. 2, row-wise branch: the clamp follows the square root).
__global__ __launch_bounds__(256) void rw_tall_finalize_kernel(const MatDesc* __restrict__ md,
                                                               const Item* __restrict__ items,
                                                               RwParams p) {
  const Item it = items[blockIdx.x];
  const MatDesc& d = md[it.mat];
  const int64_t col = (int64_t)it.tn * 256 + threadIdx.x;
  if (col >= d.n) return;
  // the loads of 16 row blocks are issued together and summed pairwise; the
  // group sums are accumulated with compensation (Kahan), so the error stays
  // at a few ulps however many row blocks a tall matrix has (fixed order)
  const float* cp = d.colpart + col;
  float s = 0.f, comp = 0.f;
  auto add = [&](float x) {
    const float y = x - comp;
    const float t = s + y;
    comp = (t - s) - y;
    s = t;
  };
  int rb = 0;
  for (; rb + 16 <= d.nrb; rb += 16) {
    float v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) v[k] = Vec<float>::load1(cp + (int64_t)(rb + k) * d.n);
#pragma unroll
    for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
      for (int k = 0; k < w; ++k) v[k] += v[k + w];
    add(v[0]);
  }
  for (; rb < d.nrb; ++rb) add(Vec<float>::load1(cp + (int64_t)rb * d.n));
  Vec<float>::store1(d.colinv + col, 1.0f / fmaxf(sqrtf(s), p.eps));
}

// Tall pass 2: D = gamma * s * U / nu_col and the parameter write, on the
// same one-shot tiles as pass 1 (n % 4 == 0).
template <DType WD, DType GD, bool NEST>
__global__ __launch_bounds__(256) void rw_tall_apply_kernel(const MatDesc* __restrict__ md,
                                                            const Item* __restrict__ items,
                                                            RwParams p) {
  using WT = typename Store<WD>::T;
  using GT = typename Store<GD>::T;
  constexpr int U = kTallRowsPerWave;
  const Item it = items[blockIdx.x];
  const MatDesc& d = md[it.mat];
  const int64_t n = d.n;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t col = (int64_t)it.tn * 256 + 4 * lane;
  if (col >= n) return;
  const int64_t r0 = (int64_t)it.tm * kTallRows + w * U;
  const GT* G = reinterpret_cast<const GT*>(d.G);
  const float* M = d.M;
  WT* W = reinterpret_cast<WT*>(d.W);
  float m[U][4], wv[U][4], g[NEST ? U : 1][4];
#pragma unroll
  for (int q = 0; q < U; ++q) {
    if (r0 + q < d.m) {
      const int64_t off = (r0 + q) * n + col;
      VecNT<float>::load4(M + off, m[q]);
      VecNT<WT>::load4(W + off, wv[q]);
      if constexpr (NEST) VecNT<GT>::load4(G + off, g[q]);
    }
  }
  float kc[4];
  Vec<float>::load4(d.colinv + col, kc);  // shared by every tile of these columns: cached
  const float gs = p.gamma * d.s;
#pragma unroll
  for (int k = 0; k < 4; ++k) kc[k] *= gs;
#pragma unroll
  for (int q = 0; q < U; ++q) {
    if (r0 + q < d.m) {
      const int64_t off = (r0 + q) * n + col;
      float dv[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        float u = m[q][k];
        if constexpr (NEST) u = g[q][k] + p.beta * m[q][k];
        dv[k] = u * kc[k];
        wv[q][k] = wv[q][k] * p.decay - p.lr * dv[k];
      }
      VecNT<WT>::store4(W + off, wv[q]);
      if (p.write_d && d.D) VecNT<float>::store4(d.D + off, dv);
    }
  }
}

// n % 4 != 0: one column per thread.
template <DType WD, DType GD>
__global__ __launch_bounds__(256) void rw_tall_apply_scalar_kernel(const MatDesc* __restrict__ md,
                                                                   const Item* __restrict__ items,
                                                                   RwParams p) {
  using WT = typename Store<WD>::T;
  using GT = typename Store<GD>::T;
  const Item it = items[blockIdx.x];
  const MatDesc& d = md[it.mat];
  const int64_t n = d.n;
  const int64_t col = (int64_t)it.tn * 256 + threadIdx.x;
  if (col >= n) return;
  const int64_t r0 = (int64_t)it.tm * kTallRows;
  const int64_t r1 = min(d.m, r0 + kTallRows);
  const GT* G = reinterpret_cast<const GT*>(d.G);
  WT* W = reinterpret_cast<WT*>(d.W);
  const float kc = p.gamma * d.s * Vec<float>::load1(d.colinv + col);
  for (int64_t r = r0; r < r1; ++r) {
    const int64_t off = r * n + col;
    const float m = Vec<float>::load1(d.M + off);
    const float u = p.nesterov ? VecNT<GT>::load1(G + off) + p.beta * m : m;
    const float dv = u * kc;
    VecNT<WT>::store1(W + off, VecNT<WT>::load1(W + off) * p.decay - p.lr * dv);
    if (p.write_d && d.D) Vec<float>::store1(d.D + off, dv);
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <int NT, int TPR, DType WD, DType GD>
static hipError_t wide_nch(int nch, const MatDesc* md, const int32_t* sm, const int32_t* ss,
                           int32_t nseg, int32_t nb, const RwParams& p, hipStream_t s) {
  dim3 g(nb), b(NT);
  switch (nch) {
    case 1: rw_wide_kernel<NT, TPR, 1, WD, GD><<<g, b, 0, s>>>(md, sm, ss, nseg, p); break;
    case 2: rw_wide_kernel<NT, TPR, 2, WD, GD><<<g, b, 0, s>>>(md, sm, ss, nseg, p); break;
    case 3: rw_wide_kernel<NT, TPR, 3, WD, GD><<<g, b, 0, s>>>(md, sm, ss, nseg, p); break;
    case 4: rw_wide_kernel<NT, TPR, 4, WD, GD><<<g, b, 0, s>>>(md, sm, ss, nseg, p); break;
    case 5: rw_wide_kernel<NT, TPR, 5, WD, GD><<<g, b, 0, s>>>(md, sm, ss, nseg, p); break;
    case 6: rw_wide_kernel<NT, TPR, 6, WD, GD><<<g, b, 0, s>>>(md, sm, ss, nseg, p); break;
    case 7: rw_wide_kernel<NT, TPR, 7, WD, GD><<<g, b, 0, s>>>(md, sm, ss, nseg, p); break;
    case 8: rw_wide_kernel<NT, TPR, 8, WD, GD><<<g, b, 0, s>>>(md, sm, ss, nseg, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <DType WD, DType GD>
static hipError_t wide_tpr(int tpr, int nch, const MatDesc* md, const int32_t* sm,
                           const int32_t* ss, int32_t nseg, int32_t nb, const RwParams& p,
                           hipStream_t s) {
  switch (tpr) {
    case 64: return wide_nch<256, 64, WD, GD>(nch, md, sm, ss, nseg, nb, p, s);
    case 256: return wide_nch<256, 256, WD, GD>(nch, md, sm, ss, nseg, nb, p, s);
    case 512: return wide_nch<512, 512, WD, GD>(nch, md, sm, ss, nseg, nb, p, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_rw_wide(int tpr, int nch, DType wt, DType gt, const MatDesc* md,
                          const int32_t* seg_mat, const int32_t* seg_start, int32_t nseg,
                          int32_t nblocks, const RwParams& p, hipStream_t s) {
  if (nblocks <= 0) return hipSuccess;
  if (wt == BF16 && gt == BF16) return wide_tpr<BF16, BF16>(tpr, nch, md, seg_mat, seg_start, nseg, nblocks, p, s);
  if (wt == BF16 && gt == F32) return wide_tpr<BF16, F32>(tpr, nch, md, seg_mat, seg_start, nseg, nblocks, p, s);
  if (wt == F32 && gt == BF16) return wide_tpr<F32, BF16>(tpr, nch, md, seg_mat, seg_start, nseg, nblocks, p, s);
  return wide_tpr<F32, F32>(tpr, nch, md, seg_mat, seg_start, nseg, nblocks, p, s);
}

hipError_t launch_rw_generic(DType wt, DType gt, const MatDesc* md, const int32_t* rows_mat,
                             const int32_t* rows_start, int32_t nseg, int32_t nrows_total,
                             const RwParams& p, hipStream_t s) {
  if (nrows_total <= 0) return hipSuccess;
  dim3 g(nrows_total), b(256);
  if (wt == BF16 && gt == BF16) rw_generic_kernel<BF16, BF16><<<g, b, 0, s>>>(md, rows_mat, rows_start, nseg, p);
  else if (wt == BF16) rw_generic_kernel<BF16, F32><<<g, b, 0, s>>>(md, rows_mat, rows_start, nseg, p);
  else if (gt == BF16) rw_generic_kernel<F32, BF16><<<g, b, 0, s>>>(md, rows_mat, rows_start, nseg, p);
  else rw_generic_kernel<F32, F32><<<g, b, 0, s>>>(md, rows_mat, rows_start, nseg, p);
  return hipGetLastError();
}

hipError_t launch_rw_tall_stats(int vec, DType gt, const MatDesc* md, const Item* items,
                                int32_t nitems, const RwParams& p, hipStream_t s) {
  if (nitems <= 0) return hipSuccess;
  dim3 g(nitems), b(256);
  if (vec == 4) {
    if (gt == BF16) rw_tall_stats_kernel<BF16><<<g, b, 0, s>>>(md, items, p);
    else rw_tall_stats_kernel<F32><<<g, b, 0, s>>>(md, items, p);
  } else {
    if (gt == BF16) rw_tall_stats_scalar_kernel<BF16><<<g, b, 0, s>>>(md, items, p);
    else rw_tall_stats_scalar_kernel<F32><<<g, b, 0, s>>>(md, items, p);
  }
  return hipGetLastError();
}

hipError_t launch_rw_tall_finalize(const MatDesc* md, const Item* items, int32_t nitems,
                                   const RwParams& p, hipStream_t s) {
  if (nitems <= 0) return hipSuccess;
  rw_tall_finalize_kernel<<<dim3(nitems), dim3(256), 0, s>>>(md, items, p);
  return hipGetLastError();
}

template <bool NEST>
static hipError_t tall_apply_tiles(DType wt, DType gt, const MatDesc* md, const Item* items,
                                   int32_t nitems, const RwParams& p, hipStream_t s) {
  dim3 g(nitems), b(256);
  if (wt == BF16 && gt == BF16) rw_tall_apply_kernel<BF16, BF16, NEST><<<g, b, 0, s>>>(md, items, p);
  else if (wt == BF16) rw_tall_apply_kernel<BF16, F32, NEST><<<g, b, 0, s>>>(md, items, p);
  else if (gt == BF16) rw_tall_apply_kernel<F32, BF16, NEST><<<g, b, 0, s>>>(md, items, p);
  else rw_tall_apply_kernel<F32, F32, NEST><<<g, b, 0, s>>>(md, items, p);
  return hipGetLastError();
}

hipError_t launch_rw_tall_apply(int vec, DType wt, DType gt, const MatDesc* md,
                                const Item* items, int32_t nitems, const RwParams& p,
                                hipStream_t s) {
  if (nitems <= 0) return hipSuccess;
  if (vec == 4)
    return p.nesterov ? tall_apply_tiles<true>(wt, gt, md, items, nitems, p, s)
                      : tall_apply_tiles<false>(wt, gt, md, items, nitems, p, s);
  dim3 g(nitems), b(256);
  if (wt == BF16 && gt == BF16) rw_tall_apply_scalar_kernel<BF16, BF16><<<g, b, 0, s>>>(md, items, p);
  else if (wt == BF16) rw_tall_apply_scalar_kernel<BF16, F32><<<g, b, 0, s>>>(md, items, p);
  else if (gt == BF16) rw_tall_apply_scalar_kernel<F32, BF16><<<g, b, 0, s>>>(md, items, p);
  else rw_tall_apply_scalar_kernel<F32, F32><<<g, b, 0, s>>>(md, items, p);
  return hipGetLastError();
}

}  // namespace prm
