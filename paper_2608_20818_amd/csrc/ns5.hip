// NS5 refresh step of Periodic Row-wise Muon on gfx950.
//
// Per matrix (oriented X in R^{r x c}, r <= c), eq. (app-ns-recurrence):
//   G_j = X_j X_j^T;   B_j = b G_j + c G_j^2;   X_{j+1} = a X_j + B_j X_j
// five times from X_0 = U~ / (||U~||_F + eps_ns), then the parameter write of
// eq. (periodic-direction) with the oriented result mapped back.
//
// Kernels, all batched over the matrices of a workspace chunk through work
// item lists (matrix, tile row, tile column):
//  * ns_prologue: momentum update, per-tile sum of squares, bf16(U) written
//    both in the oriented layout X (r x c) and transposed XT (c x r), through
//    an LDS tile transpose.  The Frobenius scale is not applied here: NS5 is
//    homogeneous, so alpha = 1/(||U||+eps) is folded into the first Gram
//    (alpha^2) and the first apply (alpha) epilogues.
//  * ns_alpha: fixed-order reduction of the tile sums into alpha.
//  * ns_gemm: C = P Q^T on bf16 operands with fp32 MFMA accumulation
//    (v_mfma_f32_32x32x16_bf16), 256 x 256 tiles, BK = 64, LDS double buffer
//    with an XOR swizzle.  Every product of the iteration has this NT form:
//      Gram   A   = X X^T              (upper tiles only, mirrored)
//      square A^2 = A A^T              (A is symmetric; upper tiles, mirrored)
//      apply  B X = B (XT)^T           (XT is the transposed copy of X)
//    The diagonals of A and B are the large entries, so they are carried in
//    fp32 and only the off-diagonal parts Ao, Bo are rounded to bf16 for the
//    next product:  A^2 = dA^2 + dA Ao + Ao dA + Ao Ao  and
//    X' = (a I + dB) X + Bo X, with the diagonal products applied in the
//    epilogues.  Epilogues also fold alpha, and at the last iteration perform
//    the parameter write W <- (1 - eta lambda) W - eta s O^{-1}(X_5).
// The workspace is padded to whole tiles and the padding stays exactly zero
// through every iteration, so the GEMMs need no bounds checks.
#include "prm_device.h"

namespace prm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

template <DType D> struct NsStore;
template <> struct NsStore<F32> { using T = float; };
template <> struct NsStore<BF16> { using T = uint16_t; };

// ---------------------------------------------------------------------------
// prologue
// ---------------------------------------------------------------------------
template <DType GD>
__global__ __launch_bounds__(256) void ns_prologue_kernel(const MatDesc* __restrict__ md,
                                                          const Item* __restrict__ items,
                                                          NsParams p) {
  using GT = typename NsStore<GD>::T;
  constexpr int T = kPrologueTile;  // 64
  __shared__ uint16_t tile[T][T + 4];
  __shared__ float red[4];
  const Item it = items[blockIdx.x];
  const MatDesc& d = md[it.mat];
  const int64_t m = d.m, n = d.n;
  // natural = stored orientation (X for wide, XT for tall); other = transposed
  uint16_t* nat = d.tall ? d.XT : d.X;
  uint16_t* tra = d.tall ? d.X : d.XT;
  const int64_t ldn = d.tall ? d.rp : d.cp;
  const int64_t ldt = d.tall ? d.cp : d.rp;
  const int64_t R0 = (int64_t)it.tm * T, C0 = (int64_t)it.tn * T;
  const int tc = (threadIdx.x & 15) * 4;
  const int tr = threadIdx.x >> 4;
  const GT* G = reinterpret_cast<const GT*>(d.G);
  float* M = d.M;
  const bool vec = (n & 3) == 0;
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = tr + 16 * i;
    const int64_t row = R0 + r, col = C0 + tc;
    float u[4] = {0.f, 0.f, 0.f, 0.f};
    if (row < m) {
      if (vec && col + 3 < n) {
        float g[4], mm[4];
        Vec<GT>::load4(G + row * n + col, g);
        Vec<float>::load4(M + row * n + col, mm);
#pragma unroll
        for (int k = 0; k < 4; ++k) mm[k] = p.beta * mm[k] + p.gcoef * g[k];
        Vec<float>::store4(M + row * n + col, mm);
#pragma unroll
        for (int k = 0; k < 4; ++k) u[k] = p.nesterov ? g[k] + p.beta * mm[k] : mm[k];
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (col + k < n) {
            const float g = Vec<GT>::load1(G + row * n + col + k);
            const float mm = p.beta * M[row * n + col + k] + p.gcoef * g;
            M[row * n + col + k] = mm;
            u[k] = p.nesterov ? g + p.beta * mm : mm;
          }
        }
      }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) ss += u[k] * u[k];
    const uint32_t h0 = f2bf(u[0]), h1 = f2bf(u[1]), h2 = f2bf(u[2]), h3 = f2bf(u[3]);
    *reinterpret_cast<uint2*>(nat + row * ldn + col) = make_uint2(h0 | (h1 << 16), h2 | (h3 << 16));
    tile[r][tc + 0] = (uint16_t)h0;
    tile[r][tc + 1] = (uint16_t)h1;
    tile[r][tc + 2] = (uint16_t)h2;
    tile[r][tc + 3] = (uint16_t)h3;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int j = tr + 16 * i;  // tile column -> transposed row
    const uint32_t v0 = tile[tc + 0][j], v1 = tile[tc + 1][j], v2 = tile[tc + 2][j],
                   v3 = tile[tc + 3][j];
    *reinterpret_cast<uint2*>(tra + (C0 + j) * ldt + R0 + tc) =
        make_uint2(v0 | (v1 << 16), v2 | (v3 << 16));
  }
  ss = block_sum<256>(ss, red);
  if (threadIdx.x == 0) d.partial[(int64_t)it.tm * d.ptiles_n + it.tn] = ss;
}

__global__ __launch_bounds__(256) void ns_alpha_kernel(const MatDesc* __restrict__ md,
                                                       const int32_t* __restrict__ mats,
                                                       NsParams p) {
  __shared__ float red[4];
  const MatDesc& d = md[mats[blockIdx.x]];
  const int nt = d.ptiles_m * d.ptiles_n;
  float s = 0.f;
  for (int i = threadIdx.x; i < nt; i += 256) s += d.partial[i];
  s = block_sum<256>(s, red);
  if (threadIdx.x == 0) *d.alpha = 1.0f / (sqrtf(s) + p.eps_ns);
}

// ---------------------------------------------------------------------------
// batched NT GEMM with fused NS5 epilogues
//
// Work-group tile 256 x 256, four waves in a 2 x 2 grid, each wave owning a
// 128 x 128 block as 4 x 4 MFMA 32x32x16 accumulators (256 fp32 per lane).
// K advances in stages of 64: global loads of stage k+1 are issued into
// registers before stage k is computed from LDS, then written to the other
// LDS buffer.  Per stage and wave: 64 MFMAs against 32 fragment reads.
// ---------------------------------------------------------------------------
namespace gemm {
constexpr int BM = kNsTile, BN = kNsTile, BK = 64;
constexpr int NTHREADS = 256;
constexpr int WM = BM / 2, WN = BN / 2;  // 2 x 2 waves
constexpr int MI = WM / 32, NI = WN / 32;
constexpr int ROW_BYTES = BK * 2;                       // 128 B per tile row
constexpr int A_BYTES = BM * ROW_BYTES;                 // 32 KB
constexpr int STAGE_BYTES = (BM + BN) * ROW_BYTES;      // 64 KB
constexpr int OP_BYTES = 2 * STAGE_BYTES;               // 128 KB
constexpr int HM = BM / 2;                              // epilogue works on half tiles
constexpr int EPI_LD = BN + 8;                          // fp32 words per staged row
constexpr int EPI_BYTES = HM * EPI_LD * 4;              // 132 KB
constexpr int LDS_BYTES = OP_BYTES > EPI_BYTES ? OP_BYTES : EPI_BYTES;
constexpr int LOADS = BM * (BK / 8) / NTHREADS;         // 16-byte chunks per thread per operand

// byte offset of 16-byte chunk `ch` of tile row `r` (XOR swizzle over 8 chunks)
__device__ __forceinline__ int swz(int r, int ch) { return r * ROW_BYTES + ((ch ^ (r & 7)) << 4); }

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(1))) u32x4* gptr4;

// One stage of both operands into registers: chunk i of this thread is tile
// row (thread/8 + 32 i), 16-byte chunk thread%8, at uint4 offset `ko` along K.
__device__ __forceinline__ void stage_load(u32x4 (&ra)[LOADS], u32x4 (&rb)[LOADS], gptr4 pa,
                                           gptr4 pb, int64_t rstep, int64_t ko) {
#pragma unroll
  for (int i = 0; i < LOADS; ++i) {
    ra[i] = pa[i * rstep + ko];
    rb[i] = pb[i * rstep + ko];
  }
}

__device__ __forceinline__ void stage_store(char* stage, const u32x4 (&ra)[LOADS],
                                            const u32x4 (&rb)[LOADS], const int (&soff)[LOADS]) {
#pragma unroll
  for (int i = 0; i < LOADS; ++i) {
    *reinterpret_cast<u32x4*>(stage + soff[i]) = ra[i];
    *reinterpret_cast<u32x4*>(stage + A_BYTES + soff[i]) = rb[i];
  }
}
}  // namespace gemm

template <int KIND, DType WD>
__global__ __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1))) void ns_gemm_kernel(const MatDesc* __restrict__ md,
                                                         const Item* __restrict__ items,
                                                         NsParams p) {
  using namespace gemm;
  using WT = typename NsStore<WD>::T;
  __shared__ __attribute__((aligned(16))) char smem[LDS_BYTES];

  const Item it = items[blockIdx.x];
  const MatDesc& d = md[it.mat];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const bool even = (p.iter & 1) == 0;
  const uint16_t* Xc = even ? d.X : d.Xn;
  const uint16_t* XTc = even ? d.XT : d.XTn;
  uint16_t* Xo = even ? d.Xn : d.X;
  uint16_t* XTo = even ? d.XTn : d.XT;
  const int64_t rp = d.rp, cp = d.cp;

  const uint16_t *P, *Q;
  int64_t ld;
  if constexpr (KIND == GEMM_GRAM) {
    P = Xc; Q = Xc; ld = cp;
  } else if constexpr (KIND == GEMM_POLY) {
    P = d.Ao; Q = d.Ao; ld = rp;
  } else {
    P = d.Bo; Q = XTc; ld = rp;
  }
  const int64_t row0 = (int64_t)it.tm * BM, col0 = (int64_t)it.tn * BN;
  const int nk = (int)(ld / BK);  // the contraction length is the leading dimension
  const uint16_t* Pt = P + row0 * ld;
  const uint16_t* Qt = Q + col0 * ld;

  // Operand loads through the global address space (global_load, not flat_load,
  // so that LDS waits do not also wait for the prefetch in flight).
  // thread -> (tile row, 16-byte chunk) pairs of its LOADS chunks per operand
  const int lrow = tid >> 3, lch = tid & 7;   // rows lrow + 32 i
  gptr4 pa = (gptr4)(Pt + (int64_t)lrow * ld + lch * 8);
  gptr4 pb = (gptr4)(Qt + (int64_t)lrow * ld + lch * 8);
  const int64_t rstep = 32 * ld / 8;          // 32 rows, in uint4 units
  int soff[LOADS];
#pragma unroll
  for (int i = 0; i < LOADS; ++i) soff[i] = swz(lrow + 32 * i, lch);

  u32x4 ra[LOADS], rb[LOADS];

  floatx16 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int arow = wm * WM + (lane & 31), brow = wn * WN + (lane & 31);
  const int khalf = lane >> 5;

  stage_load(ra, rb, pa, pb, rstep, 0);
  stage_store(smem, ra, rb, soff);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    // prefetch the next stage (the last iteration reloads its own stage into
    // the idle buffer: harmless, and it keeps the loop free of branches)
    stage_load(ra, rb, pa, pb, rstep, (int64_t)(kt + 1 < nk ? kt + 1 : kt) * (BK / 8));
    // keep the prefetch at the top of the stage: the scheduler would otherwise
    // sink it next to the LDS writes and expose the whole memory latency
    __builtin_amdgcn_sched_barrier(0);
    const char* a = smem + (kt & 1) * STAGE_BYTES;
    const char* b = a + A_BYTES;
    // fragments of k-step ks are read while the MFMAs of k-step ks-1 run
    bf16x8 a0[MI], b0[NI], a1[MI], b1[NI];
    auto frag = [&](bf16x8 (&af)[MI], bf16x8 (&bf)[NI], int ks) {
      const int ch = ks * 2 + khalf;
#pragma unroll
      for (int i = 0; i < MI; ++i) af[i] = *reinterpret_cast<const bf16x8*>(a + swz(arow + i * 32, ch));
#pragma unroll
      for (int j = 0; j < NI; ++j) bf[j] = *reinterpret_cast<const bf16x8*>(b + swz(brow + j * 32, ch));
    };
    auto mma = [&](const bf16x8 (&af)[MI], const bf16x8 (&bf)[NI]) {
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    };
    static_assert(BK / 16 == 4, "four k-steps per stage");
    frag(a0, b0, 0);
    __builtin_amdgcn_sched_barrier(0);
    frag(a1, b1, 1);
    mma(a0, b0);
    __builtin_amdgcn_sched_barrier(0);
    frag(a0, b0, 2);
    mma(a1, b1);
    __builtin_amdgcn_sched_barrier(0);
    frag(a1, b1, 3);
    mma(a0, b0);
    __builtin_amdgcn_sched_barrier(0);
    mma(a1, b1);
    __builtin_amdgcn_sched_barrier(0);
    stage_store(smem + ((kt + 1) & 1) * STAGE_BYTES, ra, rb, soff);
    __syncthreads();
  }

  const bool sym = (KIND != GEMM_APPLY);
  const bool diag = sym && it.tm == it.tn;
  const bool last = (KIND == GEMM_APPLY) && p.last;
  const float alpha = (p.iter == 0) ? *d.alpha : 1.0f;
  const bool need_t = (sym && !diag) || (KIND == GEMM_APPLY && (!last || d.tall));
  float* T = reinterpret_cast<float*>(smem);

  // Epilogue in two halves of HM rows (the whole fp32 tile does not fit in LDS).
  constexpr int EPR = 8;                    // consecutive elements per thread
  constexpr int TPRW = BN / EPR;            // threads per staged row (32)
  constexpr int RPP = NTHREADS / TPRW;      // rows per pass (8)
  const int ec = (tid % TPRW) * EPR, er = tid / TPRW;
#pragma unroll 1
  for (int h = 0; h < 2; ++h) {
    if (h) __syncthreads();   // previous half fully consumed
    if (wm == h) {
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int r = i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
            const int c = wn * WN + j * 32 + (lane & 31);
            T[r * EPI_LD + c] = acc[i][j][v];
          }
    }
    __syncthreads();
    const int64_t hrow0 = row0 + h * HM;
    // ---- pass A: row-major; final values, natural-layout outputs ----
#pragma unroll 2
    for (int ps = 0; ps < HM / RPP; ++ps) {
      const int r = ps * RPP + er;
      const int64_t gi = hrow0 + r, gj = col0 + ec;
      float v[EPR];
      Vec<float>::load8(T + r * EPI_LD + ec, v);
      if constexpr (KIND == GEMM_GRAM) {
        // A = alpha^2 acc; the diagonal goes to dA (fp32), the rest to Ao (bf16)
        const float s2 = alpha * alpha;
#pragma unroll
        for (int q = 0; q < EPR; ++q) {
          v[q] *= s2;
          if (diag && gi == gj + q) {
            d.dA[gi] = v[q];
            v[q] = 0.f;
          }
        }
        Vec<uint16_t>::store8(d.Ao + gi * rp + gj, v);
      } else if constexpr (KIND == GEMM_POLY) {
        // A^2 = dA^2 + dA Ao + Ao dA + Ao Ao;  B = b A + c A^2
        float ao[EPR], dj[EPR];
        Vec<uint16_t>::load8(d.Ao + gi * rp + gj, ao);
        Vec<float>::load8(d.dA + gj, dj);
        const float di = d.dA[gi];
#pragma unroll
        for (int q = 0; q < EPR; ++q) {
          if (diag && gi == gj + q) {
            d.dB[gi] = p.b * di + p.c * (v[q] + di * di);
            v[q] = 0.f;
          } else {
            v[q] = p.b * ao[q] + p.c * (di * ao[q] + ao[q] * dj[q] + v[q]);
          }
        }
        Vec<uint16_t>::store8(d.Bo + gi * rp + gj, v);
      } else {
        // X' = alpha ((a + dB_i) X + Bo X)
        float x[EPR];
        Vec<uint16_t>::load8(Xc + gi * cp + gj, x);
        const float ai = p.a + d.dB[gi];
#pragma unroll
        for (int q = 0; q < EPR; ++q) v[q] = alpha * (ai * x[q] + v[q]);
        if (!last) {
          Vec<uint16_t>::store8(Xo + gi * cp + gj, v);
        } else if (!d.tall) {
          // oriented (gi, gj) is stored (gi, gj): W is r x c = m x n
          const int64_t n = d.n;
          if (gi < d.m) {
            const float dc = d.s * p.dscale;
            WT* W = reinterpret_cast<WT*>(d.W) + gi * n;
            float* Dp = d.D + gi * n;
            if ((n & 7) == 0 && gj + EPR <= n) {
              float w[EPR], dv[EPR];
              Vec<WT>::load8(W + gj, w);
#pragma unroll
              for (int q = 0; q < EPR; ++q) {
                dv[q] = dc * v[q];
                w[q] = w[q] * p.decay - p.lr * dv[q];
              }
              Vec<WT>::store8(W + gj, w);
              if (p.write_d) Vec<float>::store8(Dp + gj, dv);
            } else {
#pragma unroll
              for (int q = 0; q < EPR; ++q) {
                if (gj + q < n) {
                  const float dv = dc * v[q];
                  Vec<WT>::store1(W + gj + q, Vec<WT>::load1(W + gj + q) * p.decay - p.lr * dv);
                  if (p.write_d) Dp[gj + q] = dv;
                }
              }
            }
          }
        }
      }
      if (need_t) Vec<float>::store8(T + r * EPI_LD + ec, v);  // same thread, same slots
    }
    if (!need_t) continue;
    __syncthreads();
    // ---- pass B: transposed outputs (mirror tiles, XT, tall parameter write) ----
    // thread -> one tile column j, 8 consecutive staged rows per iteration
    const int j = tid;  // BN == NTHREADS
    const int64_t orow = col0 + j;  // transposed row
#pragma unroll 2
    for (int i0 = 0; i0 < HM; i0 += EPR) {
      float v[EPR];
#pragma unroll
      for (int q = 0; q < EPR; ++q) v[q] = T[(i0 + q) * EPI_LD + j];
      const int64_t ocol = hrow0 + i0;  // transposed column start
      if constexpr (KIND == GEMM_GRAM) {
        Vec<uint16_t>::store8(d.Ao + orow * rp + ocol, v);
      } else if constexpr (KIND == GEMM_POLY) {
        Vec<uint16_t>::store8(d.Bo + orow * rp + ocol, v);
      } else {
        if (!last) {
          Vec<uint16_t>::store8(XTo + orow * rp + ocol, v);
        } else {
          // tall: oriented (i, j) is stored (j, i); W is c x r = m x n
          const int64_t n = d.n;
          if (orow < d.m) {
            const float dc = d.s * p.dscale;
            WT* W = reinterpret_cast<WT*>(d.W) + orow * n;
            float* Dp = d.D + orow * n;
            if ((n & 7) == 0 && ocol + EPR <= n) {
              float w[EPR], dv[EPR];
              Vec<WT>::load8(W + ocol, w);
#pragma unroll
              for (int q = 0; q < EPR; ++q) {
                dv[q] = dc * v[q];
                w[q] = w[q] * p.decay - p.lr * dv[q];
              }
              Vec<WT>::store8(W + ocol, w);
              if (p.write_d) Vec<float>::store8(Dp + ocol, dv);
            } else {
#pragma unroll
              for (int q = 0; q < EPR; ++q) {
                if (ocol + q < n) {
                  const float dv = dc * v[q];
                  Vec<WT>::store1(W + ocol + q, Vec<WT>::load1(W + ocol + q) * p.decay - p.lr * dv);
                  if (p.write_d) Dp[ocol + q] = dv;
                }
              }
            }
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_ns_prologue(DType gt, const MatDesc* md, const Item* items, int32_t nitems,
                              const NsParams& p, hipStream_t s) {
  if (nitems <= 0) return hipSuccess;
  if (gt == BF16) ns_prologue_kernel<BF16><<<dim3(nitems), dim3(256), 0, s>>>(md, items, p);
  else ns_prologue_kernel<F32><<<dim3(nitems), dim3(256), 0, s>>>(md, items, p);
  return hipGetLastError();
}

hipError_t launch_ns_alpha(const MatDesc* md, const int32_t* mats, int32_t nmats,
                           const NsParams& p, hipStream_t s) {
  if (nmats <= 0) return hipSuccess;
  ns_alpha_kernel<<<dim3(nmats), dim3(256), 0, s>>>(md, mats, p);
  return hipGetLastError();
}

hipError_t launch_ns_gemm(GemmKind kind, DType wt, const MatDesc* md, const Item* items,
                          int32_t nitems, const NsParams& p, hipStream_t s) {
  if (nitems <= 0) return hipSuccess;
  dim3 g(nitems), b(gemm::NTHREADS);
  switch (kind) {
    case GEMM_GRAM: ns_gemm_kernel<GEMM_GRAM, BF16><<<g, b, 0, s>>>(md, items, p); break;
    case GEMM_POLY: ns_gemm_kernel<GEMM_POLY, BF16><<<g, b, 0, s>>>(md, items, p); break;
    case GEMM_APPLY:
      if (wt == BF16) ns_gemm_kernel<GEMM_APPLY, BF16><<<g, b, 0, s>>>(md, items, p);
      else ns_gemm_kernel<GEMM_APPLY, F32><<<g, b, 0, s>>>(md, items, p);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace prm
