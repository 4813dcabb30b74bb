// NS5 refresh step of Periodic Row-wise Muon on gfx950.
//
// Per matrix (oriented X in R^{r x c}, r <= c), eq. (app-ns-recurrence):
//   G_j = X_j X_j^T;   B_j = b G_j + c G_j^2;   X_{j+1} = a X_j + B_j X_j
// five times from X_0 = U~ / (||U~||_F + eps_ns), then the parameter write of
// eq. (periodic-direction) with the oriented result mapped back.
//
// Only the transposed iterate XT = X^T (c x r, row-major) is kept.  Kernels,
// all batched over the matrices of a workspace chunk through work item lists
// (matrix, tile row, tile column):
//  * ns_prologue: momentum update, per-tile sum of squares, bf16(U~^T) written
//    as XT (through an LDS tile transpose for wide matrices).  The Frobenius
//    scale is not applied here: NS5 is homogeneous, so alpha = 1/(||U||+eps) is
//    folded into the first Gram (alpha^2) and the first apply (alpha).
//  * ns_alpha: fixed-order reduction of the tile sums into alpha.
//  * ns_gemm: bf16 MFMA products (v_mfma_f32_32x32x16_bf16) with fp32
//    accumulation on 256 x 256 tiles, K in stages of 64 streamed into a double
//    LDS buffer by direct global-to-LDS loads:
//      Gram   A   = X X^T = XT^T XT    K-major operands ("TN"), read from LDS
//                                      with transposing ds_read_b64_tr_b16;
//                                      upper tiles only, mirrored
//      square A^2 = A A^T              (A is symmetric) upper tiles, mirrored
//      split  C = X Y                  product of two commuting symmetric
//                                      matrices (C symmetric), upper tiles, mirrored
//      apply  X'^T = XT (aI + dB) + XT Bo    ("NT"; Bo is symmetric)
//    The diagonals of these symmetric matrices are the large entries, so they
//    are carried in fp32 and only the off-diagonal parts (Ao, Bo, ...) are
//    rounded to bf16 for the next product:  A^2 = dA^2 + dA Ao + Ao dA + Ao Ao,
//    with the diagonal terms applied in the epilogues.  Epilogues also fold
//    alpha, and the last apply performs the parameter write
//    W <- (1 - eta lambda) W - eta s O^{-1}(X_5).
//
// Which matrices play which role, and in what order the kinds run, is the
// dispatcher's choice (prm_api.hip): either the five iterations as written,
// or, for wide oriented shapes, the same map evaluated with r x r products
// between two explicit iterates (every B_j is a polynomial in A_0, so the
// factors aI + B_j commute: X_2 = P_1 P_0 X_0, A_{j+1} = P_j^2 A_j,
// X_5 = P_4 P_3 P_2 X_2).
// In precise mode the plain iterations carry the iterate as two bf16 parts
// (hi + lo): the prologue writes both, the Gram sums three products and the
// apply two over K segments of one accumulation, and the apply writes the next
// iterate as hi + lo.
// The workspace is padded to whole tiles and the padding stays exactly zero
// through every iteration, so the GEMMs need no bounds checks.
#include <type_traits>

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
// HILO (precise mode): the low bf16 part u - bf16(u) goes to XTl as well.
template <DType GD, bool HILO>
__global__ __launch_bounds__(256) void ns_prologue_kernel(const MatDesc* __restrict__ md,
                                                          const Item* __restrict__ items,
                                                          NsParams p) {
  using GT = typename NsStore<GD>::T;
  constexpr int T = kPrologueTile;  // 64
  __shared__ uint16_t tile[T][T + 4];
  __shared__ uint16_t tile_lo[HILO ? T : 1][T + 4];
  __shared__ float red[4];
  const Item it = items[blockIdx.x];
  const MatDesc& d = md[it.mat];
  const int64_t m = d.m, n = d.n;
  // XT (cp x rp) is the stored layout of a tall matrix and the transpose of a
  // wide one
  uint16_t* XT = d.XT;
  const int64_t ld = d.rp;
  const bool tall = d.tall;
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
        VecNT<GT>::load4(G + row * n + col, g);
        VecNT<float>::load4(M + row * n + col, mm);
#pragma unroll
        for (int k = 0; k < 4; ++k) mm[k] = p.beta * mm[k] + p.gcoef * g[k];
        VecNT<float>::store4(M + row * n + col, mm);
#pragma unroll
        for (int k = 0; k < 4; ++k) u[k] = p.nesterov ? g[k] + p.beta * mm[k] : mm[k];
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (col + k < n) {
            const float g = VecNT<GT>::load1(G + row * n + col + k);
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
    uint32_t l0 = 0, l1 = 0, l2 = 0, l3 = 0;
    if constexpr (HILO) {
      l0 = f2bf(u[0] - bf2f(h0));
      l1 = f2bf(u[1] - bf2f(h1));
      l2 = f2bf(u[2] - bf2f(h2));
      l3 = f2bf(u[3] - bf2f(h3));
    }
    if (tall) {
      *reinterpret_cast<uint2*>(XT + row * ld + col) = make_uint2(h0 | (h1 << 16), h2 | (h3 << 16));
      if constexpr (HILO) *reinterpret_cast<uint2*>(d.XTl + row * ld + col) = make_uint2(l0 | (l1 << 16), l2 | (l3 << 16));
    } else {
      tile[r][tc + 0] = (uint16_t)h0;
      tile[r][tc + 1] = (uint16_t)h1;
      tile[r][tc + 2] = (uint16_t)h2;
      tile[r][tc + 3] = (uint16_t)h3;
      if constexpr (HILO) {
        tile_lo[r][tc + 0] = (uint16_t)l0;
        tile_lo[r][tc + 1] = (uint16_t)l1;
        tile_lo[r][tc + 2] = (uint16_t)l2;
        tile_lo[r][tc + 3] = (uint16_t)l3;
      }
    }
  }
  if (!tall) {  // uniform per work group
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = tr + 16 * i;  // tile column -> transposed row
      const uint32_t v0 = tile[tc + 0][j], v1 = tile[tc + 1][j], v2 = tile[tc + 2][j],
                     v3 = tile[tc + 3][j];
      *reinterpret_cast<uint2*>(XT + (C0 + j) * ld + R0 + tc) =
          make_uint2(v0 | (v1 << 16), v2 | (v3 << 16));
      if constexpr (HILO) {
        const uint32_t w0 = tile_lo[tc + 0][j], w1 = tile_lo[tc + 1][j], w2 = tile_lo[tc + 2][j],
                       w3 = tile_lo[tc + 3][j];
        *reinterpret_cast<uint2*>(d.XTl + (C0 + j) * ld + R0 + tc) = make_uint2(w0 | (w1 << 16), w2 | (w3 << 16));
      }
    }
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
// K advances in stages of 64 through two LDS buffers.  Operands move from
// global memory straight into LDS (global_load_lds_dwordx4): each wave
// instruction fills 1 KB (8 tile rows) in lane order, and the XOR swizzle of
// the 16-byte chunks is obtained by choosing which global chunk each lane
// fetches.  Stage k+1 streams into one buffer while stage k is read from the
// other; the two buffers are distinct LDS arrays, so fragment reads never wait
// for the stage in flight.
// ---------------------------------------------------------------------------
namespace gemm {
constexpr int BM = kNsTile, BN = kNsTile, BK = 64;
// waves: 2 x 2, one per SIMD, each owning 128 x 128 of the tile.  (2 x 4, two
// waves per SIMD at 128 x 64 each, reads 1.5x more fragment bytes from LDS per
// MFMA and measured about 2% slower over the DiT-4B weight set.)
constexpr int WAVES_M = 2, WAVES_N = 2, NWAVES = WAVES_M * WAVES_N;
constexpr int NTHREADS = 64 * NWAVES;
constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
constexpr int MI = WM / 32, NI = WN / 32;
constexpr int ROW_BYTES = BK * 2;                       // 128 B per tile row
constexpr int A_BYTES = BM * ROW_BYTES;                 // 32 KB
constexpr int STAGE_BYTES = (BM + BN) * ROW_BYTES;      // 64 KB
constexpr int DMA_PER_WAVE = BM / 8 / NWAVES;           // 1 KB wave loads per operand per stage
constexpr int NDMA = 2 * DMA_PER_WAVE;                  // wave loads per stage (both operands)
constexpr int ROWS_PER_WAVE = BM / NWAVES;              // NT: tile rows one wave loads per operand
constexpr int KROWS_PER_WAVE = BK / NWAVES;             // TN: k-rows one wave loads per operand
static_assert(BM * BN * 2 <= 2 * STAGE_BYTES, "the bf16 epilogue tile fits the two stage buffers");

// byte offset of 16-byte chunk `ch` of tile row `r`: XOR swizzle of the eight
// 16-byte chunks of a row by (r / 2) % 8.  A row is 128 B, half of the 64 x 4 B
// banks, so rows 2a and 2a + 1 share no banks and 16 consecutive rows read at
// the same chunk (the fragment reads: one row per lane) hit 16 distinct
// 16-byte bank groups.
__device__ __forceinline__ int swz_f(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ int swz(int r, int ch) { return r * ROW_BYTES + ((ch ^ swz_f(r)) << 4); }

typedef __attribute__((address_space(3))) void* lds_ptr;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(1))) u32x4* gptr4;

// K-major ("TN") stage tile: 64 k-rows of 256 bf16 (512 B, 32 chunks of 16 B);
// chunk c of row r is stored at c ^ (4 (r % 4)).  A transposing fragment read
// covers 4 consecutive k-rows x 4 consecutive chunks per 32 lanes; the XOR moves
// the 4 rows to 4 different 64-byte bank quarters, so those 16 chunks occupy
// 16 distinct 16-byte bank groups.
constexpr int TN_ROW_BYTES = BM * 2;
__device__ __forceinline__ int swz_tn_f(int r) { return 4 * (r & 3); }
__device__ __forceinline__ int swz_tn(int r, int ch) { return r * TN_ROW_BYTES + ((ch ^ swz_tn_f(r)) << 4); }

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16* lds_v4i16;

}  // namespace gemm

// The operands enter the MFMAs swapped, so each lane accumulates four
// consecutive output columns of one output row (see the epilogue).  WD is the
// parameter type, used by the parameter write of the last apply.
// NSEG > 1 (precise mode): K runs over NSEG segments with their own operand
// panels, so one accumulation sums several products: the Gram (NSEG = 3)
// X_hi X_hi^T + X_hi X_lo^T + X_lo X_hi^T, the apply (NSEG = 2) the factor
// applied to X_hi and to X_lo, whose result it then writes as hi + lo.
template <int KIND, DType WD, int NSEG>
__global__ __launch_bounds__(gemm::NTHREADS, 1) void ns_gemm_kernel(const MatDesc* __restrict__ md,
                                                         const Item* __restrict__ items,
                                                         NsParams p) {
  using namespace gemm;
  __shared__ __attribute__((aligned(16))) char s0[STAGE_BYTES];
  __shared__ __attribute__((aligned(16))) char s1[STAGE_BYTES];

  const Item it = items[blockIdx.x];
  const MatDesc& d = md[it.mat];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const uint16_t* XTc = p.src == 0 ? d.XT : d.XTn;
  uint16_t* XTo = p.src == 0 ? d.XTn : d.XT;
  const uint16_t* XTcl = p.src == 0 ? d.XTl : d.XTnl;   // precise mode: low parts
  uint16_t* XTol = p.src == 0 ? d.XTnl : d.XTl;
  const int64_t rp = d.rp, cp = d.cp;
  static_assert(NSEG == 1 || (KIND == GEMM_GRAM && NSEG == 3) || (KIND == GEMM_APPLY && NSEG == 2), "segments");

  // C[row][col] = sum_k P[row][k] Q[col][k]   (NT), or
  // C[row][col] = sum_k P[k][row] Q[k][col]   (TN, the Gram on XT)
  constexpr bool TN = (KIND == GEMM_GRAM);
  const uint16_t *P, *Q;
  const int64_t ld = rp;  // every operand has rp columns
  int64_t klen;
  if constexpr (KIND == GEMM_GRAM) {
    P = XTc; Q = XTc; klen = cp;
  } else if constexpr (KIND == GEMM_POLY) {
    P = d.S[p.sx]; Q = P; klen = rp;   // Ao Ao (Ao is symmetric)
  } else if constexpr (KIND == GEMM_SPROD) {
    P = d.S[p.sx]; Q = d.S[p.sy]; klen = rp;   // Xo Yo (Yo is symmetric)
  } else {
    P = XTc; Q = d.S[p.sy]; klen = rp;   // X'^T tile: rows of XT, columns of the factor
  }
  const int64_t row0 = (int64_t)it.tm * BM, col0 = (int64_t)it.tn * BN;
  const int nk = (int)(klen / BK);  // a multiple of 4: the padded dimensions are multiples of the tile
  const int NK = NSEG * nk;         // stages over all segments
  // operand panels of each segment (segment 0: P, Q)
  const uint16_t* Ps[NSEG];
  const uint16_t* Qs[NSEG];
  Ps[0] = P;
  Qs[0] = Q;
  if constexpr (KIND == GEMM_GRAM && NSEG == 3) {
    Ps[1] = XTc; Qs[1] = XTcl;
    Ps[2] = XTcl; Qs[2] = XTc;
  } else if constexpr (KIND == GEMM_APPLY && NSEG == 2) {
    Ps[1] = XTcl; Qs[1] = Q;
  }

  // DMA sources.  NT: wave load q covers tile rows R wave + 8 q + lane / 8
  // (R = ROWS_PER_WAVE, a multiple of 16) and lane fills physical chunk lane % 8,
  // i.e. logical chunk (lane % 8) ^ swz_f(row).  TN: wave load q covers k-rows
  // KR wave + 2 q + lane / 32 (KR = KROWS_PER_WAVE, a multiple of 4) and lane
  // fills physical chunk lane % 32, i.e. logical chunk (lane % 32) ^ swz_tn_f(k-row).
  static_assert(ROWS_PER_WAVE % 16 == 0 && KROWS_PER_WAVE % 4 == 0, "swizzle phase per wave");
  // Each wave load is addressed as a wave-uniform base (scalar registers: the
  // operand, the tile, the wave and the k offset) plus a 32-bit per-lane byte
  // offset fixed for the whole tile (the row or k-row, and the swizzled chunk),
  // so issuing a load takes no 64-bit vector address arithmetic.  The offsets
  // stay below 2^31 (at most 64 rows of 2^24 bf16).
  const char *baseA[NSEG], *baseB[NSEG];
  uint32_t voff[DMA_PER_WAVE];
  if constexpr (TN) {
#pragma unroll
    for (int sg = 0; sg < NSEG; ++sg) {
      baseA[sg] = reinterpret_cast<const char*>(Ps[sg] + (int64_t)(KROWS_PER_WAVE * wave) * ld + row0);
      baseB[sg] = reinterpret_cast<const char*>(Qs[sg] + (int64_t)(KROWS_PER_WAVE * wave) * ld + col0);
    }
#pragma unroll
    for (int qq = 0; qq < DMA_PER_WAVE; ++qq) {
      const int krow = 2 * qq + (lane >> 5);  // + KR wave, which is 0 mod 4
      voff[qq] = (uint32_t)((krow * ld + (((lane & 31) ^ swz_tn_f(krow)) << 3)) * 2);
    }
  } else {
#pragma unroll
    for (int sg = 0; sg < NSEG; ++sg) {
      baseA[sg] = reinterpret_cast<const char*>(Ps[sg] + (row0 + ROWS_PER_WAVE * wave) * ld);
      baseB[sg] = reinterpret_cast<const char*>(Qs[sg] + (col0 + ROWS_PER_WAVE * wave) * ld);
    }
    // swz_f(row) = 4 (q % 2) + lane / 16, so the lane's source chunk only
    // depends on the parity of q: chunk bit 2 flips for odd q, i.e.
    // (c ^ 4) * 8 elements = c * 8 +- 32
    const int64_t lane_off = (int64_t)(lane >> 3) * ld + (((lane & 7) ^ (lane >> 4)) << 3);
#pragma unroll
    for (int qq = 0; qq < DMA_PER_WAVE; ++qq) {
      const int flip = (qq & 1) ? ((lane & 4) ? -32 : 32) : 0;
      voff[qq] = (uint32_t)((lane_off + (int64_t)(8 * qq) * ld + flip) * 2);
    }
  }
  // One 1 KB wave load of the stage at k offset `k`: block q < DMA_PER_WAVE of
  // operand A, the others of operand B.  Written as assembly because the
  // compiler folds the lane offset into a 64-bit vector address before adding
  // k (two 64-bit vector adds per load in the main loop, measured 3% of the
  // refresh step).  The compiler then does not see these LDS writes: every
  // stage wait below is an explicit vmcnt(0) before the barrier.  M0 (the LDS
  // destination of the DMA) is a register the compiler reserves and does not
  // save around the asm; in these kernels its own code reads M0 only for the
  // square epilogue's LDS DMA and writes it right before each such read (the
  // compiled assembly is checked for this by tests/test_abi.py).
  // `sg`: the K segment (0 unless NSEG > 1), `k` the offset within it
  auto dma1 = [&](char* stage, int sg, int64_t k, int q) __attribute__((always_inline)) {
    const bool isb = q >= DMA_PER_WAVE;
    const int qq = isb ? q - DMA_PER_WAVE : q;
    const char* b0 = isb ? baseB[0] : baseA[0];
    if constexpr (NSEG >= 2) {
      if (sg == 1) b0 = isb ? baseB[1] : baseA[1];
      if constexpr (NSEG >= 3) {
        if (sg == 2) b0 = isb ? baseB[NSEG - 1] : baseA[NSEG - 1];
      }
      // the segment is wave-uniform; say so, so that the base stays scalar
      const uint64_t u = (uint64_t)(uintptr_t)b0;
      b0 = (const char*)(uintptr_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(u >> 32)) << 32) |
                                    (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)u));
    }
    const char* base = b0 + (TN ? k * ld : k) * 2;
    const uint32_t lds = (uint32_t)(uintptr_t)(lds_ptr)(stage + (isb ? A_BYTES : 0) + (DMA_PER_WAVE * wave + qq) * 1024);
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"  // the M0 clobber, see above
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" : : "v"(voff[qq]), "s"(base), "s"(lds) : "m0");
#pragma clang diagnostic pop
  };
  auto stage_landed = [&]() __attribute__((always_inline)) { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };

  floatx16 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int arow = wm * WM + (lane & 31), brow = wn * WN + (lane & 31);
  const int khalf = lane >> 5;
  // TN fragment addresses (k-step 0): lane L of 16-lane group g = L / 16 reads
  // k-row 8 (g / 2) + 4 kk + (L % 16) / 4 at columns m0 + 16 (g % 2) + 4 (L % 4)
  int tn_off[MI][2], tn_offb[NI][2];
  if constexpr (TN) {
    const int g = lane >> 4, jl = lane & 15;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int kr = 8 * (g >> 1) + 4 * kk + (jl >> 2);
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const int ma = wm * WM + i * 32 + 16 * (g & 1) + 4 * (jl & 3);
        tn_off[i][kk] = swz_tn(kr, ma >> 3) + ((ma & 7) << 1);
      }
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int mb = wn * WN + j * 32 + 16 * (g & 1) + 4 * (jl & 3);
        tn_offb[j][kk] = swz_tn(kr, mb >> 3) + ((mb & 7) << 1);
      }
    }
  }

  // Apply: the term (a I + diag(dB)) applied to X^T is folded into the
  // accumulators as one more product, X^T diag(a + dB), taken while the stage
  // that holds the tile's own columns of X^T passes through LDS.  The diagonal
  // factor enters the MFMA as a synthetic operand fragment in two bf16 parts
  // (hi + lo carries 16 mantissa bits; each product is exact in fp32).  Lane L
  // supplies the diagonal entry of column 32 j + L % 32 at element
  // e = L % 32 - 16 h - 8 (L / 32) of k-step half h, when 0 <= e < 8.
  // Split product: the term diag(dX + xshift) Yo is folded the same way on
  // the other side, as a synthetic first-operand fragment (row 32 i + L % 32
  // of the wave's rows, same element rule) against the stage's Yo fragments,
  // while the stage that holds the tile's own rows as k passes through LDS
  // (Yo is symmetric, so its rows there are the needed columns).
  static_assert(MI == NI, "one fold array serves row and column blocks");
  uint32_t fold_hi[MI], fold_lo[MI];
  if constexpr (KIND == GEMM_APPLY || KIND == GEMM_SPROD) {
#pragma unroll
    for (int j = 0; j < MI; ++j) {
      const float v = (KIND == GEMM_APPLY) ? p.yshift + d.dS[p.sy][col0 + wn * WN + 32 * j + (lane & 31)]
                                           : p.xshift + d.dS[p.sx][row0 + wm * WM + 32 * j + (lane & 31)];
      fold_hi[j] = f2bf(v);
      fold_lo[j] = f2bf(v - bf2f(fold_hi[j]));
    }
  }
  auto syn = [&](uint32_t bits, int h) __attribute__((always_inline)) {
    const int e = (lane & 31) - 16 * h - 8 * (lane >> 5);
    const uint32_t word = (e & 1) ? (bits << 16) : bits;
    u32x4 f;
#pragma unroll
    for (int w = 0; w < 4; ++w) f[w] = ((unsigned)e < 8u && (e >> 1) == w) ? word : 0u;
    return __builtin_bit_cast(bf16x8, f);
  };
  auto mfma = [&](const bf16x8& x, const bf16x8& y, floatx16& c) __attribute__((always_inline)) {
    // accumulates the transposed block: (P Q^T)^T = Q P^T
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(y, x, c, 0, 0, 0);
  };

  // Fragments live across stages: the last NDEF row blocks of a stage's last
  // k-step run after the stage barrier, from set 1, while the next stage's
  // first fragments (set 0) load from LDS (measured 0.3% on the refresh step;
  // deferring two row blocks is equal).  Set 1 starts at zero, so the first
  // stage's deferred products add nothing.
  constexpr int NDEF = 1;
  bf16x8 fa[2][MI], fb[2][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i) fa[1][i] = bf16x8{};
#pragma unroll
  for (int j = 0; j < NI; ++j) fb[1][j] = bf16x8{};
  auto deferred = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = MI - NDEF; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j) mfma(fa[1][i], fb[1][j], acc[i][j]);
  };

  // Compute one stage from `cur` while streaming stage `knext` (if >= 0) into
  // `nxt`.  The vector-memory path accepts about one 1 KB wave load per 16
  // cycles, so the wave's loads are spread between MFMA sub-groups (a quarter
  // at the start, the rest over the first two k-steps) instead of stalling
  // the in-order issue behind a burst.  Sub-group i (row block i) also reads the
  // next k-step's A fragment i and, for i < NI, its B fragment i.
  // FOLD: 0 none; f = 1 or 2: the stage holds, as k, the wave's output block
  // columns (apply) or rows (split product) 2 (f - 1) and 2 (f - 1) + 1, whose
  // diagonal term is folded in when `fold` is set.
  // MORE: 1 a next stage exists, 0 none (the tile's last stage), -1 decided at
  // run time from knext; static where possible, so the main loop has no branch
  auto stage_compute = [&](const char* cur, char* nxt, int knext, auto foldc, bool fold, auto morec) __attribute__((always_inline)) {
    constexpr int FOLD = decltype(foldc)::value;
    constexpr int MORE = decltype(morec)::value;
    const char* a = cur;
    const char* b = cur + A_BYTES;
    // segment of stage knext (comparisons, not a division, so that it stays a
    // wave-uniform scalar for the load addresses)
    const int sgn = NSEG == 1 ? 0 : (int)(knext >= nk) + (NSEG >= 3 ? (int)(knext >= 2 * nk) : 0);
    const int64_t kn = (int64_t)(knext - sgn * nk) * BK;
    const bool more = MORE == 1 || (MORE == -1 && knext >= 0);
    // two transposing reads give lane L the column (L % 32) of the block at 8
    // consecutive k: k-rows 16 ks + 8 (L / 32) + 4 kk + s, s = 0..3
    auto rd_tn = [&](const char* base, const int (&off)[2], int ks) __attribute__((always_inline)) {
      v4i16 x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16)(base + off[0] + ks * 16 * TN_ROW_BYTES));
      v4i16 x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16)(base + off[1] + ks * 16 * TN_ROW_BYTES));
      return __builtin_bit_cast(bf16x8, __builtin_shufflevector(x0, x1, 0, 1, 2, 3, 4, 5, 6, 7));
    };
    auto rda = [&](int set, int i, int ks) __attribute__((always_inline)) {
      if constexpr (TN) fa[set][i] = rd_tn(a, tn_off[i], ks);
      else fa[set][i] = *reinterpret_cast<const bf16x8*>(a + swz(arow + i * 32, ks * 2 + khalf));
    };
    auto rdb = [&](int set, int j, int ks) __attribute__((always_inline)) {
      if constexpr (TN) fb[set][j] = rd_tn(b, tn_offb[j], ks);
      else fb[set][j] = *reinterpret_cast<const bf16x8*>(b + swz(brow + j * 32, ks * 2 + khalf));
    };
    // a quarter of the loads at the start, the rest spread over the sub-groups
    // of the first DMA_KSTEPS k-steps (sub-group s issues loads
    // [DMA0 + REM s / NS, DMA0 + REM (s + 1) / NS)); spreading them over one
    // or three k-steps instead measured equal or slower
    constexpr int DMA_KSTEPS = 2;
    constexpr int DMA0 = NDMA / 4, REM = NDMA - DMA0, NS = DMA_KSTEPS * MI;
    static_assert(DMA_KSTEPS >= 1 && DMA_KSTEPS <= 3, "loads must be issued before the last k-step");
    if (more) {
#pragma unroll
      for (int q = 0; q < DMA0; ++q) dma1(nxt, sgn, kn, q);
    }
#pragma unroll
    for (int i = 0; i < MI; ++i) rda(0, i, 0);
#pragma unroll
    for (int j = 0; j < NI; ++j) rdb(0, j, 0);
    deferred();  // the previous stage's last row blocks (zeros before the first stage)
    __builtin_amdgcn_sched_barrier(0);
    auto kstep = [&](auto ksc) __attribute__((always_inline)) {
      constexpr int ks = decltype(ksc)::value;
      constexpr int cs = ks & 1;
#pragma unroll
      for (int i = 0; i < (ks == 3 ? MI - NDEF : MI); ++i) {  // sub-group: row block i, NI MFMAs
        if (ks < 3) {
          if (ks < DMA_KSTEPS && more) {
            const int slot = ks * MI + i;
#pragma unroll
            for (int q = DMA0 + REM * slot / NS; q < DMA0 + REM * (slot + 1) / NS; ++q) dma1(nxt, sgn, kn, q);
          }
          rda(cs ^ 1, i, ks + 1);
          if (i < NI) rdb(cs ^ 1, i, ks + 1);
        }
#pragma unroll
        for (int j = 0; j < NI; ++j) mfma(fa[cs][i], fb[cs][j], acc[i][j]);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (FOLD != 0 && fold) {
        constexpr int J = (FOLD > 0 ? 2 * (FOLD - 1) : 0) + ks / 2;
        // opaque here, so the fragments are built in the fold stage and not
        // hoisted out of the main loop (they would hold 64 registers)
        uint32_t hb = fold_hi[J], lb = fold_lo[J];
        asm volatile("" : "+v"(hb), "+v"(lb));
        const bf16x8 hi = syn(hb, ks & 1), lo = syn(lb, ks & 1);
        if constexpr (KIND == GEMM_SPROD) {
          // J is the wave's row block here
#pragma unroll
          for (int j = 0; j < NI; ++j) mfma(hi, fb[cs][j], acc[J][j]);
#pragma unroll
          for (int j = 0; j < NI; ++j) mfma(lo, fb[cs][j], acc[J][j]);
        } else {
#pragma unroll
          for (int i = 0; i < MI; ++i) mfma(fa[cs][i], hi, acc[i][J]);
#pragma unroll
          for (int i = 0; i < MI; ++i) mfma(fa[cs][i], lo, acc[i][J]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    kstep(std::integral_constant<int, 0>{});
    kstep(std::integral_constant<int, 1>{});
    kstep(std::integral_constant<int, 2>{});
    kstep(std::integral_constant<int, 3>{});
  };
  static_assert(BK / 16 == 4 && MI == 4 && NI <= MI, "schedule assumes 4 k-steps, 4 row blocks");

  // stage 0 up front, then ping-pong: s0 holds even stages, s1 odd ones
#pragma unroll
  for (int q = 0; q < NDMA; ++q) dma1(s0, 0, 0, q);
  stage_landed();
  __syncthreads();
  constexpr std::integral_constant<int, 1> more_yes{};
  constexpr std::integral_constant<int, 0> more_no{};
  constexpr std::integral_constant<int, -1> more_rt{};
  // stages kt (in s0) and kt + 1 (in s1), counted over all segments; nk is
  // even, so stage kt + 1 exists, and m1 says whether stage kt + 2 does
  auto stage_pair = [&](int kt, auto f0, auto f1, bool fold0, bool fold1, auto m1) __attribute__((always_inline)) {
    stage_compute(s0, s1, kt + 1, f0, fold0, more_yes);
    stage_landed();
    __syncthreads();  // stage kt+1 has landed; every wave is done with s0
    stage_compute(s1, s0, kt + 2 < NK ? kt + 2 : -1, f1, fold1, m1);
    stage_landed();
    __syncthreads();
  };
  constexpr std::integral_constant<int, 0> nofold{};
  // apply: the stages that carry this wave's output columns as k; split
  // product: the stages that carry its output rows as k
  const int kfold = (KIND == GEMM_APPLY) ? (int)((col0 + wn * WN) / BK)
                    : (KIND == GEMM_SPROD) ? (int)((row0 + wm * WM) / BK) : nk;
  int kt = 0;
  // The fold (apply, split product) takes two stages (a stage pair), which run
  // between two plain loops, since one loop body holding both variants spills.
  // The pairs before the last one always stream a next stage; the last pair
  // (kt = NK - 2) runs on its own.  With several segments the fold pair recurs
  // in each (the diagonal term applies to every part of the iterate).
  constexpr bool FOLDS = KIND == GEMM_APPLY || KIND == GEMM_SPROD;
  if constexpr (FOLDS) {
    static_assert(WN == 2 * BK && WM == 2 * BK, "a wave's output columns (rows) span two stages");
#pragma unroll
    for (int sg = 0; sg < NSEG; ++sg) {
      const int kf = sg * nk + (kfold & ~1);  // kfold < nk
      for (; kt < kf; kt += 2) stage_pair(kt, nofold, nofold, false, false, more_yes);
      stage_pair(kt, std::integral_constant<int, 1>{}, std::integral_constant<int, 2>{}, true, true, more_rt);
      kt += 2;
    }
  }
  for (; kt < NK - 2; kt += 2) stage_pair(kt, nofold, nofold, false, false, more_yes);
  if (kt < NK) stage_pair(kt, nofold, nofold, false, false, more_no);

  deferred();
  // ---- epilogue ----
  // Final values are formed in registers, converted to bf16 and the whole
  // 256 x 256 tile is staged once in LDS (rows 0..127 in s0, 128..255 in s1;
  // 512 B per row, 16-byte chunk c of row r stored at c ^ (r % 32)).  It then
  // leaves as 512-byte row segments and/or as its mirror: transposing reads
  // (ds_read_b64_tr_b16) give each lane 8 consecutive tile rows of one tile
  // column, i.e. 16 bytes of a row of the mirrored tile.
  //   apply:        X'^T rows; at the last iteration the parameter write
  //                 instead (rows for a tall matrix, whose W is X^T; the
  //                 mirror for a wide one)
  //   Gram, square: rows, plus the mirror above the diagonal.
  // Lane L holds output row 32 i + L % 32 of its wave block and, for block
  // column j and q = 0..3, the 4 columns 32 j + 8 q + 4 (L / 32) + 0..3.
  const bool diag = (KIND != GEMM_APPLY) && it.tm == it.tn;  // Gram / square tile on the diagonal
  if constexpr (KIND == GEMM_POLY || KIND == GEMM_SPROD) {
    // the square (split product) needs the tile of its (first) operand at its
    // own output position: it enters the staging area (layout below) by 1 KB
    // DMA wave loads, 2 tile rows each, and every lane later reads and
    // overwrites its own 8 bytes in place
#pragma unroll 4
    for (int q = 0; q < BM / 2 / NWAVES; ++q) {
      const int r2 = 2 * ((BM / 2 / NWAVES) * wave + q);  // first row of the pair (even)
      const int R = r2 + (lane >> 5);
      const int c = (lane & 31) ^ (R & 31);
      __builtin_amdgcn_global_load_lds((const void*)(d.S[p.sx] + (row0 + R) * rp + col0 + 8 * c),
                                       (lds_ptr)((r2 < 128 ? s0 : s1) + (r2 & 127) * 512), 16, 0, 0);
    }
    __syncthreads();
  }
  const float alpha = p.use_alpha ? *d.alpha : 1.0f;
  const bool last = (KIND == GEMM_APPLY) && p.last;
  if constexpr (KIND == GEMM_APPLY && NSEG == 2) {
    if (!last) {
      // precise mode: the next iterate as hi + lo.  The tile is staged (same
      // layout as below) and written out twice, as bf16(v) into XTo and as
      // bf16(v - bf16(v)) into XTol.
      const int hl = lane >> 5, m = lane & 31;
      char* T = wm ? s1 : s0;
      auto tb = [&](int row, int col) __attribute__((always_inline)) {
        return (row < 128 ? s0 : s1) + (row & 127) * 512 + ((((col >> 3) ^ (row & 31))) << 4) + (col & 7) * 2;
      };
#pragma unroll
      for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
        for (int i = 0; i < MI; ++i) {
          const int r = 32 * i + m;
          char* trow = T + r * 512 + 8 * hl;
#pragma unroll
          for (int j = 0; j < NI; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              float v[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                v[e] = alpha * acc[i][j][4 * q + e];
                if (pass) v[e] -= bf2f(f2bf(v[e]));
              }
              const int ch = (wn * WN + 32 * j + 8 * q) >> 3;
              uint2 w;
              w.x = pack_bf2(v[0], v[1]);
              w.y = pack_bf2(v[2], v[3]);
              *reinterpret_cast<uint2*>(trow + ((ch ^ (r & 31)) << 4)) = w;
            }
        }
        __syncthreads();
        uint16_t* const dst = pass ? XTol : XTo;
        const int ch = tid & 31;
        constexpr int ROWS_PER_IT = NTHREADS / 32;
#pragma unroll 4
        for (int itr = 0; itr < BM / ROWS_PER_IT; ++itr) {
          const int row = itr * ROWS_PER_IT + (tid >> 5);
          *reinterpret_cast<u32x4*>(dst + (row0 + row) * rp + col0 + ch * 8) =
              *reinterpret_cast<const u32x4*>(tb(row, ch * 8));
        }
        __syncthreads();
      }
      return;
    }
  }
  {
    const float s2 = alpha * alpha;
    char* T = wm ? s1 : s0;
    const int hl = lane >> 5, m = lane & 31;
    // lane L holds the (r, r) entry of a diagonal block iff (L % 32) / 4 % 2
    // == L / 32, at q = (L % 32) / 8, element (L % 32) % 4
    const bool dlane = diag && wm == wn && ((m >> 2) & 1) == hl;
    const int64_t grow = row0 + wm * WM + m, gcol = col0 + wn * WN + 4 * hl;
    float* dout = d.dS[p.so];
    // square / split product: diagonal of the (second) operand at this lane's
    // columns (the same for every row block), shift included
    constexpr bool SPLIT = KIND == GEMM_POLY || KIND == GEMM_SPROD;
    const float* dX = d.dS[p.sx];
    const float* dY = (KIND == GEMM_SPROD) ? d.dS[p.sy] : dX;
    const float ys = (KIND == GEMM_SPROD) ? p.yshift : p.xshift;
    float dcol[NI][4][4];
    if constexpr (SPLIT) {
#pragma unroll
      for (int j = 0; j < NI; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          Vec<float>::load4(dY + gcol + 32 * j + 8 * q, dcol[j][q]);
#pragma unroll
          for (int e = 0; e < 4; ++e) dcol[j][q][e] += ys;
        }
    }
#pragma unroll
    for (int ih = 0; ih < MI; ih += 2) {
      // square / split product: diagonal of the first operand at rows
      // 32 i + L % 32 for two row blocks, shift included
      float drow[2];
      if constexpr (SPLIT) {
#pragma unroll
        for (int ii = 0; ii < 2; ++ii) drow[ii] = dX[grow + 32 * (ih + ii)] + p.xshift;
      }
#pragma unroll
      for (int ii = 0; ii < 2; ++ii) {
        const int i = ih + ii;
        const int r = 32 * i + m;
        char* trow = T + r * 512 + 8 * hl;
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float v[4];
            if constexpr (KIND == GEMM_GRAM) {
              // A = alpha^2 acc
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = s2 * acc[i][j][4 * q + e];
            } else if constexpr (KIND == GEMM_POLY) {
              // A^2 = dA^2 + dA Ao + Ao dA + Ao Ao;  B = b A + c A^2
              const int ch0 = (wn * WN + 32 * j + 8 * q) >> 3;
              const uint2 w2 = *reinterpret_cast<const uint2*>(trow + ((ch0 ^ (r & 31)) << 4));
              const float a4[4] = {bf2f(w2.x & 0xffffu), bf2f(w2.x >> 16), bf2f(w2.y & 0xffffu), bf2f(w2.y >> 16)};
#pragma unroll
              for (int e = 0; e < 4; ++e)
                v[e] = p.c * acc[i][j][4 * q + e] + (p.b + p.c * (drow[ii] + dcol[j][q][e])) * a4[e];
            } else if constexpr (KIND == GEMM_SPROD) {
              // (dX + Xo)(dY + Yo) = Xo Yo + dX Yo + Xo dY (+ dX dY on the
              // diagonal); Xo Yo and dX Yo are in acc (the second folded into
              // the MFMAs), Xo dY comes from the staged Xo tile
              const int ch0 = (wn * WN + 32 * j + 8 * q) >> 3;
              const uint2 w2 = *reinterpret_cast<const uint2*>(trow + ((ch0 ^ (r & 31)) << 4));
              const float a4[4] = {bf2f(w2.x & 0xffffu), bf2f(w2.x >> 16), bf2f(w2.y & 0xffffu), bf2f(w2.y >> 16)};
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * q + e] + a4[e] * dcol[j][q][e];
            } else {
              // X'^T = alpha (XT diag(a + dB) + XT Bo); both terms are in acc
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = alpha * acc[i][j][4 * q + e];
            }
            if constexpr (KIND != GEMM_APPLY) {
              if (i == j && dlane && q == (m >> 3)) {
                // the diagonal goes to dA / dB (fp32), the bf16 tile keeps 0
                float dv = acc[i][j][4 * q];
#pragma unroll
                for (int e = 1; e < 4; ++e) dv = (e == (m & 3)) ? acc[i][j][4 * q + e] : dv;
                if constexpr (KIND == GEMM_GRAM) dv = s2 * dv;
                else if constexpr (KIND == GEMM_POLY) dv = p.b * drow[ii] + p.c * (dv + drow[ii] * drow[ii]);
                else {
                  float dd = dcol[j][q][0];
#pragma unroll
                  for (int e = 1; e < 4; ++e) dd = (e == (m & 3)) ? dcol[j][q][e] : dd;
                  dv = dv + drow[ii] * dd;
                }
                dout[grow + 32 * i] = dv;
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = (e == (m & 3)) ? 0.f : v[e];
              }
            }
            const int ch = (wn * WN + 32 * j + 8 * q) >> 3;
            uint2 w;
            w.x = pack_bf2(v[0], v[1]);
            w.y = pack_bf2(v[2], v[3]);
            *reinterpret_cast<uint2*>(trow + ((ch ^ (r & 31)) << 4)) = w;
          }
      }
    }
  }
  __syncthreads();
  auto tbyte = [&](int row, int col) __attribute__((always_inline)) {
    return (row < 128 ? s0 : s1) + (row & 127) * 512 + ((((col >> 3) ^ (row & 31))) << 4) + (col & 7) * 2;
  };
  // last apply: W[wr][wc .. wc + 7] <- decay W - lr s dscale x, x = 8 bf16 outputs
  auto wupdate = [&](int64_t wr, int64_t wc, const u32x4& x) __attribute__((always_inline)) {
    using WT = typename NsStore<WD>::T;
    if (wr >= d.m) return;
    const int64_t n = d.n;
    const float dc = d.s * p.dscale;
    WT* W = reinterpret_cast<WT*>(d.W) + wr * n;
    float* const Dp = (p.write_d && d.D) ? d.D + wr * n : nullptr;
    float dv[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      dv[2 * q] = dc * bf2f(x[q] & 0xffffu);
      dv[2 * q + 1] = dc * bf2f(x[q] >> 16);
    }
    if ((n & 7) == 0 && wc + 8 <= n) {
      float w8[8];
      Vec<WT>::load8(W + wc, w8);
#pragma unroll
      for (int q = 0; q < 8; ++q) w8[q] = w8[q] * p.decay - p.lr * dv[q];
      Vec<WT>::store8(W + wc, w8);
      if (Dp) Vec<float>::store8(Dp + wc, dv);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if (wc + q < n) {
          Vec<WT>::store1(W + wc + q, Vec<WT>::load1(W + wc + q) * p.decay - p.lr * dv[q]);
          if (Dp) Vec<float>::store1(Dp + wc + q, dv[q]);
        }
      }
    }
  };
  uint16_t* const out = (KIND == GEMM_APPLY) ? XTo : d.S[p.so];
  // Last apply, bf16 W, the tile wholly inside W and W rows a multiple of 8
  // long: each thread loads the W values of 16 of its 32 chunks before it
  // writes any of them.  (The compiler cannot tell the W loads from the W
  // stores apart, so in the loops below each load waits behind the previous
  // chunk's store, and the epilogue pays the HBM latency chunk after chunk.)
  bool fastw = false;
  if constexpr (KIND == GEMM_APPLY && WD == BF16) {
    fastw = last && (d.n & 7) == 0 &&
            (d.tall ? (row0 + BM <= d.m && col0 + BN <= d.n) : (col0 + BN <= d.m && row0 + BM <= d.n));
  }
  if (fastw) {
    const float dc = d.s * p.dscale;
    const int64_t n = d.n;
    uint16_t* const W = reinterpret_cast<uint16_t*>(d.W);
    float* const Dm = (p.write_d && d.D) ? d.D : nullptr;
    // W[wr][wc .. wc + 7] <- decay W - lr dc x, from its loaded value `raw`
    auto upd = [&](int64_t wr, int64_t wc, const u32x4& raw, const u32x4& xv) __attribute__((always_inline)) {
      float dv[8], w8[8];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        dv[2 * q] = dc * bf2f(xv[q] & 0xffffu);
        dv[2 * q + 1] = dc * bf2f(xv[q] >> 16);
        w8[2 * q] = bf2f(raw[q] & 0xffffu) * p.decay - p.lr * dv[2 * q];
        w8[2 * q + 1] = bf2f(raw[q] >> 16) * p.decay - p.lr * dv[2 * q + 1];
      }
      Vec<uint16_t>::store8(W + wr * n + wc, w8);
      if (Dm) Vec<float>::store8(Dm + wr * n + wc, dv);
    };
    constexpr int NB = 16;
    if (d.tall) {
      // the tile of X^T is a tile of W: chunk itr is row 8 itr + tid / 32, columns 8 (tid % 32) ..
      const int ch = tid & 31;
#pragma unroll
      for (int b0 = 0; b0 < BM / 8; b0 += NB) {
        u32x4 raw[NB];
#pragma unroll
        for (int k = 0; k < NB; ++k)
          raw[k] = *gptr(reinterpret_cast<const u32x4*>(W + (row0 + 8 * (b0 + k) + (tid >> 5)) * n + col0 + ch * 8));
#pragma unroll
        for (int k = 0; k < NB; ++k) {
          const int row = 8 * (b0 + k) + (tid >> 5);
          upd(row0 + row, col0 + ch * 8, raw[k], *reinterpret_cast<const u32x4*>(tbyte(row, ch * 8)));
        }
      }
    } else {
      // the mirror of the X^T tile is a tile of W (same lane mapping as below)
      const int g = lane >> 4, li = lane & 15;
      constexpr int CB = BN / 16 / NWAVES;
      static_assert(CB * (BM / 32) == 2 * NB, "two batches of chunks per lane");
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        u32x4 raw[NB];
#pragma unroll
        for (int k = 0; k < NB; ++k) {
          const int cb = half * (CB / 2) + k / (BM / 32), rb = k % (BM / 32);
          const int C0 = (wave * CB + cb) * 16, R0 = 32 * rb + 8 * g;
          raw[k] = *gptr(reinterpret_cast<const u32x4*>(W + (col0 + C0 + li) * n + row0 + R0));
        }
#pragma unroll
        for (int k = 0; k < NB; ++k) {
          const int cb = half * (CB / 2) + k / (BM / 32), rb = k % (BM / 32);
          const int C0 = (wave * CB + cb) * 16, R0 = 32 * rb + 8 * g;
          const int sr = R0 + (li >> 2), sc = C0 + 4 * (li & 3);
          const v4i16 x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16)tbyte(sr, sc));
          const v4i16 x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16)tbyte(sr + 4, sc));
          upd(col0 + C0 + li, row0 + R0, raw[k],
              __builtin_bit_cast(u32x4, __builtin_shufflevector(x0, x1, 0, 1, 2, 3, 4, 5, 6, 7)));
        }
      }
    }
  }
  if (!fastw && (!last || d.tall)) {
    const int ch = tid & 31;
    constexpr int ROWS_PER_IT = NTHREADS / 32;
#pragma unroll 4
    for (int itr = 0; itr < BM / ROWS_PER_IT; ++itr) {
      const int row = itr * ROWS_PER_IT + (tid >> 5);
      const u32x4 w = *reinterpret_cast<const u32x4*>(tbyte(row, ch * 8));
      if (!last) *reinterpret_cast<u32x4*>(out + (row0 + row) * rp + col0 + ch * 8) = w;
      else wupdate(row0 + row, col0 + ch * 8, w);  // tall: the tile of X^T is a tile of W
    }
  }
  if (!fastw && ((KIND != GEMM_APPLY && !diag) || (last && !d.tall))) {
    // 16-lane group g reads tile rows R0 .. R0 + 7 (R0 = 32 rb + 8 g) of
    // columns C0 .. C0 + 15; source lane 4 a + b of the group points at
    // row R0 + a (+4), columns C0 + 4 b .. +3
    const int g = lane >> 4, li = lane & 15;
    constexpr int CB = BN / 16 / NWAVES;  // 16-column blocks per wave
#pragma unroll 2
    for (int cb = 0; cb < CB; ++cb) {
      const int C0 = (wave * CB + cb) * 16;
#pragma unroll 4
      for (int rb = 0; rb < BM / 32; ++rb) {
        const int R0 = 32 * rb + 8 * g;
        const int sr = R0 + (li >> 2), sc = C0 + 4 * (li & 3);
        const v4i16 x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16)tbyte(sr, sc));
        const v4i16 x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16)tbyte(sr + 4, sc));
        const u32x4 w = __builtin_bit_cast(u32x4, __builtin_shufflevector(x0, x1, 0, 1, 2, 3, 4, 5, 6, 7));
        if (!last) *reinterpret_cast<u32x4*>(out + (col0 + C0 + li) * rp + row0 + R0) = w;
        else wupdate(col0 + C0 + li, row0 + R0, w);  // wide: the mirror of the X^T tile is a tile of W
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
  if (p.hilo) {
    if (gt == BF16) ns_prologue_kernel<BF16, true><<<dim3(nitems), dim3(256), 0, s>>>(md, items, p);
    else ns_prologue_kernel<F32, true><<<dim3(nitems), dim3(256), 0, s>>>(md, items, p);
  } else {
    if (gt == BF16) ns_prologue_kernel<BF16, false><<<dim3(nitems), dim3(256), 0, s>>>(md, items, p);
    else ns_prologue_kernel<F32, false><<<dim3(nitems), dim3(256), 0, s>>>(md, items, p);
  }
  return hipGetLastError();
}

hipError_t launch_ns_alpha(const MatDesc* md, const int32_t* mats, int32_t nmats,
                           const NsParams& p, hipStream_t s) {
  if (nmats <= 0) return hipSuccess;
  ns_alpha_kernel<<<dim3(nmats), dim3(256), 0, s>>>(md, mats, p);
  return hipGetLastError();
}

hipError_t launch_ns_gemm(GemmKind kind, DType wt, const MatDesc* md, const Item* items,
                          int32_t nitems, const NsParams& p, hipStream_t s, bool hilo) {
  if (nitems <= 0) return hipSuccess;
  dim3 g(nitems), b(gemm::NTHREADS);
  switch (kind) {
    case GEMM_GRAM:
      if (hilo) ns_gemm_kernel<GEMM_GRAM, BF16, 3><<<g, b, 0, s>>>(md, items, p);
      else ns_gemm_kernel<GEMM_GRAM, BF16, 1><<<g, b, 0, s>>>(md, items, p);
      break;
    case GEMM_POLY: ns_gemm_kernel<GEMM_POLY, BF16, 1><<<g, b, 0, s>>>(md, items, p); break;
    case GEMM_SPROD: ns_gemm_kernel<GEMM_SPROD, BF16, 1><<<g, b, 0, s>>>(md, items, p); break;
    case GEMM_APPLY:
      if (hilo) {
        if (wt == BF16) ns_gemm_kernel<GEMM_APPLY, BF16, 2><<<g, b, 0, s>>>(md, items, p);
        else ns_gemm_kernel<GEMM_APPLY, F32, 2><<<g, b, 0, s>>>(md, items, p);
      } else {
        if (wt == BF16) ns_gemm_kernel<GEMM_APPLY, BF16, 1><<<g, b, 0, s>>>(md, items, p);
        else ns_gemm_kernel<GEMM_APPLY, F32, 1><<<g, b, 0, s>>>(md, items, p);
      }
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace prm
