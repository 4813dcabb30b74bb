// Internal definitions of libprm: the per-matrix descriptor shared by the host
// dispatcher and the gfx950 kernels, launch parameter blocks, and the
// kernel-launch entry points that the dispatcher calls.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace prm {

// One entry per matrix, in the order given to prm_init.  Caller pointers
// (W, G, M, D) are refreshed before a step whenever they change; the rest is
// fixed at prm_init.
struct MatDesc {
  // caller buffers (device, row-major m x n)
  void* W;
  const void* G;
  float* M;
  float* D;  // direction output (prm_step_debug) or nullptr
  int64_t m, n;
  float s;       // shape scale s(W)
  int32_t tall;  // m > n: oriented rows are stored columns
  // NS5 workspace (bf16 bit patterns), valid while this matrix's chunk runs.
  // Oriented r x c is padded to rp x cp (multiples of the GEMM tile); the
  // iterate is kept transposed, XT = X^T (cp x rp, row-major).
  uint16_t* XT;   // cp x rp   iterate
  uint16_t* XTn;  // cp x rp   next iterate
  // precise mode only (else nullptr): the low bf16 parts of XT and XTn, so
  // that each iterate is carried as hi + lo (16 mantissa bits)
  uint16_t* XTl;
  uint16_t* XTnl;
  // Symmetric r x r matrices in split form: S[k] (rp x rp, bf16) holds the
  // off-diagonal part (diagonal stored as zero), dS[k] (rp, fp32) the
  // diagonal.  The dispatcher assigns them roles (the Gram matrix A, B =
  // bA + cA^2, and for the chained path the products of the factors aI + B);
  // matrices on the plain five-iteration path use S[0], S[1] only.
  uint16_t* S[4];
  float* dS[4];
  float* partial; // prologue: one sum of squares per 64 x 64 tile
  float* alpha;   // 1 / (||U||_F + eps_ns)
  int64_t rp, cp;
  int32_t ptiles_m, ptiles_n;  // prologue tile grid over the padded stored shape
  // row-wise tall path
  float* colpart;  // [nrb][n] partial column sums of squares
  float* colinv;   // [n] 1 / max(||column||, eps)
  int32_t nrb;     // row blocks of the tall statistics pass
  int32_t pad0;
};

// Per-launch scalars of the row-wise kernels.
struct RwParams {
  float beta;      // momentum coefficient
  float gcoef;     // 1 (heavy-ball) or 1 - beta (dampening)
  float lr;        // eta_t
  float decay;     // 1 - eta_t * lambda
  float gamma;     // RowNorm multiplier
  float eps;       // RowNorm clamp
  int32_t nesterov;
  int32_t write_d;
};

// Per-launch scalars of the NS5 kernels.
struct NsParams {
  float beta, gcoef;
  int32_t nesterov;
  float eps_ns;
  float a, b, c;    // quintic coefficients
  float lr, decay;
  float dscale;     // 1, or gamma for the scalar-controlled ablation
  int32_t src;      // iterate read by the Gram / apply: 0 XT, 1 XTn (the apply writes the other)
  int32_t use_alpha;  // the iterate read is the unscaled X0: fold alpha (apply) or alpha^2 (Gram)
  int32_t last;     // the apply writes the parameters instead of the next iterate
  int32_t write_d;
  int32_t sx, sy, so; // split matrices: first operand, second operand, output (indices into S / dS)
  float xshift, yshift; // added to the diagonals of operands sx and sy (P = aI + B is B with shift a)
  int32_t hilo;       // precise mode: the prologue also writes the low parts (XTl)
};

// Work item of the tiled kernels.
struct Item {
  int32_t mat;
  int32_t tm;   // tile row (or row block)
  int32_t tn;   // tile column (or column slab)
  int32_t aux;
};

enum DType : int32_t { F32 = 0, BF16 = 1 };

// ---- launchers (defined in rowwise.hip / ns5.hip) -------------------------
// Wide/square matrices, whole rows held in registers.  seg_start[i] is the
// first block of segment i (matrix seg_mat[i]); nblocks blocks in total.
hipError_t launch_rw_wide(int tpr, int nch, DType wt, DType gt, const MatDesc* md,
                          const int32_t* seg_mat, const int32_t* seg_start, int32_t nseg,
                          int32_t nblocks, const RwParams& p, hipStream_t s);
// Any shape (unaligned rows, very long rows): two sweeps over the row.
hipError_t launch_rw_generic(DType wt, DType gt, const MatDesc* md, const int32_t* rows_mat,
                             const int32_t* rows_start, int32_t nseg, int32_t nrows_total,
                             const RwParams& p, hipStream_t s);
// Tall matrices: column statistics, column norms, parameter write.
hipError_t launch_rw_tall_stats(int vec, DType gt, const MatDesc* md, const Item* items,
                                int32_t nitems, const RwParams& p, hipStream_t s);
hipError_t launch_rw_tall_finalize(const MatDesc* md, const Item* items, int32_t nitems,
                                   const RwParams& p, hipStream_t s);
hipError_t launch_rw_tall_apply(int vec, DType wt, DType gt, const MatDesc* md,
                                const Item* items, int32_t nitems, const RwParams& p,
                                hipStream_t s);

// NS5 refresh.
hipError_t launch_ns_prologue(DType gt, const MatDesc* md, const Item* items, int32_t nitems,
                              const NsParams& p, hipStream_t s);  // p.hilo: also the low parts
hipError_t launch_ns_alpha(const MatDesc* md, const int32_t* mats, int32_t nmats,
                           const NsParams& p, hipStream_t s);
enum GemmKind : int32_t { GEMM_GRAM = 0, GEMM_POLY = 1, GEMM_APPLY = 2, GEMM_SPROD = 3 };
// hilo (Gram and apply only): the iterate is read as hi + lo; the Gram sums
// hi hi^T + hi lo^T + lo hi^T, the apply takes both parts and, unless it is
// the last one, writes the next iterate as hi + lo
hipError_t launch_ns_gemm(GemmKind kind, DType wt, const MatDesc* md, const Item* items,
                          int32_t nitems, const NsParams& p, hipStream_t s, bool hilo = false);

// calibration probes (probe.hip)
hipError_t launch_probe_mfma(int blocks, float* sink, unsigned long long* clk, int iters, hipStream_t s);
// kind 0: read x, 1: write y, 2: copy x -> y; n16 16-byte elements; kind 3:
// the row-wise step's traffic over n16 pieces of 4 elements (x: fp32, y: 2 x bf16)
hipError_t launch_probe_stream(int kind, int blocks, const void* x, void* y, int64_t n16, unsigned* sink,
                               hipStream_t s);

// ---- auxiliary AdamW group (adamw.hip) ------------------------------------
// One entry per tensor of the group, in the order given to prm_adamw_init;
// pointers are refreshed whenever the caller passes different ones.
struct AuxDesc {
  void* P;        // parameter (param dtype)
  const void* G;  // gradient (grad dtype)
  float* M;       // first moment
  float* V;       // second moment
  int64_t n;      // elements
  int64_t pad;
};
// A block's share: kAdamwChunk consecutive elements of one tensor.
struct AuxChunk {
  int64_t start;
  int32_t t;
  int32_t pad;
};
// Per-launch scalars (bias corrections folded in on the host, in double).
struct AdamwParams {
  float beta1, beta2;
  float omb1, omb2;      // 1 - beta1, 1 - beta2
  float eps;
  float decay;           // 1 - lr * wd
  float step_size;       // lr / (1 - beta1^t)
  float inv_sqrt_bc2;    // 1 / sqrt(1 - beta2^t)
};
constexpr int kAdamwChunk = 2048;  // elements per block: 256 threads x 2 pieces of 4
hipError_t launch_adamw(DType pt, DType gt, const AuxDesc* desc, const AuxChunk* chunks, int32_t nchunks,
                        const AdamwParams& p, hipStream_t s);

// GEMM tile edge used by the NS5 kernels; rp and cp are multiples of it.
constexpr int kNsTile = 256;
// Prologue tile edge.
constexpr int kPrologueTile = 64;
// Row block of the tall passes (rows of one 256-column tile; 8 per wave).
constexpr int kTallRows = 32;

}  // namespace prm
