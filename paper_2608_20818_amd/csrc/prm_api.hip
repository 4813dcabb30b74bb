// C ABI and host dispatcher of libprm (declared in include/prm.h).
//
// prm_init plans once: orientation and shape scale per matrix, the row-wise
// launch classes (row length -> threads per row and chunks per thread), the
// tall-matrix work lists, and the NS5 chunks (matrices grouped by oriented
// shape, packed into a bounded workspace) with their tile work lists.
// prm_step then only enqueues kernels on the context's stream: the refresh
// indicator rho_t = 1[t mod K = 0] (Sec. 3.3, Alg. 1) is decided on the host.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/prm.h"
#include "prm_internal.h"

using namespace prm;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_TRY(expr)                                                                    \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess)                                                                \
      return fail(PRM_EHIP, "%s failed: %s", #expr, hipGetErrorString(e_));              \
  } while (0)

constexpr uint64_t kAutoBudget = 48ull << 30;  // NS5 chunk workspace cap when unset
constexpr int64_t kMaxDim = 1ll << 24;

// Makes the context's device current for one entry point and restores the
// caller's device when the call returns.
struct DeviceScope {
  int prev = -1;
  hipError_t enter(int dev) {
    hipError_t e = hipGetDevice(&prev);
    if (e != hipSuccess) {
      prev = -1;
      return e;
    }
    return prev == dev ? hipSuccess : hipSetDevice(dev);
  }
  ~DeviceScope() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

// A caller buffer must be memory of the context's device (or managed
// memory): a host pointer handed to a kernel faults the GPU, so it is refused
// before anything is enqueued.  Checked when a pointer differs from the one
// the previous call passed at the same position.
int check_device_ptr(int dev, const void* p, const char* what, int i, int k) {
  hipPointerAttribute_t a;
  hipError_t e = hipPointerGetAttributes(&a, p);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(PRM_EINVAL, "%s %d: pointer %d is not device memory (%s)", what, i, k, hipGetErrorString(e));
  }
  if (a.type == hipMemoryTypeManaged || (a.type == hipMemoryTypeDevice && a.device == dev)) return PRM_OK;
  if (a.type == hipMemoryTypeDevice)
    return fail(PRM_EINVAL, "%s %d: pointer %d is memory of device %d, the context runs on device %d", what, i, k,
                a.device, dev);
  return fail(PRM_EINVAL, "%s %d: pointer %d is host memory; device memory is required", what, i, k);
}

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
inline uint64_t align256(uint64_t x) { return (x + 255) & ~uint64_t(255); }

enum KClass {
  K_RW_WIDE = 0, K_RW_GENERIC, K_RW_TALL_STATS, K_RW_TALL_FIN, K_RW_TALL_APPLY,
  K_NS_PROLOGUE, K_NS_ALPHA, K_NS_GRAM, K_NS_POLY, K_NS_APPLY, K_NS_SPROD, K_NCLASS
};
static_assert(K_NCLASS == PRM_NUM_KERNEL_CLASSES, "kernel class table");
const char* kClassName[K_NCLASS] = {"rw_wide", "rw_generic", "rw_tall_stats",
                                    "rw_tall_finalize", "rw_tall_apply", "ns_prologue",
                                    "ns_alpha", "ns_gram", "ns_poly", "ns_apply", "ns_sprod"};

struct WideClass {
  int tpr, nch;
  std::vector<int32_t> mats, starts;
  int32_t nblocks = 0;
  size_t off_mats = 0, off_starts = 0;
  double elems = 0;
};

// The matrices of a chunk that run the same NS5 sequence, with their tile
// lists: `upper` for the symmetric r x r results (Gram, square, split
// products), `apply` for the tiles of X'^T.  Per launch over the group:
// algorithmic FLOPs of an r x r times r x c product (Gram, apply) and of an
// r x r product, and the executed FLOPs of each kind.
struct NsGroup {
  std::vector<int32_t> mats;
  std::vector<Item> upper, apply;
  size_t off_upper = 0, off_apply = 0;
  double elems = 0, alg_rc = 0, alg_rr = 0, exec_gram = 0, exec_rr = 0, exec_apply = 0;
};

struct Chunk {
  std::vector<int32_t> mats;
  std::vector<Item> prologue;
  size_t off_mats = 0, off_prologue = 0;
  double elems = 0;
  NsGroup plain, chain;  // five iterations as written; the factored form
};

struct Plan {
  int32_t n = 0;
  std::vector<int64_t> m, nn, rp, cp;
  std::vector<int32_t> tall;
  std::vector<int32_t> chain;       // NS5 in the factored form (oriented c >= 2r)
  int32_t precise = 0;              // every iterate carried as hi + lo bf16 (plain path)
  std::vector<float> s;
  std::vector<uint64_t> ws_off;     // offset of the matrix's NS region inside the chunk area
  std::vector<uint64_t> small_off;  // partial sums + alpha
  std::vector<uint64_t> tall_off;   // colpart + colinv
  std::vector<int32_t> nrb;
  uint64_t chunk_bytes = 0, small_bytes = 0, tall_bytes = 0, total_bytes = 0;
  std::vector<WideClass> wide;
  WideClass generic;
  std::vector<Item> tall_items4, tall_items1, fin_items;
  size_t off_tall4 = 0, off_tall1 = 0, off_fin = 0;
  double tall_elems4 = 0, tall_elems1 = 0;
  std::vector<Chunk> chunks;
  std::vector<int32_t> ints;   // all int32 lists, uploaded once
  std::vector<Item> items;     // all item lists, uploaded once
};

int validate_cfg(const prm_config* c) {
  if (!c) return fail(PRM_EINVAL, "cfg is NULL");
  if (c->K < 1) return fail(PRM_EINVAL, "K must be >= 1 (got %d)", c->K);
  if (!(c->beta >= 0.f && c->beta < 1.f)) return fail(PRM_EINVAL, "beta must be in [0,1)");
  if (!(c->lr >= 0.f) || !std::isfinite(c->lr)) return fail(PRM_EINVAL, "lr must be finite and >= 0");
  if (!(c->wd >= 0.f) || !std::isfinite(c->wd)) return fail(PRM_EINVAL, "wd must be finite and >= 0");
  if (!(c->gamma > 0.f) || !std::isfinite(c->gamma)) return fail(PRM_EINVAL, "gamma must be > 0");
  if (!(c->eps_rownorm > 0.f) || !std::isfinite(c->eps_rownorm))
    return fail(PRM_EINVAL, "eps_rownorm must be finite and > 0");
  if (!(c->eps_ns > 0.f) || !std::isfinite(c->eps_ns)) return fail(PRM_EINVAL, "eps_ns must be finite and > 0");
  if (!std::isfinite(c->ns_a) || !std::isfinite(c->ns_b) || !std::isfinite(c->ns_c))
    return fail(PRM_EINVAL, "NS coefficients must be finite");
  if (c->nesterov != 0 && c->nesterov != 1) return fail(PRM_EINVAL, "nesterov must be 0 or 1");
  if (c->ema_dampening != 0 && c->ema_dampening != 1) return fail(PRM_EINVAL, "ema_dampening must be 0 or 1");
  if (c->never_refresh != 0 && c->never_refresh != 1) return fail(PRM_EINVAL, "never_refresh must be 0 or 1");
  if (c->gamma_on_refresh != 0 && c->gamma_on_refresh != 1) return fail(PRM_EINVAL, "gamma_on_refresh must be 0 or 1");
  if (c->ns_plain != 0 && c->ns_plain != 1) return fail(PRM_EINVAL, "ns_plain must be 0 or 1");
  if (c->ns_precise != 0 && c->ns_precise != 1) return fail(PRM_EINVAL, "ns_precise must be 0 or 1");
  if (c->scale_mode < 0 || c->scale_mode > 2) return fail(PRM_EINVAL, "unknown scale_mode %d", c->scale_mode);
  if (c->param_dtype != PRM_F32 && c->param_dtype != PRM_BF16) return fail(PRM_EDTYPE, "unsupported param_dtype %d", c->param_dtype);
  if (c->grad_dtype != PRM_F32 && c->grad_dtype != PRM_BF16) return fail(PRM_EDTYPE, "unsupported grad_dtype %d", c->grad_dtype);
  return PRM_OK;
}

float shape_scale(int64_t m, int64_t n, int mode) {
  switch (mode) {
    case PRM_SCALE_ONE: return 1.0f;
    case PRM_SCALE_RMS_0P2: return (float)(0.2 * std::sqrt((double)std::max(m, n)));
    default: return (float)std::sqrt(std::max(1.0, (double)m / (double)n));
  }
}

// NS5 workspace of one matrix: the transposed iterate and the next one (bf16;
// in precise mode also their low parts), and the split symmetric r x r
// matrices (bf16 off-diagonal part, fp32 diagonal): two on the plain path
// (A, B), four on the factored one.
int ns_splits(int chain) { return chain ? 4 : 2; }
int ns_iterates(int precise) { return precise ? 4 : 2; }
uint64_t ns_matrix_bytes(int64_t rp, int64_t cp, int chain, int precise) {
  const uint64_t xs = align256((uint64_t)rp * cp * 2), gs = align256((uint64_t)rp * rp * 2),
                 vs = align256((uint64_t)rp * 4);
  return (uint64_t)ns_iterates(precise) * xs + (uint64_t)ns_splits(chain) * (gs + vs);
}

// Row-wise launch class of a wide row of length n (0 tpr = generic path).
void wide_class(int64_t n, int& tpr, int& nch) {
  tpr = 0;
  nch = 0;
  if (n % 8 != 0) return;
  const int64_t chunks = n / 8;
  if (chunks <= 64 * 8) { tpr = 64; nch = (int)((chunks + 63) / 64); }
  else if (chunks <= 256 * 8) { tpr = 256; nch = (int)((chunks + 255) / 256); }
  else if (chunks <= 512 * 8) { tpr = 512; nch = (int)((chunks + 511) / 512); }
}

int make_plan(int32_t n_mats, const int64_t* rows, const int64_t* cols, const prm_config* cfg,
              Plan& P) {
  int rc = validate_cfg(cfg);
  if (rc) return rc;
  if (n_mats < 0) return fail(PRM_EINVAL, "n_mats must be >= 0");
  if (n_mats > 0 && (!rows || !cols)) return fail(PRM_EINVAL, "rows/cols is NULL");
  P = Plan();
  P.n = n_mats;
  P.precise = cfg->ns_precise;
  for (int i = 0; i < n_mats; ++i) {
    const int64_t m = rows[i], n = cols[i];
    if (m < 1 || n < 1 || m > kMaxDim || n > kMaxDim)
      return fail(PRM_EINVAL, "matrix %d has invalid shape %lld x %lld", i, (long long)m, (long long)n);
    const int64_t r = std::min(m, n), c = std::max(m, n);
    P.m.push_back(m);
    P.nn.push_back(n);
    P.tall.push_back(m > n ? 1 : 0);
    // the factored form needs c >= 2r: it saves work only there, and its
    // rounding stays below the plain path's only away from square shapes;
    // precise mode runs the plain path
    P.chain.push_back(!cfg->ns_plain && !cfg->ns_precise && c >= 2 * r ? 1 : 0);
    P.rp.push_back(round_up(r, kNsTile));
    P.cp.push_back(round_up(c, kNsTile));
    P.s.push_back(shape_scale(m, n, cfg->scale_mode));
  }
  // ---- small persistent buffers: prologue partial sums + alpha per matrix ----
  uint64_t off = 0;
  P.small_off.resize(n_mats);
  for (int i = 0; i < n_mats; ++i) {
    const int64_t pt = (P.rp[i] / kPrologueTile) * (P.cp[i] / kPrologueTile);
    P.small_off[i] = off;
    off = align256(off + (uint64_t)(pt + 1) * 4);
  }
  P.small_bytes = off;
  // ---- tall buffers ----
  off = 0;
  P.tall_off.assign(n_mats, 0);
  P.nrb.assign(n_mats, 0);
  for (int i = 0; i < n_mats; ++i) {
    if (!P.tall[i]) continue;
    const int64_t nrb = (P.m[i] + kTallRows - 1) / kTallRows;
    P.nrb[i] = (int32_t)nrb;
    P.tall_off[i] = off;
    off = align256(off + (uint64_t)(nrb + 1) * P.nn[i] * 4);
  }
  P.tall_bytes = off;
  // ---- NS5 chunks: group by oriented padded shape, largest first ----
  const uint64_t budget = cfg->workspace_budget_bytes ? cfg->workspace_budget_bytes : kAutoBudget;
  std::vector<int32_t> order(n_mats);
  for (int i = 0; i < n_mats; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
    if (P.rp[a] != P.rp[b]) return P.rp[a] > P.rp[b];
    return P.cp[a] > P.cp[b];
  });
  P.ws_off.assign(n_mats, 0);
  uint64_t cur = 0;
  for (int idx : order) {
    const uint64_t need = ns_matrix_bytes(P.rp[idx], P.cp[idx], P.chain[idx], P.precise);
    if (need > budget)
      return fail(PRM_ENOMEM, "matrix %d needs %llu workspace bytes, budget is %llu", idx,
                  (unsigned long long)need, (unsigned long long)budget);
    if (P.chunks.empty() || cur + need > budget) {
      P.chunks.emplace_back();
      cur = 0;
    }
    P.chunks.back().mats.push_back(idx);
    P.ws_off[idx] = cur;
    cur += need;
    P.chunk_bytes = std::max(P.chunk_bytes, cur);
  }
  P.total_bytes = align256(P.chunk_bytes) + P.small_bytes + P.tall_bytes;
  return PRM_OK;
}

// Work groups are dispatched round-robin over the eight XCDs (group b runs on
// XCD b mod 8), and each XCD has its own L2.  A GEMM work list therefore keeps
// all tiles of one matrix on one XCD (matrix k of the chunk -> XCD k mod 8) and
// orders them in super-rows of kSuperRows tile rows, so that the ~32 groups an
// XCD runs at once share a few row and column panels of the operands.  The
// per-XCD lists are then interleaved into one launch order.
constexpr int kXcds = 8;
constexpr int kSuperRows = 4;

// Tiles (tm, tn) of a tr x tc grid (upper triangle only if `upper`) in
// super-row order.
void tile_order(int32_t mat, int32_t tr, int32_t tc, bool upper, std::vector<Item>& out) {
  for (int32_t a0 = 0; a0 < tr; a0 += kSuperRows) {
    const int32_t a1 = std::min(tr, a0 + kSuperRows);
    for (int32_t b = upper ? a0 : 0; b < tc; ++b)
      for (int32_t a = a0; a < a1; ++a)
        if (!upper || b >= a) out.push_back(Item{mat, a, b, 0});
  }
}

// Interleave per-XCD item lists so that list x lands on positions = x mod 8
// while every list still has items.
std::vector<Item> interleave_xcd(const std::vector<std::vector<Item>>& per) {
  std::vector<Item> out;
  size_t total = 0;
  for (const auto& v : per) total += v.size();
  out.reserve(total);
  std::vector<size_t> pos(per.size(), 0);
  while (out.size() < total) {
    for (size_t x = 0; x < per.size(); ++x)
      if (pos[x] < per[x].size()) out.push_back(per[x][pos[x]++]);
  }
  return out;
}

// Work lists (host side); built only by prm_init.
void build_lists(Plan& P, const prm_config* cfg) {
  // row-wise wide classes
  for (int i = 0; i < P.n; ++i) {
    if (P.tall[i]) continue;
    int tpr, nch;
    wide_class(P.nn[i], tpr, nch);
    WideClass* wc = nullptr;
    if (tpr == 0) {
      wc = &P.generic;
    } else {
      for (auto& w : P.wide)
        if (w.tpr == tpr && w.nch == nch) wc = &w;
      if (!wc) {
        P.wide.emplace_back();
        wc = &P.wide.back();
        wc->tpr = tpr;
        wc->nch = nch;
      }
    }
    const int rpb = (tpr == 64) ? 4 : 1;
    wc->mats.push_back(i);
    wc->starts.push_back(wc->nblocks);
    wc->nblocks += (int32_t)((P.m[i] + rpb - 1) / rpb);
    wc->elems += (double)P.m[i] * P.nn[i];
  }
  // tall lists
  for (int i = 0; i < P.n; ++i) {
    if (!P.tall[i]) continue;
    const int vec = (P.nn[i] % 4 == 0) ? 4 : 1;
    const int64_t slabs = (P.nn[i] + 255) / 256;  // 256-column tiles
    auto& L = vec == 4 ? P.tall_items4 : P.tall_items1;
    for (int32_t rb = 0; rb < P.nrb[i]; ++rb)
      for (int32_t sb = 0; sb < slabs; ++sb) L.push_back(Item{i, rb, sb, 0});
    (vec == 4 ? P.tall_elems4 : P.tall_elems1) += (double)P.m[i] * P.nn[i];
    for (int32_t cb = 0; cb < (P.nn[i] + 255) / 256; ++cb) P.fin_items.push_back(Item{i, 0, cb, 0});
  }
  // NS5 lists per chunk and group
  for (auto& ch : P.chunks) {
    for (int i : ch.mats) {
      const int64_t pm = (P.tall[i] ? P.cp[i] : P.rp[i]) / kPrologueTile;
      const int64_t pn = (P.tall[i] ? P.rp[i] : P.cp[i]) / kPrologueTile;
      for (int32_t a = 0; a < pm; ++a)
        for (int32_t b = 0; b < pn; ++b) ch.prologue.push_back(Item{i, a, b, 0});
      ch.elems += (double)P.m[i] * P.nn[i];
    }
    for (int grp = 0; grp < 2; ++grp) {
      NsGroup& G = grp ? ch.chain : ch.plain;
      std::vector<std::vector<Item>> u(kXcds), a(kXcds);
      for (int i : ch.mats) {
        if (P.chain[i] != grp) continue;
        const size_t k = G.mats.size();
        G.mats.push_back(i);
        const double r = (double)std::min(P.m[i], P.nn[i]), c = (double)std::max(P.m[i], P.nn[i]);
        const double rp = (double)P.rp[i], cp = (double)P.cp[i], t2 = (double)kNsTile * kNsTile;
        const int32_t tr = (int32_t)(P.rp[i] / kNsTile), tc = (int32_t)(P.cp[i] / kNsTile);
        const double upper = (double)tr * (tr + 1) / 2;
        G.elems += r * c;
        G.alg_rc += 2 * r * r * c;
        G.alg_rr += 2 * r * r * r;
        G.exec_gram += upper * 2 * t2 * cp;
        G.exec_rr += upper * 2 * t2 * rp;
        // the apply's diagonal term adds 64 MFMAs per wave to 64 per stage
        G.exec_apply += (double)tc * tr * 2 * t2 * rp * (1.0 + kNsTile / 4.0 / rp);
        // symmetric products: each matrix's (upper) tiles stay on one XCD,
        // whose 32 CUs then share its r x r panels in their L2
        tile_order(i, tr, tr, true, u[k % kXcds]);
        // apply: every XCD takes a contiguous eighth of each matrix's tile
        // order, so all XCDs stream the same factor at the same time (it is
        // read by every tile row; the last-level cache serves the repeats)
        std::vector<Item> ta;
        tile_order(i, tc, tr, false, ta);  // tiles of X'^T: rows over c, columns over r
        for (int x = 0; x < kXcds; ++x)
          a[x].insert(a[x].end(), ta.begin() + ta.size() * x / kXcds, ta.begin() + ta.size() * (x + 1) / kXcds);
      }
      G.upper = interleave_xcd(u);
      G.apply = interleave_xcd(a);
    }
  }
  (void)cfg;
  // flatten
  auto put_ints = [&](const std::vector<int32_t>& v) {
    size_t o = P.ints.size();
    P.ints.insert(P.ints.end(), v.begin(), v.end());
    return o;
  };
  auto put_items = [&](const std::vector<Item>& v) {
    size_t o = P.items.size();
    P.items.insert(P.items.end(), v.begin(), v.end());
    return o;
  };
  for (auto& w : P.wide) {
    w.off_mats = put_ints(w.mats);
    w.off_starts = put_ints(w.starts);
  }
  P.generic.off_mats = put_ints(P.generic.mats);
  P.generic.off_starts = put_ints(P.generic.starts);
  P.off_tall4 = put_items(P.tall_items4);
  P.off_tall1 = put_items(P.tall_items1);
  P.off_fin = put_items(P.fin_items);
  for (auto& ch : P.chunks) {
    ch.off_mats = put_ints(ch.mats);
    ch.off_prologue = put_items(ch.prologue);
    for (NsGroup* G : {&ch.plain, &ch.chain}) {
      G->off_upper = put_items(G->upper);
      G->off_apply = put_items(G->apply);
    }
  }
  if (P.ints.empty()) P.ints.push_back(0);
  if (P.items.empty()) P.items.push_back(Item{0, 0, 0, 0});
}

// Static descriptor fields of every matrix: shape, scale, and its regions of
// the NS5 chunk area, the small per-matrix scalars and the tall statistics
// (caller pointers are filled in before a step).
void fill_descs(const Plan& P, char* chunk_base, char* small_base, char* tall_base, std::vector<MatDesc>& desc) {
  desc.assign(P.n, MatDesc{});
  for (int i = 0; i < P.n; ++i) {
    MatDesc& d = desc[i];
    d.m = P.m[i];
    d.n = P.nn[i];
    d.s = P.s[i];
    d.tall = P.tall[i];
    d.rp = P.rp[i];
    d.cp = P.cp[i];
    const uint64_t xs = align256((uint64_t)d.rp * d.cp * 2), gs = align256((uint64_t)d.rp * d.rp * 2),
                   vs = align256((uint64_t)d.rp * 4);
    char* w = chunk_base + P.ws_off[i];
    const int nx = ns_iterates(P.precise);
    d.XT = (uint16_t*)w;
    d.XTn = (uint16_t*)(w + xs);
    d.XTl = P.precise ? (uint16_t*)(w + 2 * xs) : nullptr;
    d.XTnl = P.precise ? (uint16_t*)(w + 3 * xs) : nullptr;
    const int ns = ns_splits(P.chain[i]);
    for (int k = 0; k < 4; ++k) {
      d.S[k] = k < ns ? (uint16_t*)(w + nx * xs + k * gs) : nullptr;
      d.dS[k] = k < ns ? (float*)(w + nx * xs + ns * gs + k * vs) : nullptr;
    }
    d.ptiles_m = (int32_t)((d.tall ? d.cp : d.rp) / kPrologueTile);
    d.ptiles_n = (int32_t)((d.tall ? d.rp : d.cp) / kPrologueTile);
    d.partial = (float*)(small_base + P.small_off[i]);
    d.alpha = d.partial + (int64_t)d.ptiles_m * d.ptiles_n;
    if (d.tall) {
      d.nrb = P.nrb[i];
      d.colpart = (float*)(tall_base + P.tall_off[i]);
      d.colinv = d.colpart + (int64_t)d.nrb * d.n;
    }
  }
}

struct ProfRec {
  int cls;
  hipEvent_t e0, e1;
  double bytes, flops, exec;
};

}  // namespace

struct prm_ctx {
  prm_config cfg;
  Plan plan;
  hipStream_t stream = nullptr;
  int device = 0;
  char* d_ws = nullptr;
  MatDesc* d_desc = nullptr;
  MatDesc* h_desc = nullptr;  // pinned staging of the descriptor table
  int32_t* d_ints = nullptr;
  Item* d_items = nullptr;
  hipEvent_t upload_done = nullptr;
  bool uploaded = false;
  bool debug_last = false;
  std::vector<const void*> last_ptrs;
  std::vector<MatDesc> desc;  // host copy (workspace fields filled at init)
  // profiling
  bool prof = false;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> pool;
  size_t pool_used = 0;
};

namespace {

hipEvent_t take_event(prm_ctx* c) {
  if (c->pool_used == c->pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    c->pool.push_back(e);
  }
  return c->pool[c->pool_used++];
}

// Run `launch` on the context stream, bracketed by events when profiling.
template <typename F>
int timed(prm_ctx* c, int cls, double bytes, double flops, F&& launch, double exec = 0) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (c->prof) {
    e0 = take_event(c);
    e1 = take_event(c);
    if (!e0 || !e1) return fail(PRM_EHIP, "hipEventCreate failed");
    HIP_TRY(hipEventRecord(e0, c->stream));
  }
  hipError_t e = launch();
  if (e != hipSuccess) return fail(PRM_EHIP, "%s launch failed: %s", kClassName[cls], hipGetErrorString(e));
  if (c->prof) {
    HIP_TRY(hipEventRecord(e1, c->stream));
    c->recs.push_back(ProfRec{cls, e0, e1, bytes, flops, exec});
  }
  return PRM_OK;
}

int upload_desc(prm_ctx* c, void* const* params, const void* const* grads,
                float* const* momentum, float* const* dirs) {
  const int n = c->plan.n;
  bool same = c->uploaded && c->debug_last == (dirs != nullptr);
  if (same) {
    for (int i = 0; i < n && same; ++i)
      same = c->last_ptrs[4 * i] == params[i] && c->last_ptrs[4 * i + 1] == grads[i] &&
             c->last_ptrs[4 * i + 2] == momentum[i] &&
             c->last_ptrs[4 * i + 3] == (dirs ? (const void*)dirs[i] : nullptr);
  }
  if (same) return PRM_OK;
  if (c->uploaded) HIP_TRY(hipEventSynchronize(c->upload_done));
  for (int i = 0; i < n; ++i) {
    MatDesc& d = c->desc[i];
    d.W = params[i];
    d.G = grads[i];
    d.M = momentum[i];
    d.D = dirs ? dirs[i] : nullptr;
    c->last_ptrs[4 * i] = params[i];
    c->last_ptrs[4 * i + 1] = grads[i];
    c->last_ptrs[4 * i + 2] = momentum[i];
    c->last_ptrs[4 * i + 3] = dirs ? (const void*)dirs[i] : nullptr;
  }
  std::memcpy(c->h_desc, c->desc.data(), sizeof(MatDesc) * n);
  HIP_TRY(hipMemcpyAsync(c->d_desc, c->h_desc, sizeof(MatDesc) * n, hipMemcpyHostToDevice, c->stream));
  HIP_TRY(hipEventRecord(c->upload_done, c->stream));
  c->uploaded = true;
  c->debug_last = dirs != nullptr;
  return PRM_OK;
}

int rowwise_step(prm_ctx* c, float lr, bool debug) {
  const Plan& P = c->plan;
  const prm_config& cf = c->cfg;
  RwParams p;
  p.beta = cf.beta;
  p.gcoef = cf.ema_dampening ? 1.0f - cf.beta : 1.0f;
  p.lr = lr;
  p.decay = 1.0f - lr * cf.wd;
  p.gamma = cf.gamma;
  p.eps = cf.eps_rownorm;
  p.nesterov = cf.nesterov;
  p.write_d = debug ? 1 : 0;
  const DType wt = (DType)cf.param_dtype, gt = (DType)cf.grad_dtype;
  const double gb = gt == BF16 ? 2 : 4, wb = wt == BF16 ? 2 : 4, db = debug ? 4 : 0;
  const MatDesc* md = c->d_desc;
  int rc;
  // tall matrices first (column statistics, then their parameter write)
  for (int v : {4, 1}) {
    const auto& L = v == 4 ? P.tall_items4 : P.tall_items1;
    if (L.empty()) continue;
    const Item* items = c->d_items + (v == 4 ? P.off_tall4 : P.off_tall1);
    const double el = v == 4 ? P.tall_elems4 : P.tall_elems1;
    rc = timed(c, K_RW_TALL_STATS, el * (gb + 8), 0, [&] {
      return launch_rw_tall_stats(v, gt, md, items, (int32_t)L.size(), p, c->stream);
    });
    if (rc) return rc;
  }
  if (!P.fin_items.empty()) {
    rc = timed(c, K_RW_TALL_FIN, 0, 0, [&] {
      return launch_rw_tall_finalize(md, c->d_items + P.off_fin, (int32_t)P.fin_items.size(), p, c->stream);
    });
    if (rc) return rc;
  }
  for (int v : {4, 1}) {
    const auto& L = v == 4 ? P.tall_items4 : P.tall_items1;
    if (L.empty()) continue;
    const Item* items = c->d_items + (v == 4 ? P.off_tall4 : P.off_tall1);
    const double el = v == 4 ? P.tall_elems4 : P.tall_elems1;
    rc = timed(c, K_RW_TALL_APPLY, el * (2 * wb + db), 0, [&] {
      return launch_rw_tall_apply(v, wt, gt, md, items, (int32_t)L.size(), p, c->stream);
    });
    if (rc) return rc;
  }
  for (const auto& w : P.wide) {
    rc = timed(c, K_RW_WIDE, w.elems * (gb + 8 + 2 * wb + db), 0, [&] {
      return launch_rw_wide(w.tpr, w.nch, wt, gt, md, c->d_ints + w.off_mats,
                            c->d_ints + w.off_starts, (int32_t)w.mats.size(), w.nblocks, p,
                            c->stream);
    });
    if (rc) return rc;
  }
  if (!P.generic.mats.empty()) {
    const auto& w = P.generic;
    rc = timed(c, K_RW_GENERIC, w.elems * (gb + 8 + 2 * wb + db), 0, [&] {
      return launch_rw_generic(wt, gt, md, c->d_ints + w.off_mats, c->d_ints + w.off_starts,
                               (int32_t)w.mats.size(), w.nblocks, p, c->stream);
    });
    if (rc) return rc;
  }
  return PRM_OK;
}

int refresh_step(prm_ctx* c, float lr, bool debug) {
  const Plan& P = c->plan;
  const prm_config& cf = c->cfg;
  NsParams p;
  std::memset(&p, 0, sizeof(p));
  p.beta = cf.beta;
  p.gcoef = cf.ema_dampening ? 1.0f - cf.beta : 1.0f;
  p.nesterov = cf.nesterov;
  p.eps_ns = cf.eps_ns;
  p.a = cf.ns_a;
  p.b = cf.ns_b;
  p.c = cf.ns_c;
  p.lr = lr;
  p.decay = 1.0f - lr * cf.wd;
  p.dscale = cf.gamma_on_refresh ? cf.gamma : 1.0f;
  p.write_d = debug ? 1 : 0;
  p.hilo = P.precise;
  const bool hilo = P.precise != 0;
  const DType wt = (DType)cf.param_dtype, gt = (DType)cf.grad_dtype;
  const double gb = gt == BF16 ? 2 : 4, wb = wt == BF16 ? 2 : 4, db = debug ? 4 : 0;
  const MatDesc* md = c->d_desc;
  const float a = cf.ns_a;
  int rc;
  for (const auto& ch : P.chunks) {
    rc = timed(c, K_NS_PROLOGUE, ch.elems * (gb + 8 + (hilo ? 4 : 2)), 0, [&] {  // G, M read; M, bf16 X^T (hi, lo) written
      return launch_ns_prologue(gt, md, c->d_items + ch.off_prologue, (int32_t)ch.prologue.size(), p, c->stream);
    });
    if (rc) return rc;
    rc = timed(c, K_NS_ALPHA, 0, 0, [&] {
      return launch_ns_alpha(md, c->d_ints + ch.off_mats, (int32_t)ch.mats.size(), p, c->stream);
    });
    if (rc) return rc;
    for (const NsGroup* Gp : {&ch.plain, &ch.chain}) {
      const NsGroup& G = *Gp;
      if (G.mats.empty()) continue;
      const Item* upper = c->d_items + G.off_upper;
      const Item* apply = c->d_items + G.off_apply;
      const int32_t nu = (int32_t)G.upper.size(), na = (int32_t)G.apply.size();
      // one kernel of the sequence: Gram of the iterate `src` into S[so];
      // B = bA + cA^2 from S[sx] into S[so]; the split product
      // (S[sx] + xs I)(S[sy] + ys I) into S[so]; the apply of (S[sy] + ys I)
      // to the iterate `src`, into the other iterate or, `last`, into W
      auto gram = [&](int src, int alpha, int so) {
        p.src = src; p.use_alpha = alpha; p.so = so;
        return timed(c, K_NS_GRAM, 0, G.alg_rc, [&] {
          return launch_ns_gemm(GEMM_GRAM, wt, md, upper, nu, p, c->stream, hilo);
        }, G.exec_gram * (hilo ? 3 : 1));
      };
      auto poly = [&](int sx, int so) {
        p.sx = sx; p.sy = sx; p.so = so; p.xshift = 0.f; p.yshift = 0.f;
        return timed(c, K_NS_POLY, 0, G.alg_rr, [&] {
          return launch_ns_gemm(GEMM_POLY, wt, md, upper, nu, p, c->stream);
        }, G.exec_rr);
      };
      auto sprod = [&](int sx, float xs, int sy, float ys, int so) {
        p.sx = sx; p.sy = sy; p.so = so; p.xshift = xs; p.yshift = ys;
        return timed(c, K_NS_SPROD, 0, G.alg_rr, [&] {
          return launch_ns_gemm(GEMM_SPROD, wt, md, upper, nu, p, c->stream);
        }, G.exec_rr);
      };
      auto applyk = [&](int src, int alpha, int sy, float ys, int last) {
        p.src = src; p.use_alpha = alpha; p.sy = sy; p.yshift = ys; p.last = last;
        rc = timed(c, K_NS_APPLY, last ? G.elems * (2 * wb + db) : 0, G.alg_rc, [&] {
          return launch_ns_gemm(GEMM_APPLY, wt, md, apply, na, p, c->stream, hilo);
        }, G.exec_apply * (hilo ? 2 : 1));
        p.last = 0;
        return rc;
      };
      if (Gp == &ch.plain) {
        // eq. (app-ns-recurrence) as written: A_j = X_j X_j^T in S0, B_j in S1,
        // X_{j+1} = (aI + B_j) X_j
        for (int j = 0; j < 5; ++j) {
          if ((rc = gram(j & 1, j == 0, 0)) || (rc = poly(0, 1)) || (rc = applyk(j & 1, j == 0, 1, a, j == 4)))
            return rc;
        }
      } else {
        // the factored form, with P_j = aI + B_j:
        //   j = 0: A0 (S0) = X0 X0^T, B0 (S1)
        //   j = 1: P0^2 (S2), A1 = P0^2 A0 (S3), B1 (S0), Q = P1 P0 (S2); X2 = Q X0
        //   j = 2: A2 (S0) = X2 X2^T, B2 (S1)
        //   j = 3: P2^2 (S2), A3 = P2^2 A2 (S3), B3 (S0), Q = P3 P2 (S2)
        //   j = 4: P3^2 (S1), A4 = P3^2 A3 (S0), B4 (S1), Q = P4 Q (S3); X5 = Q X2
        if ((rc = gram(0, 1, 0)) || (rc = poly(0, 1)) ||
            (rc = sprod(1, a, 1, a, 2)) || (rc = sprod(2, 0.f, 0, 0.f, 3)) || (rc = poly(3, 0)) ||
            (rc = sprod(0, a, 1, a, 2)) || (rc = applyk(0, 1, 2, 0.f, 0)) ||
            (rc = gram(1, 0, 0)) || (rc = poly(0, 1)) ||
            (rc = sprod(1, a, 1, a, 2)) || (rc = sprod(2, 0.f, 0, 0.f, 3)) || (rc = poly(3, 0)) ||
            (rc = sprod(0, a, 1, a, 2)) ||
            (rc = sprod(0, a, 0, a, 1)) || (rc = sprod(1, 0.f, 3, 0.f, 0)) || (rc = poly(0, 1)) ||
            (rc = sprod(1, a, 2, 0.f, 3)) || (rc = applyk(1, 0, 3, 0.f, 1)))
          return rc;
      }
    }
  }
  return PRM_OK;
}

// rho_t of eq. (periodic-direction) for a validated configuration and t >= 0.
int refresh_of(const prm_config& cfg, int64_t t) {
  return cfg.never_refresh ? 0 : (t % cfg.K == 0 ? 1 : 0);
}

int do_step(prm_ctx* c, void* const* params, const void* const* grads, float* const* momentum,
            int64_t t, float lr, int32_t* did_refresh, float* const* dirs, bool debug) {
  if (!c) return fail(PRM_EINVAL, "ctx is NULL");
  if (t < 0) return fail(PRM_EINVAL, "step must be >= 0 (got %lld)", (long long)t);
  const float eta = lr < 0.f ? c->cfg.lr : lr;
  if (!std::isfinite(eta)) return fail(PRM_EINVAL, "lr must be finite");
  const int n = c->plan.n;
  if (n > 0 && (!params || !grads || !momentum))
    return fail(PRM_EINVAL, "params/grads/momentum array is NULL");
  if (debug && n > 0 && !dirs) return fail(PRM_EINVAL, "direction_out array is NULL");
  for (int i = 0; i < n; ++i) {
    const void* ps[4] = {params[i], grads[i], momentum[i], debug ? (const void*)dirs[i] : nullptr};
    for (int k = 0; k < (debug ? 4 : 3); ++k) {
      if (!ps[k] && k == 3) continue;  // direction not wanted for this matrix
      if (!ps[k]) return fail(PRM_EINVAL, "matrix %d: NULL device pointer (argument %d)", i, k);
      if ((uintptr_t)ps[k] % 16) return fail(PRM_EALIGN, "matrix %d: pointer %d is not 16-byte aligned", i, k);
      if (!c->uploaded || c->last_ptrs[4 * i + k] != ps[k]) {
        const int rc = check_device_ptr(c->device, ps[k], "matrix", i, k);
        if (rc) return rc;
      }
    }
  }
  const int rho = refresh_of(c->cfg, t);
  if (did_refresh) *did_refresh = rho;
  if (n == 0) return PRM_OK;
  DeviceScope dev;
  HIP_TRY(dev.enter(c->device));
  int rc = upload_desc(c, params, grads, momentum, debug ? dirs : nullptr);
  if (rc) return rc;
  return rho ? refresh_step(c, eta, debug) : rowwise_step(c, eta, debug);
}

}  // namespace

// ---------------------------------------------------------------------------
// auxiliary AdamW group
// ---------------------------------------------------------------------------
struct prm_adamw_ctx {
  prm_adamw_config cfg;
  hipStream_t stream = nullptr;
  int device = 0;
  std::vector<int64_t> numel;
  std::vector<AuxDesc> desc;
  AuxDesc* d_desc = nullptr;
  AuxDesc* h_desc = nullptr;  // pinned staging of the pointer table
  AuxChunk* d_chunks = nullptr;
  int32_t nchunks = 0;
  hipEvent_t upload_done = nullptr;
  bool uploaded = false;
};

namespace {

int check_adamw_config(const prm_adamw_config* c) {
  if (!c) return fail(PRM_EINVAL, "cfg is NULL");
  if (!(c->lr >= 0.f) || !std::isfinite(c->lr)) return fail(PRM_EINVAL, "lr must be finite and >= 0");
  if (!(c->beta1 >= 0.f && c->beta1 < 1.f)) return fail(PRM_EINVAL, "beta1 must be in [0,1)");
  if (!(c->beta2 >= 0.f && c->beta2 < 1.f)) return fail(PRM_EINVAL, "beta2 must be in [0,1)");
  if (!(c->eps > 0.f) || !std::isfinite(c->eps)) return fail(PRM_EINVAL, "eps must be finite and > 0");
  if (!(c->wd >= 0.f) || !std::isfinite(c->wd)) return fail(PRM_EINVAL, "wd must be finite and >= 0");
  if (c->param_dtype != PRM_F32 && c->param_dtype != PRM_BF16)
    return fail(PRM_EDTYPE, "unsupported param_dtype %d", c->param_dtype);
  if (c->grad_dtype != PRM_F32 && c->grad_dtype != PRM_BF16)
    return fail(PRM_EDTYPE, "unsupported grad_dtype %d", c->grad_dtype);
  return PRM_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// allocation-free single-matrix step (prm_step_noalloc)
//
// Its descriptor, work lists and workspace live in `scratch`, a file-scope
// device array.  In host code the name `scratch` is only a stand-in for the
// symbol: its device address, which differs per GPU, comes from
// hipGetSymbolAddress (taken once per device, with that device current) and
// is the only handle host code passes on.
// ---------------------------------------------------------------------------
static __device__ __align__(256) char scratch[PRM_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on device `dev` (the current device).
int noalloc_scratch(int dev, char** out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(PRM_EINVAL, "device %d is outside the supported range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(PRM_EHIP, "hipGetSymbolAddress of the scratch array failed on device %d: %s", dev,
                  hipGetErrorString(e));
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return PRM_OK;
}

// One work list of the single matrix: `count` items from position `off`,
// enumerated row-major over a grid with `dim` columns, or (upper) over the
// tiles (a, b), b >= a, of a dim x dim grid, row by row.  The order differs
// from the context's lists (those are arranged for L2 sharing across
// matrices); each item's output tile is computed the same way either way.
struct NoallocSeg {
  int32_t off, count, dim, upper;
};
constexpr int kNoallocSegs = 4;
struct NoallocSetup {
  MatDesc d;
  NoallocSeg seg[kNoallocSegs];
  int32_t nseg;
  int32_t nints;  // int lists: all zero for one matrix (matrix 0, first block 0)
};

// Writes the descriptor, the int lists and the work lists of one call into
// the scratch array; thread i writes entry i of every list.  Everything comes
// in the kernel arguments, so no host buffer has to outlive the call.
__global__ __launch_bounds__(256) void noalloc_setup_kernel(NoallocSetup s, MatDesc* desc, int32_t* ints,
                                                            Item* items) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i == 0) *desc = s.d;
  if (i < s.nints) ints[i] = 0;
  for (int j = 0; j < s.nseg; ++j) {
    const NoallocSeg g = s.seg[j];
    if (i >= g.count) continue;
    int32_t a, b;
    if (g.upper) {
      // i < dim (dim + 1) / 2: row a holds dim - a tiles
      int32_t k = (int32_t)i;
      a = 0;
      while (k >= g.dim - a) {
        k -= g.dim - a;
        ++a;
      }
      b = a + k;
    } else {
      a = (int32_t)(i / g.dim);
      b = (int32_t)(i % g.dim);
    }
    items[g.off + i] = Item{0, a, b, 0};
  }
}

}  // namespace

extern "C" {

void prm_config_default(prm_config* cfg) {
  if (!cfg) return;
  std::memset(cfg, 0, sizeof(*cfg));
  cfg->K = 3;
  cfg->beta = 0.95f;
  cfg->lr = 5e-3f;
  cfg->wd = 0.01f;
  cfg->gamma = 0.15f;
  cfg->eps_rownorm = 1e-8f;
  cfg->eps_ns = 1e-7f;
  cfg->ns_a = 3.4445f;
  cfg->ns_b = -4.7750f;
  cfg->ns_c = 2.0315f;
  cfg->scale_mode = PRM_SCALE_SQRT_ASPECT;
  cfg->param_dtype = PRM_BF16;
  cfg->grad_dtype = PRM_BF16;
}

int prm_schedule_is_refresh(int64_t step, int32_t K) {
  if (K < 1) return fail(PRM_EINVAL, "K must be >= 1 (got %d)", K);
  if (step < 0) return fail(PRM_EINVAL, "step must be >= 0 (got %lld)", (long long)step);
  return step % K == 0 ? 1 : 0;
}

int prm_is_refresh(const prm_ctx* ctx, int64_t step) {
  if (!ctx) return fail(PRM_EINVAL, "ctx is NULL");
  if (step < 0) return fail(PRM_EINVAL, "step must be >= 0 (got %lld)", (long long)step);
  return refresh_of(ctx->cfg, step);
}

int prm_workspace_bytes(const prm_ctx* ctx, size_t* out_bytes) {
  if (!ctx || !out_bytes) return fail(PRM_EINVAL, "ctx and out_bytes must not be NULL");
  *out_bytes = (size_t)ctx->plan.total_bytes;
  return PRM_OK;
}

int prm_plan_workspace_bytes(int32_t n_mats, const int64_t* rows, const int64_t* cols,
                             const prm_config* cfg, uint64_t* out_bytes) {
  if (!out_bytes) return fail(PRM_EINVAL, "out_bytes is NULL");
  Plan P;
  int rc = make_plan(n_mats, rows, cols, cfg, P);
  if (rc) return rc;
  *out_bytes = P.total_bytes;
  return PRM_OK;
}

int prm_init(prm_ctx** out, int32_t n_mats, const int64_t* rows, const int64_t* cols,
             const prm_config* cfg, void* hip_stream) {
  if (!out) return fail(PRM_EINVAL, "out is NULL");
  *out = nullptr;
  prm_ctx* c = new prm_ctx();
  int rc = make_plan(n_mats, rows, cols, cfg, c->plan);
  if (rc) {
    delete c;
    return rc;
  }
  c->cfg = *cfg;
  c->stream = (hipStream_t)hip_stream;
  build_lists(c->plan, cfg);
  Plan& P = c->plan;
  auto cleanup = [&](int code) {
    prm_destroy(c);
    return code;
  };
  hipError_t e = hipGetDevice(&c->device);
  if (e != hipSuccess) return cleanup(fail(PRM_EHIP, "hipGetDevice failed: %s", hipGetErrorString(e)));
  if (P.total_bytes) {
    e = hipMalloc((void**)&c->d_ws, P.total_bytes);
    if (e != hipSuccess)
      return cleanup(fail(PRM_ENOMEM, "hipMalloc of %llu workspace bytes failed: %s",
                          (unsigned long long)P.total_bytes, hipGetErrorString(e)));
    e = hipMemsetAsync(c->d_ws, 0, P.total_bytes, c->stream);
    if (e != hipSuccess) return cleanup(fail(PRM_EHIP, "hipMemsetAsync failed: %s", hipGetErrorString(e)));
  }
  const size_t nd = std::max<int32_t>(P.n, 1);
  if ((e = hipMalloc((void**)&c->d_desc, sizeof(MatDesc) * nd)) != hipSuccess ||
      (e = hipHostMalloc((void**)&c->h_desc, sizeof(MatDesc) * nd, hipHostMallocDefault)) != hipSuccess ||
      (e = hipMalloc((void**)&c->d_ints, sizeof(int32_t) * P.ints.size())) != hipSuccess ||
      (e = hipMalloc((void**)&c->d_items, sizeof(Item) * P.items.size())) != hipSuccess ||
      (e = hipEventCreateWithFlags(&c->upload_done, hipEventDisableTiming)) != hipSuccess)
    return cleanup(fail(PRM_ENOMEM, "allocation failed: %s", hipGetErrorString(e)));
  e = hipMemcpy(c->d_ints, P.ints.data(), sizeof(int32_t) * P.ints.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess)
    e = hipMemcpy(c->d_items, P.items.data(), sizeof(Item) * P.items.size(), hipMemcpyHostToDevice);
  if (e != hipSuccess) return cleanup(fail(PRM_EHIP, "hipMemcpy failed: %s", hipGetErrorString(e)));
  // static descriptor fields
  c->last_ptrs.assign(4 * (size_t)P.n, nullptr);
  char* small_base = c->d_ws + align256(P.chunk_bytes);
  fill_descs(P, c->d_ws, small_base, small_base + P.small_bytes, c->desc);
  e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return cleanup(fail(PRM_EHIP, "hipStreamSynchronize failed: %s", hipGetErrorString(e)));
  *out = c;
  return PRM_OK;
}

int prm_step(prm_ctx* ctx, void* const* params, const void* const* grads, float* const* momentum,
             int64_t step, float lr, int32_t* did_refresh) {
  return do_step(ctx, params, grads, momentum, step, lr, did_refresh, nullptr, false);
}

int prm_step_debug(prm_ctx* ctx, void* const* params, const void* const* grads,
                   float* const* momentum, int64_t step, float lr, int32_t* did_refresh,
                   float* const* direction_out) {
  return do_step(ctx, params, grads, momentum, step, lr, did_refresh, direction_out, true);
}

int prm_profile_enable(prm_ctx* ctx, int32_t enable) {
  if (!ctx) return fail(PRM_EINVAL, "ctx is NULL");
  ctx->prof = enable != 0;
  return PRM_OK;
}

int prm_profile_read(prm_ctx* ctx, prm_kernel_stats* out, int32_t n) {
  if (!ctx) return fail(PRM_EINVAL, "ctx is NULL");
  if (n > 0 && !out) return fail(PRM_EINVAL, "out is NULL");
  HIP_TRY(hipStreamSynchronize(ctx->stream));
  prm_kernel_stats acc[K_NCLASS];
  std::memset(acc, 0, sizeof(acc));
  for (int k = 0; k < K_NCLASS; ++k) std::snprintf(acc[k].name, sizeof(acc[k].name), "%s", kClassName[k]);
  for (const auto& r : ctx->recs) {
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, r.e0, r.e1));
    acc[r.cls].launches += 1;
    acc[r.cls].total_ms += ms;
    acc[r.cls].alg_bytes += r.bytes;
    acc[r.cls].alg_flops += r.flops;
    acc[r.cls].exec_flops += r.exec;
  }
  ctx->recs.clear();
  ctx->pool_used = 0;
  for (int k = 0; k < std::min<int32_t>(n, K_NCLASS); ++k) out[k] = acc[k];
  return PRM_OK;
}

int prm_destroy(prm_ctx* c) {
  if (!c) return PRM_OK;
  int rc = PRM_OK;
  if (c->d_ws || c->d_desc) {
    if (hipStreamSynchronize(c->stream) != hipSuccess) rc = fail(PRM_EHIP, "hipStreamSynchronize failed in prm_destroy");
  }
  if (c->d_ws) (void)hipFree(c->d_ws);
  if (c->d_desc) (void)hipFree(c->d_desc);
  if (c->h_desc) (void)hipHostFree(c->h_desc);
  if (c->d_ints) (void)hipFree(c->d_ints);
  if (c->d_items) (void)hipFree(c->d_items);
  if (c->upload_done) (void)hipEventDestroy(c->upload_done);
  for (auto e : c->pool) (void)hipEventDestroy(e);
  delete c;
  return rc;
}

void prm_adamw_config_default(prm_adamw_config* cfg) {
  if (!cfg) return;
  std::memset(cfg, 0, sizeof(*cfg));
  cfg->lr = 1e-4f;
  cfg->beta1 = 0.9f;
  cfg->beta2 = 0.95f;
  cfg->eps = 1e-8f;
  cfg->wd = 0.01f;
  cfg->param_dtype = PRM_BF16;
  cfg->grad_dtype = PRM_BF16;
}

int prm_adamw_init(prm_adamw_ctx** out, int32_t n_tensors, const int64_t* numel,
                   const prm_adamw_config* cfg, void* hip_stream) {
  if (!out) return fail(PRM_EINVAL, "out is NULL");
  *out = nullptr;
  int rc = check_adamw_config(cfg);
  if (rc) return rc;
  if (n_tensors < 0) return fail(PRM_EINVAL, "n_tensors must be >= 0");
  if (n_tensors > 0 && !numel) return fail(PRM_EINVAL, "numel is NULL");
  std::vector<AuxChunk> chunks;
  for (int32_t i = 0; i < n_tensors; ++i) {
    if (numel[i] < 0 || numel[i] > (int64_t(1) << 40))
      return fail(PRM_EINVAL, "tensor %d has invalid size %lld", i, (long long)numel[i]);
    for (int64_t e = 0; e < numel[i]; e += kAdamwChunk) chunks.push_back(AuxChunk{e, i, 0});
    if (chunks.size() > (size_t)INT32_MAX) return fail(PRM_EINVAL, "aux group too large for one launch");
  }
  prm_adamw_ctx* c = new prm_adamw_ctx();
  c->cfg = *cfg;
  c->stream = (hipStream_t)hip_stream;
  c->numel.assign(numel, numel + n_tensors);
  c->desc.assign(n_tensors, AuxDesc{});
  for (int32_t i = 0; i < n_tensors; ++i) c->desc[i].n = numel[i];
  c->nchunks = (int32_t)chunks.size();
  hipError_t e = hipGetDevice(&c->device);
  const size_t nd = std::max<size_t>(1, (size_t)n_tensors);
  if (e == hipSuccess) e = hipMalloc((void**)&c->d_desc, sizeof(AuxDesc) * nd);
  if (e == hipSuccess) e = hipHostMalloc((void**)&c->h_desc, sizeof(AuxDesc) * nd, hipHostMallocDefault);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->upload_done, hipEventDisableTiming);
  if (e == hipSuccess && !chunks.empty()) {
    e = hipMalloc((void**)&c->d_chunks, sizeof(AuxChunk) * chunks.size());
    if (e == hipSuccess)
      e = hipMemcpy(c->d_chunks, chunks.data(), sizeof(AuxChunk) * chunks.size(), hipMemcpyHostToDevice);
  }
  if (e != hipSuccess) {
    rc = fail(e == hipErrorOutOfMemory ? PRM_ENOMEM : PRM_EHIP, "prm_adamw_init: %s", hipGetErrorString(e));
    prm_adamw_destroy(c);
    return rc;
  }
  *out = c;
  return PRM_OK;
}

int prm_adamw_step(prm_adamw_ctx* c, void* const* params, const void* const* grads, float* const* exp_avg,
                   float* const* exp_avg_sq, int64_t t, float lr) {
  if (!c) return fail(PRM_EINVAL, "ctx is NULL");
  if (t < 1) return fail(PRM_EINVAL, "t must be >= 1 (got %lld)", (long long)t);
  const float eta = lr < 0.f ? c->cfg.lr : lr;
  if (!std::isfinite(eta)) return fail(PRM_EINVAL, "lr must be finite");
  const int n = (int)c->numel.size();
  if (n > 0 && (!params || !grads || !exp_avg || !exp_avg_sq))
    return fail(PRM_EINVAL, "params/grads/exp_avg/exp_avg_sq array is NULL");
  bool same = c->uploaded;
  for (int i = 0; i < n; ++i) {
    if (c->numel[i] == 0) continue;
    const void* ps[4] = {params[i], grads[i], exp_avg[i], exp_avg_sq[i]};
    for (int k = 0; k < 4; ++k) {
      if (!ps[k]) return fail(PRM_EINVAL, "tensor %d: NULL device pointer (argument %d)", i, k);
      if ((uintptr_t)ps[k] % 16) return fail(PRM_EALIGN, "tensor %d: pointer %d is not 16-byte aligned", i, k);
    }
    const AuxDesc& d = c->desc[i];
    const void* prev[4] = {d.P, d.G, d.M, d.V};
    for (int k = 0; k < 4; ++k) {
      if (!c->uploaded || prev[k] != ps[k]) {
        const int rc = check_device_ptr(c->device, ps[k], "tensor", i, k);
        if (rc) return rc;
      }
    }
    same = same && d.P == params[i] && d.G == grads[i] && d.M == exp_avg[i] && d.V == exp_avg_sq[i];
  }
  if (c->nchunks == 0) return PRM_OK;
  DeviceScope dev;
  HIP_TRY(dev.enter(c->device));
  if (!same) {
    if (c->uploaded) HIP_TRY(hipEventSynchronize(c->upload_done));
    for (int i = 0; i < n; ++i) {
      AuxDesc& d = c->desc[i];
      if (c->numel[i] == 0) {
        d.P = nullptr; d.G = nullptr; d.M = nullptr; d.V = nullptr;
        continue;
      }
      d.P = params[i];
      d.G = grads[i];
      d.M = exp_avg[i];
      d.V = exp_avg_sq[i];
    }
    std::memcpy(c->h_desc, c->desc.data(), sizeof(AuxDesc) * n);
    HIP_TRY(hipMemcpyAsync(c->d_desc, c->h_desc, sizeof(AuxDesc) * n, hipMemcpyHostToDevice, c->stream));
    HIP_TRY(hipEventRecord(c->upload_done, c->stream));
    c->uploaded = true;
  }
  const double b1 = c->cfg.beta1, b2 = c->cfg.beta2;
  const double bc1 = 1.0 - std::pow(b1, (double)t), bc2 = 1.0 - std::pow(b2, (double)t);
  AdamwParams a;
  a.beta1 = (float)b1;
  a.beta2 = (float)b2;
  a.omb1 = (float)(1.0 - b1);
  a.omb2 = (float)(1.0 - b2);
  a.eps = c->cfg.eps;
  a.decay = (float)(1.0 - (double)eta * (double)c->cfg.wd);
  a.step_size = (float)((double)eta / bc1);
  a.inv_sqrt_bc2 = (float)(1.0 / std::sqrt(bc2));
  hipError_t e = launch_adamw((DType)c->cfg.param_dtype, (DType)c->cfg.grad_dtype, c->d_desc, c->d_chunks,
                              c->nchunks, a, c->stream);
  if (e != hipSuccess) return fail(PRM_EHIP, "adamw launch failed: %s", hipGetErrorString(e));
  return PRM_OK;
}

int prm_adamw_destroy(prm_adamw_ctx* c) {
  if (!c) return PRM_OK;
  int rc = PRM_OK;
  if (c->d_desc && hipStreamSynchronize(c->stream) != hipSuccess)
    rc = fail(PRM_EHIP, "hipStreamSynchronize failed in prm_adamw_destroy");
  if (c->d_desc) (void)hipFree(c->d_desc);
  if (c->h_desc) (void)hipHostFree(c->h_desc);
  if (c->d_chunks) (void)hipFree(c->d_chunks);
  if (c->upload_done) (void)hipEventDestroy(c->upload_done);
  delete c;
  return rc;
}

int prm_peak_mfma(void* hip_stream, int32_t iters, double* tflops, double* clock_ghz) {
  if (!tflops || !clock_ghz) return fail(PRM_EINVAL, "tflops and clock_ghz must not be NULL");
  if (iters < 1 || iters > (1 << 24)) return fail(PRM_EINVAL, "iters must be in [1, 2^24] (got %d)", iters);
  hipStream_t s = (hipStream_t)hip_stream;
  int dev = 0, cus = 0;
  HIP_TRY(hipGetDevice(&dev));
  HIP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  const int blocks = 4 * cus;  // 16 waves per CU
  float* sink = nullptr;
  unsigned long long* clk = nullptr;
  HIP_TRY(hipMalloc(&sink, (size_t)blocks * 256 * sizeof(float)));
  if (hipMalloc(&clk, (size_t)blocks * 2 * sizeof(unsigned long long)) != hipSuccess) {
    (void)hipFree(sink);
    return fail(PRM_ENOMEM, "hipMalloc of the probe clocks failed");
  }
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = PRM_OK;
  std::vector<unsigned long long> h((size_t)blocks * 2);
  float ms = 0.f;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess ||
      launch_probe_mfma(blocks, sink, clk, 64, s) != hipSuccess ||  // warm-up
      hipEventRecord(e0, s) != hipSuccess || launch_probe_mfma(blocks, sink, clk, iters, s) != hipSuccess ||
      hipEventRecord(e1, s) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
      hipEventElapsedTime(&ms, e0, e1) != hipSuccess ||
      hipMemcpy(h.data(), clk, h.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost) != hipSuccess)
    rc = fail(PRM_EHIP, "MFMA probe failed: %s", hipGetErrorString(hipGetLastError()));
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  (void)hipFree(sink);
  (void)hipFree(clk);
  if (rc) return rc;
  double cyc = 0, ref = 0;
  for (int b = 0; b < blocks; ++b) { cyc += (double)h[2 * b]; ref += (double)h[2 * b + 1]; }
  // 4 waves per block, 8 MFMAs of 32 x 32 x 16 (2 FLOPs per MAC) per iteration
  const double flops = (double)blocks * 4 * (double)iters * 8 * (32.0 * 32 * 16 * 2);
  *tflops = flops / (ms * 1e-3) / 1e12;
  *clock_ghz = ref > 0 ? cyc / ref * 0.1 : 0.0;  // reference clock: 100 MHz
  return PRM_OK;
}

int prm_peak_hbm(void* hip_stream, uint64_t bytes, double* read_gbs, double* write_gbs, double* copy_gbs,
                 double* rowwise_gbs) {
  if (!read_gbs || !write_gbs || !copy_gbs || !rowwise_gbs) return fail(PRM_EINVAL, "output pointers must not be NULL");
  if (bytes < (1u << 20) || bytes % 16) return fail(PRM_EINVAL, "bytes must be >= 1 MiB and a multiple of 16");
  hipStream_t s = (hipStream_t)hip_stream;
  int dev = 0, cus = 0;
  HIP_TRY(hipGetDevice(&dev));
  HIP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  void *x = nullptr, *y = nullptr;
  unsigned* sink = nullptr;
  if (hipMalloc(&x, bytes) != hipSuccess || hipMalloc(&y, bytes) != hipSuccess ||
      hipMalloc(&sink, 256) != hipSuccess) {
    if (x) (void)hipFree(x);
    if (y) (void)hipFree(y);
    return fail(PRM_ENOMEM, "hipMalloc of 2 x %llu probe bytes failed", (unsigned long long)bytes);
  }
  const int64_t n16 = (int64_t)(bytes / 16);
  // one 16-byte element per thread: the dispatcher then walks the buffers in
  // address order, which streams faster than a few grid-striding blocks
  const int64_t nb = (n16 + 255) / 256;
  if (nb > (int64_t)INT32_MAX) {
    (void)hipFree(x);
    (void)hipFree(y);
    (void)hipFree(sink);
    return fail(PRM_EINVAL, "bytes too large for one probe grid");
  }
  (void)cus;
  // the row-wise pass: pieces of 4 elements (16 bytes of x), 512 per block
  const int grid[4] = {(int)nb, (int)nb, (int)nb, (int)((n16 + 511) / 512)};
  const int64_t count[4] = {n16, n16, n16, n16};
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = PRM_OK;
  double* out[4] = {read_gbs, write_gbs, copy_gbs, rowwise_gbs};
  const double moved[4] = {(double)bytes, (double)bytes, 2.0 * (double)bytes, 4.0 * 14.0 * (double)n16};
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess ||
      launch_probe_stream(1, grid[1], nullptr, x, n16, sink, s) != hipSuccess)  // defined contents of x
    rc = fail(PRM_EHIP, "HBM probe setup failed");
  for (int kind = 0; kind < 4 && rc == PRM_OK; ++kind) {
    float best = 0.f;
    for (int rep = 0; rep < 4 && rc == PRM_OK; ++rep) {  // first repetition is a warm-up
      float ms = 0.f;
      if (hipEventRecord(e0, s) != hipSuccess || launch_probe_stream(kind, grid[kind], x, y, count[kind], sink, s) != hipSuccess ||
          hipEventRecord(e1, s) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
          hipEventElapsedTime(&ms, e0, e1) != hipSuccess) {
        rc = fail(PRM_EHIP, "HBM probe kernel %d failed: %s", kind, hipGetErrorString(hipGetLastError()));
        break;
      }
      if (rep > 0 && (best == 0.f || ms < best)) best = ms;
    }
    if (rc == PRM_OK) *out[kind] = moved[kind] / (best * 1e-3) / 1e9;
  }
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  (void)hipFree(x);
  (void)hipFree(y);
  (void)hipFree(sink);
  return rc;
}

int prm_step_noalloc(const prm_config* cfg, int64_t rows, int64_t cols, void* param, const void* grad,
                     float* momentum, int64_t step, float lr, int32_t* did_refresh, void* hip_stream) {
  if (!cfg) return fail(PRM_EINVAL, "cfg is NULL");
  if (step < 0) return fail(PRM_EINVAL, "step must be >= 0 (got %lld)", (long long)step);
  if (cfg->ns_precise) return fail(PRM_EINVAL, "ns_precise is not available in the allocation-free step");
  const float eta = lr < 0.f ? cfg->lr : lr;
  if (!std::isfinite(eta)) return fail(PRM_EINVAL, "lr must be finite");
  // the workspace cap is the scratch array, checked below
  prm_config c2 = *cfg;
  c2.workspace_budget_bytes = 1ull << 62;
  Plan P;
  int rc = make_plan(1, &rows, &cols, &c2, P);
  if (rc) return rc;
  const void* ps[3] = {param, grad, momentum};
  for (int k = 0; k < 3; ++k) {
    if (!ps[k]) return fail(PRM_EINVAL, "NULL device pointer (argument %d)", k);
    if ((uintptr_t)ps[k] % 16) return fail(PRM_EALIGN, "pointer %d is not 16-byte aligned", k);
  }
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  for (int k = 0; k < 3; ++k) {
    rc = check_device_ptr(dev, ps[k], "matrix", 0, k);
    if (rc) return rc;
  }
  const int rho = refresh_of(c2, step);
  // scratch layout: descriptor | int lists | work lists | per-matrix scalars |
  // NS5 workspace (refresh) or tall column statistics (row-wise)
  const int64_t T = P.rp[0] / kNsTile, tc = P.cp[0] / kNsTile;
  const int64_t pn = (P.tall[0] ? P.rp[0] : P.cp[0]) / kPrologueTile;
  const int64_t pm = (P.tall[0] ? P.cp[0] : P.rp[0]) / kPrologueTile;
  const int64_t slabs = (P.nn[0] + 255) / 256;
  const int64_t nitems = rho ? pm * pn + T * (T + 1) / 2 + tc * T : (P.tall[0] ? (int64_t)P.nrb[0] * slabs + slabs : 0);
  const uint64_t off_ints = align256(sizeof(MatDesc)), off_items = off_ints + 256;
  const uint64_t off_small = off_items + align256((uint64_t)std::max<int64_t>(nitems, 1) * sizeof(Item));
  const uint64_t off_big = off_small + align256(P.small_bytes);
  const uint64_t need = off_big + (rho ? P.chunk_bytes : P.tall_bytes);
  if (need > PRM_NOALLOC_SCRATCH_BYTES)
    return fail(PRM_ENOMEM, "a %s step of a %lld x %lld matrix needs %llu scratch bytes; the allocation-free step has %llu",
                rho ? "refresh" : "row-wise", (long long)rows, (long long)cols, (unsigned long long)need,
                (unsigned long long)PRM_NOALLOC_SCRATCH_BYTES);
  build_lists(P, &c2);
  if (P.ints.size() > 64) return fail(PRM_EHIP, "internal: %zu int list entries", P.ints.size());
  for (int32_t v : P.ints)
    if (v != 0) return fail(PRM_EHIP, "internal: nonzero int list entry for one matrix");
  // the work lists this step launches, packed from item 0
  NoallocSetup s;
  std::memset(&s, 0, sizeof(s));
  int32_t pos = 0;
  auto add = [&](size_t& off, size_t count, int64_t want, int64_t dim, int upper) {
    if ((int64_t)count != want || s.nseg == kNoallocSegs) return false;
    off = (size_t)pos;
    s.seg[s.nseg++] = NoallocSeg{pos, (int32_t)count, (int32_t)dim, upper};
    pos += (int32_t)count;
    return true;
  };
  bool ok = true;
  if (rho) {
    Chunk& ch = P.chunks[0];
    NsGroup& G = P.chain[0] ? ch.chain : ch.plain;  // the other group is empty
    ok = add(ch.off_prologue, ch.prologue.size(), pm * pn, pn, 0) &&
         add(G.off_upper, G.upper.size(), T * (T + 1) / 2, T, 1) &&
         add(G.off_apply, G.apply.size(), tc * T, T, 0);
  } else if (P.tall[0]) {
    const bool v4 = !P.tall_items4.empty();
    ok = add(v4 ? P.off_tall4 : P.off_tall1, v4 ? P.tall_items4.size() : P.tall_items1.size(),
             (int64_t)P.nrb[0] * slabs, slabs, 0) &&
         add(P.off_fin, P.fin_items.size(), slabs, slabs, 0);
  }
  if (!ok || pos != nitems) return fail(PRM_EHIP, "internal: work list sizes disagree with the plan");
  s.nints = (int32_t)P.ints.size();
  char* base = nullptr;
  rc = noalloc_scratch(dev, &base);
  if (rc) return rc;
  std::vector<MatDesc> desc;
  fill_descs(P, base + off_big, base + off_small, base + off_big, desc);
  s.d = desc[0];
  s.d.W = param;
  s.d.G = grad;
  s.d.M = momentum;
  s.d.D = nullptr;
  if (did_refresh) *did_refresh = rho;
  prm_ctx c;
  c.cfg = c2;
  c.stream = (hipStream_t)hip_stream;
  c.device = dev;
  c.d_desc = reinterpret_cast<MatDesc*>(base);
  c.d_ints = reinterpret_cast<int32_t*>(base + off_ints);
  c.d_items = reinterpret_cast<Item*>(base + off_items);
  const int64_t threads = std::max<int64_t>({(int64_t)pos, (int64_t)s.nints, 1});
  noalloc_setup_kernel<<<dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, c.stream>>>(s, c.d_desc, c.d_ints,
                                                                                           c.d_items);
  HIP_TRY(hipGetLastError());
  c.plan = std::move(P);
  return rho ? refresh_step(&c, eta, false) : rowwise_step(&c, eta, false);
}

const char* prm_last_error(void) { return g_err.c_str(); }

}  // extern "C"
