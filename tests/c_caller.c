/*
 * A caller of libprm written in plain C: the HIP runtime for device memory and
 * a stream, the C ABI of include/prm.h for the optimizer, nothing else (no
 * PyTorch, no Python objects).  The GPU tests load it as a shared object and
 * compare what it writes with the oracle.
 *
 * prm_c_run_case(dir) reads a case from `dir`:
 *   case.txt      line 1: n_mats K steps t0 param_dtype grad_dtype (0 f32, 1 bf16)
 *                 line 2: beta lr wd gamma
 *                 then one line "m n" per matrix
 *   W<i>.bin      initial parameters (param_dtype, row-major m x n)
 *   M<i>.bin      initial momentum (fp32)
 *   G<i>_<s>.bin  gradient of step s = 0 .. steps-1 (grad_dtype)
 * runs steps t0 .. t0 + steps - 1 through prm_step_debug on one stream, and
 * writes W<i>.out, M<i>.out (after the last step), D<i>.out (the direction of
 * the last step, fp32) and rho.txt (rho_t of every step: from prm_step_debug,
 * from prm_is_refresh on the context and from prm_schedule_is_refresh).
 * Returns 0, or -1 with a message in `msg`.
 */
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "prm.h"

typedef struct {
  char* msg;
  int msglen;
} Err;

static int failf(Err* e, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(e->msg, (size_t)e->msglen, fmt, ap);
  va_end(ap);
  return -1;
}

static size_t dsize(int dt) { return dt == PRM_BF16 ? 2 : 4; }

/* Reads exactly `bytes` from dir/name into a new host buffer. */
static void* read_file(const char* dir, const char* name, size_t bytes, Err* e) {
  char path[1024];
  snprintf(path, sizeof(path), "%s/%s", dir, name);
  FILE* f = fopen(path, "rb");
  if (!f) {
    failf(e, "cannot open %s", path);
    return NULL;
  }
  void* buf = malloc(bytes ? bytes : 1);
  size_t got = buf ? fread(buf, 1, bytes, f) : 0;
  fclose(f);
  if (!buf || got != bytes) {
    free(buf);
    failf(e, "%s: expected %zu bytes, read %zu", path, bytes, got);
    return NULL;
  }
  return buf;
}

static int write_file(const char* dir, const char* name, const void* buf, size_t bytes, Err* e) {
  char path[1024];
  snprintf(path, sizeof(path), "%s/%s", dir, name);
  FILE* f = fopen(path, "wb");
  if (!f) return failf(e, "cannot create %s", path);
  size_t put = fwrite(buf, 1, bytes, f);
  fclose(f);
  return put == bytes ? 0 : failf(e, "short write to %s", path);
}

/* Host file -> new device buffer of the same size. */
static void* upload(const char* dir, const char* name, size_t bytes, Err* e) {
  void* h = read_file(dir, name, bytes, e);
  if (!h) return NULL;
  void* d = NULL;
  hipError_t he = hipMalloc(&d, bytes);
  if (he == hipSuccess) he = hipMemcpy(d, h, bytes, hipMemcpyHostToDevice);
  free(h);
  if (he != hipSuccess) {
    if (d) (void)hipFree(d);
    failf(e, "%s: %s", name, hipGetErrorString(he));
    return NULL;
  }
  return d;
}

/* Device buffer -> dir/name. */
static int download(const char* dir, const char* name, const void* d, size_t bytes, Err* e) {
  void* h = malloc(bytes ? bytes : 1);
  if (!h) return failf(e, "out of host memory");
  hipError_t he = hipMemcpy(h, d, bytes, hipMemcpyDeviceToHost);
  int rc = he == hipSuccess ? write_file(dir, name, h, bytes, e) : failf(e, "%s: %s", name, hipGetErrorString(he));
  free(h);
  return rc;
}

int prm_c_run_case(const char* dir, char* msg, int msglen) {
  Err e = {msg, msglen};
  if (msg && msglen > 0) msg[0] = '\0';
  char path[1024];
  snprintf(path, sizeof(path), "%s/case.txt", dir);
  FILE* f = fopen(path, "r");
  if (!f) return failf(&e, "cannot open %s", path);
  int n = 0, K = 0, steps = 0, pdt = 0, gdt = 0;
  long long t0 = 0;
  float beta = 0.f, lr = 0.f, wd = 0.f, gamma = 0.f;
  if (fscanf(f, "%d %d %d %lld %d %d", &n, &K, &steps, &t0, &pdt, &gdt) != 6 ||
      fscanf(f, "%f %f %f %f", &beta, &lr, &wd, &gamma) != 4 || n < 1 || n > 4096 || steps < 1) {
    fclose(f);
    return failf(&e, "malformed %s", path);
  }
  int64_t* rows = calloc((size_t)n, sizeof(int64_t));
  int64_t* cols = calloc((size_t)n, sizeof(int64_t));
  void** W = calloc((size_t)n, sizeof(void*));
  void** G = calloc((size_t)n, sizeof(void*));
  float** M = calloc((size_t)n, sizeof(float*));
  float** D = calloc((size_t)n, sizeof(float*));
  int rc = 0;
  if (!rows || !cols || !W || !G || !M || !D) rc = failf(&e, "out of host memory");
  for (int i = 0; i < n && rc == 0; ++i) {
    long long m = 0, c = 0;
    if (fscanf(f, "%lld %lld", &m, &c) != 2 || m < 1 || c < 1) rc = failf(&e, "malformed shape line %d", i);
    rows[i] = m;
    cols[i] = c;
  }
  fclose(f);

  hipStream_t stream = NULL;
  prm_ctx* ctx = NULL;
  if (rc == 0 && hipStreamCreate(&stream) != hipSuccess) rc = failf(&e, "hipStreamCreate failed");
  if (rc == 0) {
    prm_config cfg;
    prm_config_default(&cfg);
    cfg.K = K;
    cfg.beta = beta;
    cfg.lr = lr;
    cfg.wd = wd;
    cfg.gamma = gamma;
    cfg.param_dtype = pdt;
    cfg.grad_dtype = gdt;
    if (prm_init(&ctx, n, rows, cols, &cfg, (void*)stream) != PRM_OK)
      rc = failf(&e, "prm_init: %s", prm_last_error());
  }
  char name[64];
  for (int i = 0; i < n && rc == 0; ++i) {
    const size_t el = (size_t)rows[i] * (size_t)cols[i];
    snprintf(name, sizeof(name), "W%d.bin", i);
    if (!(W[i] = upload(dir, name, el * dsize(pdt), &e))) rc = -1;
    snprintf(name, sizeof(name), "M%d.bin", i);
    if (rc == 0 && !(M[i] = (float*)upload(dir, name, el * 4, &e))) rc = -1;
    if (rc == 0 && (hipMalloc((void**)&G[i], el * dsize(gdt)) != hipSuccess ||
                    hipMalloc((void**)&D[i], el * 4) != hipSuccess))
      rc = failf(&e, "hipMalloc failed for matrix %d", i);
  }
  FILE* rf = NULL;
  if (rc == 0) {
    snprintf(path, sizeof(path), "%s/rho.txt", dir);
    if (!(rf = fopen(path, "w"))) rc = failf(&e, "cannot create %s", path);
  }
  for (int s = 0; s < steps && rc == 0; ++s) {
    for (int i = 0; i < n && rc == 0; ++i) {
      const size_t bytes = (size_t)rows[i] * (size_t)cols[i] * dsize(gdt);
      snprintf(name, sizeof(name), "G%d_%d.bin", i, s);
      void* h = read_file(dir, name, bytes, &e);
      if (!h) {
        rc = -1;
        break;
      }
      /* the previous step may still read G: order the copy on the same stream */
      hipError_t he = hipMemcpyAsync(G[i], h, bytes, hipMemcpyHostToDevice, stream);
      if (he == hipSuccess) he = hipStreamSynchronize(stream);
      free(h);
      if (he != hipSuccess) rc = failf(&e, "gradient upload: %s", hipGetErrorString(he));
    }
    if (rc) break;
    const long long t = t0 + s;
    int32_t rho = -1;
    if (prm_step_debug(ctx, W, (const void* const*)G, M, t, -1.0f, &rho, D) != PRM_OK) {
      rc = failf(&e, "prm_step_debug(t=%lld): %s", t, prm_last_error());
      break;
    }
    fprintf(rf, "%lld %d %d %d\n", t, rho, prm_is_refresh(ctx, t), prm_schedule_is_refresh(t, K));
  }
  if (rf) fclose(rf);
  if (rc == 0 && hipStreamSynchronize(stream) != hipSuccess) rc = failf(&e, "hipStreamSynchronize failed");
  for (int i = 0; i < n && rc == 0; ++i) {
    const size_t el = (size_t)rows[i] * (size_t)cols[i];
    snprintf(name, sizeof(name), "W%d.out", i);
    rc = download(dir, name, W[i], el * dsize(pdt), &e);
    snprintf(name, sizeof(name), "M%d.out", i);
    if (rc == 0) rc = download(dir, name, M[i], el * 4, &e);
    snprintf(name, sizeof(name), "D%d.out", i);
    if (rc == 0) rc = download(dir, name, D[i], el * 4, &e);
  }
  if (ctx && prm_destroy(ctx) != PRM_OK && rc == 0) rc = failf(&e, "prm_destroy: %s", prm_last_error());
  for (int i = 0; i < n; ++i) {
    if (W && W[i]) (void)hipFree(W[i]);
    if (G && G[i]) (void)hipFree(G[i]);
    if (M && M[i]) (void)hipFree(M[i]);
    if (D && D[i]) (void)hipFree(D[i]);
  }
  if (stream) (void)hipStreamDestroy(stream);
  free(rows);
  free(cols);
  free(W);
  free(G);
  free(M);
  free(D);
  return rc;
}
