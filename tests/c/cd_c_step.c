/*
 * A plain C99 client of the CurvaDion C ABI (include/curvadion.h): it uses
 * nothing but that header, the HIP runtime's C API for device memory, and
 * libcurvadion.so.  The tests run it in two modes:
 *
 *   cd_c_step check
 *       no device needed: the ABI version, invalid descriptors and NULL
 *       arguments rejected with CD_EINVAL and a message, cd_destroy(NULL).
 *
 *   cd_c_step run DIR M N R STEPS DTYPE POLICY TAU MU ETA
 *       one layer (DTYPE f32 or bf16, POLICY 0..3) stepped STEPS times on
 *       the default stream.  Reads DIR/M0.bin, X0.bin (m x n fp32), Q0.bin
 *       (n x r fp32) and G<t>.bin (m x n, fp32 or bf16 bits), all row-major;
 *       writes DIR/M.bin, X.bin, Q.bin and DIR/steps.txt (one line per step:
 *       RMMC, branch, status).
 *
 *   cd_c_step async DIR ...
 *       the same steps, each asynchronous (no result argument: the call
 *       enqueues the whole step and returns), every gradient in its own
 *       device buffer; then cd_layer_last_result, whose outcome is the one
 *       line of DIR/steps.txt.
 *
 * Exit status 0 on success; any unexpected status prints the library's
 * message and exits 1.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "curvadion.h"

static int fail_hip(const char* what, hipError_t e) {
  fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
  return 1;
}

static cd_layer_desc base_desc(void) {
  cd_layer_desc d;
  memset(&d, 0, sizeof(d));
  d.m = 64;
  d.n = 32;
  d.r_max = 8;
  d.grad_dtype = CD_F32;
  d.tau = 0.5;
  d.eps = 1e-8;
  d.eta_local_scale = 1.0;
  d.policy = CD_POLICY_RMMC;
  d.H = 1;
  d.weight_decay = 0.0;
  return d;
}

static int expect_einval(const cd_layer_desc* d, const char* what) {
  cd_layer* L = (cd_layer*)(uintptr_t)1;   /* must come back NULL */
  const cd_status st = cd_layer_create(d, &L);
  if (st != CD_EINVAL || L != NULL || cd_last_error()[0] == '\0') {
    fprintf(stderr, "%s: status %d, layer %p, message '%s'\n", what, (int)st, (void*)L, cd_last_error());
    return 1;
  }
  printf("%-18s CD_EINVAL: %s\n", what, cd_last_error());
  return 0;
}

static int check(void) {
  cd_layer_desc d;
  int bad = 0;
  if (cd_abi_version() != CD_ABI_VERSION) {
    fprintf(stderr, "library ABI %d, header %d\n", cd_abi_version(), CD_ABI_VERSION);
    return 1;
  }
  d = base_desc(); d.m = 0;                bad |= expect_einval(&d, "m = 0");
  d = base_desc(); d.r_max = 33;           bad |= expect_einval(&d, "r_max > min(m,n)");
  d = base_desc(); d.grad_dtype = (cd_dtype)7; bad |= expect_einval(&d, "dtype");
  d = base_desc(); d.policy = (cd_policy)9;    bad |= expect_einval(&d, "policy");
  d = base_desc(); d.eps = -1.0;           bad |= expect_einval(&d, "eps < 0");
  d = base_desc(); d.weight_decay = -0.1;  bad |= expect_einval(&d, "weight_decay < 0");
  d = base_desc(); d.policy = CD_POLICY_EVERY_H; d.H = 0; bad |= expect_einval(&d, "H = 0");
  bad |= expect_einval(NULL, "NULL desc");
  if (cd_step(NULL, NULL, NULL, NULL, NULL, 0.9f, 0.01f, 4, NULL, NULL) != CD_EINVAL) bad = 1;
  if (cd_group_create(NULL, 1, NULL) != CD_EINVAL) bad = 1;
  if (cd_destroy(NULL) != CD_OK || cd_group_destroy(NULL) != CD_OK) bad = 1;
  if (cd_layer_last_result(NULL, NULL) != CD_EINVAL || cd_group_last_result(NULL, NULL, NULL) != CD_EINVAL) bad = 1;
  if (!bad) printf("check ok (ABI %d)\n", cd_abi_version());
  return bad;
}

static void* read_file(const char* dir, const char* name, size_t bytes) {
  char path[4096];
  FILE* f;
  void* buf;
  snprintf(path, sizeof(path), "%s/%s", dir, name);
  f = fopen(path, "rb");
  if (!f) { fprintf(stderr, "cannot open %s\n", path); return NULL; }
  buf = malloc(bytes ? bytes : 1);
  if (buf && fread(buf, 1, bytes, f) != bytes) {
    fprintf(stderr, "%s: short read\n", path);
    free(buf);
    buf = NULL;
  }
  fclose(f);
  return buf;
}

static int write_file(const char* dir, const char* name, const void* buf, size_t bytes) {
  char path[4096];
  FILE* f;
  size_t w;
  snprintf(path, sizeof(path), "%s/%s", dir, name);
  f = fopen(path, "wb");
  if (!f) { fprintf(stderr, "cannot create %s\n", path); return 1; }
  w = fwrite(buf, 1, bytes, f);
  fclose(f);
  return w != bytes;
}

static int run(int argc, char** argv, int async) {
  const char* dir;
  int m, n, r, steps, policy, t, rc = 1;
  void** dGs = NULL;
  int bf16;
  double tau;
  float mu, eta;
  size_t mn_bytes, g_bytes, q_bytes;
  float *hM = NULL, *hX = NULL, *hQ = NULL;
  void *dG = NULL, *dM = NULL, *dX = NULL, *dQ = NULL;
  cd_layer* L = NULL;
  cd_layer_desc d;
  FILE* log = NULL;
  char path[4096];
  hipError_t e;

  if (argc != 12) {
    fprintf(stderr, "usage: %s run|async DIR M N R STEPS f32|bf16 POLICY TAU MU ETA\n", argv[0]);
    return 2;
  }
  dir = argv[2];
  m = atoi(argv[3]); n = atoi(argv[4]); r = atoi(argv[5]); steps = atoi(argv[6]);
  bf16 = strcmp(argv[7], "bf16") == 0;
  policy = atoi(argv[8]);
  tau = atof(argv[9]);
  mu = (float)atof(argv[10]);
  eta = (float)atof(argv[11]);
  if (m < 1 || n < 1 || r < 1 || steps < 1) { fprintf(stderr, "bad sizes\n"); return 2; }
  mn_bytes = (size_t)m * (size_t)n * sizeof(float);
  g_bytes = (size_t)m * (size_t)n * (bf16 ? 2u : 4u);
  q_bytes = (size_t)n * (size_t)r * sizeof(float);

  hM = (float*)read_file(dir, "M0.bin", mn_bytes);
  hX = (float*)read_file(dir, "X0.bin", mn_bytes);
  hQ = (float*)read_file(dir, "Q0.bin", q_bytes);
  if (!hM || !hX || !hQ) goto done;
  if ((e = hipMalloc(&dG, g_bytes)) != hipSuccess) { rc = fail_hip("hipMalloc G", e); goto done; }
  if ((e = hipMalloc(&dM, mn_bytes)) != hipSuccess) { rc = fail_hip("hipMalloc M", e); goto done; }
  if ((e = hipMalloc(&dX, mn_bytes)) != hipSuccess) { rc = fail_hip("hipMalloc X", e); goto done; }
  if ((e = hipMalloc(&dQ, q_bytes)) != hipSuccess) { rc = fail_hip("hipMalloc Q", e); goto done; }
  if ((e = hipMemcpy(dM, hM, mn_bytes, hipMemcpyHostToDevice)) != hipSuccess) { rc = fail_hip("copy M", e); goto done; }
  if ((e = hipMemcpy(dX, hX, mn_bytes, hipMemcpyHostToDevice)) != hipSuccess) { rc = fail_hip("copy X", e); goto done; }
  if ((e = hipMemcpy(dQ, hQ, q_bytes, hipMemcpyHostToDevice)) != hipSuccess) { rc = fail_hip("copy Q", e); goto done; }

  d = base_desc();
  d.m = m; d.n = n; d.r_max = r;
  d.grad_dtype = bf16 ? CD_BF16 : CD_F32;
  d.tau = tau;
  d.policy = (cd_policy)policy;
  if (cd_layer_create(&d, &L) != CD_OK) { fprintf(stderr, "create: %s\n", cd_last_error()); goto done; }

  snprintf(path, sizeof(path), "%s/steps.txt", dir);
  log = fopen(path, "w");
  if (!log) { fprintf(stderr, "cannot create %s\n", path); goto done; }
  if (async) {
    /* every gradient in a buffer of its own, copied before the first step:
       an asynchronous step may still read its G when the next one is
       enqueued */
    dGs = (void**)calloc((size_t)steps, sizeof(void*));
    if (!dGs) goto done;
    for (t = 0; t < steps; ++t) {
      char name[64];
      void* hG;
      snprintf(name, sizeof(name), "G%d.bin", t);
      hG = read_file(dir, name, g_bytes);
      if (!hG) goto done;
      if ((e = hipMalloc(&dGs[t], g_bytes)) != hipSuccess) { free(hG); rc = fail_hip("hipMalloc G", e); goto done; }
      e = hipMemcpy(dGs[t], hG, g_bytes, hipMemcpyHostToDevice);
      free(hG);
      if (e != hipSuccess) { rc = fail_hip("copy G", e); goto done; }
    }
  }
  for (t = 0; t < steps; ++t) {
    char name[64];
    void* hG;
    cd_result res;
    cd_status st;
    if (async) {
      st = cd_step(L, dGs[t], (float*)dM, (float*)dX, (float*)dQ, mu, eta, r, NULL, NULL);
      if (st != CD_OK) { fprintf(stderr, "async step %d: %s\n", t, cd_last_error()); goto done; }
      continue;
    }
    snprintf(name, sizeof(name), "G%d.bin", t);
    hG = read_file(dir, name, g_bytes);
    if (!hG) goto done;
    e = hipMemcpy(dG, hG, g_bytes, hipMemcpyHostToDevice);
    free(hG);
    if (e != hipSuccess) { rc = fail_hip("copy G", e); goto done; }
    st = cd_step(L, dG, (float*)dM, (float*)dX, (float*)dQ, mu, eta, r, NULL, &res);
    if (st != CD_OK && st != CD_ENONFINITE) { fprintf(stderr, "step %d: %s\n", t, cd_last_error()); goto done; }
    fprintf(log, "%.17g %d %d\n", res.rmmc, res.sync_flag, (int)st);
    printf("step %d: rmmc %.6g %s\n", t + 1, res.rmmc, res.sync_flag ? "sync" : "local");
  }
  if (async) {
    cd_result res;
    const cd_status st = cd_layer_last_result(L, &res);
    if (st != CD_OK && st != CD_ENONFINITE && st != CD_ERANKDEF) {
      fprintf(stderr, "last result: %s\n", cd_last_error());
      goto done;
    }
    fprintf(log, "%.17g %d %d\n", res.rmmc, res.sync_flag, (int)st);
    printf("%d asynchronous steps; last: rmmc %.6g %s\n", steps, res.rmmc, res.sync_flag ? "sync" : "local");
  }
  if ((e = hipDeviceSynchronize()) != hipSuccess) { rc = fail_hip("synchronize", e); goto done; }
  if ((e = hipMemcpy(hM, dM, mn_bytes, hipMemcpyDeviceToHost)) != hipSuccess) { rc = fail_hip("copy M back", e); goto done; }
  if ((e = hipMemcpy(hX, dX, mn_bytes, hipMemcpyDeviceToHost)) != hipSuccess) { rc = fail_hip("copy X back", e); goto done; }
  if ((e = hipMemcpy(hQ, dQ, q_bytes, hipMemcpyDeviceToHost)) != hipSuccess) { rc = fail_hip("copy Q back", e); goto done; }
  if (write_file(dir, "M.bin", hM, mn_bytes) || write_file(dir, "X.bin", hX, mn_bytes) ||
      write_file(dir, "Q.bin", hQ, q_bytes))
    goto done;
  rc = 0;
done:
  if (log) fclose(log);
  if (L) cd_destroy(L);
  if (dG) (void)hipFree(dG);
  if (dM) (void)hipFree(dM);
  if (dX) (void)hipFree(dX);
  if (dQ) (void)hipFree(dQ);
  if (dGs) {
    for (t = 0; t < steps; ++t)
      if (dGs[t]) (void)hipFree(dGs[t]);
    free(dGs);
  }
  free(hM); free(hX); free(hQ);
  return rc;
}

int main(int argc, char** argv) {
  if (argc >= 2 && strcmp(argv[1], "check") == 0) return check();
  if (argc >= 2 && strcmp(argv[1], "run") == 0) return run(argc, argv, 0);
  if (argc >= 2 && strcmp(argv[1], "async") == 0) return run(argc, argv, 1);
  fprintf(stderr, "usage: %s check | run|async DIR M N R STEPS f32|bf16 POLICY TAU MU ETA\n", argv[0]);
  return 2;
}
