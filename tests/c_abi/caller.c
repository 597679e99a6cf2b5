/*
 * A plain C caller of the library: no PyTorch, the HIP runtime only for device
 * memory and a stream.  It runs the hot path as a C user would: separately
 * allocated leaves, a segment table, one batched flatten of the params tree
 * and the K gradient trees, the K-step Adam driver forward and VJP with only
 * the final moment state stored (the VJP recomputes the rest), and one batched
 * unflatten of p_K and the K gradient cotangents.
 *
 * usage: caller IN OUT
 *   IN  (little-endian): int64 S, K, count0; double lr, b1, b2, eps, eps_root;
 *       int64 numel[S]; float p leaves, then the K gradient trees, each as
 *       its leaves back to back; then the output cotangent of p_K as a flat
 *       array of n = sum(numel) floats.
 *   OUT: float p_K leaves, mu_K[n], nu_K[n], the K gradient-cotangent trees
 *       (leaves back to back), dmu0[n], dnu0[n].
 * Exit status 0 on success; on a failing call it prints the call, its code
 * and diffopt_last_error() and exits 1.
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "diffopt.h"

#define MAXK DIFFOPT_REMAT_SPAN

static void die(const char* what) {
  fprintf(stderr, "caller: %s\n", what);
  exit(1);
}

static void check_hip(hipError_t e, const char* what) {
  if (e != hipSuccess) {
    fprintf(stderr, "caller: %s: %s\n", what, hipGetErrorString(e));
    exit(1);
  }
}

static void check(int rc, const char* what) {
  if (rc != DIFFOPT_OK) {
    fprintf(stderr, "caller: %s returned %d: %s\n", what, rc, diffopt_last_error());
    exit(1);
  }
}

static void rd(void* p, size_t sz, size_t cnt, FILE* f) {
  if (cnt && fread(p, sz, cnt, f) != cnt) die("short input file");
}

static void wr(const void* p, size_t sz, size_t cnt, FILE* f) {
  if (cnt && fwrite(p, sz, cnt, f) != cnt) die("short write");
}

static void* dalloc(size_t bytes) {
  void* p = NULL;
  if (bytes) check_hip(hipMalloc(&p, bytes), "hipMalloc");
  return p;
}

/* one tree instance: a device allocation per nonempty leaf, and the device
 * array of their addresses in table order */
typedef struct {
  float** leaf;
  uint64_t* d_addr;
} Tree;

static Tree tree_new(int64_t S, const int64_t* numel) {
  Tree t;
  uint64_t* h = (uint64_t*)calloc((size_t)(S ? S : 1), sizeof(uint64_t));
  t.leaf = (float**)calloc((size_t)(S ? S : 1), sizeof(float*));
  if (!h || !t.leaf) die("out of host memory");
  for (int64_t j = 0; j < S; ++j) {
    t.leaf[j] = (float*)dalloc((size_t)numel[j] * sizeof(float));
    h[j] = (uint64_t)(uintptr_t)t.leaf[j];
  }
  t.d_addr = (uint64_t*)dalloc((size_t)(S ? S : 1) * sizeof(uint64_t));
  check_hip(hipMemcpy(t.d_addr, h, (size_t)S * sizeof(uint64_t), hipMemcpyHostToDevice), "upload addresses");
  free(h);
  return t;
}

int main(int argc, char** argv) {
  if (argc != 3) die("usage: caller IN OUT");
  FILE* in = fopen(argv[1], "rb");
  if (!in) die("cannot open input");
  int64_t hdr[3];
  double hp[5];
  rd(hdr, sizeof(int64_t), 3, in);
  rd(hp, sizeof(double), 5, in);
  const int64_t S = hdr[0], K = hdr[1], count0 = hdr[2];
  if (S < 0 || K < 1 || K > MAXK) die("need S >= 0 and 1 <= K <= DIFFOPT_REMAT_SPAN");
  int64_t* numel = (int64_t*)calloc((size_t)(S ? S : 1), sizeof(int64_t));
  if (!numel) die("out of host memory");
  rd(numel, sizeof(int64_t), (size_t)S, in);
  int64_t n = 0;
  for (int64_t j = 0; j < S; ++j) n += numel[j];
  float* host = (float*)malloc((size_t)(n ? n : 1) * sizeof(float));
  if (!host) die("out of host memory");

  diffopt_segtable* table = NULL;
  check(diffopt_segtable_create(S, numel, NULL, 4, &table), "diffopt_segtable_create");
  if (diffopt_segtable_total(table) != n) die("table total differs from sum(numel)");

  /* input trees: p, then K gradient trees, filled leaf by leaf */
  Tree trees[1 + MAXK];
  for (int64_t t = 0; t <= K; ++t) {
    trees[t] = tree_new(S, numel);
    for (int64_t j = 0; j < S; ++j) {
      rd(host, sizeof(float), (size_t)numel[j], in);
      if (numel[j])
        check_hip(hipMemcpy(trees[t].leaf[j], host, (size_t)numel[j] * sizeof(float), hipMemcpyHostToDevice),
                  "upload leaf");
    }
  }
  float* cot = (float*)dalloc((size_t)n * sizeof(float));
  rd(host, sizeof(float), (size_t)n, in);
  if (n) check_hip(hipMemcpy(cot, host, (size_t)n * sizeof(float), hipMemcpyHostToDevice), "upload cotangent");
  fclose(in);

  hipStream_t st;
  check_hip(hipStreamCreate(&st), "hipStreamCreate");

  /* flat buffers */
  const size_t nb = (size_t)n * sizeof(float);
  float* flat[1 + MAXK];
  for (int64_t t = 0; t <= K; ++t) flat[t] = (float*)dalloc(nb);
  float *m0 = (float*)dalloc(nb), *v0 = (float*)dalloc(nb), *mK = (float*)dalloc(nb), *vK = (float*)dalloc(nb);
  float *pK = (float*)dalloc(nb), *dm0 = (float*)dalloc(nb), *dv0 = (float*)dalloc(nb);
  float* dg[MAXK];
  for (int64_t k = 0; k < K; ++k) dg[k] = (float*)dalloc(nb);
  if (n) {
    check_hip(hipMemsetAsync(m0, 0, nb, st), "zero mu0");
    check_hip(hipMemsetAsync(v0, 0, nb, st), "zero nu0");
  }

  /* pack p and the K gradient trees in one launch */
  const uint64_t* addr[1 + MAXK];
  void* flats[1 + MAXK];
  for (int64_t t = 0; t <= K; ++t) {
    addr[t] = trees[t].d_addr;
    flats[t] = flat[t];
  }
  check(diffopt_tree_flatten_batch(table, K + 1, addr, flats, st), "diffopt_tree_flatten_batch");

  /* K fused Adam steps; only the initial and final moment states are stored */
  const float* grads[MAXK];
  const float* mu_in[MAXK + 1];
  const float* nu_in[MAXK + 1];
  float* mu_tr[MAXK + 1];
  float* nu_tr[MAXK + 1];
  for (int64_t k = 0; k < K; ++k) grads[k] = flat[1 + k];
  for (int64_t k = 0; k <= K; ++k) {
    mu_tr[k] = k == 0 ? m0 : (k == K ? mK : NULL);
    nu_tr[k] = k == 0 ? v0 : (k == K ? vK : NULL);
    mu_in[k] = mu_tr[k];
    nu_in[k] = nu_tr[k];
  }
  check(diffopt_adam_unrolled_fwd(K, n, flat[0], grads, mu_tr, nu_tr, pK, count0, hp[0], hp[1], hp[2], hp[3],
                                  hp[4], st),
        "diffopt_adam_unrolled_fwd");
  check(diffopt_adam_unrolled_bwd(K, n, cot, grads, mu_in, nu_in, dg, dm0, dv0, count0, hp[0], hp[1], hp[2], hp[3],
                                  hp[4], st),
        "diffopt_adam_unrolled_bwd");

  /* unpack p_K and the K gradient cotangents into new leaves */
  Tree outs[1 + MAXK];
  const void* oflat[1 + MAXK];
  const uint64_t* oaddr[1 + MAXK];
  for (int64_t t = 0; t <= K; ++t) {
    outs[t] = tree_new(S, numel);
    oaddr[t] = outs[t].d_addr;
    oflat[t] = t == 0 ? (const void*)pK : (const void*)dg[t - 1];
  }
  check(diffopt_tree_unflatten_batch(table, K + 1, oflat, oaddr, st), "diffopt_tree_unflatten_batch");
  check_hip(hipStreamSynchronize(st), "hipStreamSynchronize");

  FILE* out = fopen(argv[2], "wb");
  if (!out) die("cannot open output");
  for (int64_t t = 0; t <= K; ++t) {
    for (int64_t j = 0; j < S; ++j) {
      if (numel[j])
        check_hip(hipMemcpy(host, outs[t].leaf[j], (size_t)numel[j] * sizeof(float), hipMemcpyDeviceToHost),
                  "download leaf");
      wr(host, sizeof(float), (size_t)numel[j], out);
    }
    if (t == 0) { /* mu_K, nu_K right after p_K */
      const float* st2[2] = {mK, vK};
      for (int q = 0; q < 2; ++q) {
        if (n) check_hip(hipMemcpy(host, st2[q], nb, hipMemcpyDeviceToHost), "download state");
        wr(host, sizeof(float), (size_t)n, out);
      }
    }
  }
  const float* tail[2] = {dm0, dv0};
  for (int q = 0; q < 2; ++q) {
    if (n) check_hip(hipMemcpy(host, tail[q], nb, hipMemcpyDeviceToHost), "download cotangent");
    wr(host, sizeof(float), (size_t)n, out);
  }
  if (fclose(out) != 0) die("cannot close output");
  diffopt_segtable_destroy(table);
  check_hip(hipStreamDestroy(st), "hipStreamDestroy");
  return 0;
}
