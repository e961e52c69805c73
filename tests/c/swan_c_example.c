/*
 * A C program that uses libswan through include/swan.h alone (plus the HIP
 * runtime's C API for device memory): the boundary as a C caller sees it.
 *
 *   swan_c_example sizes   host only: size queries and argument checks
 *   swan_c_example run     GPU: compress of the context, then one decode step
 *                          (swan_decode_step: the last token's append and the
 *                          attention) through the C ABI, checked against a
 *                          reference computed here in double
 *
 * The reference restates Algorithm 1 for this case: fp32 storage, rotations that
 * are signed permutations (so the rotated vectors are exact in fp32), tokens older
 * than the last b pruned to their k largest magnitudes (ties to the lower index),
 * softmax with 1/sqrt(128), and the output rotated back with P_vo^T.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "swan.h"

#define D 128
#define B 2
#define HQ 4
#define HKV 2
#define L 300
#define BUF 16
#define K 40

static int fails = 0;
#define CHECK(cond, ...)                  \
  do {                                    \
    if (!(cond)) {                        \
      fprintf(stderr, "FAIL: " __VA_ARGS__); \
      fprintf(stderr, "\n");              \
      ++fails;                            \
    }                                     \
  } while (0)

static uint64_t lcg = 88172645463325252ull;
static double uniform(void) {  /* in [-1, 1) */
  lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
  return (double)(lcg >> 11) / (double)(1ull << 53) * 2.0 - 1.0;
}

/* P[i][j] = sign[i] if j == perm[i]: x_hat[perm[i]] = sign[i] * x[i] */
static void signed_permutation(float* P, int seed) {
  int perm[D];
  for (int i = 0; i < D; ++i) perm[i] = i;
  for (int i = D - 1; i > 0; --i) {
    const int j = (int)((uniform() * 0.5 + 0.5) * (i + 1) + seed) % (i + 1);
    const int t = perm[i];
    perm[i] = perm[j];
    perm[j] = t;
  }
  memset(P, 0, sizeof(float) * D * D);
  for (int i = 0; i < D; ++i) P[i * D + perm[i]] = uniform() < 0 ? -1.f : 1.f;
}

static void rotate(const float* x, const float* P, double* y) {
  for (int j = 0; j < D; ++j) {
    double s = 0.0;
    for (int i = 0; i < D; ++i) s += (double)x[i] * (double)P[i * D + j];
    y[j] = s;
  }
}

/* zero all but the k largest |y| (ties: lower index) */
static void prune(double* y, int k) {
  int keep[D];
  memset(keep, 0, sizeof(keep));
  for (int n = 0; n < k; ++n) {
    int best = -1;
    for (int j = 0; j < D; ++j)
      if (!keep[j] && (best < 0 || fabs(y[j]) > fabs(y[best]))) best = j;
    keep[best] = 1;
  }
  for (int j = 0; j < D; ++j)
    if (!keep[j]) y[j] = 0.0;
}

static int host_checks(void) {
  size_t pb = 0;
  CHECK(swan_page_bytes(SWAN_F16, 48, &pb) == SWAN_OK && pb == 64 * 48 * 3, "page bytes %zu", pb);
  CHECK(swan_page_bytes(SWAN_F16_E4M3, 41, &pb) == SWAN_OK && pb == 64 * 48 * 2,
        "e4m3 page bytes %zu", pb);
  CHECK(swan_page_bytes(SWAN_F16, 0, &pb) == SWAN_ERR_INVALID_ARG, "k = 0 accepted");
  CHECK(strlen(swan_last_error()) > 0, "no error message");
  swan_cache c;
  memset(&c, 0, sizeof(c));
  c.batch = B;
  c.n_q_heads = HQ;
  c.n_kv_heads = HKV;
  c.head_dim = D;
  c.buffer_tokens = BUF;
  c.sparse_capacity = L;
  c.dtype = SWAN_F32;
  const int32_t kk[B] = {K, 64}, kv[B] = {24, 64};
  size_t kb = 0, vb = 0, rb = 0;
  CHECK(swan_cache_bytes(&c, kk, kv, &kb, &vb, &rb) == SWAN_OK, "cache bytes: %s",
        swan_last_error());
  const size_t npc = (L + 63) / 64;
  CHECK(kb == HKV * npc * 64 * 5 * (40 + 64), "k pages %zu", kb);
  CHECK(vb == HKV * npc * 64 * 5 * (24 + 64), "v pages %zu", vb);
  CHECK(rb == (size_t)B * HKV * BUF * D * 4, "ring %zu", rb);
  const int32_t lens[B] = {L, 100};
  size_t ws = 0;
  CHECK(swan_decode_workspace_bytes(&c, lens, kk, kv, &ws) == SWAN_OK && ws > 0, "workspace");
  /* arguments are checked before anything is enqueued: no device pointers needed */
  CHECK(swan_decode_attention(&c, lens, kk, kv, NULL, NULL, NULL, 0.f, NULL, NULL, ws, NULL) ==
            SWAN_ERR_INVALID_ARG,
        "null operands accepted");
  c.n_q_heads = 3;
  CHECK(swan_cache_bytes(&c, kk, kv, &kb, &vb, &rb) == SWAN_ERR_INVALID_ARG,
        "bad head counts accepted");
  c.n_q_heads = HQ;
  const int32_t kbad[B] = {K, 129};
  CHECK(swan_cache_bytes(&c, kbad, NULL, &kb, &vb, &rb) == SWAN_ERR_INVALID_ARG,
        "k > 128 accepted");
  CHECK(swan_version() >= 200, "version %d", swan_version());
  return fails;
}

#define HIP(x)                                                              \
  do {                                                                      \
    hipError_t e_ = (x);                                                    \
    if (e_ != hipSuccess) {                                                 \
      fprintf(stderr, "HIP error %s at %s:%d\n", hipGetErrorString(e_), __FILE__, __LINE__); \
      exit(2);                                                              \
    }                                                                       \
  } while (0)

static int gpu_run(void) {
  const size_t nkv = (size_t)B * HKV * L * D;
  float* kh = malloc(sizeof(float) * nkv);
  float* vh = malloc(sizeof(float) * nkv);
  float* qh = malloc(sizeof(float) * B * HQ * D);
  float* P = malloc(sizeof(float) * 2 * HKV * D * D);
  for (size_t i = 0; i < nkv; ++i) kh[i] = (float)uniform();
  for (size_t i = 0; i < nkv; ++i) vh[i] = (float)uniform();
  for (size_t i = 0; i < (size_t)B * HQ * D; ++i) qh[i] = (float)(2.0 * uniform());
  for (int h = 0; h < 2 * HKV; ++h) signed_permutation(P + (size_t)h * D * D, h);
  const float* Pqk_h = P;
  const float* Pvo_h = P + (size_t)HKV * D * D;

  swan_cache c;
  memset(&c, 0, sizeof(c));
  c.batch = B;
  c.n_q_heads = HQ;
  c.n_kv_heads = HKV;
  c.head_dim = D;
  c.buffer_tokens = BUF;
  c.sparse_capacity = L - BUF;
  c.dtype = SWAN_F32;
  const int32_t kact[B] = {K, K};
  size_t kb, vb, rb;
  if (swan_cache_bytes(&c, kact, NULL, &kb, &vb, &rb) != SWAN_OK) return 1;
  void *kp, *vp, *kr, *vr, *kn, *vn, *kl, *vl, *q, *out, *Pd, *ws;
  HIP(hipMalloc(&kp, kb));
  HIP(hipMalloc(&vp, vb));
  HIP(hipMalloc(&kr, rb));
  HIP(hipMalloc(&vr, rb));
  HIP(hipMalloc(&kn, sizeof(float) * nkv));
  HIP(hipMalloc(&vn, sizeof(float) * nkv));
  HIP(hipMalloc(&kl, sizeof(float) * B * HKV * D));
  HIP(hipMalloc(&vl, sizeof(float) * B * HKV * D));
  HIP(hipMalloc(&q, sizeof(float) * B * HQ * D));
  HIP(hipMalloc(&out, sizeof(float) * B * HQ * D));
  HIP(hipMalloc(&Pd, sizeof(float) * 2 * HKV * D * D));
  HIP(hipMemcpy(kn, kh, sizeof(float) * nkv, hipMemcpyHostToDevice));
  HIP(hipMemcpy(vn, vh, sizeof(float) * nkv, hipMemcpyHostToDevice));
  HIP(hipMemcpy(q, qh, sizeof(float) * B * HQ * D, hipMemcpyHostToDevice));
  /* the last token of every (sequence, kv head): the decode step's new key and value */
  for (int bh = 0; bh < B * HKV; ++bh) {
    const size_t src = ((size_t)bh * L + (L - 1)) * D;
    HIP(hipMemcpy((float*)kl + (size_t)bh * D, kh + src, sizeof(float) * D, hipMemcpyHostToDevice));
    HIP(hipMemcpy((float*)vl + (size_t)bh * D, vh + src, sizeof(float) * D, hipMemcpyHostToDevice));
  }
  HIP(hipMemcpy(Pd, P, sizeof(float) * 2 * HKV * D * D, hipMemcpyHostToDevice));
  c.k_pages = kp;
  c.v_pages = vp;
  c.k_ring = kr;
  c.v_ring = vr;
  const float* Pqk = (const float*)Pd;
  const float* Pvo = (const float*)Pd + (size_t)HKV * D * D;
  /* the context: the first L - 1 rows of each sequence's L; then the decode step appends the
     last token and attends in one call */
  const int32_t zero[B] = {0, 0}, first[B] = {L - 1, L - 1}, lens[B] = {L, L};
  swan_status st = swan_compress_append(&c, zero, kact, NULL, kn, vn, L, first, Pqk, Pvo, NULL);
  CHECK(st == SWAN_OK, "compress: %s", swan_last_error());
  size_t wsb = 0;
  CHECK(swan_decode_workspace_bytes(&c, lens, kact, NULL, &wsb) == SWAN_OK, "ws bytes");
  HIP(hipMalloc(&ws, wsb));
  st = swan_decode_step(&c, first, kact, NULL, kl, vl, q, Pqk, Pvo, 0.f, out, ws, wsb, NULL);
  CHECK(st == SWAN_OK, "decode step: %s", swan_last_error());
  HIP(hipDeviceSynchronize());
  float* got = malloc(sizeof(float) * B * HQ * D);
  HIP(hipMemcpy(got, out, sizeof(float) * B * HQ * D, hipMemcpyDeviceToHost));

  double worst = 0.0;
  double* kt = malloc(sizeof(double) * L * D);
  double* vt = malloc(sizeof(double) * L * D);
  for (int b = 0; b < B; ++b)
    for (int hq = 0; hq < HQ; ++hq) {
      const int h = hq / (HQ / HKV);
      for (int t = 0; t < L; ++t) {
        const size_t row = (((size_t)b * HKV + h) * L + t) * D;
        rotate(kh + row, Pqk_h + (size_t)h * D * D, kt + (size_t)t * D);
        rotate(vh + row, Pvo_h + (size_t)h * D * D, vt + (size_t)t * D);
        if (t < L - BUF) {
          prune(kt + (size_t)t * D, K);
          prune(vt + (size_t)t * D, K);
        }
      }
      double qr[D], s[L], oh[D];
      rotate(qh + ((size_t)b * HQ + hq) * D, Pqk_h + (size_t)h * D * D, qr);
      double m = -INFINITY, z = 0.0;
      for (int t = 0; t < L; ++t) {
        double a = 0.0;
        for (int j = 0; j < D; ++j) a += qr[j] * kt[(size_t)t * D + j];
        s[t] = a / sqrt((double)D);
        if (s[t] > m) m = s[t];
      }
      for (int j = 0; j < D; ++j) oh[j] = 0.0;
      for (int t = 0; t < L; ++t) {
        const double p = exp(s[t] - m);
        z += p;
        for (int j = 0; j < D; ++j) oh[j] += p * vt[(size_t)t * D + j];
      }
      double omax = 0.0, emax = 0.0;
      for (int i = 0; i < D; ++i) {  /* o = o_hat . P_vo^T */
        double a = 0.0;
        for (int j = 0; j < D; ++j) a += oh[j] / z * (double)Pvo_h[(size_t)h * D * D + i * D + j];
        if (fabs(a) > omax) omax = fabs(a);
        const double e = fabs((double)got[((size_t)b * HQ + hq) * D + i] - a);
        if (e > emax) emax = e;
      }
      if (emax / omax > worst) worst = emax / omax;
    }
  printf("max relative error %.3e\n", worst);
  CHECK(worst <= 2e-3, "output error %.3e", worst);
  HIP(hipFree(kp));
  HIP(hipFree(vp));
  HIP(hipFree(kr));
  HIP(hipFree(vr));
  HIP(hipFree(kn));
  HIP(hipFree(vn));
  HIP(hipFree(kl));
  HIP(hipFree(vl));
  HIP(hipFree(q));
  HIP(hipFree(out));
  HIP(hipFree(Pd));
  HIP(hipFree(ws));
  free(kh);
  free(vh);
  free(qh);
  free(P);
  free(got);
  free(kt);
  free(vt);
  return fails;
}

int main(int argc, char** argv) {
  if (argc < 2) {
    fprintf(stderr, "usage: %s sizes|run\n", argv[0]);
    return 2;
  }
  const int r = strcmp(argv[1], "run") == 0 ? gpu_run() : host_checks();
  printf("%s\n", r ? "FAILED" : "ok");
  return r ? 1 : 0;
}
