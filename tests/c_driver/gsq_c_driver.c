/*
 * A plain C user of the GSQ library: no Python, no torch, only the HIP runtime and the C ABI of
 * include/gsq.h.  It builds a small synthetic layer on the host, optimises it for a few steps on
 * the GPU, hardens and packs it, and writes its inputs and results to a file, so that a test can
 * run the same layer through the Python binding and compare the two bit for bit.
 *
 * Layer: W 96 x 384 ~ N(0, 0.02^2) (fp32, passed as fp32), calibration X of 512 tokens whose
 * channels are N(0, 1) times a LogNormal(0, 0.5) scale, H = X^T X; 4 levels {-1.5, -0.5, 0.5,
 * 1.5}, groups of 128, bf16 precision, Philox seed 7.  Five Adam steps with tau annealed
 * linearly from 1.0 to 0.05, the loss requested every step and the next sample fused.
 *
 * File layout (little-endian): int32 O, I, T, steps; uint64 packed bytes; float W[O*I],
 * H[I*I], tau[steps], loss[steps], hard_loss; uint8 codes[O*I], packed[packed bytes].
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "gsq.h"

enum { O = 96, I = 384, T = 512, STEPS = 5 };

static uint64_t lcg_state;
static double unif(void) {   /* 53-bit uniform in (0, 1) from a 64-bit LCG (Knuth's MMIX) */
  lcg_state = lcg_state * 6364136223846793005ull + 1442695040888963407ull;
  return ((double)(lcg_state >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}
static double normal(void) {  /* Box-Muller */
  const double u = unif(), v = unif();
  return sqrt(-2.0 * log(u)) * cos(6.283185307179586 * v);
}

#define FAIL(...) do { snprintf(msg, (size_t)msg_len, __VA_ARGS__); rc = 1; goto done; } while (0)
#define HIPCALL(x) do { hipError_t e_ = (x); if (e_ != hipSuccess) FAIL("%s: %s", #x, hipGetErrorString(e_)); } while (0)
#define GSQCALL(x) do { gsq_status s_ = (x); if (s_ != GSQ_OK) FAIL("%s: status %d: %s", #x, (int)s_, gsq_last_error()); } while (0)

int gsq_c_driver_run(const char* out_path, char* msg, int msg_len) {
  int rc = 0;
  float *W = NULL, *H = NULL, tau[STEPS], loss[STEPS], hard = 0.f;
  double *X = NULL, *Hd = NULL;
  uint8_t *codes = NULL, *packed = NULL;
  void *dW = NULL, *dH = NULL, *dloss = NULL, *dhard = NULL, *dcodes = NULL, *dpacked = NULL;
  hipStream_t stream = NULL;
  gsq_layer* layer = NULL;
  FILE* f = NULL;
  size_t psize = 0;
  msg[0] = 0;

  /* inputs */
  lcg_state = 0x243F6A8885A308D3ull;
  W = (float*)malloc(sizeof(float) * O * I);
  H = (float*)malloc(sizeof(float) * I * I);
  X = (double*)malloc(sizeof(double) * T * I);
  Hd = (double*)calloc((size_t)I * I, sizeof(double));
  codes = (uint8_t*)malloc(O * I);
  if (!W || !H || !X || !Hd || !codes) FAIL("host allocation failed");
  for (int i = 0; i < O * I; ++i) W[i] = (float)(0.02 * normal());
  for (int c = 0; c < I; ++c) {
    const double scale = exp(0.5 * normal());
    for (int t = 0; t < T; ++t) X[(size_t)t * I + c] = normal() * scale;
  }
  for (int t = 0; t < T; ++t)
    for (int a = 0; a < I; ++a) {
      const double xa = X[(size_t)t * I + a];
      for (int b = 0; b < I; ++b) Hd[(size_t)a * I + b] += xa * X[(size_t)t * I + b];
    }
  for (size_t i = 0; i < (size_t)I * I; ++i) H[i] = (float)Hd[i];

  gsq_config cfg;
  memset(&cfg, 0, sizeof cfg);
  cfg.batch = 1;
  cfg.out_features = O;
  cfg.in_features = I;
  cfg.n_levels = 4;
  cfg.levels[0] = -1.5f; cfg.levels[1] = -0.5f; cfg.levels[2] = 0.5f; cfg.levels[3] = 1.5f;
  cfg.group_size = 128;
  cfg.layout = GSQ_LAYOUT_GROUP;
  cfg.precision = GSQ_PREC_BF16;
  cfg.seed = 7;
  cfg.alpha = 6.0f;
  cfg.sigma_init = 1.0f;
  cfg.init_noise = 1;
  cfg.relaxation = GSQ_RELAX_GRID;
  psize = gsq_packed_size(&cfg);
  if (psize == 0) FAIL("gsq_packed_size rejected the configuration: %s", gsq_last_error());
  packed = (uint8_t*)malloc(psize);
  if (!packed) FAIL("host allocation failed");

  /* device buffers, the caller's own */
  HIPCALL(hipStreamCreate(&stream));
  HIPCALL(hipMalloc(&dW, sizeof(float) * O * I));
  HIPCALL(hipMalloc(&dH, sizeof(float) * I * I));
  HIPCALL(hipMalloc(&dloss, sizeof(float) * STEPS));
  HIPCALL(hipMalloc(&dhard, sizeof(float)));
  HIPCALL(hipMalloc(&dcodes, O * I));
  HIPCALL(hipMalloc(&dpacked, psize));
  HIPCALL(hipMemcpyAsync(dW, W, sizeof(float) * O * I, hipMemcpyHostToDevice, stream));
  HIPCALL(hipMemcpyAsync(dH, H, sizeof(float) * I * I, hipMemcpyHostToDevice, stream));

  GSQCALL(gsq_layer_init(&cfg, dW, GSQ_DT_FP32, (const float*)dH, NULL, stream, &layer));
  for (int t = 0; t < STEPS; ++t) tau[t] = 1.0f + (0.05f - 1.0f) * (float)t / (float)(STEPS - 1);
  for (int t = 0; t < STEPS; ++t) {
    gsq_step_params p;
    memset(&p, 0, sizeof p);
    p.tau = tau[t];
    p.kappa = 1.0f;
    p.lr_logits = 1e-2f;
    p.lr_scales = 5e-5f;
    p.beta1 = 0.9f;
    p.beta2 = 0.95f;
    p.eps = 1e-8f;
    p.gumbel_noise = 1;
    p.tau_next = t + 1 < STEPS ? tau[t + 1] : 0.0f;
    p.kappa_next = 1.0f;
    p.optimizer = GSQ_OPT_ADAM;
    p.weight_decay = 0.0f;
    p.samples = 1;
    GSQCALL(gsq_step(layer, &p, (float*)dloss + t, stream));
  }
  GSQCALL(gsq_harden(layer, (uint8_t*)dcodes, NULL, (float*)dhard, stream));
  GSQCALL(gsq_pack(layer, dpacked, psize, stream));
  HIPCALL(hipMemcpyAsync(loss, dloss, sizeof(float) * STEPS, hipMemcpyDeviceToHost, stream));
  HIPCALL(hipMemcpyAsync(&hard, dhard, sizeof(float), hipMemcpyDeviceToHost, stream));
  HIPCALL(hipMemcpyAsync(codes, dcodes, O * I, hipMemcpyDeviceToHost, stream));
  HIPCALL(hipMemcpyAsync(packed, dpacked, psize, hipMemcpyDeviceToHost, stream));
  HIPCALL(hipStreamSynchronize(stream));
  GSQCALL(gsq_check(layer, stream));

  f = fopen(out_path, "wb");
  if (!f) FAIL("cannot open %s", out_path);
  {
    const int32_t hdr[4] = {O, I, T, STEPS};
    const uint64_t pb = psize;
    if (fwrite(hdr, sizeof hdr, 1, f) != 1 || fwrite(&pb, sizeof pb, 1, f) != 1 ||
        fwrite(W, sizeof(float), O * I, f) != (size_t)(O * I) ||
        fwrite(H, sizeof(float), (size_t)I * I, f) != (size_t)I * I ||
        fwrite(tau, sizeof(float), STEPS, f) != STEPS || fwrite(loss, sizeof(float), STEPS, f) != STEPS ||
        fwrite(&hard, sizeof hard, 1, f) != 1 ||
        fwrite(codes, 1, O * I, f) != (size_t)(O * I) || fwrite(packed, 1, psize, f) != psize)
      FAIL("short write to %s", out_path);
  }

done:
  if (f) fclose(f);
  if (layer) gsq_layer_destroy(layer);
  if (dW) hipFree(dW);
  if (dH) hipFree(dH);
  if (dloss) hipFree(dloss);
  if (dhard) hipFree(dhard);
  if (dcodes) hipFree(dcodes);
  if (dpacked) hipFree(dpacked);
  if (stream) hipStreamDestroy(stream);
  free(W); free(H); free(X); free(Hd); free(codes); free(packed);
  return rc;
}
