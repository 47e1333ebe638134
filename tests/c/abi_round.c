/*
 * abi_round.c -- the C ABI used from plain C, with no Python or torch: one
 * fl_round (Section 4.2: A local steps, then FedAvg) on device buffers from
 * hipMalloc, compared bit for bit with the oracle's orc_round on the same
 * host inputs, plus an error path that must be reported before any launch.
 * Test code: it links the library and the oracle side by side.  Inputs come
 * from a local xorshift generator; nothing the oracle sees comes from the
 * device.  Exit status 0 when everything matches.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "flround.h"
#include "oracle.h"

#define NEL 100003
#define NSEG 4
#define NPEER 3
#define NGRP 3
#define NSTEP 2

static uint64_t rng_state = 0x9E3779B97F4A7C15ULL;

static double uniform(void) { /* xorshift64*, in [0, 1) */
  rng_state ^= rng_state >> 12;
  rng_state ^= rng_state << 25;
  rng_state ^= rng_state >> 27;
  return (double)((rng_state * 0x2545F4914F6CDD1DULL) >> 11) / 9007199254740992.0;
}

static uint16_t bf16_bits(float x) { /* any valid bf16 pattern near x */
  uint32_t u;
  memcpy(&u, &x, 4);
  return (uint16_t)(u >> 16);
}

#define CHECK_HIP(call)                                                       \
  do {                                                                        \
    hipError_t e_ = (call);                                                   \
    if (e_ != hipSuccess) {                                                   \
      fprintf(stderr, "abi_round: %s failed: %s\n", #call, hipGetErrorString(e_)); \
      return 2;                                                               \
    }                                                                         \
  } while (0)

int main(void) {
  const int64_t off[NSEG + 1] = {0, 30000, 30001, 65536, NEL};
  const uint8_t decay[NSEG] = {1, 0, 1, 1};
  const float weights[NGRP] = {1.0f, 2.0f, 3.0f};
  const int self_group = 1;
  const int64_t step0 = 5;
  const float grad_scale = 1.0f / 3.0f;

  static uint16_t grads[NSTEP * NPEER][NEL], reps[NGRP][NEL];
  static uint16_t working[NEL], working_ref[NEL], working_out[NEL];
  static float master[NEL], master_ref[NEL], master_out[NEL], m_out[NEL], v_out[NEL];
  static float zeros[NEL], m_ref[NEL], v_ref[NEL];
  static float ss_out[NSTEP * NSEG];
  static double ss_ref[NSTEP * NSEG];

  for (int k = 0; k < NSTEP * NPEER; ++k)
    for (int i = 0; i < NEL; ++i) grads[k][i] = bf16_bits((float)(2e-3 * (uniform() - 0.5)));
  for (int i = 0; i < NEL; ++i) {
    master[i] = (float)(0.04 * (uniform() - 0.5));
    working[i] = bf16_bits(master[i]);
  }
  for (int g = 0; g < NGRP; ++g)
    for (int i = 0; i < NEL; ++i) reps[g][i] = bf16_bits((float)(0.04 * (uniform() - 0.5)));

  /* device side */
  fl_layout* lay = NULL;
  int rc = fl_layout_create(NEL, NSEG, off, decay, &lay);
  if (rc != FL_OK) {
    fprintf(stderr, "abi_round: fl_layout_create: %s\n", fl_status_string(rc));
    return 1;
  }
  uint16_t* d_grads[NSTEP * NPEER];
  uint16_t* d_reps[NGRP];
  for (int k = 0; k < NSTEP * NPEER; ++k) {
    CHECK_HIP(hipMalloc((void**)&d_grads[k], sizeof(uint16_t) * NEL));
    CHECK_HIP(hipMemcpy(d_grads[k], grads[k], sizeof(uint16_t) * NEL, hipMemcpyHostToDevice));
  }
  for (int g = 0; g < NGRP; ++g) {
    CHECK_HIP(hipMalloc((void**)&d_reps[g], sizeof(uint16_t) * NEL));
    CHECK_HIP(hipMemcpy(d_reps[g], reps[g], sizeof(uint16_t) * NEL, hipMemcpyHostToDevice));
  }
  float *d_master, *d_m, *d_v, *d_ss;
  uint16_t* d_working;
  CHECK_HIP(hipMalloc((void**)&d_master, sizeof(float) * NEL));
  CHECK_HIP(hipMalloc((void**)&d_m, sizeof(float) * NEL));
  CHECK_HIP(hipMalloc((void**)&d_v, sizeof(float) * NEL));
  CHECK_HIP(hipMalloc((void**)&d_working, sizeof(uint16_t) * NEL));
  CHECK_HIP(hipMalloc((void**)&d_ss, sizeof(float) * NSTEP * NSEG));
  CHECK_HIP(hipMemcpy(d_master, master, sizeof(float) * NEL, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_m, zeros, sizeof(float) * NEL, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_v, zeros, sizeof(float) * NEL, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_working, working, sizeof(uint16_t) * NEL, hipMemcpyHostToDevice));

  fl_round_cfg cfg;
  memset(&cfg, 0, sizeof cfg);
  cfg.R = NPEER;
  cfg.G = NGRP;
  cfg.A = NSTEP;
  cfg.self_group = self_group;
  cfg.grad_scale = grad_scale;
  cfg.h.lr = 3e-4f;
  cfg.h.beta1 = 0.9f;
  cfg.h.beta2 = 0.95f;
  cfg.h.eps = 1e-8f;
  cfg.h.weight_decay = 0.1f;
  cfg.step0 = step0;
  cfg.weights = weights;

  /* an invalid configuration is refused before anything is enqueued */
  fl_round_cfg bad = cfg;
  bad.R = 0;
  rc = fl_round(lay, &bad, (const uint16_t* const*)d_grads, (const uint16_t* const*)d_reps,
                d_master, d_m, d_v, d_working, d_ss, NULL);
  if (rc != FL_ERR_INVALID) {
    fprintf(stderr, "abi_round: R = 0 gave %d, expected FL_ERR_INVALID\n", rc);
    return 1;
  }

  rc = fl_round(lay, &cfg, (const uint16_t* const*)d_grads, (const uint16_t* const*)d_reps,
                d_master, d_m, d_v, d_working, d_ss, NULL);
  if (rc != FL_OK) {
    fprintf(stderr, "abi_round: fl_round: %s\n", fl_status_string(rc));
    return 1;
  }
  CHECK_HIP(hipDeviceSynchronize());
  CHECK_HIP(hipMemcpy(master_out, d_master, sizeof(float) * NEL, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(m_out, d_m, sizeof(float) * NEL, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(v_out, d_v, sizeof(float) * NEL, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(working_out, d_working, sizeof(uint16_t) * NEL, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(ss_out, d_ss, sizeof(float) * NSTEP * NSEG, hipMemcpyDeviceToHost));

  /* oracle on the same host inputs */
  memcpy(master_ref, master, sizeof master);
  memcpy(working_ref, working, sizeof working);
  const uint16_t* h_grads[NSTEP * NPEER];
  const uint16_t* h_reps[NGRP];
  for (int k = 0; k < NSTEP * NPEER; ++k) h_grads[k] = grads[k];
  for (int g = 0; g < NGRP; ++g) h_reps[g] = reps[g];
  orc_hparams oh = {3e-4f, 0.9f, 0.95f, 1e-8f, 0.1f};
  rc = orc_round(NSEG, off, decay, NPEER, NGRP, NSTEP, self_group, grad_scale, &oh, step0,
                 weights, h_grads, h_reps, master_ref, m_ref, v_ref, working_ref, ss_ref, NULL,
                 0.0f, NULL);
  if (rc != 0) {
    fprintf(stderr, "abi_round: orc_round returned %d\n", rc);
    return 1;
  }

  int bad_elems = 0;
  bad_elems += memcmp(master_out, master_ref, sizeof master_ref) != 0;
  bad_elems += memcmp(m_out, m_ref, sizeof m_ref) != 0;
  bad_elems += memcmp(v_out, v_ref, sizeof v_ref) != 0;
  bad_elems += memcmp(working_out, working_ref, sizeof working_ref) != 0;
  double worst = 0.0;
  for (int k = 0; k < NSTEP * NSEG; ++k) {
    const double rel = fabs((double)ss_out[k] - ss_ref[k]) / (ss_ref[k] > 0 ? ss_ref[k] : 1.0);
    if (rel > worst) worst = rel;
  }
  fl_layout_destroy(lay);
  for (int k = 0; k < NSTEP * NPEER; ++k) hipFree(d_grads[k]);
  for (int g = 0; g < NGRP; ++g) hipFree(d_reps[g]);
  hipFree(d_master);
  hipFree(d_m);
  hipFree(d_v);
  hipFree(d_working);
  hipFree(d_ss);
  if (bad_elems || worst > 1e-5) {
    fprintf(stderr, "abi_round: mismatch (%d state arrays differ, seg_sumsq rel err %.3g)\n",
            bad_elems, worst);
    return 1;
  }
  printf("abi_round ok: fl_round (N=%d, R=%d, G=%d, A=%d) bitwise equal to the oracle; "
         "seg_sumsq rel err %.3g; library version 0x%x\n", NEL, NPEER, NGRP, NSTEP, worst,
         fl_version());
  return 0;
}
