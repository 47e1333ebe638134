/*
 * oracle.c -- plain, slow, obviously-correct CPU oracle.  TEST INFRASTRUCTURE
 * ONLY (see oracle.h for what is computed and which passages of the paper
 * each step follows).  Scalar loops, one thread, no SIMD, no FMA.
 */
#include "oracle.h"

#ifndef M_PI
#define M_PI 3.14159265358979323846
#endif

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* bf16 is the upper half of a binary32. */
float orc_bf16_to_f32(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

/* binary32 -> bf16, round to nearest, ties to even.  A NaN keeps its sign
 * and upper payload bits and is made quiet. */
uint16_t orc_f32_to_bf16(float x) {
  uint32_t u;
  memcpy(&u, &x, sizeof u);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu) != 0u)
    return (uint16_t)((u >> 16) | 0x0040u);
  uint32_t lower = u & 0xFFFFu;
  uint32_t upper = u >> 16;
  if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u))) upper += 1u;
  return (uint16_t)upper;
}

int orc_shard_reduce(int64_t n, int R, const uint16_t* const* grads, float grad_scale,
                     float* g) {
  if (n < 0 || R < 1 || (n > 0 && (!grads || !g))) return -1;
  for (int64_t i = 0; i < n; ++i) {
    float acc = 0.0f;
    for (int r = 0; r < R; ++r) acc = acc + orc_bf16_to_f32(grads[r][i]);
    g[i] = acc * grad_scale;
  }
  return 0;
}

int orc_seg_sumsq(int64_t n_seg, const int64_t* seg_off, const float* g, double* out) {
  if (n_seg < 0 || !seg_off || (n_seg > 0 && !out)) return -1;
  for (int64_t s = 0; s < n_seg; ++s) {
    double sum = 0.0;
    for (int64_t i = seg_off[s]; i < seg_off[s + 1]; ++i) sum += (double)g[i] * (double)g[i];
    out[s] = sum;
  }
  return 0;
}

double orc_total_sumsq(int64_t n, const float* g) {
  double sum = 0.0;
  for (int64_t i = 0; i < n; ++i) sum += (double)g[i] * (double)g[i];
  return sum;
}

float orc_clip_coef(double total_sumsq, float max_norm) {
  const double c = (double)max_norm / (sqrt(total_sumsq) + 1e-6);
  /* min(1, c) as torch's clamp takes it: a NaN norm gives a NaN coefficient */
  return (float)(c >= 1.0 ? 1.0 : c);
}

double orc_grad_total(int64_t n, int R, const uint16_t* const* grads, float grad_scale,
                      double acc0) {
  double sum = acc0;
  for (int64_t i = 0; i < n; ++i) {
    float acc = 0.0f;
    for (int r = 0; r < R; ++r) acc = acc + orc_bf16_to_f32(grads[r][i]);
    const float g = acc * grad_scale;
    sum += (double)g * (double)g;
  }
  return sum;
}

/* (n5) scale g in place by the clip coefficient of the whole-shard norm:
 * that of g itself, or the given total. */
static void orc_clip(int64_t n, float* g, float max_norm, const double* total) {
  const float coef = orc_clip_coef(total ? *total : orc_total_sumsq(n, g), max_norm);
  for (int64_t i = 0; i < n; ++i) g[i] = g[i] * coef;
}

int orc_adamw_step(int64_t n_seg, const int64_t* seg_off, const uint8_t* seg_decay,
                   const orc_hparams* h, int64_t t, const float* g, float* master, float* m,
                   float* v, uint16_t* working) {
  if (n_seg < 0 || !seg_off || !h || t < 1) return -1;
  const double lr = (double)h->lr;
  const double bc1 = 1.0 - pow((double)h->beta1, (double)t);
  const double bc2 = 1.0 - pow((double)h->beta2, (double)t);
  const float step_size = (float)(lr / bc1);
  const float bc2_sqrt = (float)sqrt(bc2);
  const float b1 = h->beta1;
  const float b2 = h->beta2;
  const float omb1 = (float)(1.0 - (double)h->beta1);
  const float omb2 = (float)(1.0 - (double)h->beta2);
  const float eps = h->eps;
  const float decay_on = (float)(1.0 - lr * (double)h->weight_decay);

  for (int64_t s = 0; s < n_seg; ++s) {
    const float decay = (seg_decay == NULL || seg_decay[s]) ? decay_on : 1.0f;
    for (int64_t i = seg_off[s]; i < seg_off[s + 1]; ++i) {
      const float gi = g[i];
      float p = master[i] * decay;
      const float mn = (b1 * m[i]) + (omb1 * gi);
      const float vn = (b2 * v[i]) + (omb2 * (gi * gi));
      const float den = (sqrtf(vn) / bc2_sqrt) + eps;
      p = p - (step_size * (mn / den));
      master[i] = p;
      m[i] = mn;
      v[i] = vn;
      if (working) working[i] = orc_f32_to_bf16(p);
    }
  }
  return 0;
}

/* Normalised FedAvg weights: w_g / sum(w) with the sum taken in double in
 * index order, each quotient rounded to float.  -1 if a weight is negative
 * or not finite or the sum is not positive. */
static int orc_norm_weights(int G, const float* w, float* out) {
  double sum = 0.0;
  for (int k = 0; k < G; ++k) {
    if (!(w[k] >= 0.0f) || !isfinite(w[k])) return -1;
    sum += (double)w[k];
  }
  if (!(sum > 0.0) || !isfinite(sum)) return -1;
  for (int k = 0; k < G; ++k) out[k] = (float)((double)w[k] / sum);
  return 0;
}

int orc_fedavg(int64_t n, int G, const uint16_t* const* replicas, const float* weights,
               float* master_out, uint16_t* working_out) {
  if (n < 0 || G < 1 || !weights || (n > 0 && (!replicas || !master_out || !working_out)))
    return -1;
  float* wn = (float*)malloc(sizeof(float) * (size_t)G);
  if (!wn) return -1;
  if (orc_norm_weights(G, weights, wn) != 0) {
    free(wn);
    return -1;
  }
  for (int64_t i = 0; i < n; ++i) {
    float acc = 0.0f;
    for (int k = 0; k < G; ++k) acc = acc + (wn[k] * orc_bf16_to_f32(replicas[k][i]));
    master_out[i] = acc;
    working_out[i] = orc_f32_to_bf16(acc);
  }
  free(wn);
  return 0;
}

int orc_round(int64_t n_seg, const int64_t* seg_off, const uint8_t* seg_decay, int R, int G,
              int A, int self_group, float grad_scale, const orc_hparams* h, int64_t step0,
              const float* weights, const uint16_t* const* grads,
              const uint16_t* const* replicas, float* master, float* m, float* v,
              uint16_t* working, double* seg_sumsq, const float* step_lr,
              float max_grad_norm, const double* clip_totals) {
  if (n_seg < 0 || !seg_off || R < 1 || G < 1 || A < 1 || self_group < 0 ||
      self_group >= G || !h || step0 < 1 || !weights || !grads || !replicas)
    return -1;
  const int64_t n = seg_off[n_seg];
  if (n > 0 && (!master || !m || !v || !working)) return -1;
  float* g = (float*)malloc(sizeof(float) * (size_t)(n > 0 ? n : 1));
  const uint16_t** reps = (const uint16_t**)malloc(sizeof(uint16_t*) * (size_t)G);
  if (!g || !reps) {
    free(g);
    free(reps);
    return -1;
  }
  int rc = 0;
  for (int a = 0; a < A && rc == 0; ++a) {
    rc = orc_shard_reduce(n, R, grads + (size_t)a * (size_t)R, grad_scale, g);
    if (rc == 0 && seg_sumsq)
      rc = orc_seg_sumsq(n_seg, seg_off, g, seg_sumsq + (size_t)a * (size_t)n_seg);
    if (rc == 0 && max_grad_norm > 0.0f)
      orc_clip(n, g, max_grad_norm, clip_totals ? clip_totals + a : NULL);
    orc_hparams ha = *h;
    if (step_lr) ha.lr = step_lr[a];
    if (rc == 0)
      rc = orc_adamw_step(n_seg, seg_off, seg_decay, &ha, step0 + a, g, master, m, v, working);
  }
  if (rc == 0) {
    for (int k = 0; k < G; ++k) reps[k] = (k == self_group) ? working : replicas[k];
    rc = orc_fedavg(n, G, reps, weights, master, working);
  }
  free(g);
  free(reps);
  return rc;
}

int orc_shard_reduce_wire(int64_t n, int R, const uint16_t* const* grads, float grad_scale,
                          uint16_t* wire) {
  if (n < 0 || R < 1 || (n > 0 && (!grads || !wire))) return -1;
  for (int64_t i = 0; i < n; ++i) {
    float acc = 0.0f;
    for (int r = 0; r < R; ++r) acc = acc + orc_bf16_to_f32(grads[r][i]);
    wire[i] = orc_f32_to_bf16(acc * grad_scale);
  }
  return 0;
}

int orc_broadcast_recv(int64_t n, const float* recv, float* master, uint16_t* working) {
  if (n < 0 || (n > 0 && (!recv || !master || !working))) return -1;
  for (int64_t i = 0; i < n; ++i) {
    master[i] = recv[i];
    working[i] = orc_f32_to_bf16(recv[i]);
  }
  return 0;
}

int orc_round_hsdp(int64_t n_seg, const int64_t* seg_off, const uint8_t* seg_decay, int R, int H,
                   int replica, float hsdp_scale, int member, int G, int A, int self_group,
                   float grad_scale, const orc_hparams* h, int64_t step0, const float* weights,
                   const uint16_t* const* grads, const uint16_t* const* replica_wires,
                   const uint16_t* const* replicas, const float* bcast, float* master, float* m,
                   float* v, uint16_t* working, double* seg_sumsq, const float* step_lr,
                   float max_grad_norm, const double* clip_totals) {
  if (n_seg < 0 || !seg_off || R < 1 || H < 1 || replica < 0 || replica >= H || A < 1 ||
      !h || step0 < 1 || !grads)
    return -1;
  if (H > 1 && !replica_wires) return -1;
  if (member && (G < 1 || self_group < 0 || self_group >= G || !weights || !replicas)) return -1;
  if (!member && !bcast && seg_off[n_seg] > 0) return -1;
  const int64_t n = seg_off[n_seg];
  if (n > 0 && (!master || !m || !v || !working)) return -1;
  float* g = (float*)malloc(sizeof(float) * (size_t)(n > 0 ? n : 1));
  uint16_t* wire = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)(n > 0 ? n : 1));
  const uint16_t** wires = (const uint16_t**)malloc(sizeof(uint16_t*) * (size_t)H);
  const uint16_t** reps = (const uint16_t**)malloc(sizeof(uint16_t*) * (size_t)(G > 0 ? G : 1));
  int rc = (g && wire && wires && reps) ? 0 : -1;
  for (int a = 0; a < A && rc == 0; ++a) {
    const uint16_t* const* ga = grads + (size_t)a * (size_t)R;
    if (H == 1) {
      rc = orc_shard_reduce(n, R, ga, grad_scale, g);
    } else {
      rc = orc_shard_reduce_wire(n, R, ga, grad_scale, wire);
      for (int k = 0; k < H; ++k)
        wires[k] = (k == replica) ? wire : replica_wires[(size_t)a * (size_t)H + (size_t)k];
      if (rc == 0) rc = orc_shard_reduce(n, H, wires, hsdp_scale, g);
    }
    if (rc == 0 && seg_sumsq)
      rc = orc_seg_sumsq(n_seg, seg_off, g, seg_sumsq + (size_t)a * (size_t)n_seg);
    if (rc == 0 && max_grad_norm > 0.0f)
      orc_clip(n, g, max_grad_norm, clip_totals ? clip_totals + a : NULL);
    orc_hparams ha = *h;
    if (step_lr) ha.lr = step_lr[a];
    if (rc == 0)
      rc = orc_adamw_step(n_seg, seg_off, seg_decay, &ha, step0 + a, g, master, m, v, working);
  }
  if (rc == 0) {
    if (member) {
      for (int k = 0; k < G; ++k) reps[k] = (k == self_group) ? working : replicas[k];
      rc = orc_fedavg(n, G, reps, weights, master, working);
    } else {
      rc = orc_broadcast_recv(n, bcast, master, working);
    }
  }
  free(g);
  free(wire);
  free(wires);
  free(reps);
  return rc;
}

int orc_fedopt(int64_t n, int G, const uint16_t* const* replicas, const float* weights,
               const orc_outer* o, float* prev, float* buf, float* master_out,
               uint16_t* working_out) {
  if (n < 0 || G < 1 || !weights || !o ||
      (n > 0 && (!replicas || !prev || !buf || !master_out || !working_out)))
    return -1;
  float* wn = (float*)malloc(sizeof(float) * (size_t)G);
  if (!wn) return -1;
  if (orc_norm_weights(G, weights, wn) != 0) {
    free(wn);
    return -1;
  }
  const float eta = o->lr;
  const float mu = o->momentum;
  for (int64_t i = 0; i < n; ++i) {
    float xbar = 0.0f;
    for (int k = 0; k < G; ++k) xbar = xbar + (wn[k] * orc_bf16_to_f32(replicas[k][i]));
    const float delta = prev[i] - xbar;
    const float b = (mu * buf[i]) + delta;
    const float d = o->nesterov ? (delta + (mu * b)) : b;
    const float p = prev[i] - (eta * d);
    buf[i] = b;
    prev[i] = p;
    master_out[i] = p;
    working_out[i] = orc_f32_to_bf16(p);
  }
  free(wn);
  return 0;
}

int orc_round_outer(int64_t n_seg, const int64_t* seg_off, const uint8_t* seg_decay, int R, int G,
                    int A, int self_group, float grad_scale, const orc_hparams* h, int64_t step0,
                    const float* weights, const orc_outer* o, const uint16_t* const* grads,
                    const uint16_t* const* replicas, float* prev, float* buf, float* master,
                    float* m, float* v, uint16_t* working, double* seg_sumsq,
                    const float* step_lr, float max_grad_norm, const double* clip_totals) {
  if (n_seg < 0 || !seg_off || R < 1 || G < 1 || A < 1 || self_group < 0 ||
      self_group >= G || !h || !o || step0 < 1 || !weights || !grads || !replicas)
    return -1;
  const int64_t n = seg_off[n_seg];
  if (n > 0 && (!master || !m || !v || !working || !prev || !buf)) return -1;
  float* g = (float*)malloc(sizeof(float) * (size_t)(n > 0 ? n : 1));
  const uint16_t** reps = (const uint16_t**)malloc(sizeof(uint16_t*) * (size_t)G);
  int rc = (g && reps) ? 0 : -1;
  for (int a = 0; a < A && rc == 0; ++a) {
    rc = orc_shard_reduce(n, R, grads + (size_t)a * (size_t)R, grad_scale, g);
    if (rc == 0 && seg_sumsq)
      rc = orc_seg_sumsq(n_seg, seg_off, g, seg_sumsq + (size_t)a * (size_t)n_seg);
    if (rc == 0 && max_grad_norm > 0.0f)
      orc_clip(n, g, max_grad_norm, clip_totals ? clip_totals + a : NULL);
    orc_hparams ha = *h;
    if (step_lr) ha.lr = step_lr[a];
    if (rc == 0)
      rc = orc_adamw_step(n_seg, seg_off, seg_decay, &ha, step0 + a, g, master, m, v, working);
  }
  if (rc == 0) {
    for (int k = 0; k < G; ++k) reps[k] = (k == self_group) ? working : replicas[k];
    rc = orc_fedopt(n, G, reps, weights, o, prev, buf, master, working);
  }
  free(g);
  free(reps);
  return rc;
}

float orc_lr_cosine(int64_t t, int64_t total_steps, int64_t warmup_steps, float lr_max,
                    float lr_min) {
  const double s = (double)(t - 1);
  const double w = (double)warmup_steps;
  double f;
  if (s < w) {
    f = s / (w > 1.0 ? w : 1.0);
  } else {
    const double span = (double)(total_steps - warmup_steps);
    const double q = (s - w) / (span > 1.0 ? span : 1.0);
    const double rho = (double)lr_min / (double)lr_max;
    f = 0.5 * (1.0 + cos(M_PI * q));
    f = f * (1.0 - rho) + rho;
    if (f < 0.0) f = 0.0;
  }
  return (float)((double)lr_max * f);
}

/* Array forms of the two conversions, for the tests. */
void orc_f32_to_bf16_array(int64_t n, const float* x, uint16_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_f32_to_bf16(x[i]);
}

void orc_bf16_to_f32_array(int64_t n, const uint16_t* x, float* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_bf16_to_f32(x[i]);
}
