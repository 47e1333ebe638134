/*
 * oracle.h -- plain CPU oracle for one GPU's share of FL+FSDP / FL+HSDP
 * parameter synchronisation.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this code; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no source, header, table or helper with the
 * GPU library.
 *
 * What it computes, per element i of a flat shard of n elements split into
 * segments (each a slice of one layer, the unit FSDP shards equally over a
 * sharding group -- Section 2, FSDP):
 *
 *  (a1) local arithmetic of the gradient reduce-scatter over the R peers of
 *       the sharding group (Section 2, FSDP; Section 5.1 notes that the
 *       collectives average gradients and that the order of the floating-
 *       point operations changes bf16 results, so the order is fixed here):
 *         acc = 0; for r = 0..R-1: acc = acc + f32(grad_r[i])   (fp32)
 *         g = acc * grad_scale
 *  (a2) one AdamW step (Section 5 setup: AdamW, lr 3e-4, bf16 training)
 *       on the fp32 master copy with decoupled weight decay and bias
 *       correction, then the bf16 working copy for the next forward:
 *         p  = master[i] * decay_s
 *         mn = b1 * m[i] + omb1 * g
 *         vn = b2 * v[i] + omb2 * (g * g)
 *         den = sqrt(vn) / bc2_sqrt + eps
 *         p  = p - step_size * (mn / den)
 *         master = p; m = mn; v = vn; working = bf16_rne(p)
 *       with host scalars (double, then rounded to float):
 *         step_size = lr / (1 - beta1^t), bc2_sqrt = sqrt(1 - beta2^t),
 *         omb1 = 1 - beta1, omb2 = 1 - beta2,
 *         decay_s = 1 - lr * weight_decay if segment s decays, else 1.
 *  (a3) FedAvg: the weighted average of the G federation groups' replicas
 *       of the shard (Section 2, Federated Learning; Section 4.1, Eq. (3);
 *       Section 4.2, Eq. (4): once aggregated, a shard is the mean of the
 *       matching shards of all groups):
 *         w_g' = w_g / sum_g w_g          (double, then float)
 *         acc = 0; for g = 0..G-1: acc = acc + w_g' * f32(rep_g[i])   (fp32)
 *         master = acc; working = bf16_rne(acc); m and v unchanged.
 *  (a4) one round: A local steps (a1 then a2 at step t = step0 + a), then
 *       FedAvg with the own replica taken from the bf16 working copy
 *       (Section 4.2: groups aggregate once per A local optimiser steps).
 *  (a5) per-segment sum of squares of g for each local step, accumulated in
 *       double in index order.
 *  (n4) learning-rate schedule (Section 5: cosine decay with 10 % warm-up):
 *       for optimiser step t (1-based), s = t - 1:
 *         s < W: f = s / max(1, W)
 *         else:  q = (s - W) / max(1, T - W); f = 0.5 (1 + cos(pi q));
 *                f = f (1 - lr_min / lr_max) + lr_min / lr_max; f = max(0, f)
 *         lr_t = (float)(lr_max * f)                      (all in double)
 *       A round may give each of its A local steps its own lr.
 *  (n5) global-norm clipping of each local step's gradient (the clipping of
 *       torch.nn.utils.clip_grad_norm_), driven by the sum of squares that
 *       (a5) computes: total = sum_i (double)g[i]^2 (index order);
 *       coef = (float)min(1, max_norm / (sqrt(total) + 1e-6)) (double);
 *       g[i] = g[i] * coef (fp32) before AdamW.  The per-segment sums of (a5)
 *       are those of the unclipped g.  max_norm <= 0: no clipping.
 *
 * FL+HSDP (Section 2, HSDP; Section 4.1, Eq. (2); Section 4.2, Eq. (5)): the
 * gradient is averaged in two tiers (Section 5.1), first over the sharding
 * group, then over the H replicas of the replication group, whose all-reduce
 * carries bf16 shards:
 *  (n1) wire[i] = bf16_rne(g1[i]), g1 from (a1) over the sharding group;
 *       g[i] = hsdp_scale * sum_{h=0..H-1} f32(wire_h[i]), h ascending, the own
 *       replica's wire at its index; with H = 1 the second tier is skipped
 *       and g = g1 (HSDP with one replica is FSDP).
 *  (n2) after FedAvg among one replica per group, that replica broadcasts its
 *       fp32 master shard to the others of its group: master = received,
 *       working = bf16_rne(received).
 *
 * Outer optimiser (Section 3: DiLoCo and Photon pair the inner AdamW with an
 * outer Nesterov-momentum step; Section 4.1: other aggregation strategies
 * build on FedAvg).  The outer gradient is the global model at the start of
 * the round minus the weighted average of the groups' models:
 *  (n3) xbar = FedAvg sum of (a3); delta = prev - xbar;
 *       buf = mu * buf + delta;
 *       d = nesterov ? delta + mu * buf : buf;
 *       p = prev - eta * d;
 *       master = p; working = bf16_rne(p); prev = p   (fp32, in this order)
 *       With eta = 1 and mu = 0 this is FedAvg up to the rounding of
 *       prev - (prev - xbar).
 *
 * Every fp32 operation above is one IEEE-754 binary32 operation rounded to
 * nearest even, evaluated in the written order; the file is compiled with
 * -ffp-contract=off and without fast-math, and subnormals are kept.
 */
#ifndef FL_ORACLE_H
#define FL_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  float lr, beta1, beta2, eps, weight_decay;
} orc_hparams;

float orc_bf16_to_f32(uint16_t h);
uint16_t orc_f32_to_bf16(float x);
void orc_f32_to_bf16_array(int64_t n, const float* x, uint16_t* out);
void orc_bf16_to_f32_array(int64_t n, const uint16_t* x, float* out);

/* (a1) g[i] for i in [0, n). grads: R host arrays of n bf16 values. */
int orc_shard_reduce(int64_t n, int R, const uint16_t* const* grads, float grad_scale,
                     float* g);

/* (a5) out[s] = sum over segment s of (double)g[i]^2, i ascending. */
int orc_seg_sumsq(int64_t n_seg, const int64_t* seg_off, const float* g, double* out);

/* (a2) One AdamW step at step number t (1-based) over n = seg_off[n_seg]
 * elements; working may be NULL (not written). */
int orc_adamw_step(int64_t n_seg, const int64_t* seg_off, const uint8_t* seg_decay,
                   const orc_hparams* h, int64_t t, const float* g, float* master, float* m,
                   float* v, uint16_t* working);

/* (a3) FedAvg of G bf16 replicas; working_out may be one of replicas[]. */
int orc_fedavg(int64_t n, int G, const uint16_t* const* replicas, const float* weights,
               float* master_out, uint16_t* working_out);

/* (n5) sum of (double)g[i]^2 over [0, n), index order; clip coefficient.
 * orc_grad_total: acc0 + the same sum for the reduced gradient of R peers
 * (g[i] as in (a1)), so a caller can stream a long shard chunk by chunk and
 * still add in index order. */
double orc_total_sumsq(int64_t n, const float* g);
float orc_clip_coef(double total_sumsq, float max_norm);
double orc_grad_total(int64_t n, int R, const uint16_t* const* grads, float grad_scale,
                      double acc0);

/* (n4) scheduled learning rate of optimiser step t. */
float orc_lr_cosine(int64_t t, int64_t total_steps, int64_t warmup_steps, float lr_max,
                    float lr_min);

/* (a4) One round.  grads: A*R arrays, step-major.  replicas: G arrays, the
 * entry at self_group is ignored (the working copy is used).  step_lr: NULL
 * (every step uses h->lr) or A learning rates.  seg_sumsq: NULL or A*n_seg
 * doubles.  clip_totals: NULL (the norm of each step is that of this
 * shard's g), or A whole-shard sums of squares to clip against (a shard
 * evaluated on a sample of its elements). */
int orc_round(int64_t n_seg, const int64_t* seg_off, const uint8_t* seg_decay, int R, int G,
              int A, int self_group, float grad_scale, const orc_hparams* h, int64_t step0,
              const float* weights, const uint16_t* const* grads,
              const uint16_t* const* replicas, float* master, float* m, float* v,
              uint16_t* working, double* seg_sumsq, const float* step_lr,
              float max_grad_norm, const double* clip_totals);

/* (n1) tier 1 to the bf16 wire format. */
int orc_shard_reduce_wire(int64_t n, int R, const uint16_t* const* grads, float grad_scale,
                          uint16_t* wire);

/* (n2) receive side of the intra-group broadcast. */
int orc_broadcast_recv(int64_t n, const float* recv, float* master, uint16_t* working);

/* One FL+HSDP round on one replica.  grads: A*R sharding-peer arrays;
 * replica_wires: A*H arrays of the other replicas' tier-1 wire shards
 * (entry a*H + replica ignored); member != 0: this replica takes part in
 * FedAvg with the G replicas (entry self_group ignored); member == 0: it
 * receives bcast (fp32) instead.  seg_sumsq: NULL or A*n_seg (of the
 * tier-2 gradient). */
int orc_round_hsdp(int64_t n_seg, const int64_t* seg_off, const uint8_t* seg_decay, int R, int H,
                   int replica, float hsdp_scale, int member, int G, int A, int self_group,
                   float grad_scale, const orc_hparams* h, int64_t step0, const float* weights,
                   const uint16_t* const* grads, const uint16_t* const* replica_wires,
                   const uint16_t* const* replicas, const float* bcast, float* master, float* m,
                   float* v, uint16_t* working, double* seg_sumsq, const float* step_lr,
                   float max_grad_norm, const double* clip_totals);

typedef struct {
  float lr, momentum;
  int nesterov;
} orc_outer;

/* (n3) outer step.  prev, buf: fp32 state (in/out); working_out may be one
 * of replicas[]. */
int orc_fedopt(int64_t n, int G, const uint16_t* const* replicas, const float* weights,
               const orc_outer* o, float* prev, float* buf, float* master_out,
               uint16_t* working_out);

/* A local steps as in orc_round, then the outer step (n3) instead of FedAvg. */
int orc_round_outer(int64_t n_seg, const int64_t* seg_off, const uint8_t* seg_decay, int R, int G,
                    int A, int self_group, float grad_scale, const orc_hparams* h, int64_t step0,
                    const float* weights, const orc_outer* o, const uint16_t* const* grads,
                    const uint16_t* const* replicas, float* prev, float* buf, float* master,
                    float* m, float* v, uint16_t* working, double* seg_sumsq,
                    const float* step_lr, float max_grad_norm, const double* clip_totals);

#ifdef __cplusplus
}
#endif

#endif
