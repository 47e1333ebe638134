/*
 * flround.h -- C ABI of libflround: one GPU's share of the parameter
 * synchronisation in FL+FSDP and FL+HSDP training, on AMD Instinct MI355X
 * (gfx950).
 *
 * The method (Section 4.2) runs F federation groups, each an FSDP (or HSDP)
 * deployment with the same sharding policy.  Every local step, each rank
 * reduce-scatters the gradients of its sharding group and applies the inner
 * optimiser (AdamW, Section 5) to its shard; every A steps the ranks that hold
 * corresponding shards in the F groups replace them by their weighted average
 * (FedAvg, Section 2 and Section 4.1 Eq. (3); Eq. (4) and Eq. (5) for the
 * FSDP and HSDP variants).  This library computes, for one rank's flat shard
 * of N elements, the arithmetic of that schedule with the collectives already
 * done: the peers' gradient contributions and the other groups' replicas are
 * plain device buffers.
 *
 * Notation: N shard elements, split into n_seg segments (slices of layers,
 * the unit FSDP shards equally -- Section 2); R peers of the sharding group
 * (the paper's S); G federation groups (the paper's F); A local steps
 * between aggregations.
 *
 * Conventions, for every function below:
 *  - Return value: an fl_status.  Nothing throws, aborts or prints.
 *  - Every argument is checked before anything is enqueued; on an error
 *    nothing has been launched and no output has been touched.
 *  - "Device pointer" arguments point to device memory of the device that
 *    was current when the layout was created; that device must be current at
 *    the call (else FL_ERR_DEVICE).  They must be 16-byte aligned
 *    (FL_ERR_ALIGN).  They may be NULL only when N == 0.  The caller owns all
 *    of them; the library keeps no pointer after a call returns.
 *  - Arrays of pointers ("host array of device pointers") and weight or
 *    fingerprint arrays live in host memory and are read during the call.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream)
 *    and the call returns without waiting for it.  A launch failure returns
 *    FL_ERR_HIP.
 *  - bf16 values are passed as their 16-bit patterns (uint16_t).
 *  - Arithmetic: fp32, in the operation order stated per function, each
 *    operation correctly rounded (no contraction into FMA, subnormals kept);
 *    bf16 results are rounded to nearest even from fp32, NaN stays NaN.
 *    Results are bitwise independent of the launch configuration.
 *  - Calls that write the same buffers must not overlap in time.
 */
#ifndef FLROUND_H
#define FLROUND_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FL_OK = 0,
  FL_ERR_INVALID = -1, /* NULL where not allowed, value out of range, non-finite */
  FL_ERR_ALIGN = -2,   /* a device pointer is not 16-byte aligned               */
  FL_ERR_LAYOUT = -3,  /* a replica's layout fingerprint differs from ours      */
  FL_ERR_DEVICE = -4,  /* current device is not the layout's device             */
  FL_ERR_HIP = -5,     /* a HIP runtime call or a kernel launch failed          */
  FL_ERR_NOMEM = -6,   /* host or device allocation failed                      */
  FL_ERR_SCRATCH = -7  /* fl_round_noalloc: the layout's per-segment workspace
                          exceeds the library's static scratch                 */
} fl_status;

#define FL_MAX_PEERS 64  /* upper bound on R */
#define FL_MAX_GROUPS 64 /* upper bound on G */

/* Human-readable name of a status code (static storage). */
const char* fl_status_string(int status);

/* ABI version: (major << 16) | minor.  Minor versions add entry points or
 * append fields to the end of a configuration struct; a caller built against
 * minor k needs a library of minor >= k.  Minor 1: the FL+HSDP entry
 * points; 2: the outer step; 3: fl_lr_cosine and fl_round_cfg.step_lr;
 * 4: fl_round_cfg.max_grad_norm and the clipping entry points;
 * 5: fl_round_cfg.grad_scratch. */
int fl_version(void);

/* ------------------------------------------------------------------------
 * Shard layout.  The flat shard of N elements is the concatenation of
 * n_seg segments; segment s covers [seg_offsets[s], seg_offsets[s+1]) and
 * takes weight decay iff seg_decay[s] != 0.  All federation groups must use
 * the same layout (the alignment constraint of Section 4.2); the
 * fingerprint lets a caller check that before averaging.
 *
 * fl_layout_create: n >= 0; n_seg >= 1 when n > 0 (n_seg == 0 allowed only
 *   for n == 0); seg_offsets: host array of n_seg + 1 values, [0] == 0,
 *   strictly increasing, [n_seg] == n; seg_decay: host array of n_seg flags,
 *   or NULL for "every segment decays".  Uploads small per-segment and
 *   per-tile tables (about 16 bytes per 2048 elements) to the current device,
 *   and allocates the workspace of the per-segment sums of squares (32 bytes
 *   per (2048-element tile, segment) pair -- twice that when there are at
 *   most 8 segments of at most 1024 tiles each -- plus 8 per segment and per
 *   1024-tile chunk of a segment; zeroed once); returns FL_ERR_NOMEM /
 *   FL_ERR_HIP if that fails.  *out receives a handle that may be used from
 *   several streams at once.
 *   The workspace serves one call at a time: a call that needs it (seg_sumsq
 *   given, or clipping) uses it when no other host thread's call holds it,
 *   after making its stream wait for the kernels of the last call that used
 *   it when that call ran on another stream; a call made while it is held,
 *   or on a stream being captured into a HIP graph, takes a stream-ordered
 *   temporary of the same size instead, allocated and freed on its stream.
 * fl_layout_destroy: frees the handle and its device tables (NULL is OK).
 *   The caller must ensure no enqueued call still uses it.
 * ---------------------------------------------------------------------- */
typedef struct fl_layout fl_layout;

int fl_layout_create(int64_t n, int64_t n_seg, const int64_t* seg_offsets,
                     const uint8_t* seg_decay, fl_layout** out);
int fl_layout_destroy(fl_layout* layout);
int64_t fl_layout_numel(const fl_layout* layout);        /* N, or -1 on NULL     */
int64_t fl_layout_num_segments(const fl_layout* layout); /* n_seg, or -1 on NULL */

/* 64-bit FNV-1a hash of (n, n_seg, seg_offsets, decay flags as 0/1).
 * fl_fingerprint computes it on the host without a GPU (0 if the arguments
 * would not make a valid layout); fl_layout_fingerprint returns the
 * layout's (0 on NULL). */
uint64_t fl_fingerprint(int64_t n, int64_t n_seg, const int64_t* seg_offsets,
                        const uint8_t* seg_decay);
uint64_t fl_layout_fingerprint(const fl_layout* layout);

/* AdamW hyperparameters (Section 5: AdamW, lr 3e-4).  Requirements:
 * finite; lr >= 0; 0 <= beta1 < 1; 0 <= beta2 < 1; eps > 0;
 * weight_decay >= 0. */
typedef struct {
  float lr, beta1, beta2, eps, weight_decay;
} fl_adamw_hparams;

/* ------------------------------------------------------------------------
 * fl_shard_reduce -- local arithmetic of the intra-group gradient
 * reduce-scatter (Section 2, FSDP; Eq. (1)): the R peers' bf16 contributions
 * to this rank's shard, summed in fp32 in ascending peer order and scaled
 * (grad_scale = 1/R averages, as the collectives of Section 5.1 do):
 *     acc = 0; for r in 0..R-1: acc = acc + f32(peer_grads[r][i]);
 *     grad_out[i] = acc * grad_scale
 * peer_grads: host array of R device pointers to N bf16 values (may repeat).
 * grad_out: device pointer, N floats (must not overlap an input).
 * seg_sumsq: NULL, or device pointer to n_seg floats receiving, per segment,
 *   the sum of grad_out[i]^2 (exact double squares, fixed-tree double sums,
 *   rounded once to float): per-layer gradient-norm telemetry.  Uses the
 *   layout's workspace (see fl_layout_create).  A small finalize kernel
 *   folds the pass's per-tile partials into the per-segment totals.  In
 *   fl_round, fl_round_outer, fl_round_noalloc and fl_round_hsdp, when every
 *   segment spans at most 1024 tiles and there are at most 8 segments, one
 *   extra workgroup of the round's next kernel (the next step, or the
 *   FedAvg or broadcast pass) does that fold instead, with the same fixed
 *   trees and the same bits, while the rest of the kernel streams.
 * 1 <= R <= FL_MAX_PEERS; grad_scale finite.
 * ---------------------------------------------------------------------- */
int fl_shard_reduce(const fl_layout* layout, int R, const uint16_t* const* peer_grads,
                    float grad_scale, float* grad_out, float* seg_sumsq, void* stream);

/* ------------------------------------------------------------------------
 * fl_adamw_step -- one AdamW step (Section 5) of the fp32 master shard at
 * step number `step` (1-based), decoupled weight decay first, bias-corrected
 * moments, eps outside the square root; then the bf16 working copy that the
 * next forward pass all-gathers (Section 2, FSDP):
 *     p  = master[i] * decay_s            (decay_s = 1 - lr*wd if segment s
 *                                          decays, else 1)
 *     mn = beta1 * m[i] + (1 - beta1) * g[i]
 *     vn = beta2 * v[i] + (1 - beta2) * (g[i] * g[i])
 *     p  = p - step_size * (mn / (sqrt(vn) / bc2_sqrt + eps))
 *     master[i] = p; m[i] = mn; v[i] = vn; working[i] = bf16(p)
 * with step_size = lr / (1 - beta1^step), bc2_sqrt = sqrt(1 - beta2^step),
 * 1 - beta and decay_s computed on the host in double and rounded to float.
 * grad: device, N floats.  master, m, v: device, N floats each, updated in
 * place, pairwise distinct.  working: device, N bf16, or NULL to skip.
 * ---------------------------------------------------------------------- */
int fl_adamw_step(const fl_layout* layout, const fl_adamw_hparams* h, int64_t step,
                  const float* grad, float* master, float* m, float* v, uint16_t* working,
                  void* stream);

/* ------------------------------------------------------------------------
 * fl_local_step -- fl_shard_reduce followed by fl_adamw_step in one pass:
 * the reduced gradient stays in registers (nothing runs between the
 * reduce-scatter's completion and the optimiser on the shard).  Bitwise
 * equal to the two-call chain.  working is required here.
 * ---------------------------------------------------------------------- */
int fl_local_step(const fl_layout* layout, const fl_adamw_hparams* h, int64_t step, int R,
                  const uint16_t* const* peer_grads, float grad_scale, float* master, float* m,
                  float* v, uint16_t* working, float* seg_sumsq, void* stream);

/* ------------------------------------------------------------------------
 * fl_fedavg -- FedAvg of G federation-group replicas of this shard
 * (Section 2, Federated Learning; Section 4.1 Eq. (3); Section 4.2: once
 * aggregated, a shard is the mean of the matching shards of all groups, so
 * every group sums the same bf16 inputs in the same ascending order and
 * ends bit-identical):
 *     w'_g = w_g / sum_g w_g        (host, double, rounded to float)
 *     acc = 0; for g in 0..G-1: acc = acc + w'_g * f32(replicas[g][i])
 *     master_out[i] = acc; working_out[i] = bf16(acc)
 * Optimiser moments are not touched.
 * replicas: host array of G device pointers to N bf16 values; the caller's
 *   own replica is its working copy and may be passed as one entry, and
 *   working_out may then be that same pointer (in-place average).  Any
 *   other overlap of outputs with inputs is undefined.
 * weights: host array of G finite values >= 0 with a positive sum
 *   (e.g. per-group sample counts).
 * replica_fp: NULL, or host array of G layout fingerprints, one per replica;
 *   any entry that differs from this layout's -> FL_ERR_LAYOUT.
 * master_out: device, N floats.  working_out: device, N bf16.
 * 1 <= G <= FL_MAX_GROUPS.
 * ---------------------------------------------------------------------- */
int fl_fedavg(const fl_layout* layout, int G, const uint16_t* const* replicas,
              const float* weights, const uint64_t* replica_fp, float* master_out,
              uint16_t* working_out, void* stream);

/* ------------------------------------------------------------------------
 * fl_round -- one federated round on this shard (Section 4.2, Eq. (4) and
 * Eq. (5)): A local steps, then FedAvg after the A-th local update:
 *     for a in 0..A-1: fl_local_step(step = step0 + a,
 *                                    peer_grads = grads[a*R .. a*R+R-1])
 *     fl_fedavg(replicas with replicas[self_group] := working,
 *               master_out = master, working_out = working)
 * Bitwise equal to that chain of calls.
 * grads: host array of A*R device pointers (step-major; entries may repeat).
 * replicas: host array of G device pointers; entry self_group is ignored
 *   (may be NULL).
 * master, m, v: device, N floats; working: device, N bf16; all updated in
 *   place and pairwise distinct.
 * seg_sumsq: NULL, or device pointer to A*n_seg floats (row a = local step a;
 *   see fl_shard_reduce).
 * Allocation: with seg_sumsq or max_grad_norm > 0 the round uses the
 *   layout's workspace for all its steps, or one stream-ordered temporary
 *   when that is not available to this stream (see fl_layout_create); under
 *   graph capture the temporary becomes a graph allocation.  Without them it
 *   allocates nothing.  fl_round_noalloc never allocates.
 * Configuration: 1 <= R <= FL_MAX_PEERS, 1 <= G <= FL_MAX_GROUPS, A >= 1,
 *   0 <= self_group < G, step0 >= 1, grad_scale finite, h and weights as
 *   above, replica_fp as in fl_fedavg, step_lr entries finite and >= 0,
 *   max_grad_norm finite and >= 0.
 * phase_events: NULL, or host array of A+2 hipEvent_t created by the caller;
 *   event a (a < A) is recorded on `stream` before local step a, event A
 *   before FedAvg, event A+1 after it (per-phase timing of the round, like
 *   the optimiser / aggregation split of Table 4).  A NULL entry records
 *   nothing at its point (e.g. only events 0, A and A+1: every event
 *   recorded between kernels costs GPU time).
 * ---------------------------------------------------------------------- */
typedef struct {
  int R;                     /* peers in the sharding group                 */
  int G;                     /* federation groups                           */
  int A;                     /* local steps between aggregations            */
  int self_group;            /* index of this rank's group among the G      */
  float grad_scale;          /* 1/R for averaging                           */
  fl_adamw_hparams h;        /* inner optimiser                             */
  int64_t step0;             /* step number of the round's first local step */
  const float* weights;      /* host, G FedAvg weights                      */
  const uint64_t* replica_fp;/* NULL or host, G fingerprints                */
  void* const* phase_events; /* NULL or host, A+2 hipEvent_t (entries may  */
                             /* be NULL)                                    */
  const float* step_lr;      /* NULL or host, A learning rates, one per local
                                step (overrides h.lr; e.g. fl_lr_cosine)   */
  float max_grad_norm;       /* > 0: clip each local step's gradient to this
                                global norm (fl_local_step_clipped); 0: off;
                                negative or non-finite: FL_ERR_INVALID      */
  float* grad_scratch;       /* NULL, or device, N floats distinct from every
                                other buffer: with max_grad_norm > 0 the
                                sum-of-squares pass also stores each step's
                                reduced gradient there and the step reads it
                                back, so the peer gradients are read once:
                                2R + 34 bytes per element instead of 4R + 26
                                (faster for R >= 6).  Same results bit for
                                bit.  Ignored without clipping and by
                                fl_round_hsdp with H > 1.                   */
} fl_round_cfg;

int fl_round(const fl_layout* layout, const fl_round_cfg* cfg, const uint16_t* const* grads,
             const uint16_t* const* replicas, float* master, float* m, float* v,
             uint16_t* working, float* seg_sumsq, void* stream);

/* ------------------------------------------------------------------------
 * fl_round_noalloc -- fl_round for callers that cannot allocate device
 * memory: code being captured into a HIP graph, tight serving loops, and
 * harnesses that forbid allocation.  Same arguments, same arithmetic, same
 * bits as fl_round; it calls no allocator, and the workspace of the
 * per-segment sums of squares (seg_sumsq given, or clipping) is a static
 * device array of the library, FL_NOALLOC_SCRATCH_BYTES (32 MiB) per GPU,
 * held from the library's first use of that GPU until the process ends.
 * Every fl_round_noalloc call on one GPU shares that array: calls that
 * overlap in time on one GPU (two streams, two host threads) race and give
 * undefined results; calls on one stream are ordered and safe.
 * A layout whose workspace (as in fl_layout_create, plus 8 bytes) exceeds
 * the array returns FL_ERR_SCRATCH before anything is enqueued, when the call
 * needs the workspace; with neither seg_sumsq nor clipping any layout is
 * accepted.  Nothing in the array needs clearing: every slot a call reads it
 * has written first.  The array's address on a GPU is looked up by the first
 * fl_layout_create on that GPU.
 * fl_noalloc_workspace_bytes returns the bytes a layout would need (0 for
 * NULL or an empty layout).
 * ---------------------------------------------------------------------- */
#define FL_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

int fl_round_noalloc(const fl_layout* layout, const fl_round_cfg* cfg,
                     const uint16_t* const* grads, const uint16_t* const* replicas,
                     float* master, float* m, float* v, uint16_t* working, float* seg_sumsq,
                     void* stream);
size_t fl_noalloc_workspace_bytes(const fl_layout* layout);

/* ------------------------------------------------------------------------
 * fl_lr_cosine -- the learning rate of optimiser step t (1-based) under
 * cosine decay with linear warm-up (Section 5 decays the learning rate on a
 * cosine after warming it up over the first tenth of the run), in double,
 * rounded once to float; s = t - 1:
 *     s < warmup:  f = s / max(1, warmup)
 *     otherwise:   q = (s - warmup) / max(1, total - warmup);
 *                  f = 0.5 (1 + cos(pi q)); f = f (1 - lr_min/lr_max) + lr_min/lr_max;
 *                  f = max(0, f)
 *     returns lr_max * f
 * The usual warm-up for a 10 % ratio is ceil(0.1 * total).  Host only; a
 * caller fills fl_round_cfg.step_lr with it for the A steps of a round.
 * ---------------------------------------------------------------------- */
float fl_lr_cosine(int64_t t, int64_t total_steps, int64_t warmup_steps, float lr_max,
                   float lr_min);

/* ------------------------------------------------------------------------
 * Global-norm gradient clipping of a local step (the rule of
 * torch.nn.utils.clip_grad_norm_), driven by the sum of squares of the
 * reduced gradient:
 *     coef = (float)min(1, max_norm / (sqrt(total_sumsq) + 1e-6))   (double;
 *            a NaN total gives a NaN coef, as torch's clamp does)
 *     g[i] = (acc[i] * grad_scale) * coef, then AdamW as fl_local_step
 * The norm is over the whole model, i.e. over every shard of the sharding
 * group: a multi-GPU caller computes its shard's sum with fl_grad_sumsq,
 * all-reduces it, then calls fl_local_step_clipped.  Within one GPU,
 * fl_round_cfg.max_grad_norm does both for the local shard (the per-segment
 * sums then report the unclipped gradient).  coef == 1 leaves the step
 * bitwise equal to the unclipped one.
 *
 * fl_grad_sumsq: total_sumsq = sum_i (double)g[i]^2 of this shard's reduced
 *   gradient (exact double squares, fixed-tree double sums), written to a
 *   device double (8-byte aligned); seg_sumsq: NULL or n_seg floats as in
 *   fl_shard_reduce.  Reads the R gradients once and writes no gradient.
 * fl_local_step_clipped: fl_local_step with the coefficient above, from a
 *   device double total_sumsq; max_norm > 0 and finite.
 * ---------------------------------------------------------------------- */
int fl_grad_sumsq(const fl_layout* layout, int R, const uint16_t* const* peer_grads,
                  float grad_scale, double* total_sumsq, float* seg_sumsq, void* stream);
int fl_local_step_clipped(const fl_layout* layout, const fl_adamw_hparams* h, int64_t step, int R,
                          const uint16_t* const* peer_grads, float grad_scale,
                          const double* total_sumsq, float max_norm, float* master, float* m,
                          float* v, uint16_t* working, void* stream);

/* ------------------------------------------------------------------------
 * Outer optimiser (Section 3: DiLoCo and Photon pair the inner AdamW with an
 * outer Nesterov-momentum step, FedOpt / FedMom; Section 4.1: aggregation
 * strategies that build on FedAvg).  The outer gradient is the global model
 * at the start of the round (prev) minus the FedAvg average of the groups'
 * models:
 *     xbar = the FedAvg sum of fl_fedavg, in the same order
 *     delta = prev[i] - xbar
 *     buf[i] = momentum * buf[i] + delta
 *     d = nesterov ? delta + momentum * buf[i] : buf[i]
 *     p = prev[i] - lr * d
 *     master_out[i] = prev[i] = p; working_out[i] = bf16(p)
 * (torch's SGD with dampening 0 on the outer gradient; with lr = 1 and
 * momentum = 0 it is FedAvg up to the rounding of prev - (prev - xbar)).
 * prev, buf: device, N floats each, caller-owned outer state (start: prev =
 * the global model every group began the round from, buf = 0).
 *
 * fl_fedopt: arguments as fl_fedavg plus the outer state; prev, buf and
 *   master_out pairwise distinct.  Requirements: finite lr >= 0,
 *   0 <= momentum <= 1.
 * fl_round_outer: fl_round with the outer step in place of FedAvg; prev and
 *   buf distinct from master, m, v and each other.
 * ---------------------------------------------------------------------- */
typedef struct {
  float lr;       /* outer learning rate (DiLoCo: 0.7)   */
  float momentum; /* outer momentum (DiLoCo: 0.9)        */
  int nesterov;   /* nonzero: Nesterov form              */
} fl_outer_hparams;

int fl_fedopt(const fl_layout* layout, int G, const uint16_t* const* replicas,
              const float* weights, const uint64_t* replica_fp, const fl_outer_hparams* outer,
              float* prev, float* buf, float* master_out, uint16_t* working_out, void* stream);
int fl_round_outer(const fl_layout* layout, const fl_round_cfg* cfg, const fl_outer_hparams* outer,
                   const uint16_t* const* grads, const uint16_t* const* replicas, float* prev,
                   float* buf, float* master, float* m, float* v, uint16_t* working,
                   float* seg_sumsq, void* stream);

/* ------------------------------------------------------------------------
 * FL+HSDP (Section 2, HSDP; Section 4.1, Eq. (2); Section 4.2, Eq. (5)).
 * Each federation group is an HSDP deployment: H replicas of an S-way
 * sharding group.  Gradients are averaged in two tiers (Section 5.1): over
 * the sharding group (reduce-scatter), then over the H replicas of the shard
 * (all-reduce, whose messages are bf16 shards).  After the A-th local step
 * one replica per group joins FedAvg and then broadcasts its shard to the
 * other replicas of its group.
 *
 * fl_shard_reduce_wire -- tier 1 in the wire format:
 *     acc = 0; for r in 0..R-1: acc = acc + f32(peer_grads[r][i]);
 *     wire_out[i] = bf16(acc * grad_scale)
 *   wire_out: device, N bf16.  Tier 2 is fl_local_step over the H wire
 *   shards (own included at its index) with grad_scale = 1/H.
 *
 * fl_broadcast_recv -- receive side of the broadcast, which carries the fp32
 *   master shard so that all replicas stay bit-identical:
 *     master[i] = recv_master[i]; working[i] = bf16(recv_master[i])
 *   recv_master, master: device, N floats; working: device, N bf16.
 *
 * fl_round_hsdp -- one FL+HSDP round on one replica:
 *     for a in 0..A-1:
 *       H == 1: fl_local_step(R peers grads[a*R ..])      (FL+FSDP)
 *       H  > 1: fl_shard_reduce_wire(grads[a*R ..], grad_scale) -> wire;
 *               fl_local_step(H shards: replica_wires[a*H + k], with
 *                             wire at k == replica; hsdp_scale)
 *     then fedavg_member ? fl_fedavg (as in fl_round) : fl_broadcast_recv.
 *   cfg: as for fl_round (G, self_group, weights, replica_fp are used only
 *   by a FedAvg member).  replica_wires: host array of A*H device pointers
 *   (entry a*H + replica ignored), or NULL when H == 1.  wire: device, N
 *   bf16 scratch that receives this replica's tier-1 shard of each step (the
 *   message it would send); unused when H == 1.  replicas: as for fl_round
 *   (member only).  bcast_master: device, N floats (non-member only).
 *   seg_sumsq: NULL or A*n_seg floats of the tier-2 gradient.
 *   1 <= H <= FL_MAX_PEERS, 0 <= replica < H, hsdp_scale finite.
 *   H == 1 is bitwise fl_round.
 * ---------------------------------------------------------------------- */
typedef struct {
  int H;             /* replicas in the replication group (the paper's R) */
  int replica;       /* this rank's index among the H                     */
  float hsdp_scale;  /* 1/H for averaging                                 */
  int fedavg_member; /* nonzero: joins FedAvg; zero: receives the broadcast */
} fl_hsdp_cfg;

int fl_shard_reduce_wire(const fl_layout* layout, int R, const uint16_t* const* peer_grads,
                         float grad_scale, uint16_t* wire_out, void* stream);
int fl_broadcast_recv(const fl_layout* layout, const float* recv_master, float* master,
                      uint16_t* working, void* stream);
int fl_round_hsdp(const fl_layout* layout, const fl_round_cfg* cfg, const fl_hsdp_cfg* hc,
                  const uint16_t* const* grads, const uint16_t* const* replica_wires,
                  uint16_t* wire, const uint16_t* const* replicas, const float* bcast_master,
                  float* master, float* m, float* v, uint16_t* working, float* seg_sumsq,
                  void* stream);

/* ------------------------------------------------------------------------
 * Launch-shape control, for tuning sweeps and for tests that check that
 * results do not depend on the launch shape.  blocks_per_cu > 0 caps the
 * grid of every streaming kernel at blocks_per_cu * (number of CUs); 0
 * restores the defaults (one workgroup per CU for the fused step and the
 * FedAvg-side passes, more for the passes that only read the peer gradients,
 * by R).  Process-wide; returns the previous value.
 * ---------------------------------------------------------------------- */
int fl_set_blocks_per_cu(int blocks_per_cu);

#ifdef __cplusplus
}
#endif

#endif /* FLROUND_H */
