/*
 * synth_host.c -- host build of the synthetic-input generator.
 *
 * Evaluates the value kinds of synth_rng.h on the CPU, either over a
 * contiguous index range or at an arbitrary list of indices (to rebuild the
 * inputs of sampled elements for the oracle).  Must be compiled with
 * -ffp-contract=off so that its bits equal the device build's.
 */
#include <pthread.h>
#include <stddef.h>
#include <stdint.h>

#define SYNTH_FN static inline
#include "synth_rng.h"

static int synth_is_bf16(int kind) {
  return kind == SYN_NORMAL_BF16 || kind == SYN_DRIFT_BF16 ||
         kind == SYN_STUDENT3_BF16;
}

/* One value; returns its bits in the low 32 (f32) or 16 (bf16) bits. */
static uint32_t synth_value(const synth_spec* sp, uint64_t k1, uint64_t k2,
                            uint64_t i) {
  switch (sp->kind) {
    case SYN_NORMAL_F32:
      return synth_fbits((float)(sp->mean + sp->std * synth_normal(k1, i, 0)));
    case SYN_NORMAL_BF16:
      return synth_bf16((float)(sp->mean + sp->std * synth_normal(k1, i, 0)));
    case SYN_DRIFT_F32:
      return synth_fbits(synth_drift_f32(sp, k1, k2, i));
    case SYN_DRIFT_BF16:
      return synth_bf16(synth_drift_f32(sp, k1, k2, i));
    case SYN_STUDENT3_BF16:
      return synth_bf16(synth_student3(sp, k1, i));
    default:
      return 0;
  }
}

static int synth_kind_ok(int kind) {
  return kind >= SYN_NORMAL_F32 && kind <= SYN_STUDENT3_BF16;
}

/* Fill out[0..n) with the values at indices i0..i0+n-1.
 * out is float* for f32 kinds and uint16_t* for bf16 kinds.
 * Returns 0, or -1 on a bad kind or argument. */
int synth_host_fill(const synth_spec* sp, int64_t i0, int64_t n, void* out) {
  if (!sp || !synth_kind_ok(sp->kind) || n < 0 || i0 < 0 || (n > 0 && !out))
    return -1;
  uint64_t k1 = synth_stream_key(sp->seed, sp->stream);
  uint64_t k2 = synth_stream_key(sp->seed, sp->stream2);
  if (synth_is_bf16(sp->kind)) {
    uint16_t* o = (uint16_t*)out;
    for (int64_t j = 0; j < n; ++j)
      o[j] = (uint16_t)synth_value(sp, k1, k2, (uint64_t)(i0 + j));
  } else {
    uint32_t* o = (uint32_t*)out;
    for (int64_t j = 0; j < n; ++j)
      o[j] = synth_value(sp, k1, k2, (uint64_t)(i0 + j));
  }
  return 0;
}

/* out[j] = value at index idx[j], j in [0, n). */
int synth_host_gather(const synth_spec* sp, const int64_t* idx, int64_t n,
                      void* out) {
  if (!sp || !synth_kind_ok(sp->kind) || n < 0 || (n > 0 && (!out || !idx)))
    return -1;
  uint64_t k1 = synth_stream_key(sp->seed, sp->stream);
  uint64_t k2 = synth_stream_key(sp->seed, sp->stream2);
  for (int64_t j = 0; j < n; ++j) {
    if (idx[j] < 0) return -1;
  }
  if (synth_is_bf16(sp->kind)) {
    uint16_t* o = (uint16_t*)out;
    for (int64_t j = 0; j < n; ++j)
      o[j] = (uint16_t)synth_value(sp, k1, k2, (uint64_t)idx[j]);
  } else {
    uint32_t* o = (uint32_t*)out;
    for (int64_t j = 0; j < n; ++j)
      o[j] = synth_value(sp, k1, k2, (uint64_t)idx[j]);
  }
  return 0;
}

/* Raw 64-bit draws, for tests of the generator itself. */
int synth_host_draws(uint64_t seed, uint64_t stream, uint32_t sub, int64_t i0,
                     int64_t n, uint64_t* out) {
  if (n < 0 || i0 < 0 || (n > 0 && !out)) return -1;
  uint64_t k = synth_stream_key(seed, stream);
  for (int64_t j = 0; j < n; ++j) out[j] = synth_draw(k, (uint64_t)(i0 + j), sub);
  return 0;
}

/* Standard-normal draws as doubles, for distribution tests. */
int synth_host_normals(uint64_t seed, uint64_t stream, int64_t i0, int64_t n,
                       double* out) {
  if (n < 0 || i0 < 0 || (n > 0 && !out)) return -1;
  uint64_t k = synth_stream_key(seed, stream);
  for (int64_t j = 0; j < n; ++j) out[j] = synth_normal(k, (uint64_t)(i0 + j), 0);
  return 0;
}

/* The series helpers, exported so a test can compare them with libm. */
double synth_host_log(double x) { return synth_log(x); }
double synth_host_cos2pi(double u) { return synth_cos2pi(u); }
double synth_host_sqrt(double x) { return synth_sqrt(x); }

/* synth_host_fill split over `threads` POSIX threads (same values). */
typedef struct {
  const synth_spec* sp;
  int64_t i0, n;
  void* out;
  int rc;
} synth_job;

static void* synth_job_run(void* p) {
  synth_job* j = (synth_job*)p;
  j->rc = synth_host_fill(j->sp, j->i0, j->n, j->out);
  return NULL;
}

int synth_host_fill_mt(const synth_spec* sp, int64_t i0, int64_t n, void* out, int threads) {
  if (threads <= 1 || n < 65536) return synth_host_fill(sp, i0, n, out);
  if (threads > 64) threads = 64;
  if (!sp || !synth_kind_ok(sp->kind) || n < 0 || i0 < 0 || !out) return -1;
  const size_t esz = synth_is_bf16(sp->kind) ? 2 : 4;
  pthread_t tid[64];
  synth_job job[64];
  const int64_t chunk = (n + threads - 1) / threads;
  int started = 0;
  int rc = 0;
  for (int t = 0; t < threads; ++t) {
    const int64_t lo = (int64_t)t * chunk;
    if (lo >= n) break;
    const int64_t cnt = (lo + chunk <= n) ? chunk : n - lo;
    job[t].sp = sp;
    job[t].i0 = i0 + lo;
    job[t].n = cnt;
    job[t].out = (char*)out + (size_t)lo * esz;
    job[t].rc = 0;
    if (pthread_create(&tid[t], NULL, synth_job_run, &job[t]) != 0) {
      job[t].rc = synth_host_fill(sp, i0 + lo, cnt, job[t].out);
      tid[t] = 0;
    }
    started = t + 1;
  }
  for (int t = 0; t < started; ++t) {
    if (tid[t]) pthread_join(tid[t], NULL);
    if (job[t].rc) rc = job[t].rc;
  }
  return rc;
}
