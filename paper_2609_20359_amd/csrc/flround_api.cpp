// flround_api.cpp -- the C ABI of libflround (declared in include/flround.h).
//
// This layer validates every argument before anything is enqueued, turns the
// paper-level description of a round (group size, number of groups, local
// steps between aggregations, per-group weights) into per-step scalars on the
// host in double, and enqueues the gfx950 kernels on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "flr_internal.h"
#include "flround.h"

using flr::kTile;

struct fl_layout {
  int device = 0;
  int num_cus = 0;
  uint64_t fingerprint = 0;
  void* dev_mem = nullptr;  // one allocation holding all device tables
  flr::LayoutDev L{};
  // Workspace of the per-segment sums of squares (see Workspace below),
  // allocated with the layout and zeroed once.  One call holds it at a time
  // (ws_busy); the last one ran on ws_stream and recorded ws_done after its
  // kernels, which a call on another stream waits for.  A call made while
  // it is held, or one being captured into a graph, takes a stream-ordered
  // allocation of its own.
  void* ws_mem = nullptr;
  std::atomic<bool> ws_busy{false};
  hipStream_t ws_stream = nullptr;
  hipEvent_t ws_done = nullptr;
  bool ws_recorded = false;
  // This device's static scratch of fl_round_noalloc (null if the lookup
  // failed; fl_round_noalloc then reports FL_ERR_HIP when it needs it).
  void* noalloc = nullptr;
};

namespace {

std::atomic<int> g_blocks_per_cu{0};  // 0: the per-pass defaults below

// Default workgroups per CU.  One 256-thread workgroup per CU keeps enough
// 16-byte loads in flight for the passes that stream many arrays (the fused
// step, FedAvg, the optimiser-only and broadcast passes).  A pass that only
// reads the R peer gradients (the sum-of-squares pass, and the reductions when
// R is small) has fewer loads in flight per thread and needs more workgroups
// to cover HBM latency.  Chosen by occupancy sweeps on a 1.0e9-element shard.
constexpr int kDefaultBlocksPerCu = 1;
int sumsq_blocks_per_cu(int R) {
  return R >= 8 ? 2 : R >= 4 ? 3 : R == 3 ? 4 : R == 2 ? 6 : 8;
}
int reduce_blocks_per_cu(int R) { return R >= 8 ? 1 : 2; }
int wire_blocks_per_cu(int R) {
  const bool two_vector_kernel = R == 1 || R == 2 || R == 4 || R == 8 || R == 16;
  if (two_vector_kernel) return R <= 2 ? 2 : 1;
  return R >= 8 ? 1 : 2;
}

constexpr uint64_t kFnvOffset = 0xCBF29CE484222325ULL;
constexpr uint64_t kFnvPrime = 0x100000001B3ULL;

uint64_t fnv_bytes(uint64_t h, const void* p, size_t n) {
  const unsigned char* b = static_cast<const unsigned char*>(p);
  for (size_t i = 0; i < n; ++i) {
    h ^= b[i];
    h *= kFnvPrime;
  }
  return h;
}

bool layout_args_ok(int64_t n, int64_t n_seg, const int64_t* off) {
  if (n < 0 || n_seg < 0 || !off) return false;
  if (n > 0 && n_seg < 1) return false;
  if (n == 0 && n_seg != 0) return false;
  if (n_seg > (int64_t)INT32_MAX - 1) return false;
  if (off[0] != 0 || off[n_seg] != n) return false;
  for (int64_t s = 0; s < n_seg; ++s)
    if (off[s + 1] <= off[s]) return false;
  return true;
}

uint64_t fingerprint_of(int64_t n, int64_t n_seg, const int64_t* off, const uint8_t* decay) {
  uint64_t h = kFnvOffset;
  h = fnv_bytes(h, &n, sizeof n);
  h = fnv_bytes(h, &n_seg, sizeof n_seg);
  h = fnv_bytes(h, off, sizeof(int64_t) * (size_t)(n_seg + 1));
  for (int64_t s = 0; s < n_seg; ++s) {
    const unsigned char f = (decay == nullptr || decay[s] != 0) ? 1 : 0;
    h = fnv_bytes(h, &f, 1);
  }
  return h;
}

bool finite(float x) { return std::isfinite(x); }

bool hparams_ok(const fl_adamw_hparams* h) {
  if (!h) return false;
  if (!finite(h->lr) || !finite(h->beta1) || !finite(h->beta2) || !finite(h->eps) ||
      !finite(h->weight_decay))
    return false;
  if (!(h->lr >= 0.f)) return false;
  if (!(h->beta1 >= 0.f && h->beta1 < 1.f)) return false;
  if (!(h->beta2 >= 0.f && h->beta2 < 1.f)) return false;
  if (!(h->eps > 0.f)) return false;
  if (!(h->weight_decay >= 0.f)) return false;
  return true;
}

// Per-step scalars: double on the host, each rounded once to float.
flr::AdamScalars adam_scalars(const fl_adamw_hparams& h, int64_t step) {
  const double lr = (double)h.lr;
  const double t = (double)step;
  flr::AdamScalars s;
  s.b1 = h.beta1;
  s.b2 = h.beta2;
  s.omb1 = (float)(1.0 - (double)h.beta1);
  s.omb2 = (float)(1.0 - (double)h.beta2);
  s.step_size = (float)(lr / (1.0 - std::pow((double)h.beta1, t)));
  s.bc2_sqrt = (float)std::sqrt(1.0 - std::pow((double)h.beta2, t));
  s.eps = h.eps;
  s.decay = (float)(1.0 - lr * (double)h.weight_decay);
  return s;
}

// FedAvg weights w / sum(w): sum in double in index order.
int normalise_weights(int G, const float* w, float* out) {
  if (!w) return FL_ERR_INVALID;
  double sum = 0.0;
  for (int g = 0; g < G; ++g) {
    if (!finite(w[g]) || !(w[g] >= 0.f)) return FL_ERR_INVALID;
    sum += (double)w[g];
  }
  if (!(sum > 0.0) || !std::isfinite(sum)) return FL_ERR_INVALID;
  for (int g = 0; g < G; ++g) out[g] = (float)((double)w[g] / sum);
  return FL_OK;
}

// Hyperparameters of local step a of a round: step_lr overrides lr.
fl_adamw_hparams step_hparams(const fl_round_cfg& c, int a) {
  fl_adamw_hparams h = c.h;
  if (c.step_lr) h.lr = c.step_lr[a];
  return h;
}

bool step_lrs_ok(const fl_round_cfg& c) {
  if (!std::isfinite(c.max_grad_norm) || !(c.max_grad_norm >= 0.f)) return false;
  if (!c.step_lr) return true;
  for (int a = 0; a < c.A; ++a)
    if (!std::isfinite(c.step_lr[a]) || !(c.step_lr[a] >= 0.f)) return false;
  return true;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// A device pointer argument: must be non-null and 16-byte aligned when n > 0.
int dev_ptr(const void* p, int64_t n) {
  if (n == 0) return FL_OK;
  if (!p) return FL_ERR_INVALID;
  return aligned16(p) ? FL_OK : FL_ERR_ALIGN;
}

int check_device(const fl_layout* lay) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return FL_ERR_HIP;
  return dev == lay->device ? FL_OK : FL_ERR_DEVICE;
}

// Workgroups of a pass over `units` tiles or vector groups: a grid-stride
// loop over a grid of bpc workgroups per CU; a shard whose units all fit on
// the chip at once (at most kResidentPerCu per CU) gets one workgroup per unit
// instead, so that a small shard is not spread over fewer workgroups than it
// has tiles.  An explicit fl_set_blocks_per_cu applies to every pass.
constexpr int kResidentPerCu = 4;
int grid_for(const fl_layout* lay, int64_t units, int default_bpc = kDefaultBlocksPerCu) {
  const int set = g_blocks_per_cu.load(std::memory_order_relaxed);
  if (set <= 0 && units <= (int64_t)kResidentPerCu * lay->num_cus) return (int)(units < 1 ? 1 : units);
  const int bpc = set > 0 ? set : default_bpc;
  int64_t cap = (int64_t)bpc * (int64_t)lay->num_cus;
  if (cap < 1) cap = 1;
  int64_t g = units < cap ? units : cap;
  return (int)(g < 1 ? 1 : g);
}

int fedavg_grid(const fl_layout* lay) {
  const int64_t nvec = (lay->L.n + flr::kVec - 1) / flr::kVec;
  return grid_for(lay, (nvec + flr::kBlock - 1) / flr::kBlock);
}

int status_of(hipError_t e) {
  if (e == hipSuccess) return FL_OK;
  if (e == hipErrorOutOfMemory) return FL_ERR_NOMEM;
  return FL_ERR_HIP;
}

int check_peers(int R, const uint16_t* const* peers, int64_t n) {
  if (R < 1 || R > FL_MAX_PEERS || !peers) return FL_ERR_INVALID;
  for (int r = 0; r < R; ++r) {
    const int rc = dev_ptr(peers[r], n);
    if (rc != FL_OK) return rc;
  }
  return FL_OK;
}

// Whether a pass's finalize may be carried by the next kernel of the same
// call (see flr::Carry): every segment one finalize chunk, few of them.
bool carry_ok(const flr::LayoutDev& L) {
  return L.n_chunks == L.n_seg && L.n_chunks >= 1 && L.n_chunks <= flr::kCarryMaxChunks;
}

// Workspace of the per-segment sums of squares: the (piece, wave) partials
// (kWaves doubles per piece; two sets where the finalize may be carried, so
// that a pass writes one while the next kernel's carried finalize reads the
// other), one double per finalize chunk, one per segment, and the
// whole-shard total.
size_t ws_slots(const flr::LayoutDev& L) {
  return (size_t)(L.n_pieces > 0 ? L.n_pieces : 1) * flr::kWaves;
}
size_t ws_bytes(const flr::LayoutDev& L) {
  const size_t nch = (size_t)(L.n_chunks > 0 ? L.n_chunks : 1);
  const size_t nseg = (size_t)(L.n_seg > 0 ? L.n_seg : 1);
  return (ws_slots(L) * (carry_ok(L) ? 2 : 1) + nch + nseg + 1) * sizeof(double);
}

struct Workspace {
  double* p = nullptr;
  double* p2 = nullptr;         // the second set of partials (null: no carry)
  double* chunks = nullptr;
  double* seg = nullptr;
  double* total = nullptr;
  hipStream_t st = nullptr;
  fl_layout* owner = nullptr;   // the layout whose workspace this is (or null)
  void* own = nullptr;          // a stream-ordered allocation of this call

  // The static scratch of fl_round_noalloc.  Nothing is allocated and
  // nothing needs releasing.
  int use_static(const fl_layout* lay, hipStream_t stream) {
    st = stream;
    if (!lay->noalloc) return FL_ERR_HIP;
    carve(lay->L, lay->noalloc);
    return FL_OK;
  }

  void carve(const flr::LayoutDev& L, void* mem) {
    p = static_cast<double*>(mem);
    p2 = carry_ok(L) ? p + ws_slots(L) : nullptr;
    chunks = p + ws_slots(L) * (p2 ? 2 : 1);
    seg = chunks + (L.n_chunks > 0 ? L.n_chunks : 1);
    total = seg + (L.n_seg > 0 ? L.n_seg : 1);
  }

  // The layout's workspace when this stream may use it, else a stream-ordered
  // allocation.
  int acquire(const fl_layout* layc, hipStream_t stream) {
    fl_layout* lay = const_cast<fl_layout*>(layc);
    st = stream;
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &cs) != hipSuccess) return FL_ERR_HIP;
    bool expected = false;
    if (cs == hipStreamCaptureStatusNone && lay->ws_mem &&
        lay->ws_busy.compare_exchange_strong(expected, true, std::memory_order_acquire)) {
      if (!lay->ws_recorded || lay->ws_stream == stream) {
        // the last call that used it ran on this stream: stream order
        // already puts its kernels first
        owner = lay;
        carve(lay->L, lay->ws_mem);
        return FL_OK;
      }
      if (hipStreamWaitEvent(stream, lay->ws_done, 0) == hipSuccess) {
        // another stream used it last: this stream waits for those kernels
        owner = lay;
        carve(lay->L, lay->ws_mem);
        return FL_OK;
      }
      lay->ws_busy.store(false, std::memory_order_release);
      return FL_ERR_HIP;
    }
    const hipError_t e = hipMallocAsync(&own, ws_bytes(lay->L), st);
    if (e != hipSuccess) {
      own = nullptr;
      return status_of(e);
    }
    carve(lay->L, own);
    return FL_OK;
  }

  int release() {
    int rc = FL_OK;
    if (owner) {
      if (hipEventRecord(owner->ws_done, st) == hipSuccess) {
        owner->ws_stream = st;
        owner->ws_recorded = true;
      } else {
        // nothing marks where this call's kernels end: wait for them here,
        // so that the next call may take the workspace on any stream
        (void)hipStreamSynchronize(st);
        owner->ws_recorded = false;
        owner->ws_stream = nullptr;
        rc = FL_ERR_HIP;
      }
      owner->ws_busy.store(false, std::memory_order_release);
      owner = nullptr;
    } else if (own) {
      rc = status_of(hipFreeAsync(own, st));
      own = nullptr;
    }
    p = p2 = chunks = seg = total = nullptr;
    return rc;
  }
};

// Bytes of the static scratch a layout's workspace needs in fl_round_noalloc.
size_t noalloc_bytes(const flr::LayoutDev& L) { return ws_bytes(L); }

// The partials set for a pass: the one a carried finalize in the same launch
// does not read.
double* free_slot(const Workspace& ws, const flr::Carry& c) {
  return (ws.p2 && c.partials == ws.p) ? ws.p2 : ws.p;
}

// Move a pending carried finalize into a kernel's arguments.
template <typename Args>
void take_carry(Args& a, flr::Carry* pending) {
  if (pending && pending->partials) {
    a.carry = *pending;
    pending->partials = nullptr;
  }
}

// After a pass with per-segment sums: leave the finalize to the next kernel
// of the call (pending non-null and the layout allows it), else enqueue the
// finalize kernels now.
int finish_sums(const fl_layout* lay, const Workspace& ws, double* partials, float* out,
                flr::Carry* pending, hipStream_t st) {
  if (pending && ws.p2) {
    pending->partials = partials;
    pending->chunk_p0 = lay->L.chunk_p0;
    pending->n_chunks = lay->L.n_chunks;
    pending->out = out;
    return FL_OK;
  }
  return status_of(flr::launch_seg_finalize(lay->L, partials, ws.chunks, ws.seg, out, nullptr,
                                            st));
}

flr::StepArgs step_args(const fl_layout* lay) {
  flr::StepArgs a;
  std::memset(&a, 0, sizeof a);
  a.L = lay->L;
  return a;
}

// Enqueue one fused local step (and, with seg_sumsq, its per-segment sums).
// With clip_max > 0 the step first runs a sum-of-squares pass over the same
// inputs (whole-shard total and, if asked, the per-segment sums), then the
// fused step with the gradient scaled by the clip coefficient.  Given
// g_scratch (N floats), the first pass also stores the reduced gradient and
// the step is the AdamW-only pass over it, so the peer gradients are read
// once: 2R + 4 then 30 bytes per element instead of 2R then 2R + 26.
// pending (may be null): the finalize carried between the kernels of one
// call; the first kernel enqueued here runs the one pending, and an
// unclipped step with per-segment sums may leave its own there.
int enqueue_local_step(const fl_layout* lay, const fl_adamw_hparams& h, int64_t step, int R,
                       const uint16_t* const* peers, float grad_scale, float* master, float* m,
                       float* v, uint16_t* working, const Workspace& ws, float* seg_sumsq,
                       hipStream_t st, float clip_max = 0.f, float* g_scratch = nullptr,
                       flr::Carry* pending = nullptr) {
  flr::StepArgs a = step_args(lay);
  for (int r = 0; r < R; ++r) a.grads[r] = peers[r];
  a.R = R;
  a.grad_scale = grad_scale;
  const int grid = grid_for(lay, lay->L.n_tiles);
  int rc = FL_OK;
  take_carry(a, pending);
  if (clip_max > 0.f && g_scratch) {
    a.partials = free_slot(ws, a.carry);
    a.g_out = g_scratch;
    rc = status_of(flr::launch_reduce(a, grid_for(lay, lay->L.n_tiles, reduce_blocks_per_cu(R)),
                                      st));
    if (rc == FL_OK)
      rc = status_of(flr::launch_seg_finalize(lay->L, a.partials, ws.chunks, ws.seg, seg_sumsq,
                                              ws.total, st));
    flr::StepArgs b = step_args(lay);
    b.s = adam_scalars(h, step);
    b.g_in = g_scratch;
    b.master = master;
    b.m = m;
    b.v = v;
    b.working = working;
    b.clip_total = ws.total;
    b.clip_max = clip_max;
    if (rc == FL_OK) rc = status_of(flr::launch_adamw(b, grid, st));
    return rc;
  }
  if (clip_max > 0.f) {
    a.partials = free_slot(ws, a.carry);
    rc = status_of(flr::launch_sumsq_only(a, grid_for(lay, lay->L.n_tiles,
                                                      sumsq_blocks_per_cu(R)), st));
    if (rc == FL_OK)
      rc = status_of(flr::launch_seg_finalize(lay->L, a.partials, ws.chunks, ws.seg, seg_sumsq,
                                              ws.total, st));
    a.partials = nullptr;
    a.carry = flr::Carry{};
    a.clip_total = ws.total;
    a.clip_max = clip_max;
    seg_sumsq = nullptr;
  }
  a.s = adam_scalars(h, step);
  a.master = master;
  a.m = m;
  a.v = v;
  a.working = working;
  if (seg_sumsq) a.partials = free_slot(ws, a.carry);
  if (rc == FL_OK) rc = status_of(flr::launch_local_step(a, grid, st));
  if (rc == FL_OK && seg_sumsq) rc = finish_sums(lay, ws, a.partials, seg_sumsq, pending, st);
  return rc;
}

bool outer_ok(const fl_outer_hparams* o) {
  return o && finite(o->lr) && finite(o->momentum) && o->lr >= 0.f && o->momentum >= 0.f &&
         o->momentum <= 1.f;
}

int enqueue_fedavg(const fl_layout* lay, int G, const uint16_t* const* reps, const float* wn,
                   float* master, uint16_t* working, hipStream_t st,
                   const fl_outer_hparams* outer = nullptr, float* prev = nullptr,
                   float* buf = nullptr, flr::Carry* pending = nullptr) {
  flr::FedArgs f;
  std::memset(&f, 0, sizeof f);
  take_carry(f, pending);
  if (outer) {
    f.prev = prev;
    f.buf = buf;
    f.eta = outer->lr;
    f.mu = outer->momentum;
    f.nesterov = outer->nesterov ? 1 : 0;
  }
  f.n = lay->L.n;
  f.G = G;
  for (int g = 0; g < G; ++g) {
    f.reps[g] = reps[g];
    f.w[g] = wn[g];
  }
  f.master = master;
  f.working = working;
  return status_of(flr::launch_fedavg(f, fedavg_grid(lay), st));
}

int enqueue_bcast(const fl_layout* lay, const float* recv, float* master, uint16_t* working,
                  hipStream_t st, flr::Carry* pending = nullptr) {
  flr::BcastArgs b;
  std::memset(&b, 0, sizeof b);
  take_carry(b, pending);
  b.n = lay->L.n;
  b.recv = recv;
  b.master = master;
  b.working = working;
  return status_of(flr::launch_bcast_recv(b, fedavg_grid(lay), st));
}

}  // namespace

extern "C" {

const char* fl_status_string(int status) {
  switch (status) {
    case FL_OK: return "FL_OK";
    case FL_ERR_INVALID: return "FL_ERR_INVALID: invalid argument";
    case FL_ERR_ALIGN: return "FL_ERR_ALIGN: device pointer not 16-byte aligned";
    case FL_ERR_LAYOUT: return "FL_ERR_LAYOUT: replica layout fingerprint mismatch";
    case FL_ERR_DEVICE: return "FL_ERR_DEVICE: current device is not the layout's device";
    case FL_ERR_HIP: return "FL_ERR_HIP: HIP runtime or launch failure";
    case FL_ERR_NOMEM: return "FL_ERR_NOMEM: allocation failed";
    case FL_ERR_SCRATCH:
      return "FL_ERR_SCRATCH: the layout's per-segment workspace exceeds fl_round_noalloc's "
             "static scratch";
    default: return "unknown fl_status";
  }
}

int fl_version(void) { return (1 << 16) | 7; }

float fl_lr_cosine(int64_t t, int64_t total_steps, int64_t warmup_steps, float lr_max,
                   float lr_min) {
  const double s = (double)(t - 1);
  const double w = (double)warmup_steps;
  double f;
  if (s < w) {
    f = s / std::max(1.0, w);
  } else {
    const double q = (s - w) / std::max(1.0, (double)(total_steps - warmup_steps));
    const double rho = (double)lr_min / (double)lr_max;
    f = 0.5 * (1.0 + std::cos(M_PI * q));
    f = f * (1.0 - rho) + rho;
    f = std::max(0.0, f);
  }
  return (float)((double)lr_max * f);
}

int fl_set_blocks_per_cu(int blocks_per_cu) {
  return g_blocks_per_cu.exchange(blocks_per_cu > 0 ? blocks_per_cu : 0);
}

uint64_t fl_fingerprint(int64_t n, int64_t n_seg, const int64_t* seg_offsets,
                        const uint8_t* seg_decay) {
  if (!layout_args_ok(n, n_seg, seg_offsets)) return 0;
  return fingerprint_of(n, n_seg, seg_offsets, seg_decay);
}

int fl_layout_create(int64_t n, int64_t n_seg, const int64_t* seg_offsets,
                     const uint8_t* seg_decay, fl_layout** out) {
  if (!out) return FL_ERR_INVALID;
  *out = nullptr;
  if (!layout_args_ok(n, n_seg, seg_offsets)) return FL_ERR_INVALID;
  const int64_t n_tiles = (n + kTile - 1) / kTile;
  if (n_tiles > (int64_t)INT32_MAX / 2) return FL_ERR_INVALID;

  // Per-tile segment tables.
  std::vector<flr::TileInfo> tiles((size_t)n_tiles);
  std::vector<int64_t> seg_piece0((size_t)n_seg + 1, 0);
  int64_t s = 0;
  int64_t pieces = 0;
  for (int64_t t = 0; t < n_tiles; ++t) {
    const int64_t lo = t * kTile;
    const int64_t hi = (lo + kTile < n ? lo + kTile : n) - 1;
    while (seg_offsets[s + 1] <= lo) ++s;
    int64_t s1 = s;
    while (seg_offsets[s1 + 1] <= hi) ++s1;
    flr::TileInfo ti;
    ti.seg0 = (int32_t)s;
    ti.nseg = (int32_t)(s1 - s + 1);
    if (pieces > (int64_t)INT32_MAX - ti.nseg) return FL_ERR_INVALID;
    ti.piece0 = (int32_t)pieces;
    ti.decay = (ti.nseg == 1 && (seg_decay == nullptr || seg_decay[s] != 0)) ? 1 : 0;
    tiles[(size_t)t] = ti;
    for (int64_t k = s; k <= s1; ++k)
      if (seg_offsets[k] >= lo) seg_piece0[(size_t)k] = pieces + (k - s);
    pieces += ti.nseg;
  }
  seg_piece0[(size_t)n_seg] = pieces;
  // Finalize chunks: each segment's pieces in runs of at most kChunkPieces.
  std::vector<int64_t> chunk_p0;
  std::vector<int64_t> seg_chunk0((size_t)n_seg + 1, 0);
  for (int64_t k = 0; k < n_seg; ++k) {
    seg_chunk0[(size_t)k] = (int64_t)chunk_p0.size();
    for (int64_t p = seg_piece0[(size_t)k]; p < seg_piece0[(size_t)k + 1]; p += flr::kChunkPieces)
      chunk_p0.push_back(p);
  }
  const int64_t n_chunks = (int64_t)chunk_p0.size();
  seg_chunk0[(size_t)n_seg] = n_chunks;
  chunk_p0.push_back(pieces);
  std::vector<uint8_t> decay((size_t)n_seg);
  for (int64_t k = 0; k < n_seg; ++k) decay[(size_t)k] = (seg_decay == nullptr || seg_decay[k]) ? 1 : 0;

  fl_layout* lay = new (std::nothrow) fl_layout();
  if (!lay) return FL_ERR_NOMEM;
  if (hipGetDevice(&lay->device) != hipSuccess) {
    delete lay;
    return FL_ERR_HIP;
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, lay->device) !=
          hipSuccess || cus < 1) {
    delete lay;
    return FL_ERR_HIP;
  }
  lay->num_cus = cus;
  lay->fingerprint = fingerprint_of(n, n_seg, seg_offsets, seg_decay);
  lay->L.n = n;
  lay->L.n_seg = n_seg;
  lay->L.n_tiles = n_tiles;
  lay->L.n_pieces = pieces;
  lay->L.n_chunks = n_chunks;

  // One device allocation:
  // [seg_off | seg_piece0 | seg_chunk0 | chunk_p0 | tiles | seg_decay | workspace].
  const size_t b_off = sizeof(int64_t) * (size_t)(n_seg + 1);
  const size_t b_pp = sizeof(int64_t) * (size_t)(n_seg + 1);
  const size_t b_sc = sizeof(int64_t) * (size_t)(n_seg + 1);
  const size_t b_cp = sizeof(int64_t) * (size_t)(n_chunks + 1);
  const size_t b_tiles = sizeof(flr::TileInfo) * (size_t)n_tiles;
  const size_t b_dec = (size_t)n_seg;
  const size_t b_tables = (b_off + b_pp + b_sc + b_cp + b_tiles + b_dec + 255) & ~(size_t)255;
  const size_t b_ws = n > 0 ? ws_bytes(lay->L) : 0;
  const size_t total = b_tables + b_ws + 64;
  void* mem = nullptr;
  hipError_t e = hipMalloc(&mem, total);
  if (e != hipSuccess) {
    delete lay;
    return status_of(e);
  }
  if (b_ws) {
    e = hipMemset(static_cast<char*>(mem) + b_tables, 0, b_ws);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&lay->ws_done, hipEventDisableTiming);
    if (e != hipSuccess) {
      (void)hipFree(mem);
      delete lay;
      return status_of(e);
    }
    lay->ws_mem = static_cast<char*>(mem) + b_tables;
  }
  char* base = static_cast<char*>(mem);
  char* p_off = base;
  char* p_pp = p_off + b_off;
  char* p_sc = p_pp + b_pp;
  char* p_cp = p_sc + b_sc;
  char* p_tiles = p_cp + b_cp;
  char* p_dec = p_tiles + b_tiles;
  e = hipMemcpy(p_off, seg_offsets, b_off, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(p_pp, seg_piece0.data(), b_pp, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(p_sc, seg_chunk0.data(), b_sc, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(p_cp, chunk_p0.data(), b_cp, hipMemcpyHostToDevice);
  if (e == hipSuccess && b_tiles) e = hipMemcpy(p_tiles, tiles.data(), b_tiles, hipMemcpyHostToDevice);
  if (e == hipSuccess && b_dec) e = hipMemcpy(p_dec, decay.data(), b_dec, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    if (lay->ws_done) (void)hipEventDestroy(lay->ws_done);
    (void)hipFree(mem);
    delete lay;
    return status_of(e);
  }
  lay->dev_mem = mem;
  // set-up of fl_round_noalloc's static scratch on this device (once per
  // device; a failure here only disables fl_round_noalloc's workspace)
  if (flr::noalloc_scratch(lay->device, &lay->noalloc) != hipSuccess) {
    (void)hipGetLastError();
    lay->noalloc = nullptr;
  }
  lay->L.seg_off = reinterpret_cast<const int64_t*>(p_off);
  lay->L.seg_piece0 = reinterpret_cast<const int64_t*>(p_pp);
  lay->L.seg_chunk0 = reinterpret_cast<const int64_t*>(p_sc);
  lay->L.chunk_p0 = reinterpret_cast<const int64_t*>(p_cp);
  lay->L.tiles = reinterpret_cast<const flr::TileInfo*>(p_tiles);
  lay->L.seg_decay = reinterpret_cast<const uint8_t*>(p_dec);
  *out = lay;
  return FL_OK;
}

int fl_layout_destroy(fl_layout* layout) {
  if (!layout) return FL_OK;
  int rc = FL_OK;
  if (layout->dev_mem) {
    int cur = -1;
    (void)hipGetDevice(&cur);
    if (cur != layout->device) (void)hipSetDevice(layout->device);
    if (layout->ws_done && hipEventDestroy(layout->ws_done) != hipSuccess) rc = FL_ERR_HIP;
    if (hipFree(layout->dev_mem) != hipSuccess) rc = FL_ERR_HIP;
    if (cur >= 0 && cur != layout->device) (void)hipSetDevice(cur);
  }
  delete layout;
  return rc;
}

int64_t fl_layout_numel(const fl_layout* layout) { return layout ? layout->L.n : -1; }

int64_t fl_layout_num_segments(const fl_layout* layout) { return layout ? layout->L.n_seg : -1; }

uint64_t fl_layout_fingerprint(const fl_layout* layout) {
  return layout ? layout->fingerprint : 0;
}

int fl_shard_reduce(const fl_layout* layout, int R, const uint16_t* const* peer_grads,
                    float grad_scale, float* grad_out, float* seg_sumsq, void* stream) {
  if (!layout) return FL_ERR_INVALID;
  const int64_t n = layout->L.n;
  int rc = check_peers(R, peer_grads, n);
  if (rc != FL_OK) return rc;
  if (!finite(grad_scale)) return FL_ERR_INVALID;
  if ((rc = dev_ptr(grad_out, n)) != FL_OK) return rc;
  if (seg_sumsq && (reinterpret_cast<uintptr_t>(seg_sumsq) & 3u)) return FL_ERR_ALIGN;
  if ((rc = check_device(layout)) != FL_OK) return rc;
  if (n == 0) return FL_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  Workspace ws;
  if (seg_sumsq && (rc = ws.acquire(layout, st)) != FL_OK) return rc;
  flr::StepArgs a = step_args(layout);
  for (int r = 0; r < R; ++r) a.grads[r] = peer_grads[r];
  a.R = R;
  a.grad_scale = grad_scale;
  a.g_out = grad_out;
  a.partials = ws.p;
  rc = status_of(flr::launch_reduce(a, grid_for(layout, layout->L.n_tiles,
                                                reduce_blocks_per_cu(R)), st));
  if (rc == FL_OK && seg_sumsq)
    rc = status_of(flr::launch_seg_finalize(layout->L, ws.p, ws.chunks, ws.seg, seg_sumsq,
                                            nullptr, st));
  const int rc2 = ws.release();
  return rc != FL_OK ? rc : rc2;
}

int fl_adamw_step(const fl_layout* layout, const fl_adamw_hparams* h, int64_t step,
                  const float* grad, float* master, float* m, float* v, uint16_t* working,
                  void* stream) {
  if (!layout || !hparams_ok(h) || step < 1) return FL_ERR_INVALID;
  const int64_t n = layout->L.n;
  int rc;
  if ((rc = dev_ptr(grad, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(master, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(m, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(v, n)) != FL_OK) return rc;
  if (working && (rc = dev_ptr(working, n)) != FL_OK) return rc;
  if (n > 0 && (master == m || master == v || m == v)) return FL_ERR_INVALID;
  if ((rc = check_device(layout)) != FL_OK) return rc;
  if (n == 0) return FL_OK;
  flr::StepArgs a = step_args(layout);
  a.s = adam_scalars(*h, step);
  a.g_in = grad;
  a.master = master;
  a.m = m;
  a.v = v;
  a.working = working;
  return status_of(flr::launch_adamw(a, grid_for(layout, layout->L.n_tiles),
                                     static_cast<hipStream_t>(stream)));
}

int fl_local_step(const fl_layout* layout, const fl_adamw_hparams* h, int64_t step, int R,
                  const uint16_t* const* peer_grads, float grad_scale, float* master, float* m,
                  float* v, uint16_t* working, float* seg_sumsq, void* stream) {
  if (!layout || !hparams_ok(h) || step < 1 || !finite(grad_scale)) return FL_ERR_INVALID;
  const int64_t n = layout->L.n;
  int rc = check_peers(R, peer_grads, n);
  if (rc != FL_OK) return rc;
  if ((rc = dev_ptr(master, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(m, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(v, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(working, n)) != FL_OK) return rc;
  if (n > 0 && (master == m || master == v || m == v)) return FL_ERR_INVALID;
  if (seg_sumsq && (reinterpret_cast<uintptr_t>(seg_sumsq) & 3u)) return FL_ERR_ALIGN;
  if ((rc = check_device(layout)) != FL_OK) return rc;
  if (n == 0) return FL_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  Workspace ws;
  if (seg_sumsq && (rc = ws.acquire(layout, st)) != FL_OK) return rc;
  rc = enqueue_local_step(layout, *h, step, R, peer_grads, grad_scale, master, m, v, working, ws,
                          seg_sumsq, st);
  const int rc2 = ws.release();
  return rc != FL_OK ? rc : rc2;
}

int fl_fedavg(const fl_layout* layout, int G, const uint16_t* const* replicas,
              const float* weights, const uint64_t* replica_fp, float* master_out,
              uint16_t* working_out, void* stream) {
  if (!layout || G < 1 || G > FL_MAX_GROUPS || !replicas) return FL_ERR_INVALID;
  const int64_t n = layout->L.n;
  float wn[FL_MAX_GROUPS];
  int rc = normalise_weights(G, weights, wn);
  if (rc != FL_OK) return rc;
  for (int g = 0; g < G; ++g)
    if ((rc = dev_ptr(replicas[g], n)) != FL_OK) return rc;
  if ((rc = dev_ptr(master_out, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(working_out, n)) != FL_OK) return rc;
  if (replica_fp)
    for (int g = 0; g < G; ++g)
      if (replica_fp[g] != layout->fingerprint) return FL_ERR_LAYOUT;
  if ((rc = check_device(layout)) != FL_OK) return rc;
  if (n == 0) return FL_OK;
  return enqueue_fedavg(layout, G, replicas, wn, master_out, working_out,
                        static_cast<hipStream_t>(stream));
}

int fl_grad_sumsq(const fl_layout* layout, int R, const uint16_t* const* peer_grads,
                  float grad_scale, double* total_sumsq, float* seg_sumsq, void* stream) {
  if (!layout || !total_sumsq) return FL_ERR_INVALID;
  const int64_t n = layout->L.n;
  int rc = check_peers(R, peer_grads, n);
  if (rc != FL_OK) return rc;
  if (!finite(grad_scale)) return FL_ERR_INVALID;
  if (reinterpret_cast<uintptr_t>(total_sumsq) & 7u) return FL_ERR_ALIGN;
  if (seg_sumsq && (reinterpret_cast<uintptr_t>(seg_sumsq) & 3u)) return FL_ERR_ALIGN;
  if ((rc = check_device(layout)) != FL_OK) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (n == 0) return status_of(flr::launch_zero_total(total_sumsq, st));
  Workspace ws;
  if ((rc = ws.acquire(layout, st)) != FL_OK) return rc;
  flr::StepArgs a = step_args(layout);
  for (int r = 0; r < R; ++r) a.grads[r] = peer_grads[r];
  a.R = R;
  a.grad_scale = grad_scale;
  a.partials = ws.p;
  rc = status_of(flr::launch_sumsq_only(a, grid_for(layout, layout->L.n_tiles,
                                                    sumsq_blocks_per_cu(R)), st));
  if (rc == FL_OK)
    rc = status_of(flr::launch_seg_finalize(layout->L, ws.p, ws.chunks, ws.seg, seg_sumsq,
                                            total_sumsq, st));
  const int rc2 = ws.release();
  return rc != FL_OK ? rc : rc2;
}

int fl_local_step_clipped(const fl_layout* layout, const fl_adamw_hparams* h, int64_t step, int R,
                          const uint16_t* const* peer_grads, float grad_scale,
                          const double* total_sumsq, float max_norm, float* master, float* m,
                          float* v, uint16_t* working, void* stream) {
  if (!layout || !hparams_ok(h) || step < 1 || !finite(grad_scale) || !total_sumsq ||
      !finite(max_norm) || !(max_norm > 0.f))
    return FL_ERR_INVALID;
  const int64_t n = layout->L.n;
  int rc = check_peers(R, peer_grads, n);
  if (rc != FL_OK) return rc;
  if ((rc = dev_ptr(master, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(m, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(v, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(working, n)) != FL_OK) return rc;
  if (reinterpret_cast<uintptr_t>(total_sumsq) & 7u) return FL_ERR_ALIGN;
  if (n > 0 && (master == m || master == v || m == v)) return FL_ERR_INVALID;
  if ((rc = check_device(layout)) != FL_OK) return rc;
  if (n == 0) return FL_OK;
  flr::StepArgs a = step_args(layout);
  for (int r = 0; r < R; ++r) a.grads[r] = peer_grads[r];
  a.R = R;
  a.grad_scale = grad_scale;
  a.s = adam_scalars(*h, step);
  a.master = master;
  a.m = m;
  a.v = v;
  a.working = working;
  a.clip_total = total_sumsq;
  a.clip_max = max_norm;
  return status_of(flr::launch_local_step(a, grid_for(layout, layout->L.n_tiles),
                                          static_cast<hipStream_t>(stream)));
}

int fl_shard_reduce_wire(const fl_layout* layout, int R, const uint16_t* const* peer_grads,
                         float grad_scale, uint16_t* wire_out, void* stream) {
  if (!layout) return FL_ERR_INVALID;
  const int64_t n = layout->L.n;
  int rc = check_peers(R, peer_grads, n);
  if (rc != FL_OK) return rc;
  if (!finite(grad_scale)) return FL_ERR_INVALID;
  if ((rc = dev_ptr(wire_out, n)) != FL_OK) return rc;
  if ((rc = check_device(layout)) != FL_OK) return rc;
  if (n == 0) return FL_OK;
  flr::StepArgs a = step_args(layout);
  for (int r = 0; r < R; ++r) a.grads[r] = peer_grads[r];
  a.R = R;
  a.grad_scale = grad_scale;
  a.wire_out = wire_out;
  return status_of(flr::launch_reduce_wire(a, grid_for(layout, layout->L.n_tiles,
                                                        wire_blocks_per_cu(R)),
                                           static_cast<hipStream_t>(stream)));
}

int fl_broadcast_recv(const fl_layout* layout, const float* recv_master, float* master,
                      uint16_t* working, void* stream) {
  if (!layout) return FL_ERR_INVALID;
  const int64_t n = layout->L.n;
  int rc;
  if ((rc = dev_ptr(recv_master, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(master, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(working, n)) != FL_OK) return rc;
  if ((rc = check_device(layout)) != FL_OK) return rc;
  if (n == 0) return FL_OK;
  return enqueue_bcast(layout, recv_master, master, working, static_cast<hipStream_t>(stream));
}

int fl_round_hsdp(const fl_layout* layout, const fl_round_cfg* cfg, const fl_hsdp_cfg* hc,
                  const uint16_t* const* grads, const uint16_t* const* replica_wires,
                  uint16_t* wire, const uint16_t* const* replicas, const float* bcast_master,
                  float* master, float* m, float* v, uint16_t* working, float* seg_sumsq,
                  void* stream) {
  if (!layout || !cfg || !hc || !grads) return FL_ERR_INVALID;
  const fl_round_cfg& c = *cfg;
  const int64_t n = layout->L.n;
  const bool member = hc->fedavg_member != 0;
  if (c.R < 1 || c.R > FL_MAX_PEERS || c.A < 1 || c.step0 < 1 || !finite(c.grad_scale) ||
      !hparams_ok(&c.h) || !step_lrs_ok(c))
    return FL_ERR_INVALID;
  if (hc->H < 1 || hc->H > FL_MAX_PEERS || hc->replica < 0 || hc->replica >= hc->H ||
      !finite(hc->hsdp_scale))
    return FL_ERR_INVALID;
  if (c.step0 > INT64_MAX - c.A) return FL_ERR_INVALID;
  if ((int64_t)c.A * (c.R > hc->H ? c.R : hc->H) > (int64_t)INT32_MAX) return FL_ERR_INVALID;
  int rc = FL_OK;
  float wn[FL_MAX_GROUPS];
  const uint16_t* reps[FL_MAX_GROUPS];
  if (member) {
    if (c.G < 1 || c.G > FL_MAX_GROUPS || c.self_group < 0 || c.self_group >= c.G || !replicas)
      return FL_ERR_INVALID;
    if ((rc = normalise_weights(c.G, c.weights, wn)) != FL_OK) return rc;
    for (int g = 0; g < c.G; ++g) {
      if (g == c.self_group) {
        reps[g] = working;
        continue;
      }
      if ((rc = dev_ptr(replicas[g], n)) != FL_OK) return rc;
      reps[g] = replicas[g];
    }
    if (c.replica_fp)
      for (int g = 0; g < c.G; ++g)
        if (g != c.self_group && c.replica_fp[g] != layout->fingerprint) return FL_ERR_LAYOUT;
  } else if ((rc = dev_ptr(bcast_master, n)) != FL_OK) {
    return rc;
  }
  for (int64_t k = 0; k < (int64_t)c.A * c.R; ++k)
    if ((rc = dev_ptr(grads[k], n)) != FL_OK) return rc;
  if (hc->H > 1) {
    if (!replica_wires) return FL_ERR_INVALID;
    for (int a = 0; a < c.A; ++a)
      for (int k = 0; k < hc->H; ++k)
        if (k != hc->replica &&
            (rc = dev_ptr(replica_wires[(size_t)a * (size_t)hc->H + (size_t)k], n)) != FL_OK)
          return rc;
    if ((rc = dev_ptr(wire, n)) != FL_OK) return rc;
  }
  if ((rc = dev_ptr(master, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(m, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(v, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(working, n)) != FL_OK) return rc;
  if (n > 0 && (master == m || master == v || m == v)) return FL_ERR_INVALID;
  if (n > 0 && hc->H > 1 && (wire == working)) return FL_ERR_INVALID;
  if (seg_sumsq && (reinterpret_cast<uintptr_t>(seg_sumsq) & 3u)) return FL_ERR_ALIGN;
  // the gradient scratch of a clipped step pays off only for the R-peer
  // reduction, i.e. with one replica
  float* g_scratch = (c.max_grad_norm > 0.f && hc->H == 1) ? c.grad_scratch : nullptr;
  if (g_scratch) {
    if ((rc = dev_ptr(g_scratch, n)) != FL_OK) return rc;
    const void* others[] = {master, m, v, working};
    for (const void* o : others)
      if (n > 0 && o == g_scratch) return FL_ERR_INVALID;
  }
  if ((rc = check_device(layout)) != FL_OK) return rc;

  hipStream_t st = static_cast<hipStream_t>(stream);
  auto record = [&](int k) -> int {
    if (!c.phase_events || !c.phase_events[k]) return FL_OK;
    return status_of(hipEventRecord(static_cast<hipEvent_t>(c.phase_events[k]), st));
  };
  Workspace ws;
  if (n > 0 && (seg_sumsq || c.max_grad_norm > 0.f) && (rc = ws.acquire(layout, st)) != FL_OK)
    return rc;
  flr::Carry pending{};  // a step's finalize, run by the call's next kernel
  for (int a = 0; a < c.A && rc == FL_OK; ++a) {
    rc = record(a);
    if (rc != FL_OK || n == 0) continue;
    float* ss = seg_sumsq ? seg_sumsq + (size_t)a * (size_t)layout->L.n_seg : nullptr;
    const uint16_t* const* ga = grads + (size_t)a * (size_t)c.R;
    if (hc->H == 1) {
      rc = enqueue_local_step(layout, step_hparams(c, a), c.step0 + a, c.R, ga, c.grad_scale,
                              master, m, v, working, ws, ss, st, c.max_grad_norm, g_scratch,
                              &pending);
      continue;
    }
    // tier 1: the sharding group's reduction, in the bf16 wire format
    flr::StepArgs t1 = step_args(layout);
    for (int r = 0; r < c.R; ++r) t1.grads[r] = ga[r];
    t1.R = c.R;
    t1.grad_scale = c.grad_scale;
    t1.wire_out = wire;
    rc = status_of(flr::launch_reduce_wire(
        t1, grid_for(layout, layout->L.n_tiles, wire_blocks_per_cu(c.R)), st));
    // tier 2: the replication group's average of the H wire shards, fused
    // with the optimiser step
    const uint16_t* wires[FL_MAX_PEERS];
    for (int k = 0; k < hc->H; ++k)
      wires[k] = (k == hc->replica) ? wire : replica_wires[(size_t)a * (size_t)hc->H + (size_t)k];
    if (rc == FL_OK)
      rc = enqueue_local_step(layout, step_hparams(c, a), c.step0 + a, hc->H, wires,
                              hc->hsdp_scale, master, m, v, working, ws, ss, st, c.max_grad_norm,
                              nullptr, &pending);
  }
  if (rc == FL_OK) rc = record(c.A);
  if (rc == FL_OK && n > 0) {
    if (member)
      rc = enqueue_fedavg(layout, c.G, reps, wn, master, working, st, nullptr, nullptr, nullptr,
                          &pending);
    else
      rc = enqueue_bcast(layout, bcast_master, master, working, st, &pending);
  }
  if (rc == FL_OK) rc = record(c.A + 1);
  const int rc2 = ws.release();
  return rc != FL_OK ? rc : rc2;
}

int fl_fedopt(const fl_layout* layout, int G, const uint16_t* const* replicas,
              const float* weights, const uint64_t* replica_fp, const fl_outer_hparams* outer,
              float* prev, float* buf, float* master_out, uint16_t* working_out, void* stream) {
  if (!layout || G < 1 || G > FL_MAX_GROUPS || !replicas || !outer_ok(outer))
    return FL_ERR_INVALID;
  const int64_t n = layout->L.n;
  float wn[FL_MAX_GROUPS];
  int rc = normalise_weights(G, weights, wn);
  if (rc != FL_OK) return rc;
  for (int g = 0; g < G; ++g)
    if ((rc = dev_ptr(replicas[g], n)) != FL_OK) return rc;
  if ((rc = dev_ptr(prev, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(buf, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(master_out, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(working_out, n)) != FL_OK) return rc;
  if (n > 0 && (prev == buf || prev == master_out || buf == master_out)) return FL_ERR_INVALID;
  if (replica_fp)
    for (int g = 0; g < G; ++g)
      if (replica_fp[g] != layout->fingerprint) return FL_ERR_LAYOUT;
  if ((rc = check_device(layout)) != FL_OK) return rc;
  if (n == 0) return FL_OK;
  return enqueue_fedavg(layout, G, replicas, wn, master_out, working_out,
                        static_cast<hipStream_t>(stream), outer, prev, buf);
}

// Shared body of fl_round and fl_round_outer (outer == nullptr: FedAvg).
static int round_impl(const fl_layout* layout, const fl_round_cfg* cfg,
                      const fl_outer_hparams* outer, const uint16_t* const* grads,
                      const uint16_t* const* replicas, float* prev, float* buf, float* master,
                      float* m, float* v, uint16_t* working, float* seg_sumsq, void* stream,
                      bool noalloc = false);

int fl_round_outer(const fl_layout* layout, const fl_round_cfg* cfg, const fl_outer_hparams* outer,
                   const uint16_t* const* grads, const uint16_t* const* replicas, float* prev,
                   float* buf, float* master, float* m, float* v, uint16_t* working,
                   float* seg_sumsq, void* stream) {
  if (!outer_ok(outer)) return FL_ERR_INVALID;
  return round_impl(layout, cfg, outer, grads, replicas, prev, buf, master, m, v, working,
                    seg_sumsq, stream);
}

int fl_round(const fl_layout* layout, const fl_round_cfg* cfg, const uint16_t* const* grads,
             const uint16_t* const* replicas, float* master, float* m, float* v,
             uint16_t* working, float* seg_sumsq, void* stream) {
  return round_impl(layout, cfg, nullptr, grads, replicas, nullptr, nullptr, master, m, v,
                    working, seg_sumsq, stream);
}

int fl_round_noalloc(const fl_layout* layout, const fl_round_cfg* cfg,
                     const uint16_t* const* grads, const uint16_t* const* replicas,
                     float* master, float* m, float* v, uint16_t* working, float* seg_sumsq,
                     void* stream) {
  return round_impl(layout, cfg, nullptr, grads, replicas, nullptr, nullptr, master, m, v,
                    working, seg_sumsq, stream, true);
}

size_t fl_noalloc_workspace_bytes(const fl_layout* layout) {
  if (!layout || layout->L.n == 0) return 0;
  return noalloc_bytes(layout->L);
}

static int round_impl(const fl_layout* layout, const fl_round_cfg* cfg,
                      const fl_outer_hparams* outer, const uint16_t* const* grads,
                      const uint16_t* const* replicas, float* prev, float* buf, float* master,
                      float* m, float* v, uint16_t* working, float* seg_sumsq, void* stream,
                      bool noalloc) {
  if (!layout || !cfg || !grads || !replicas) return FL_ERR_INVALID;
  const fl_round_cfg& c = *cfg;
  const int64_t n = layout->L.n;
  if (c.R < 1 || c.R > FL_MAX_PEERS || c.G < 1 || c.G > FL_MAX_GROUPS || c.A < 1 ||
      c.self_group < 0 || c.self_group >= c.G || c.step0 < 1 || !finite(c.grad_scale) ||
      !hparams_ok(&c.h) || !step_lrs_ok(c))
    return FL_ERR_INVALID;
  if (c.step0 > INT64_MAX - c.A) return FL_ERR_INVALID;
  if ((int64_t)c.A * c.R > (int64_t)INT32_MAX) return FL_ERR_INVALID;
  float wn[FL_MAX_GROUPS];
  int rc = normalise_weights(c.G, c.weights, wn);
  if (rc != FL_OK) return rc;
  for (int64_t k = 0; k < (int64_t)c.A * c.R; ++k)
    if ((rc = dev_ptr(grads[k], n)) != FL_OK) return rc;
  const uint16_t* reps[FL_MAX_GROUPS];
  for (int g = 0; g < c.G; ++g) {
    if (g == c.self_group) {
      reps[g] = working;
      continue;
    }
    if ((rc = dev_ptr(replicas[g], n)) != FL_OK) return rc;
    reps[g] = replicas[g];
  }
  if ((rc = dev_ptr(master, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(m, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(v, n)) != FL_OK) return rc;
  if ((rc = dev_ptr(working, n)) != FL_OK) return rc;
  if (n > 0 && (master == m || master == v || m == v)) return FL_ERR_INVALID;
  if (outer) {
    if ((rc = dev_ptr(prev, n)) != FL_OK) return rc;
    if ((rc = dev_ptr(buf, n)) != FL_OK) return rc;
    if (n > 0) {
      const void* state[] = {master, m, v, prev, buf};
      for (int i = 0; i < 5; ++i)
        for (int j = i + 1; j < 5; ++j)
          if (state[i] == state[j]) return FL_ERR_INVALID;
    }
  }
  if (seg_sumsq && (reinterpret_cast<uintptr_t>(seg_sumsq) & 3u)) return FL_ERR_ALIGN;
  float* g_scratch = c.max_grad_norm > 0.f ? c.grad_scratch : nullptr;
  if (g_scratch) {
    if ((rc = dev_ptr(g_scratch, n)) != FL_OK) return rc;
    const void* others[] = {master, m, v, working, prev, buf};
    for (const void* o : others)
      if (n > 0 && o == g_scratch) return FL_ERR_INVALID;
  }
  if (c.replica_fp)
    for (int g = 0; g < c.G; ++g)
      if (g != c.self_group && c.replica_fp[g] != layout->fingerprint) return FL_ERR_LAYOUT;
  if ((rc = check_device(layout)) != FL_OK) return rc;
  const bool needs_ws = n > 0 && (seg_sumsq || c.max_grad_norm > 0.f);
  if (noalloc && needs_ws && noalloc_bytes(layout->L) > flr::kNoallocScratchBytes)
    return FL_ERR_SCRATCH;

  hipStream_t st = static_cast<hipStream_t>(stream);
  auto record = [&](int k) -> int {
    if (!c.phase_events || !c.phase_events[k]) return FL_OK;
    return status_of(hipEventRecord(static_cast<hipEvent_t>(c.phase_events[k]), st));
  };
  Workspace ws;
  if (needs_ws && (rc = noalloc ? ws.use_static(layout, st) : ws.acquire(layout, st)) != FL_OK)
    return rc;
  flr::Carry pending{};  // a step's finalize, run by the call's next kernel
  for (int a = 0; a < c.A && rc == FL_OK; ++a) {
    rc = record(a);
    if (rc == FL_OK && n > 0)
      rc = enqueue_local_step(layout, step_hparams(c, a), c.step0 + a, c.R,
                              grads + (size_t)a * (size_t)c.R, c.grad_scale, master, m, v, working, ws,
                              seg_sumsq ? seg_sumsq + (size_t)a * (size_t)layout->L.n_seg : nullptr,
                              st, c.max_grad_norm, g_scratch, &pending);
  }
  if (rc == FL_OK) rc = record(c.A);
  if (rc == FL_OK && n > 0)
    rc = enqueue_fedavg(layout, c.G, reps, wn, master, working, st, outer, prev, buf, &pending);
  if (rc == FL_OK) rc = record(c.A + 1);
  const int rc2 = ws.release();
  return rc != FL_OK ? rc : rc2;
}

}  // extern "C"
