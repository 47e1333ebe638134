// flround_kernels.hip -- gfx950 kernels of the parameter-sync path.
//
// Every kernel here is a bandwidth-bound stream over the flat shard: an
// element is read once, updated with a few dozen fp32 operations and written
// once, so the kernels are built for HBM, not for the matrix cores:
//   * a workgroup of 256 threads (4 wave64) owns one 2048-element tile per
//     iteration of a grid-stride loop; each thread owns 8 consecutive
//     elements, i.e. one 16-byte load per bf16 stream and two per fp32 stream
//     (global_load_dwordx4), so every wave touches whole 128-byte lines;
//   * all loads of a tile are issued before its arithmetic (memory-level
//     parallelism), with compile-time peer / group counts where common;
//   * sums over peers and replicas run in ascending index order in fp32, one
//     correctly rounded operation at a time (the file is built with
//     -ffp-contract=off), so results are bitwise those of the definition and
//     do not depend on the grid;
//   * per-segment sums of squares use wave64 butterfly reductions only: each
//     lane squares its elements exactly in double, and each wave writes one
//     double partial per (tile, segment) piece it covers, with no workgroup
//     barrier in the streaming loop; a small finalize folds the partials per
//     segment (and, for clipping, over the shard) in fixed trees; only tiles
//     that straddle a segment boundary (rare) resolve segments per element.
#include "flr_internal.h"

#include <mutex>

// Workspace of fl_round_noalloc, for callers that cannot allocate: one array
// per GPU in the code object, held until the process ends.  Host code uses
// only the per-device address that noalloc_scratch() looks up, never this
// name (which on the host side is a stand-in, not a device address).
static __device__ __align__(256) unsigned char scratch[flr::kNoallocScratchBytes];

namespace flr {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef double f64x2 __attribute__((ext_vector_type(2)));

// Cache hints.  ld_once: streams read once per pass (peer gradients, FedAvg
// replicas); ld: the read-modify-write state (master, m, v, fp32 gradient);
// st: every store.
#ifndef FLR_NT_ONCE
#define FLR_NT_ONCE 1
#endif
#ifndef FLR_NT_LOADS
#define FLR_NT_LOADS 0
#endif
#ifndef FLR_NT_STORES
#define FLR_NT_STORES 1
#endif

template <typename T>
__device__ __forceinline__ T ld_once(const T* p) {
#if FLR_NT_ONCE
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

template <typename T>
__device__ __forceinline__ T ld(const T* p) {
#if FLR_NT_LOADS
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

template <typename T>
__device__ __forceinline__ void st(T* p, T v) {
#if FLR_NT_STORES
  __builtin_nontemporal_store(v, p);
#else
  *p = v;
#endif
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16 bits, round to nearest even; NaN -> quiet NaN, sign kept.
__device__ __forceinline__ uint32_t to_bf16(float x) {
  const uint32_t u = __float_as_uint(x);
  const uint32_t r = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
  return ((u & 0x7FFFFFFFu) > 0x7F800000u) ? ((u >> 16) | 0x40u) : r;
}

__device__ __forceinline__ u32x4 pack_bf16x8(const float x[8]) {
  u32x4 o;
  o.x = to_bf16(x[0]) | (to_bf16(x[1]) << 16);
  o.y = to_bf16(x[2]) | (to_bf16(x[3]) << 16);
  o.z = to_bf16(x[4]) | (to_bf16(x[5]) << 16);
  o.w = to_bf16(x[6]) | (to_bf16(x[7]) << 16);
  return o;
}

// acc[e] = acc[e] + bf16 element e of w (ascending e).
__device__ __forceinline__ void add_bf16x8(float acc[8], u32x4 w) {
  acc[0] = acc[0] + bf16_lo(w.x);
  acc[1] = acc[1] + bf16_hi(w.x);
  acc[2] = acc[2] + bf16_lo(w.y);
  acc[3] = acc[3] + bf16_hi(w.y);
  acc[4] = acc[4] + bf16_lo(w.z);
  acc[5] = acc[5] + bf16_hi(w.z);
  acc[6] = acc[6] + bf16_lo(w.w);
  acc[7] = acc[7] + bf16_hi(w.w);
}

// acc[e] = acc[e] + wt * bf16 element e of w.
__device__ __forceinline__ void fma_free_bf16x8(float acc[8], float wt, u32x4 w) {
  acc[0] = acc[0] + (wt * bf16_lo(w.x));
  acc[1] = acc[1] + (wt * bf16_hi(w.x));
  acc[2] = acc[2] + (wt * bf16_lo(w.y));
  acc[3] = acc[3] + (wt * bf16_hi(w.y));
  acc[4] = acc[4] + (wt * bf16_lo(w.z));
  acc[5] = acc[5] + (wt * bf16_hi(w.z));
  acc[6] = acc[6] + (wt * bf16_lo(w.w));
  acc[7] = acc[7] + (wt * bf16_hi(w.w));
}

__device__ __forceinline__ void load_f32x8(const float* p, float x[8]) {
  const f32x4 a = ld(reinterpret_cast<const f32x4*>(p));
  const f32x4 b = ld(reinterpret_cast<const f32x4*>(p + 4));
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

__device__ __forceinline__ void store_f32x8(float* p, const float x[8]) {
  st(reinterpret_cast<f32x4*>(p), f32x4{x[0], x[1], x[2], x[3]});
  st(reinterpret_cast<f32x4*>(p + 4), f32x4{x[4], x[5], x[6], x[7]});
}

// Reduced gradient of 8 elements (full vector): peers in ascending order.
template <int RT>
__device__ __forceinline__ void reduce_vec(const StepArgs& a, int64_t base, float g[8]) {
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if constexpr (RT > 0) {
    u32x4 w[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r) w[r] = ld_once(reinterpret_cast<const u32x4*>(a.grads[r] + base));
#pragma unroll
    for (int r = 0; r < RT; ++r) add_bf16x8(acc, w[r]);
  } else {
    constexpr int kChunk = 4;
    for (int r0 = 0; r0 < a.R; r0 += kChunk) {
      u32x4 w[kChunk];
#pragma unroll
      for (int k = 0; k < kChunk; ++k)
        if (r0 + k < a.R) w[k] = ld_once(reinterpret_cast<const u32x4*>(a.grads[r0 + k] + base));
#pragma unroll
      for (int k = 0; k < kChunk; ++k)
        if (r0 + k < a.R) add_bf16x8(acc, w[k]);
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) g[e] = acc[e] * a.grad_scale;
}

// Same for the last, partial vector: elements base .. base + cnt - 1.
__device__ __forceinline__ void reduce_tail(const StepArgs& a, int64_t base, int cnt,
                                            float g[8]) {
  for (int e = 0; e < 8; ++e) {
    float acc = 0.f;
    if (e < cnt) {
      for (int r = 0; r < a.R; ++r)
        acc = acc + __uint_as_float((uint32_t)a.grads[r][base + e] << 16);
    }
    g[e] = acc * a.grad_scale;
  }
}

// Fixed-tree sum over one wave64: butterfly exchange, after which every lane
// holds the same bits (each step adds the same two partials in both lanes).
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = v + __shfl_xor(v, off, 64);
  return v;
}

// Clip coefficient from the whole-shard sum of squares: min(1, max / (norm +
// 1e-6)) in double, rounded once to float; a NaN norm gives NaN, as torch's
// clamp does.
__device__ __forceinline__ float clip_coef(const double* total, float max_norm) {
  const double c = (double)max_norm / (__builtin_sqrt(*total) + 1e-6);
  return (float)(c >= 1.0 ? 1.0 : c);
}

// Segment of element `i`, searching [lo, hi] (segments overlapping the tile).
__device__ __forceinline__ int find_seg(const int64_t* off, int lo, int hi, int64_t i) {
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (off[mid] <= i) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Fixed-tree total of the (piece, wave) partials of finalize chunk c: thread
// j folds pieces j, j + 256, ... (each piece's kWaves slots in order), a
// wave64 butterfly, then the 4 wave totals in order.  Called by all threads
// of the workgroup; the result is valid in thread 0.  The partials were
// written by an earlier kernel.
__device__ __forceinline__ double chunk_fold(const int64_t* chunk_p0, const double* partials,
                                             int64_t c, double* red) {
  const int64_t p0 = chunk_p0[c];
  const int64_t p1 = chunk_p0[c + 1];
  double acc = 0.0;
  for (int64_t p = p0 + threadIdx.x; p < p1; p += kBlock) {
    const double* q = partials + p * kWaves;
    const f64x2 w0 = *reinterpret_cast<const f64x2*>(q);
    const f64x2 w1 = *reinterpret_cast<const f64x2*>(q + 2);
    acc = acc + w0.x;
    acc = acc + w0.y;
    acc = acc + w1.x;
    acc = acc + w1.y;
  }
  acc = wave_sum(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  const double sum = ((red[0] + red[1]) + red[2]) + red[3];
  __syncthreads();
  return sum;
}

// Fixed-tree total of n_seg per-segment values: thread t adds values t,
// t + 256, ... in order, a wave64 butterfly, then the 4 wave totals in order.
// Called by all threads; the result is valid in thread 0.
template <typename Get>
__device__ __forceinline__ double total_fold(int64_t n_seg, Get get, double* red) {
  double acc = 0.0;
  for (int64_t s = threadIdx.x; s < n_seg; s += kBlock) acc = acc + get(s);
  acc = wave_sum(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  const double sum = ((red[0] + red[1]) + red[2]) + red[3];
  __syncthreads();
  return sum;
}

// A carried finalize (see Carry): the last workgroup of a kernel launched
// with one extra workgroup folds the previous pass's partials, chunk by
// chunk, with the tree of k_seg_chunks, and writes each segment's float sum;
// returns true in that workgroup (which then has nothing else to do).  Every
// workgroup calls it first; the others stream over work units blockIdx.x ..
// in steps of gridDim.x - carried, exactly as without the extra workgroup.
// That keeps the workgroup -> tile mapping, and so the XCD that touches each
// tile, the same in consecutive kernels: at small shard sizes the next pass
// then finds the tile in that XCD's L2.  The partials come from an earlier
// kernel of the same stream, so plain loads see them.
__device__ __forceinline__ bool run_carry(const Carry& c) {
  if (c.partials == nullptr || blockIdx.x != gridDim.x - 1) return false;
  __shared__ double red[4];
  for (int64_t k = 0; k < c.n_chunks; ++k) {
    const double sum = chunk_fold(c.chunk_p0, c.partials, k, red);
    if (threadIdx.x == 0) c.out[k] = (float)sum;
  }
  return true;
}

__device__ __forceinline__ int carried(const Carry& c) { return c.partials != nullptr ? 1 : 0; }

// MODE 0: fused reduce + AdamW + working copy; 1: reduce only (g_out); 2:
// AdamW only (g_in); 3: reduce to the bf16 wire format (wire_out); 4: reduce
// with no output but the sums of squares.  In MODE 0 and 2 the gradient is
// scaled by the clip coefficient when a.clip_total is set.  SUMSQ: per-piece
// sums of squares of g (before clipping).
template <int RT, int MODE, bool SUMSQ>
__global__ void __launch_bounds__(kBlock) k_step(const StepArgs a) {
  const int tid = threadIdx.x;
  const bool clip = (MODE == 0 || MODE == 2) && a.clip_total != nullptr;
  const float coef = clip ? clip_coef(a.clip_total, a.clip_max) : 1.0f;
  if (run_carry(a.carry)) return;
  const int cw = carried(a.carry);
  for (int64_t t = blockIdx.x; t < a.L.n_tiles; t += (int64_t)gridDim.x - cw) {
    const TileInfo ti = a.L.tiles[t];
    const int64_t base = t * kTile + (int64_t)tid * kVec;
    const int64_t left = a.L.n - base;
    const int cnt = left >= kVec ? kVec : (left > 0 ? (int)left : 0);

    // segment of each element (only needed where the tile straddles segments)
    int seg[8];
    if (ti.nseg > 1 && (SUMSQ || MODE == 0 || MODE == 2)) {
      int s = cnt > 0 ? find_seg(a.L.seg_off, ti.seg0, ti.seg0 + ti.nseg - 1, base) : ti.seg0;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (e < cnt)
          while (base + e >= a.L.seg_off[s + 1]) ++s;
        seg[e] = s;
      }
    }

    float g[8];
    float p[8], m[8], v[8];
    if (cnt == kVec) {
      if constexpr (MODE == 0 || MODE == 2) {
        load_f32x8(a.master + base, p);
        load_f32x8(a.m + base, m);
        load_f32x8(a.v + base, v);
      }
      if constexpr (MODE == 2) load_f32x8(a.g_in + base, g);
      else reduce_vec<RT>(a, base, g);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[e] = 0.f; m[e] = 0.f; v[e] = 0.f; g[e] = 0.f;
        if constexpr (MODE == 0 || MODE == 2) {
          if (e < cnt) { p[e] = a.master[base + e]; m[e] = a.m[base + e]; v[e] = a.v[base + e]; }
        }
        if constexpr (MODE == 2) {
          if (e < cnt) g[e] = a.g_in[base + e];
        }
      }
      if constexpr (MODE != 2) {
        if (cnt > 0) reduce_tail(a, base, cnt, g);
      }
    }

    if constexpr (MODE == 4) {
      // sums of squares only
    } else if constexpr (MODE == 1) {
      if (cnt == kVec) {
        store_f32x8(a.g_out + base, g);
      } else {
        for (int e = 0; e < cnt; ++e) a.g_out[base + e] = g[e];
      }
    } else if constexpr (MODE == 3) {
      if (cnt == kVec) {
        st(reinterpret_cast<u32x4*>(a.wire_out + base), pack_bf16x8(g));
      } else {
        for (int e = 0; e < cnt; ++e) a.wire_out[base + e] = (uint16_t)to_bf16(g[e]);
      }
    } else {
      const AdamScalars& s = a.s;
      float gc[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) gc[e] = clip ? g[e] * coef : g[e];
      float d[8];
      if (ti.nseg == 1) {
        const float du = ti.decay ? s.decay : 1.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) d[e] = du;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) d[e] = a.L.seg_decay[seg[e]] ? s.decay : 1.0f;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float pe = p[e] * d[e];
        const float mn = (s.b1 * m[e]) + (s.omb1 * gc[e]);
        const float vn = (s.b2 * v[e]) + (s.omb2 * (gc[e] * gc[e]));
        const float den = (__builtin_sqrtf(vn) / s.bc2_sqrt) + s.eps;
        pe = pe - (s.step_size * (mn / den));
        p[e] = pe; m[e] = mn; v[e] = vn;
      }
      if (cnt == kVec) {
        store_f32x8(a.master + base, p);
        store_f32x8(a.m + base, m);
        store_f32x8(a.v + base, v);
        if (MODE == 0 || a.working) st(reinterpret_cast<u32x4*>(a.working + base), pack_bf16x8(p));
      } else {
        for (int e = 0; e < cnt; ++e) {
          a.master[base + e] = p[e];
          a.m[base + e] = m[e];
          a.v[base + e] = v[e];
          if (MODE == 0 || a.working) a.working[base + e] = (uint16_t)to_bf16(p[e]);
        }
      }
    }

    if constexpr (SUMSQ) {
      // One partial per (piece, wave): the wave's share of the piece, the
      // exact double squares of its 8 elements per lane summed in order, then
      // the wave butterfly; no barrier.
      const int wid = tid >> 6;
      if (ti.nseg == 1) {
        double acc = 0.0;
#pragma unroll
        for (int e = 0; e < 8; ++e) if (e < cnt) acc = acc + (double)g[e] * (double)g[e];
        const double tot = wave_sum(acc);
        if ((tid & 63) == 0) a.partials[(int64_t)ti.piece0 * kWaves + wid] = tot;
      } else {
        for (int j = 0; j < ti.nseg; ++j) {
          const int sj = ti.seg0 + j;
          double acc = 0.0;
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (e < cnt && seg[e] == sj) acc = acc + (double)g[e] * (double)g[e];
          const double tot = wave_sum(acc);
          if ((tid & 63) == 0) a.partials[((int64_t)ti.piece0 + j) * kWaves + wid] = tot;
        }
      }
    }
  }
}

// Reduction to the bf16 wire format with compile-time R (MODE 3 of k_step
// for other R).  It needs no segment data, so it strides over 8-element
// vectors and takes two per thread per iteration, issuing all 2R loads before
// the arithmetic of either: a read-mostly pass needs that many loads in
// flight to cover HBM latency at one workgroup per CU.  Same arithmetic and
// bits as MODE 3.
template <int RT>
__global__ void __launch_bounds__(kBlock) k_wire(const StepArgs a) {
  if (run_carry(a.carry)) return;
  const int cw = carried(a.carry);
  const int64_t nvec = (a.L.n + kVec - 1) / kVec;
  const int64_t stride = ((int64_t)gridDim.x - cw) * kBlock;
  for (int64_t v0 = (int64_t)blockIdx.x * kBlock + threadIdx.x; v0 < nvec; v0 += 2 * stride) {
    const int64_t v1 = v0 + stride;
    const int64_t b0 = v0 * kVec, b1 = v1 * kVec;
    if (b1 + kVec <= a.L.n) {  // both vectors full (b0 < b1)
      u32x4 w0[RT], w1[RT];
#pragma unroll
      for (int r = 0; r < RT; ++r) w0[r] = ld_once(reinterpret_cast<const u32x4*>(a.grads[r] + b0));
#pragma unroll
      for (int r = 0; r < RT; ++r) w1[r] = ld_once(reinterpret_cast<const u32x4*>(a.grads[r] + b1));
      float g0[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      float g1[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int r = 0; r < RT; ++r) add_bf16x8(g0, w0[r]);
#pragma unroll
      for (int r = 0; r < RT; ++r) add_bf16x8(g1, w1[r]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        g0[e] = g0[e] * a.grad_scale;
        g1[e] = g1[e] * a.grad_scale;
      }
      st(reinterpret_cast<u32x4*>(a.wire_out + b0), pack_bf16x8(g0));
      st(reinterpret_cast<u32x4*>(a.wire_out + b1), pack_bf16x8(g1));
      continue;
    }
    for (int k = 0; k < 2; ++k) {  // the last vectors of the shard
      const int64_t vi = k == 0 ? v0 : v1;
      if (vi >= nvec) break;
      const int64_t base = vi * kVec;
      const int64_t left = a.L.n - base;
      float g[8];
      if (left >= kVec) {
        reduce_vec<RT>(a, base, g);
        st(reinterpret_cast<u32x4*>(a.wire_out + base), pack_bf16x8(g));
      } else {
        reduce_tail(a, base, (int)left, g);
        for (int e = 0; e < (int)left; ++e) a.wire_out[base + e] = (uint16_t)to_bf16(g[e]);
      }
    }
  }
}

// FedAvg: master = sum_g w_g * f32(rep_g), ascending g; working = bf16(master).
// OUTER: the outer optimiser step on that average instead:
//   delta = prev - xbar; buf = mu * buf + delta;
//   d = nesterov ? delta + mu * buf : buf; p = prev - eta * d;
//   master = prev = p; working = bf16(p).
template <int GT, bool OUTER>
__global__ void __launch_bounds__(kBlock) k_fedavg(const FedArgs a) {
  if (run_carry(a.carry)) return;
  const int cw = carried(a.carry);
  const int64_t nvec = (a.n + kVec - 1) / kVec;
  const int64_t stride = ((int64_t)gridDim.x - cw) * kBlock;
  for (int64_t vi = (int64_t)blockIdx.x * kBlock + threadIdx.x; vi < nvec; vi += stride) {
    const int64_t base = vi * kVec;
    const int64_t left = a.n - base;
    const int cnt = left >= kVec ? kVec : (int)left;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    float prev[8], buf[8];
    if (cnt == kVec) {
      if constexpr (OUTER) {
        load_f32x8(a.prev + base, prev);
        load_f32x8(a.buf + base, buf);
      }
      if constexpr (GT > 0) {
        u32x4 w[GT];
#pragma unroll
        for (int k = 0; k < GT; ++k) w[k] = ld_once(reinterpret_cast<const u32x4*>(a.reps[k] + base));
#pragma unroll
        for (int k = 0; k < GT; ++k) fma_free_bf16x8(acc, a.w[k], w[k]);
      } else {
        constexpr int kChunk = 4;
        for (int k0 = 0; k0 < a.G; k0 += kChunk) {
          u32x4 w[kChunk];
#pragma unroll
          for (int k = 0; k < kChunk; ++k)
            if (k0 + k < a.G) w[k] = ld_once(reinterpret_cast<const u32x4*>(a.reps[k0 + k] + base));
#pragma unroll
          for (int k = 0; k < kChunk; ++k)
            if (k0 + k < a.G) fma_free_bf16x8(acc, a.w[k0 + k], w[k]);
        }
      }
    } else {
      for (int e = 0; e < cnt; ++e) {
        float s = 0.f;
        for (int k = 0; k < a.G; ++k)
          s = s + (a.w[k] * __uint_as_float((uint32_t)a.reps[k][base + e] << 16));
        acc[e] = s;
        if constexpr (OUTER) {
          prev[e] = a.prev[base + e];
          buf[e] = a.buf[base + e];
        }
      }
    }
    if constexpr (OUTER) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (e < cnt) {
          const float delta = prev[e] - acc[e];
          const float b = (a.mu * buf[e]) + delta;
          const float d = a.nesterov ? (delta + (a.mu * b)) : b;
          acc[e] = prev[e] - (a.eta * d);
          buf[e] = b;
        }
      }
    }
    if (cnt == kVec) {
      store_f32x8(a.master + base, acc);
      st(reinterpret_cast<u32x4*>(a.working + base), pack_bf16x8(acc));
      if constexpr (OUTER) {
        store_f32x8(a.prev + base, acc);
        store_f32x8(a.buf + base, buf);
      }
    } else {
      for (int e = 0; e < cnt; ++e) {
        a.master[base + e] = acc[e];
        a.working[base + e] = (uint16_t)to_bf16(acc[e]);
        if constexpr (OUTER) {
          a.prev[base + e] = acc[e];
          a.buf[base + e] = buf[e];
        }
      }
    }
  }
}

// Per-segment totals of the (piece, wave) partials, in double, in fixed
// trees that do not depend on the grid.  Stage 1: one workgroup per chunk of
// up to kChunkPieces pieces of one segment; thread j folds pieces j, j+256,
// ... (each piece's kWaves slots in order), then a wave64 butterfly and the 4
// wave totals in order.  Stage 2: one thread per segment adds its chunks in
// order (double per segment, and its float rounding if requested); skipped
// when every segment is one chunk.  Stage 3 (whole-shard total, for
// clipping): one workgroup folds the segments.
// DIRECT (every segment is a single chunk, so chunk c is segment c): the
// chunk sum is the segment's total; write it, and its float rounding if
// requested, in place of stage 2 (which would add it to 0.0: the same bits).
template <bool DIRECT>
__global__ void __launch_bounds__(kBlock) k_seg_chunks(const LayoutDev L, const double* partials,
                                                       double* chunk_sums, float* out) {
  __shared__ double red[4];
  for (int64_t c = blockIdx.x; c < L.n_chunks; c += gridDim.x) {
    const double sum = chunk_fold(L.chunk_p0, partials, c, red);
    if (threadIdx.x == 0) {
      chunk_sums[c] = sum;
      if (DIRECT && out) out[c] = (float)sum;
    }
  }
}

__global__ void __launch_bounds__(kBlock) k_seg_totals(const LayoutDev L, const double* chunk_sums,
                                                       double* seg_dbl, float* out) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t s = (int64_t)blockIdx.x * kBlock + threadIdx.x; s < L.n_seg; s += stride) {
    double acc = 0.0;
    for (int64_t c = L.seg_chunk0[s]; c < L.seg_chunk0[s + 1]; ++c) acc = acc + chunk_sums[c];
    seg_dbl[s] = acc;
    if (out) out[s] = (float)acc;
  }
}

__global__ void __launch_bounds__(kBlock) k_total(const int64_t n_seg, const double* seg_dbl,
                                                  double* total) {
  __shared__ double red[4];
  const double tot = total_fold(n_seg, [&](int64_t s) { return seg_dbl[s]; }, red);
  if (threadIdx.x == 0) *total = tot;
}

// Broadcast receive: master = recv; working = bf16(recv).
__global__ void __launch_bounds__(kBlock) k_bcast_recv(const BcastArgs a) {
  if (run_carry(a.carry)) return;
  const int cw = carried(a.carry);
  const int64_t n = a.n;
  const int64_t nvec = (n + kVec - 1) / kVec;
  const int64_t stride = ((int64_t)gridDim.x - cw) * kBlock;
  for (int64_t vi = (int64_t)blockIdx.x * kBlock + threadIdx.x; vi < nvec; vi += stride) {
    const int64_t base = vi * kVec;
    const int64_t left = n - base;
    if (left >= kVec) {
      float x[8];
      const f32x4 u = ld_once(reinterpret_cast<const f32x4*>(a.recv + base));
      const f32x4 w = ld_once(reinterpret_cast<const f32x4*>(a.recv + base + 4));
      x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
      x[4] = w.x; x[5] = w.y; x[6] = w.z; x[7] = w.w;
      store_f32x8(a.master + base, x);
      st(reinterpret_cast<u32x4*>(a.working + base), pack_bf16x8(x));
    } else {
      for (int e = 0; e < (int)left; ++e) {
        const float x = a.recv[base + e];
        a.master[base + e] = x;
        a.working[base + e] = (uint16_t)to_bf16(x);
      }
    }
  }
}

// grid workgroups for the stream, plus one for a carried finalize.
template <typename Args>
hipError_t launch(const void* fn, const Args& a, int grid, hipStream_t st) {
  void* args[] = {const_cast<Args*>(&a)};
  const unsigned g = (unsigned)grid + (a.carry.partials != nullptr ? 1u : 0u);
  return hipLaunchKernel(fn, dim3(g), dim3(kBlock), args, 0, st);
}

template <int MODE, bool SUMSQ>
hipError_t dispatch_step(const StepArgs& a, int grid, hipStream_t st) {
  switch (a.R) {
    case 1: return launch((const void*)k_step<1, MODE, SUMSQ>, a, grid, st);
    case 2: return launch((const void*)k_step<2, MODE, SUMSQ>, a, grid, st);
    case 4: return launch((const void*)k_step<4, MODE, SUMSQ>, a, grid, st);
    case 8: return launch((const void*)k_step<8, MODE, SUMSQ>, a, grid, st);
    case 16: return launch((const void*)k_step<16, MODE, SUMSQ>, a, grid, st);
    default: return launch((const void*)k_step<0, MODE, SUMSQ>, a, grid, st);
  }
}

}  // namespace

hipError_t launch_local_step(const StepArgs& a, int grid, hipStream_t st) {
  return a.partials ? dispatch_step<0, true>(a, grid, st) : dispatch_step<0, false>(a, grid, st);
}

hipError_t launch_reduce(const StepArgs& a, int grid, hipStream_t st) {
  return a.partials ? dispatch_step<1, true>(a, grid, st) : dispatch_step<1, false>(a, grid, st);
}

hipError_t launch_reduce_wire(const StepArgs& a, int grid, hipStream_t st) {
  switch (a.R) {
    case 1: return launch((const void*)k_wire<1>, a, grid, st);
    case 2: return launch((const void*)k_wire<2>, a, grid, st);
    case 4: return launch((const void*)k_wire<4>, a, grid, st);
    case 8: return launch((const void*)k_wire<8>, a, grid, st);
    case 16: return launch((const void*)k_wire<16>, a, grid, st);
    default: return dispatch_step<3, false>(a, grid, st);
  }
}

hipError_t launch_bcast_recv(const BcastArgs& a, int grid, hipStream_t st) {
  return launch((const void*)k_bcast_recv, a, grid, st);
}

hipError_t launch_adamw(const StepArgs& a, int grid, hipStream_t st) {
  return launch((const void*)k_step<1, 2, false>, a, grid, st);
}

template <bool OUTER>
hipError_t dispatch_fedavg(const FedArgs& a, int grid, hipStream_t st) {
  switch (a.G) {
    case 1: return launch((const void*)k_fedavg<1, OUTER>, a, grid, st);
    case 2: return launch((const void*)k_fedavg<2, OUTER>, a, grid, st);
    case 4: return launch((const void*)k_fedavg<4, OUTER>, a, grid, st);
    case 8: return launch((const void*)k_fedavg<8, OUTER>, a, grid, st);
    case 16: return launch((const void*)k_fedavg<16, OUTER>, a, grid, st);
    default: return launch((const void*)k_fedavg<0, OUTER>, a, grid, st);
  }
}

hipError_t launch_fedavg(const FedArgs& a, int grid, hipStream_t st) {
  return a.prev ? dispatch_fedavg<true>(a, grid, st) : dispatch_fedavg<false>(a, grid, st);
}

hipError_t launch_seg_finalize(const LayoutDev& L, const double* partials, double* chunk_sums,
                               double* seg_dbl, float* out, double* total, hipStream_t st) {
  if (L.n_seg == 0) return hipSuccess;
  const int g1 = (int)(L.n_chunks < 65535 ? L.n_chunks : 65535);
  const bool direct = L.n_chunks == L.n_seg;
  double* stage1 = direct ? seg_dbl : chunk_sums;
  void* a1[] = {const_cast<LayoutDev*>(&L), &partials, &stage1, &out};
  hipError_t e = hipLaunchKernel(direct ? (const void*)k_seg_chunks<true>
                                        : (const void*)k_seg_chunks<false>,
                                 dim3((unsigned)g1), dim3(kBlock), a1, 0, st);
  if (e != hipSuccess) return e;
  if (direct) {
    if (!total) return hipSuccess;
    int64_t n_seg = L.n_seg;
    void* a3[] = {&n_seg, &seg_dbl, &total};
    return hipLaunchKernel((const void*)k_total, dim3(1), dim3(kBlock), a3, 0, st);
  }
  const int64_t b2 = (L.n_seg + kBlock - 1) / kBlock;
  const int g2 = (int)(b2 < 65535 ? b2 : 65535);
  void* a2[] = {const_cast<LayoutDev*>(&L), &chunk_sums, &seg_dbl, &out};
  e = hipLaunchKernel((const void*)k_seg_totals, dim3((unsigned)g2), dim3(kBlock), a2, 0, st);
  if (e != hipSuccess || !total) return e;
  int64_t n_seg = L.n_seg;
  void* a3[] = {&n_seg, &seg_dbl, &total};
  return hipLaunchKernel((const void*)k_total, dim3(1), dim3(kBlock), a3, 0, st);
}

hipError_t launch_zero_total(double* total, hipStream_t st) {
  int64_t n_seg = 0;
  const double* none = nullptr;
  void* a3[] = {&n_seg, &none, &total};
  return hipLaunchKernel((const void*)k_total, dim3(1), dim3(kBlock), a3, 0, st);
}

hipError_t launch_sumsq_only(const StepArgs& a, int grid, hipStream_t st) {
  return dispatch_step<4, true>(a, grid, st);
}

hipError_t noalloc_scratch(int device, void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  if (device < 0 || device >= kMaxDevices || !ptr) return hipErrorInvalidValue;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[device]) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[device] = p;
  }
  *ptr = addr[device];
  return hipSuccess;
}

}  // namespace flr
