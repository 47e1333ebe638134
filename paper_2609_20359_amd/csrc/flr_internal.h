// flr_internal.h -- types shared by the C-ABI layer (flround_api.cpp) and the
// gfx950 kernels (flround_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace flr {

constexpr int kBlock = 256;            // threads per workgroup (4 wave64)
constexpr int kVec = 8;                // elements per thread per tile (16 B of bf16)
constexpr int kTile = kBlock * kVec;   // elements per tile: 2048
constexpr int kWaves = kBlock / 64;    // wave64s per workgroup: one partial slot each
constexpr int kChunkPieces = 1024;    // pieces folded by one workgroup in the finalize
constexpr int kCarryMaxChunks = 8;    // finalize carried by the next kernel up to this many chunks
constexpr int kMaxPeers = 64;
constexpr int kMaxGroups = 64;

// Per-tile descriptor of the segment structure, 16 bytes.
//   seg0   first segment overlapping the tile
//   nseg   number of segments overlapping it (1: the whole tile is in seg0)
//   piece0 index of the tile's first (tile, segment) piece; the tile owns
//          pieces piece0 .. piece0 + nseg - 1, one per overlapping segment
//   decay  when nseg == 1: seg0's weight-decay flag
struct TileInfo {
  int32_t seg0;
  int32_t nseg;
  int32_t piece0;
  int32_t decay;
};

// Device view of a layout.
struct LayoutDev {
  int64_t n;
  int64_t n_seg;
  int64_t n_tiles;
  int64_t n_pieces;
  const int64_t* seg_off;     // n_seg + 1
  const uint8_t* seg_decay;   // n_seg, 0/1
  const TileInfo* tiles;      // n_tiles
  const int64_t* seg_piece0;  // n_seg + 1: pieces of segment s are
                              // [seg_piece0[s], seg_piece0[s+1])
  int64_t n_chunks;
  const int64_t* chunk_p0;    // n_chunks + 1: chunk c folds pieces
                              // [chunk_p0[c], chunk_p0[c+1]), all of one segment
  const int64_t* seg_chunk0;  // n_seg + 1: chunks of segment s are
                              // [seg_chunk0[s], seg_chunk0[s+1])
};

// The finalize of the previous pass of a call, carried by the call's next
// kernel: that kernel runs one extra workgroup (its last) which folds the
// (piece, wave) partials the previous pass wrote, with the trees of
// k_seg_chunks, while the other workgroups stream.  Only for layouts whose
// every segment is one finalize chunk (chunk c is segment c) and that have at
// most kCarryMaxChunks of them.  partials == null: nothing carried.
struct Carry {
  const double* partials;
  const int64_t* chunk_p0;  // n_chunks + 1
  int64_t n_chunks;
  float* out;               // n_chunks floats: the per-segment sums
};

// Per-step AdamW scalars, computed on the host in double, rounded to float.
struct AdamScalars {
  float b1, omb1, b2, omb2;
  float step_size, bc2_sqrt, eps, decay;
};

// Arguments of the local-step family (reduce, AdamW, fused step).
struct StepArgs {
  LayoutDev L;
  const uint16_t* grads[kMaxPeers];
  int R;
  float grad_scale;
  AdamScalars s;
  float* master;
  float* m;
  float* v;
  uint16_t* working;   // may be null for the standalone AdamW step
  float* g_out;        // standalone reduce: fp32 reduced gradient
  const float* g_in;   // standalone AdamW: fp32 gradient
  uint16_t* wire_out;  // reduce to the bf16 wire format
  double* partials;    // per-(piece, wave) sums of squares, kWaves per piece
                       // (null: not requested)
  const double* clip_total;  // MODE 0: whole-shard sum of squares, clipping on
  float clip_max;            // its max norm
  Carry carry;
};

struct FedArgs {
  int64_t n;
  const uint16_t* reps[kMaxGroups];
  float w[kMaxGroups];
  int G;
  float* master;
  uint16_t* working;
  // outer optimiser step (prev == null: plain FedAvg)
  float* prev;
  float* buf;
  float eta, mu;
  int nesterov;
  Carry carry;
};

struct BcastArgs {
  int64_t n;
  const float* recv;
  float* master;
  uint16_t* working;
  Carry carry;
};

hipError_t launch_local_step(const StepArgs& a, int grid, hipStream_t st);
hipError_t launch_reduce(const StepArgs& a, int grid, hipStream_t st);
hipError_t launch_adamw(const StepArgs& a, int grid, hipStream_t st);
hipError_t launch_reduce_wire(const StepArgs& a, int grid, hipStream_t st);
hipError_t launch_bcast_recv(const BcastArgs& a, int grid, hipStream_t st);
hipError_t launch_fedavg(const FedArgs& a, int grid, hipStream_t st);
// The launch helpers take `grid` workgroups for the stream and add one for a
// carried finalize (a.carry.partials set).
// Per-segment totals from the (piece, wave) partials: chunk_sums
// (L.n_chunks doubles) and seg_dbl (L.n_seg doubles) are temporaries; out
// (n_seg floats) and total (one double, the whole shard) may be null.
hipError_t launch_seg_finalize(const LayoutDev& L, const double* partials, double* chunk_sums,
                               double* seg_dbl, float* out, double* total, hipStream_t st);
hipError_t launch_sumsq_only(const StepArgs& a, int grid, hipStream_t st);

// The static scratch of fl_round_noalloc (kNoallocScratchBytes per GPU).
// The first call for a device, with that device current, looks up the
// array's address on it; later calls return the cached address.  Nothing in
// it needs to start at zero: every slot is written before it is read.
constexpr size_t kNoallocScratchBytes = (size_t)32 << 20;
hipError_t noalloc_scratch(int device, void** ptr);
hipError_t launch_zero_total(double* total, hipStream_t st);

}  // namespace flr
