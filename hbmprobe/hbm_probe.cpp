// hbm_probe -- attainable HBM bandwidth on this GPU for the access patterns of
// the parameter-sync kernels, with no arithmetic: the ceiling that the local
// step and FedAvg kernels are compared with, besides the 8 TB/s datasheet
// peak.  Not part of the library.
//
// Patterns (every stream a separate buffer; each thread moves 16 B of every
// stream per grid-stride iteration, 256-thread workgroups):
//   read1      1 stream read
//   write1     1 stream written
//   copy       1 read, 1 written
//   triad      2 read, 1 written (STREAM's triad traffic)
//   step_R8    8 bf16 streams read, 3 fp32 streams read and written, 1 bf16
//              stream written: the traffic of one fused local step (R = 8)
//   step_R4, step_R2  the same with 4 and 2 peer streams (R = 4; the FL+HSDP
//              second tier averages H = 2 bf16 wire shards, the R = 2 pattern)
//   sumsq_R8, sumsq_R4  8 or 4 bf16 streams read, nothing written: the
//              sum-of-squares pass before a clipped step
//   wire_R4    4 bf16 streams read, 1 bf16 stream written: the FL+HSDP
//              first-tier reduction to the wire format
//   reduce_R8  8 bf16 streams read, 1 fp32 stream written: the reduction
//              that stores the gradient of a clipped step in its scratch
//   fedavg_G4  4 bf16 streams read, 1 fp32 and 1 bf16 stream written
//   fedopt_G4  as fedavg_G4 plus 2 fp32 streams read and written (the outer
//              step's round-start model and momentum buffer)
//   bcast      4 bytes read (two 2-byte streams), 1 fp32 and 1 bf16 stream
//              written: the FL+HSDP broadcast receive
//   rmw3       3 fp32 streams read and written in place: the optimiser state
//              of the fused step alone
//   step_R8_tiled  as step_R8, but the three fp32 state arrays interleaved per
//              2048-element tile ([tile][master | m | v]), i.e. one 24 KB
//              read-modify-write chunk per tile instead of three streams
//   <pattern>_w  a pattern whose every wave waits for its previous
//              iteration's stores to complete before issuing its next loads
//              (copy, triad, step_R8/R4/R2, wire_R4, reduce_R8, fedavg_G4,
//              fedopt_G4, bcast, rmw3)
// each with plain and nontemporal stores, for 1, 2, 3, 4 and 8 workgroups per CU
// (or the one count given).
// Buffers are sized for the given element count (default: the
// 1,003,782,144-element shard of Llama-3.1-8B at S = 8; the S = 4 shard has
// 2,007,564,288 elements and needs about 120 GB).
//
// usage: hbm_probe [elements [pattern[,pattern...] [workgroups per CU [stagger]]]]
//   with a pattern list only those patterns run (an empty list: all, and
//   the runtime copy line, which is printed only without a list); a counter
//   run names one pattern and one workgroup count so that every dispatch of
//   the run is that pattern; a workgroup count of 0 keeps the default set.
//   stagger (bytes, a multiple of 256; default 0): place the streams in one
//   allocation, stream k at a 2 MiB boundary plus k * stagger, as the
//   library's staggered placement places a shard's arrays.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

#define CK(x)                                                                         \
  do {                                                                                \
    hipError_t e_ = (x);                                                              \
    if (e_ != hipSuccess) {                                                           \
      std::printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);      \
      std::exit(1);                                                                   \
    }                                                                                 \
  } while (0)

template <typename F>
float time_ms(F launch, int reps);

// Patterns and workgroup counts selected on the command line (empty: all).
static std::vector<std::string> g_only;
static std::vector<int> g_bpc = {1, 2, 3, 4, 8};

static bool selected(const char* name) {
  if (g_only.empty()) return true;
  for (const std::string& o : g_only)
    if (o == name) return true;
  return false;
}

struct Streams {
  const u32x4* rd[12];  // read-only 16-byte streams, in units of u32x4
  u32x4* rmw[4];        // read-modify-write streams (fp32, 2 x 16 B per thread)
  u32x4* wr[2];         // write-only streams: wr[0] bf16 (2 B per element), wr[1] fp32
  u32x4* tiled;         // 3 fp32 arrays interleaved per 2048-element tile
  long nvec;            // 16-byte vectors per bf16 stream
};

// 8 bf16 streams read; master/m/v tile-interleaved (read and written); one
// bf16 stream written.  Tile of vector i: i / 256; its state block holds
// 3 x 512 vectors.  Indices stay below 6 * nvec.
template <bool NTS>
__global__ void __launch_bounds__(256) k_step_tiled(Streams s) {
  const long stride = (long)gridDim.x * 256;
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < s.nvec; i += stride) {
    u32x4 x = {(unsigned)i, 0u, 0u, 0u};
#pragma unroll
    for (int k = 0; k < 8; ++k) x += __builtin_nontemporal_load(s.rd[k] + i);
    const long base = (i / 256) * 1536 + (i % 256) * 2;
    u32x4 a[6];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      a[2 * k] = s.tiled[base + 512 * k];
      a[2 * k + 1] = s.tiled[base + 512 * k + 1];
    }
#pragma unroll
    for (int k = 0; k < 6; ++k) {
      u32x4* q = s.tiled + base + 512 * (k / 2) + (k & 1);
      if (NTS) __builtin_nontemporal_store(a[k] + x, q); else *q = a[k] + x;
    }
    if (NTS) __builtin_nontemporal_store(x, s.wr[0] + i); else s.wr[0][i] = x;
  }
}

void run_tiled(Streams s, int cus, long elems) {
  if (!selected("step_R8_tiled")) return;
  const double bytes = (double)elems * 42.0;
  for (int nts = 0; nts < 2; ++nts) {
    double best = 0.0;
    int best_bpc = 0;
    std::printf("| %-9s | %-5s |", "step_R8_tiled", nts ? "nt" : "plain");
    for (int bpc : g_bpc) {
      const int grid = bpc * cus;
      float ms = nts ? time_ms([&] { k_step_tiled<true><<<grid, 256>>>(s); }, 5)
                     : time_ms([&] { k_step_tiled<false><<<grid, 256>>>(s); }, 5);
      CK(hipGetLastError());
      const double gbs = bytes / (ms * 1e-3) / 1e9;
      std::printf(" %7.1f |", gbs);
      if (gbs > best) {
        best = gbs;
        best_bpc = bpc;
      }
    }
    std::printf(" %7.1f (%d/CU) | %5.1f %% |\n", best, best_bpc, 100.0 * best / 8000.0);
    std::fflush(stdout);
  }
}

// NRD bf16 streams read, NRMW fp32 streams read+written, NWH bf16 streams
// written, NWF fp32 streams written.  fp32 streams hold 2 vectors per bf16
// vector.  All indices < nvec (bf16) or < 2 * nvec (fp32).
template <int NRD, int NRMW, int NWH, int NWF, bool NTS, bool WAIT = false>
__global__ void __launch_bounds__(256) k_pattern(Streams s) {
  static_assert(NWF <= 1 && NWH <= 1, "wr[1] is the one fp32 and wr[0] the one bf16 stream");
  const long stride = (long)gridDim.x * 256;
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < s.nvec; i += stride) {
    // WAIT: the previous iteration's stores complete before this
    // iteration's loads are issued (s_waitcnt vmcnt(0))
    if (WAIT) __builtin_amdgcn_s_waitcnt(0xF70);
    u32x4 x = {(unsigned)i, 0u, 0u, 0u};
#pragma unroll
    for (int k = 0; k < NRD; ++k) x += __builtin_nontemporal_load(s.rd[k] + i);
    u32x4 a[NRMW > 0 ? NRMW : 1], b[NRMW > 0 ? NRMW : 1];
#pragma unroll
    for (int k = 0; k < NRMW; ++k) {
      a[k] = s.rmw[k][2 * i];
      b[k] = s.rmw[k][2 * i + 1];
    }
#pragma unroll
    for (int k = 0; k < NRMW; ++k) {
      if (NTS) {
        __builtin_nontemporal_store(a[k] + x, s.rmw[k] + 2 * i);
        __builtin_nontemporal_store(b[k] + x, s.rmw[k] + 2 * i + 1);
      } else {
        s.rmw[k][2 * i] = a[k] + x;
        s.rmw[k][2 * i + 1] = b[k] + x;
      }
    }
#pragma unroll
    for (int k = 0; k < NWH; ++k) {
      if (NTS) __builtin_nontemporal_store(x, s.wr[k] + i); else s.wr[k][i] = x;
    }
#pragma unroll
    for (int k = 0; k < NWF; ++k) {
      if (NTS) {
        __builtin_nontemporal_store(x, s.wr[1 - k] + 2 * i);
        __builtin_nontemporal_store(x, s.wr[1 - k] + 2 * i + 1);
      } else {
        s.wr[1 - k][2 * i] = x;
        s.wr[1 - k][2 * i + 1] = x;
      }
    }
    if (NRD + NRMW + NWH + NWF == NRD && x.y == 0xFFFFFFFFu && x.z == 0x12345u)
      s.wr[0][0] = x;  // keep read-only loads alive
  }
}

template <typename F>
float time_ms(F launch, int reps) {
  hipEvent_t a, b;
  CK(hipEventCreate(&a));
  CK(hipEventCreate(&b));
  launch();
  CK(hipDeviceSynchronize());
  CK(hipEventRecord(a));
  for (int r = 0; r < reps; ++r) launch();
  CK(hipEventRecord(b));
  CK(hipEventSynchronize(b));
  float ms = 0.f;
  CK(hipEventElapsedTime(&ms, a, b));
  CK(hipEventDestroy(a));
  CK(hipEventDestroy(b));
  return ms / reps;
}

template <int NRD, int NRMW, int NWH, int NWF, bool WAIT = false>
void run(const char* name, Streams s, int cus, long elems) {
  if (!selected(name)) return;
  const double bytes = (double)elems * (2.0 * NRD + 8.0 * NRMW + 2.0 * NWH + 4.0 * NWF);
  for (int nts = 0; nts < 2; ++nts) {
    double best = 0.0;
    int best_bpc = 0;
    std::printf("| %-9s | %-5s |", name, nts ? "nt" : "plain");
    for (int bpc : g_bpc) {
      const int grid = bpc * cus;
      float ms =
          nts ? time_ms([&] { k_pattern<NRD, NRMW, NWH, NWF, true, WAIT><<<grid, 256>>>(s); }, 5)
              : time_ms([&] { k_pattern<NRD, NRMW, NWH, NWF, false, WAIT><<<grid, 256>>>(s); }, 5);
      CK(hipGetLastError());
      const double gbs = bytes / (ms * 1e-3) / 1e9;
      std::printf(" %7.1f |", gbs);
      if (gbs > best) {
        best = gbs;
        best_bpc = bpc;
      }
    }
    std::printf(" %7.1f (%d/CU) | %5.1f %% |\n", best, best_bpc, 100.0 * best / 8000.0);
    std::fflush(stdout);
  }
}

int main(int argc, char** argv) {
  long elems = argc > 1 ? std::atol(argv[1]) : 1003782144L;
  elems -= elems % 8;
  if (argc > 2) {
    std::string list = argv[2];
    size_t pos = 0;
    while (pos <= list.size()) {
      const size_t c = list.find(',', pos);
      const std::string item = list.substr(pos, c == std::string::npos ? std::string::npos : c - pos);
      if (!item.empty()) g_only.push_back(item);
      if (c == std::string::npos) break;
      pos = c + 1;
    }
  }
  if (argc > 3) {
    const int b = std::atoi(argv[3]);
    if (b < 0 || b > 16) {
      std::printf("workgroups per CU must be 1..16 (0: the default set)\n");
      return 2;
    }
    if (b > 0) g_bpc = {b};
  }
  // stagger > 0: every stream carved from one allocation, stream k at a
  // 2 MiB boundary plus k * stagger bytes, in the order of the library's
  // staggered placement of a shard (master, m, v, working copy, then the
  // peer gradients); 0: one allocation per stream
  const long stagger = argc > 4 ? std::atol(argv[4]) : 0;
  if (stagger < 0 || stagger % 256 != 0) {
    std::printf("stagger must be a non-negative multiple of 256 bytes\n");
    return 2;
  }
  int cus = 0;
  CK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0));
  hipDeviceProp_t prop;
  CK(hipGetDeviceProperties(&prop, 0));
  Streams s;
  s.nvec = elems / 8;
  std::vector<void*> bufs;
  // the streams in placement order: the three state arrays, the written
  // bf16 stream, the twelve read streams, then the rest
  const size_t tiled_bytes = (size_t)elems * 12 + 3 * 2048 * 4;
  std::vector<size_t> sizes;
  for (int k = 0; k < 3; ++k) sizes.push_back((size_t)elems * 4);   // rmw[0..2]
  sizes.push_back((size_t)elems * 2);                                 // wr[0] (bf16 writes)
  for (int k = 0; k < 12; ++k) sizes.push_back((size_t)elems * 2);  // rd[0..11]
  sizes.push_back((size_t)elems * 4);                                 // rmw[3]
  sizes.push_back((size_t)elems * 4);                                 // wr[1]
  sizes.push_back(tiled_bytes);                                       // tiled
  std::vector<void*> ptrs;
  if (stagger == 0) {
    for (size_t b : sizes) {
      void* p = nullptr;
      CK(hipMalloc(&p, b));
      CK(hipMemset(p, 0, b));
      bufs.push_back(p);
      ptrs.push_back(p);
    }
  } else {
    const size_t align = (size_t)2 << 20;
    size_t total = align;
    for (size_t b : sizes) total += (b + align - 1) / align * align + align;
    void* pool = nullptr;
    CK(hipMalloc(&pool, total));
    CK(hipMemset(pool, 0, total));
    bufs.push_back(pool);
    char* base = static_cast<char*>(pool);
    size_t off = (align - reinterpret_cast<uintptr_t>(base) % align) % align;
    for (size_t k = 0; k < sizes.size(); ++k) {
      // slot k: [off, off + roundup(size) + align); the stream starts
      // (k * stagger) % align into it, so it ends inside the slot
      ptrs.push_back(base + off + (k * (size_t)stagger) % align);
      off += (sizes[k] + align - 1) / align * align + align;
    }
  }
  for (int k = 0; k < 3; ++k) s.rmw[k] = static_cast<u32x4*>(ptrs[k]);
  s.wr[0] = static_cast<u32x4*>(ptrs[3]);
  for (int k = 0; k < 12; ++k) s.rd[k] = static_cast<const u32x4*>(ptrs[4 + k]);
  s.rmw[3] = static_cast<u32x4*>(ptrs[16]);
  s.wr[1] = static_cast<u32x4*>(ptrs[17]);
  s.tiled = static_cast<u32x4*>(ptrs[18]);
  std::printf("# HBM ceiling probe: %s, %d CUs, %ld-element streams\n\n", prop.gcnArchName, cus,
              elems);
  std::printf("GB/s by workgroups per CU; bytes = bytes the pattern moves; peak 8000 GB/s.\n\n");
  std::printf("| pattern | stores |");
  for (int b : g_bpc) std::printf(" %d/CU |", b);
  std::printf(" best | of peak |\n|---|---|");
  for (size_t k = 0; k < g_bpc.size(); ++k) std::printf("---|");
  std::printf("---|---|\n");
  run<1, 0, 0, 0>("read1", s, cus, elems);
  run<0, 0, 1, 0>("write1", s, cus, elems);
  run<1, 0, 1, 0>("copy", s, cus, elems);
  run<2, 0, 1, 0>("triad", s, cus, elems);
  run<8, 3, 1, 0>("step_R8", s, cus, elems);
  run<4, 3, 1, 0>("step_R4", s, cus, elems);
  run<2, 3, 1, 0>("step_R2", s, cus, elems);
  run<8, 0, 0, 0>("sumsq_R8", s, cus, elems);
  run<4, 0, 0, 0>("sumsq_R4", s, cus, elems);
  run<4, 0, 1, 0>("wire_R4", s, cus, elems);
  run<8, 0, 0, 1>("reduce_R8", s, cus, elems);
  run<4, 0, 1, 1>("fedavg_G4", s, cus, elems);
  run<4, 2, 1, 1>("fedopt_G4", s, cus, elems);
  run<2, 0, 1, 1>("bcast", s, cus, elems);
  run<0, 3, 0, 0>("rmw3", s, cus, elems);
  run_tiled(s, cus, elems);
  // the same patterns with each wave's stores completing before its next loads
  run<1, 0, 1, 0, true>("copy_w", s, cus, elems);
  run<2, 0, 1, 0, true>("triad_w", s, cus, elems);
  run<8, 3, 1, 0, true>("step_R8_w", s, cus, elems);
  run<4, 3, 1, 0, true>("step_R4_w", s, cus, elems);
  run<2, 3, 1, 0, true>("step_R2_w", s, cus, elems);
  run<4, 0, 1, 0, true>("wire_R4_w", s, cus, elems);
  run<8, 0, 0, 1, true>("reduce_R8_w", s, cus, elems);
  run<4, 0, 1, 1, true>("fedavg_G4_w", s, cus, elems);
  run<4, 2, 1, 1, true>("fedopt_G4_w", s, cus, elems);
  run<2, 0, 1, 1, true>("bcast_w", s, cus, elems);
  run<0, 3, 0, 0, true>("rmw3_w", s, cus, elems);

  // the runtime's own device-to-device copy of one fp32 stream, as a vendor
  // reference point for the copy pattern (bytes read + written)
  if (g_only.empty()) {
    void* src = static_cast<void*>(s.rmw[0]);
    void* dst = static_cast<void*>(s.wr[1]);
    const size_t bytes = (size_t)elems * 4;
    const float ms =
        time_ms([&] { CK(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, 0)); }, 5);
    const double gbs = 2.0 * (double)bytes / (ms * 1e-3) / 1e9;
    std::printf("\nhipMemcpyAsync device to device, %zu bytes: %.3f ms, %.1f GB/s moved "
                "(%.1f %% of peak)\n", bytes, ms, gbs, 100.0 * gbs / 8000.0);
  }
  for (void* p : bufs) CK(hipFree(p));
  return 0;
}
