// Host-side internals shared by the translation units of libjanus.
#pragma once

#include <vector>

#include "common.h"
#include "gemm.h"

// Device memory owned by a context, grown on demand and never shrunk.
struct janus_buffer {
  void* ptr = nullptr;
  size_t bytes = 0;
};

// Kernel families timed by the optional profiler (janus_profile_*).
enum JanusProfClass {
  PROF_EXPERT_GEMM = 0,   // expert token x weight products (forward and the three backward passes)
  PROF_EXPERT_WGRAD,      // expert weight gradients (chunked products and their fixed-order reduction)
  PROF_DENSE_GEMM,        // readout and radial-filter products and their gradients
  PROF_EDGE,              // per-edge gather / dispatch / adjoint kernels
  PROF_ATOM,              // per-atom combine / scatter kernels
  PROF_ROUTE,             // routing and the expert permutation
  PROF_GRAPH,             // neighbour list, reverse map, geometry and basis
  PROF_OTHER,             // validation, readout, loss, forces, router and embedding gradients
  PROF_ATTN,              // neighbourhood self-attention (per-atom query / key passes)
  PROF_NCLASS
};

struct janus_prof_rec {
  int cls;
  hipEvent_t a, b;
  double flops, bytes;
};

struct janus_ctx {
  janus_config cfg;
  int device = 0;
  janus_buffer ws;        // per-step workspace of janus_step
  janus_buffer aux;       // tables and partials of the standalone GEMM entry points
  janus_buffer nl;        // per-atom counts and flags of janus_build_edges
  janus_buffer gbuf;      // whole-batch arrays of janus_step (flags, structure ids, loss shares)
  int* host_word = nullptr;   // 4 pinned host ints for the flag / count reads
  int* host_plan = nullptr;   // pinned host ints for the chunk plan
  size_t host_plan_n = 0;
  long long ws_limit = 0;     // workspace cap in bytes (0: from free device memory)
  int last_chunks = 0;        // chunks used by the last janus_step
  int edge_builder = 0;       // janus_set_edge_builder mode (0 auto, 1 cell lists, 2 all pairs)
  long long last_triplets = 0; // triplets of the last janus_step's batch
  // profiler: event pairs recorded around kernel families while enabled
  bool prof_on = false;
  unsigned prof_mask = 0;     // families recorded (bit = JanusProfClass)
  std::vector<janus_prof_rec> prof_recs;
  std::vector<hipEvent_t> prof_pool;
  size_t prof_used = 0;
  // second stream for the expert weight gradients, which then run beside the
  // memory-bound double-backward products (janus_set_concurrency)
  int concurrent = 0;
  hipStream_t side = nullptr;
  std::vector<hipEvent_t> sync_pool;   // fork / join events, reused every step
  size_t sync_used = 0;
};

namespace janus {

// Records an event pair around the launches issued during its lifetime.
struct ProfScope {
  janus_ctx* c;
  hipStream_t st;
  janus_prof_rec rec;
  bool on;
  ProfScope(janus_ctx* ctx, hipStream_t s, int cls, double flops, double bytes);
  ~ProfScope();
};

// Fork / join between the caller's stream and the context's side stream.
// side_stream() is the stream the weight gradients go to: the side stream when
// concurrency is on, else the caller's stream itself (then every fork, mark and
// wait below is a no-op and the step runs in one stream, in the same order).
struct SideSync {
  janus_ctx* c;
  hipStream_t st, sd;
  hipError_t err = hipSuccess;
  SideSync(janus_ctx* ctx, hipStream_t main);
  // event recorded on `from` now (nullptr when both streams are one)
  hipEvent_t record(hipStream_t from);
  // `to` waits for everything issued to `from` so far
  void order(hipStream_t from, hipStream_t to);
  void fork() { order(st, sd); }
  void join() { order(sd, st); }
  hipEvent_t mark() { return record(sd); }
  void wait(hipEvent_t e);
};

// Grow `b` to at least `bytes` (contents are not preserved).
int ensure(janus_buffer& b, size_t bytes);

// Bump allocator over one device buffer; every region is 256-byte aligned.
struct Carver {
  uintptr_t base;
  size_t off = 0;
  explicit Carver(void* p) : base(reinterpret_cast<uintptr_t>(p)) {}
  template <class T>
  T* take(size_t n) {
    off = (off + 255) & ~size_t(255);
    T* p = reinterpret_cast<T*>(base + off);
    off += n * sizeof(T);
    return p;
  }
  size_t size() const { return (off + 255) & ~size_t(255); }
};

// Upper bounds on the tile / chunk tables of a grouped GEMM over M rows.
inline int max_rows_tiles(long long M, int groups) { return (int)((M + GBM - 1) / GBM) + groups; }
inline int max_wchunks(long long M, int groups, int kc) { return (int)((M + kc - 1) / kc) + groups; }

// Chunk length of the weight-gradient contraction, a power of two from 128 to
// 2048 rows.  A 2048-row chunk is 128 LDS stages, the K loop of the K = 2048
// expert products.  Longer chunks are slower at full size (512 x 2048 blocks
// over 1.8 M rows: 16384-row chunks take 16 % longer, partial reduction
// included): the tiles of one chunk share its operand rows through L2 only
// while they run in step, and the last round of long workgroups leaves most
// of the GPU idle.  Shorter chunks are taken while the grid has fewer than
// 4096 workgroups (four rounds of the 1024 that are resident at once), as long
// as the partial tiles of the halved chunk (written and read back once by the
// reduction) stay within half of the operand bytes.
inline int wgrad_chunk_rows(long long M, int P, int Q) {
  const long long tiles = (long long)((P + GBM - 1) / GBM) * ((Q + GBN - 1) / GBN);
  const double operand_bytes = 4.0 * (double)M * (P + Q);
  auto blocks = [&](long long kc) { return ((M + kc - 1) / kc) * tiles; };
  auto partial_bytes = [&](long long kc) { return 8.0 * (double)((M + kc - 1) / kc) * P * Q; };
  long long kc = 2048;
  while (kc > 128 && blocks(kc) < 4096 && partial_bytes(kc / 2) <= 0.5 * operand_bytes) kc /= 2;
  return (int)kc;
}

// Chunk length of the skinny weight gradient (wgrad_skinny_kernel, one workgroup
// per chunk): a multiple of the rows of one of its steps, long enough that all
// chunks fit in one set of resident workgroups (CUs x workgroups per CU at the
// kernel instance's register and LDS use, queried from the runtime), so no
// second, mostly idle round runs.
int skinny_chunk_rows(long long M, int P, int Q);

// Instance of the skinny weight gradient for P x Q: P rounded up to 8, 16 or 32,
// and the columns per lane.
template <int PM, int CW>
const void* skinny_instance() { return (const void*)wgrad_skinny_kernel<PM, CW>; }
inline const void* skinny_kernel(int P, int Q) {
  const int cw = skinny_cw(Q);
#define JANUS_SKINNY_CW(PM) (cw == 4 ? skinny_instance<PM, 4>() : cw == 2 ? skinny_instance<PM, 2>() : skinny_instance<PM, 1>())
  return P <= 8 ? JANUS_SKINNY_CW(8) : P <= 16 ? JANUS_SKINNY_CW(16) : JANUS_SKINNY_CW(32);
#undef JANUS_SKINNY_CW
}

void launch_wgrad_reduce(hipStream_t st, const float* partial, const int* chunk_first, int groups,
                         long long PQ, float* G, int accumulate);

// Launch helpers (the tables must have been built on `st` beforehand).
template <bool NT, class ALoad, class Epi>
void launch_rows(hipStream_t st, const ALoad& al, const float* B, int K, int N, const RowsTile* tiles,
                 const int* n_tiles, int max_tiles, const Epi& epi, float* rowsum = nullptr) {
  if (max_tiles <= 0) return;
  dim3 grid(xcd_grid(max_tiles, (N + GBN - 1) / GBN));
  hipLaunchKernelGGL((gemm_rows_kernel<NT, ALoad, Epi>), grid, dim3(256), 0, st, al, B, K, N, tiles,
                     n_tiles, epi, rowsum);
}

template <class ALoad, class BLoad>
void launch_wgrad(hipStream_t st, const ALoad& al, const BLoad& bl, int P, int Q, const WChunk* chunks,
                  const int* n_chunks, const int* chunk_first, int max_chunks, int groups,
                  float* partial, float* G, int accumulate) {
  if (max_chunks > 0) {
    dim3 grid(xcd_grid(max_chunks, ((P + GBM - 1) / GBM) * ((Q + GBN - 1) / GBN)));
    hipLaunchKernelGGL((gemm_wgrad_kernel<ALoad, BLoad>), grid, dim3(256), 0, st, al, bl, P, Q, chunks,
                       n_chunks, partial);
  }
  launch_wgrad_reduce(st, partial, chunk_first, groups, (long long)P * Q, G, accumulate);
}

// Skinny weight gradient (P <= 32, Q <= 512, P and Q multiples of 4, one group):
// G (+)= (s * A)^T B over the chunks of the table.
inline void launch_wgrad_skinny(hipStream_t st, const float* A, const float* s, const float* B, int P, int Q,
                                const WChunk* chunks, const int* n_chunks, const int* chunk_first, int max_chunks,
                                float* partial, float* G, int accumulate) {
  if (max_chunks > 0) {
    void* args[] = {(void*)&A, (void*)&s, (void*)&B, (void*)&P, (void*)&Q, (void*)&chunks, (void*)&n_chunks,
                    (void*)&partial};
    (void)hipLaunchKernel(skinny_kernel(P, Q), dim3(max_chunks), dim3(256), args, sizeof(float) * P * Q, st);
  }
  launch_wgrad_reduce(st, partial, chunk_first, 1, (long long)P * Q, G, accumulate);
}

void build_tables(hipStream_t st, const int* row_off, int groups, int kc, RowsTile* tiles, int* n_tiles,
                  WChunk* chunks, int* n_chunks, int* chunk_first);

}  // namespace janus
