// Element-type top-k routing and the stable expert-grouped permutation of
// edge tokens.
//
// Paper Sec. "Algorithmic innovation" (sparse MoE routing): edge tokens are
// routed by the element types of their atoms, and all routing decisions are
// made before the interaction blocks run.  Reading: the router logits of an
// edge are the fp32 sum (Pc[Z_i] + Pn[Z_j]) + beta; the top-k experts are
// taken in descending logit order with the lower index first on ties; the
// gate of a chosen expert is its probability under the softmax over all
// experts.  Because the logits depend only on the species pair, the decision
// is made once per pair and looked up per edge.  Tokens are then grouped by
// expert with a stable counting sort on (expert, edge, choice), which fixes
// the slot of every (edge, choice) pair exactly.
#include "internal.h"
#include "route.h"

namespace janus {

constexpr int kSortChunk = 4096;

// One thread per species pair p = a * n_species + b.
__global__ void route_pairs_kernel(const float* __restrict__ Pc, const float* __restrict__ Pn,
                                   const float* __restrict__ beta, int nsp, int E, int k,
                                   int* __restrict__ peid, float* __restrict__ pgate, float* __restrict__ pprob) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= nsp * nsp) return;
  const int a = p / nsp, b = p % nsp;
  float l[64];
  double mx = -1e300;
  for (int x = 0; x < E; ++x) {
    l[x] = __fadd_rn(__fadd_rn(Pc[a * E + x], Pn[b * E + x]), beta[x]);
    double ld = ((double)Pc[a * E + x] + (double)Pn[b * E + x]) + (double)beta[x];
    mx = ld > mx ? ld : mx;
  }
  double den = 0.0;
  for (int x = 0; x < E; ++x) den += exp((((double)Pc[a * E + x] + (double)Pn[b * E + x]) + (double)beta[x]) - mx);
  for (int x = 0; x < E; ++x)
    pprob[(long long)p * E + x] =
        (float)(exp((((double)Pc[a * E + x] + (double)Pn[b * E + x]) + (double)beta[x]) - mx) / den);
  unsigned long long taken = 0;
  for (int c = 0; c < k; ++c) {
    int best = -1;
    for (int x = 0; x < E; ++x) {
      if (taken >> x & 1ull) continue;
      if (best < 0 || l[x] > l[best]) best = x;
    }
    taken |= 1ull << best;
    peid[p * k + c] = best;
    pgate[p * k + c] =
        (float)(exp((((double)Pc[a * E + best] + (double)Pn[b * E + best]) + (double)beta[best]) - mx) / den);
  }
}

// Per edge: species pair, chosen experts and gates.
__global__ void route_edges_kernel(const int* __restrict__ species, const int* __restrict__ ei,
                                   const int* __restrict__ ej, int Ne, int nsp, int k,
                                   const int* __restrict__ peid, const float* __restrict__ pgate,
                                   int* __restrict__ pair, int* __restrict__ eid, float* __restrict__ gate) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne) return;
  const int p = species[ei[e]] * nsp + species[ej[e]];
  pair[e] = p;
  for (int c = 0; c < k; ++c) {
    eid[(long long)e * k + c] = peid[p * k + c];
    gate[(long long)e * k + c] = pgate[p * k + c];
  }
}

// Histogram of expert ids per chunk of kSortChunk flattened (edge, choice) entries.
__global__ void sort_count_kernel(const int* __restrict__ eid, long long M, int E, int* __restrict__ cnt) {
  __shared__ int hist[64];
  const int ch = blockIdx.x;
  if (threadIdx.x < 64) hist[threadIdx.x] = 0;
  __syncthreads();
  const long long f0 = (long long)ch * kSortChunk;
  const long long f1 = min(M, f0 + kSortChunk);
  for (long long f = f0 + threadIdx.x; f < f1; f += blockDim.x) atomicAdd(&hist[eid[f]], 1);
  __syncthreads();
  if (threadIdx.x < E) cnt[(long long)ch * E + threadIdx.x] = hist[threadIdx.x];
}

// Exclusive scan of one expert's column of chunk counts (one workgroup per expert).
__global__ void sort_colscan_kernel(const int* __restrict__ cnt, int nch, int E, int* __restrict__ colpre,
                                    int* __restrict__ total) {
  __shared__ int part[256];
  const int x = blockIdx.x, t = threadIdx.x;
  const int per = (nch + 255) / 256;
  const int lo = min(nch, t * per), hi = min(nch, lo + per);
  int s = 0;
  for (int c = lo; c < hi; ++c) s += cnt[(long long)c * E + x];
  part[t] = s;
  __syncthreads();
  for (int o = 1; o < 256; o <<= 1) {
    int v = t >= o ? part[t - o] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int run = part[t] - s;
  for (int c = lo; c < hi; ++c) {
    colpre[(long long)c * E + x] = run;
    run += cnt[(long long)c * E + x];
  }
  if (t == 255) total[x] = part[255];
}

__global__ void sort_offsets_kernel(const int* __restrict__ total, int E, int* __restrict__ off) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  int acc = 0;
  for (int x = 0; x < E; ++x) {
    off[x] = acc;
    acc += total[x];
  }
  off[E] = acc;
}

// One wave per chunk walks its entries in order, 64 at a time; the rank of
// an entry among equal keys comes from a ballot match, so the order is stable.
__global__ __launch_bounds__(64) void sort_scatter_kernel(const int* __restrict__ eid, const float* __restrict__ gate,
                                                          long long M, int E, const int* __restrict__ off,
                                                          const int* __restrict__ colpre, int* __restrict__ pos,
                                                          float* __restrict__ slot_gate) {
  __shared__ int run[64];
  const int ch = blockIdx.x, lane = threadIdx.x;
  run[lane] = 0;
  __syncthreads();
  const long long f0 = (long long)ch * kSortChunk;
  const long long f1 = min(M, f0 + kSortChunk);
  const unsigned long long lt = (1ull << lane) - 1ull;
  for (long long g = f0; g < f1; g += 64) {
    const long long f = g + lane;
    const bool valid = f < f1;
    const int key = valid ? eid[f] : 0;
    unsigned long long mm = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 6; ++b) {
      const bool bit = (key >> b) & 1;
      const unsigned long long bb = __ballot(bit);
      mm &= bit ? bb : ~bb;
    }
    const int rank = __popcll(mm & lt);
    const int base = run[key];
    __syncthreads();
    if (valid) {
      const int p = off[key] + colpre[(long long)ch * E + key] + base + rank;
      pos[f] = p;
      slot_gate[p] = gate[f];
      if ((mm >> lane) == 1ull) run[key] = base + __popcll(mm);   // last entry of its key
    }
    __syncthreads();
  }
}

void route_block(hipStream_t st, const RouteArgs& a) {
  const int np = a.nsp * a.nsp;
  hipLaunchKernelGGL(route_pairs_kernel, dim3(cdiv(np, 128)), dim3(128), 0, st, a.Pc, a.Pn, a.beta, a.nsp, a.E, a.k,
                     a.peid, a.pgate, a.pprob);
  if (a.Ne > 0)
    hipLaunchKernelGGL(route_edges_kernel, dim3(cdiv(a.Ne, 256)), dim3(256), 0, st, a.species, a.ei, a.ej, a.Ne,
                       a.nsp, a.k, a.peid, a.pgate, a.pair, a.eid, a.gate);
  sort_tokens(st, a.eid, a.gate, (long long)a.Ne * a.k, a.E, a.cnt, a.colpre, a.total, a.off, a.pos, a.slot_gate);
}

void sort_tokens(hipStream_t st, const int* eid, const float* gate, long long M, int E, int* cnt, int* colpre,
                 int* total, int* off, int* pos, float* slot_gate) {
  const int nch = (int)((M + kSortChunk - 1) / kSortChunk);
  if (nch > 0) {
    hipLaunchKernelGGL(sort_count_kernel, dim3(nch), dim3(256), 0, st, eid, M, E, cnt);
    hipLaunchKernelGGL(sort_colscan_kernel, dim3(E), dim3(256), 0, st, cnt, nch, E, colpre, total);
  } else {
    hipLaunchKernelGGL(zero_ints_kernel, dim3(1), dim3(64), 0, st, total, E);
  }
  hipLaunchKernelGGL(sort_offsets_kernel, dim3(1), dim3(1), 0, st, total, E, off);
  if (nch > 0)
    hipLaunchKernelGGL(sort_scatter_kernel, dim3(nch), dim3(64), 0, st, eid, gate, M, E, off, colpre, pos,
                       slot_gate);
}

int sort_chunks(long long M) { return (int)((M + kSortChunk - 1) / kSortChunk); }

__global__ void zero_ints_kernel(int* p, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0;
}

}  // namespace janus
