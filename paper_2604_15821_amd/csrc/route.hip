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
// is made once per pair and looked up per edge.  The feature-update MoE
// routes atom tokens the same way with logits Pf[Z_i] + betaf, decided once
// per species.  Tokens are then grouped by
// expert with a stable counting sort on (expert, edge, choice), which fixes
// the slot of every (edge, choice) pair exactly.
#include "internal.h"
#include "route.h"

namespace janus {

constexpr int kSortChunk = 1024;

// Top-k (descending fp32 logit, lower index first on ties) and gates (softmax
// over all E experts, evaluated in fp64) of one logit row; l32(x) and l64(x)
// give the logit of expert x in fp32 and fp64.
template <class L32, class L64>
__device__ void topk_softmax(L32 l32, L64 l64, int E, int k, int* __restrict__ eid, float* __restrict__ gate,
                             float* __restrict__ prob) {
  float l[64];
  double mx = -1e300;
  for (int x = 0; x < E; ++x) {
    l[x] = l32(x);
    const double ld = l64(x);
    mx = ld > mx ? ld : mx;
  }
  double den = 0.0;
  for (int x = 0; x < E; ++x) den += exp(l64(x) - mx);
  for (int x = 0; x < E; ++x) prob[x] = (float)(exp(l64(x) - mx) / den);
  unsigned long long taken = 0;
  for (int c = 0; c < k; ++c) {
    int best = -1;
    for (int x = 0; x < E; ++x) {
      if (taken >> x & 1ull) continue;
      if (best < 0 || l[x] > l[best]) best = x;
    }
    taken |= 1ull << best;
    eid[c] = best;
    gate[c] = (float)(exp(l64(best) - mx) / den);
  }
}

// One thread per species pair p = a * n_species + b.
__global__ void route_pairs_kernel(const float* __restrict__ Pc, const float* __restrict__ Pn,
                                   const float* __restrict__ beta, int nsp, int E, int k,
                                   int* __restrict__ peid, float* __restrict__ pgate, float* __restrict__ pprob) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= nsp * nsp) return;
  const float* pa = Pc + (long long)(p / nsp) * E;
  const float* pb = Pn + (long long)(p % nsp) * E;
  topk_softmax([&](int x) { return __fadd_rn(__fadd_rn(pa[x], pb[x]), beta[x]); },
               [&](int x) { return ((double)pa[x] + (double)pb[x]) + (double)beta[x]; }, E, k, peid + p * k,
               pgate + p * k, pprob + (long long)p * E);
}

// Feature-update MoE, one thread per species a: logits Pf[a] + betaf.
__global__ void route_species_kernel(const float* __restrict__ Pf, const float* __restrict__ beta, int nsp, int E,
                                     int k, int* __restrict__ seid, float* __restrict__ sgate,
                                     float* __restrict__ sprob) {
  const int a = blockIdx.x * blockDim.x + threadIdx.x;
  if (a >= nsp) return;
  const float* pa = Pf + (long long)a * E;
  topk_softmax([&](int x) { return __fadd_rn(pa[x], beta[x]); },
               [&](int x) { return (double)pa[x] + (double)beta[x]; }, E, k, seid + a * k, sgate + a * k,
               sprob + (long long)a * E);
}

// Per atom: chosen experts and gates of its species.
__global__ void route_atoms_kernel(const int* __restrict__ species, int N, int k, const int* __restrict__ seid,
                                   const float* __restrict__ sgate, int* __restrict__ eid, float* __restrict__ gate) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N) return;
  const int z = species[i];
  for (int c = 0; c < k; ++c) {
    eid[(long long)i * k + c] = seid[z * k + c];
    gate[(long long)i * k + c] = sgate[z * k + c];
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

void route_atoms(hipStream_t st, const AtomRouteArgs& a) {
  hipLaunchKernelGGL(route_species_kernel, dim3(cdiv(a.nsp, 64)), dim3(64), 0, st, a.Pf, a.beta, a.nsp, a.E, a.k,
                     a.seid, a.sgate, a.sprob);
  if (a.N > 0)
    hipLaunchKernelGGL(route_atoms_kernel, dim3(cdiv(a.N, 256)), dim3(256), 0, st, a.species, a.N, a.k, a.seid,
                       a.sgate, a.eid, a.gate);
  sort_tokens(st, a.eid, a.gate, (long long)a.N * a.k, a.E, a.cnt, a.colpre, a.total, a.off, a.pos, a.slot_gate);
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
