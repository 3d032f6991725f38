// Routing launchers (route.hip).
#pragma once

#include "common.h"

namespace janus {

struct RouteArgs {
  const float* Pc;        // [nsp, E]
  const float* Pn;        // [nsp, E]
  const float* beta;      // [E]
  const int* species;     // [N]
  const int* ei;
  const int* ej;
  int Ne, nsp, E, k;
  int* peid;              // [nsp*nsp, k]  chosen experts per species pair
  float* pgate;           // [nsp*nsp, k]  their gates
  float* pprob;           // [nsp*nsp, E]  full softmax per pair
  int* pair;              // [Ne]          species pair of each edge
  int* eid;               // [Ne, k]
  float* gate;            // [Ne, k]
  int* cnt;               // [sort_chunks(Ne*k), E] scratch
  int* colpre;            // [sort_chunks(Ne*k), E] scratch
  int* total;             // [E]           tokens per expert
  int* off;               // [E+1]         first slot of each expert
  int* pos;               // [Ne, k]       slot of (edge, choice)
  float* slot_gate;       // [Ne*k]        gate of the token in each slot
};

// Routing of the atom tokens of the feature-update MoE (logits Pf[Z_i] + beta).
struct AtomRouteArgs {
  const float* Pf;        // [nsp, E]
  const float* beta;      // [E]
  const int* species;     // [N]
  int N, nsp, E, k;
  int* seid;              // [nsp, k]      chosen experts per species
  float* sgate;           // [nsp, k]      their gates
  float* sprob;           // [nsp, E]      full softmax per species
  int* eid;               // [N, k]
  float* gate;            // [N, k]
  int* cnt;               // [sort_chunks(N*k), E] scratch
  int* colpre;            // [sort_chunks(N*k), E] scratch
  int* total;             // [E]
  int* off;               // [E+1]
  int* pos;               // [N, k]        slot of (atom, choice)
  float* slot_gate;       // [N*k]
};

__global__ void zero_ints_kernel(int* p, int n);
void route_atoms(hipStream_t st, const AtomRouteArgs& a);
void route_block(hipStream_t st, const RouteArgs& a);
// Stable counting sort of M tokens (flattened (token, choice) entries with
// expert ids eid) into expert-grouped slots: total[E], off[E+1], pos[M],
// slot_gate[M]; cnt and colpre are scratch of sort_chunks(M) * E ints.
void sort_tokens(hipStream_t st, const int* eid, const float* gate, long long M, int E, int* cnt, int* colpre,
                 int* total, int* off, int* pos, float* slot_gate);
int sort_chunks(long long M);

}  // namespace janus
