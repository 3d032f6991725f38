// The training step (paper Sec. "Runtime for multi-phase double-backward
// execution"): forward to the energy, first backward to the forces, double
// backward of the force loss, final backward of the energy loss; and the
// context / layout entry points of the C ABI.
//
// The batch is processed in chunks of whole structures.  Structures only
// interact through the loss normalisation (1/S and 1/(3N) of the whole
// batch), which every chunk uses, so the chunked step computes the same
// loss, energies, forces and weight gradients as one pass over the batch;
// weight gradients and the loss accumulate over chunks in chunk order.
#include "step_kernels.h"

using namespace janus;

static thread_local int g_last_hip = 0;

int janus_set_hip_error(hipError_t e) {
  g_last_hip = (int)e;
  return JANUS_EHIP;
}

extern "C" const char* janus_strerror(int code) {
  switch (code) {
    case JANUS_OK: return "ok";
    case JANUS_EINVAL: return "invalid argument (sizes, offsets, species or edge indices)";
    case JANUS_ECAPACITY: return "edge buffers too small";
    case JANUS_ENOMEM:
      return "device allocation failed, a structure does not fit the workspace, or the sizes exceed a fixed scratch";
    case JANUS_EHIP: return "HIP runtime error";
    case JANUS_EUNSUPPORTED: return "configuration or input not supported by this library";
    default: return "unknown error";
  }
}

extern "C" int janus_create(const janus_config* cfg, janus_ctx** out) {
  if (!out) return JANUS_EINVAL;
  *out = nullptr;
  int rc = check_config(cfg);
  if (rc) return rc;
  janus_ctx* c = new janus_ctx();
  c->cfg = *cfg;
  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return JANUS_EHIP;
  }
  if (hipHostMalloc((void**)&c->host_word, 4 * sizeof(int), hipHostMallocDefault) != hipSuccess) {
    delete c;
    return JANUS_EHIP;
  }
  *out = c;
  return JANUS_OK;
}

extern "C" void janus_destroy(janus_ctx* c) {
  if (!c) return;
  if (c->ws.ptr) (void)hipFree(c->ws.ptr);
  if (c->aux.ptr) (void)hipFree(c->aux.ptr);
  if (c->nl.ptr) (void)hipFree(c->nl.ptr);
  if (c->gbuf.ptr) (void)hipFree(c->gbuf.ptr);
  if (c->host_word) (void)hipHostFree(c->host_word);
  if (c->host_plan) (void)hipHostFree(c->host_plan);
  for (hipEvent_t e : c->prof_pool) (void)hipEventDestroy(e);
  for (hipEvent_t e : c->sync_pool) (void)hipEventDestroy(e);
  if (c->side) (void)hipStreamDestroy(c->side);
  delete c;
}

extern "C" int janus_set_workspace_limit(janus_ctx* ctx, int64_t bytes) {
  if (!ctx || bytes < 0) return JANUS_EINVAL;
  ctx->ws_limit = bytes;
  return JANUS_OK;
}

extern "C" int janus_set_concurrency(janus_ctx* ctx, int on) {
  if (!ctx || (on != 0 && on != 1)) return JANUS_EINVAL;
  ctx->concurrent = on;
  return JANUS_OK;
}

extern "C" int janus_last_chunks(const janus_ctx* ctx) { return ctx ? ctx->last_chunks : 0; }
extern "C" int64_t janus_last_triplets(const janus_ctx* ctx) { return ctx ? ctx->last_triplets : 0; }

extern "C" int janus_weight_layout(const janus_config* cfg, janus_tensor_desc* out, int32_t* n_tensors,
                                   int64_t* n_floats) {
  if (!cfg || !n_tensors || !n_floats) return JANUS_EINVAL;
  int rc = check_config(cfg);
  if (rc == JANUS_EINVAL) return rc;
  Layout L = make_layout(*cfg);
  const int cap = *n_tensors;
  *n_tensors = (int)L.ents.size();
  *n_floats = L.total;
  if (!out) return JANUS_OK;
  if (cap < (int)L.ents.size()) return JANUS_EINVAL;
  for (size_t q = 0; q < L.ents.size(); ++q) {
    std::memset(&out[q], 0, sizeof(janus_tensor_desc));
    std::strncpy(out[q].name, L.ents[q].name.c_str(), sizeof(out[q].name) - 1);
    out[q].offset = L.ents[q].off;
    out[q].ndim = L.ents[q].ndim;
    for (int k = 0; k < 3; ++k) out[q].shape[k] = L.ents[q].shape[k];
  }
  return JANUS_OK;
}

#define JANUS_CAT2(a, b) a##b
#define JANUS_CAT(a, b) JANUS_CAT2(a, b)
#define PROF(cls, fl, by) ProfScope JANUS_CAT(ps_, __LINE__)(ctx, st, cls, (double)(fl), (double)(by))
#define PROFS(strm, cls, fl, by) ProfScope JANUS_CAT(ps_, __LINE__)(ctx, strm, cls, (double)(fl), (double)(by))

namespace {

__global__ void add_ints_kernel(int* __restrict__ dst, const int* __restrict__ src, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) dst[i] += src[i];
}

// One chunk: structures [s0, s0+S), atoms [a0, a0+N), edges [e0, e0+Ne).
struct ChunkArgs {
  int s0, a0, S, N;
  long long e0, Ne;
  int S_tot, N_tot;
  long long Ne_tot;
  int index;
  long long Nt;                  // triplets of the chunk (three-body term)
  long long t0, Nt_tot;          // first triplet of the chunk, triplets of the batch
  const unsigned char* tshort;   // whole-batch short-bond flags
  // robust loss: ROBUST_ONE (the batch is this one chunk: base losses, statistics
  // and seeds here), ROBUST_LOSSES (forward and force backward only, then this
  // chunk's base losses), ROBUST_SEEDS (seeds from the batch statistics, then the
  // double and final backward); robust_g: whole-batch [S] base losses, [S] dL/dL_s,
  // then the loss
  int robust_mode;
  double* robust_g;
};
enum { ROBUST_OFF = 0, ROBUST_ONE, ROBUST_LOSSES, ROBUST_SEEDS };

__global__ void copy_add_kernel(int* __restrict__ dst, const int* __restrict__ src, long long n, int add) {
  const long long q = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (q < n) dst[q] = src[q] + add;
}

int run_chunk(janus_ctx* ctx, hipStream_t st, Plan& p, const Layout& L, const ChunkArgs& ca, const float* pos_g,
              const float* cell_g, const int32_t* species_g, const int32_t* offsets_g, const janus_edges* nl,
              const float* W, const float* E_ref_g, const float* F_ref_g, const float* S_ref_g,
              const janus_labels* labels, double* loss_part, float* E_g, float* F_g, float* stress_g, float* dLdW,
              float* dLdR_g, const janus_debug* dbg) {
  const janus_config& cfg = ctx->cfg;
  const int T = p.T, Ee = p.E, k = p.k, d = p.d, h = p.hdim, nb = p.nb, nsp = p.nsp;
  const int N = ca.N, S = ca.S;
  const long long Ne = ca.Ne, M = p.M, Nd = (long long)N * d;

  // chunk views of the caller's arrays
  const float* pos = pos_g + 3LL * ca.a0;
  const float* cell = cell_g + 9LL * ca.s0;
  const int* species = species_g + ca.a0;
  const int8_t* shift = nl->shift ? nl->shift + 3 * ca.e0 : nullptr;
  const float* E_ref = E_ref_g + ca.s0;
  const float* F_ref = F_ref_g + 3LL * ca.a0;
  float* E = E_g + ca.s0;
  float* F = F_g + 3LL * ca.a0;
  const float* S_ref = S_ref_g ? S_ref_g + 9LL * ca.s0 : nullptr;
  float* stress_out = stress_g ? stress_g + 9LL * ca.s0 : nullptr;
  {
    PROF(PROF_OTHER, 0, Ne * 24.0);
    const long long nthr = std::max<long long>(Ne, std::max(N, S) + 1);
    hipLaunchKernelGGL(rebase_kernel, dim3(cdiv(nthr, 256)), dim3(256), 0, st, nl->ei, nl->ej, nl->rev, nl->rowptr,
                       offsets_g, ca.a0, (int)ca.e0, ca.s0, N, Ne, S, p.cei, p.cej, p.crev, p.crow, p.coff);
    launch_atom_struct(st, p.coff, S, N, p.sid);
  }
  const int* ei = p.cei;
  const int* ej = p.cej;
  const int* rowptr = p.crow;
  const int* rev = p.crev;
  const int* offsets = p.coff;

  auto Wp = [&](const std::string& n) { return W + L.at(n); };
  auto Gp = [&](const std::string& n) { return dLdW + L.at(n); };
  auto blk = [](int t, const char* n) { return "blocks." + std::to_string(t) + "." + n; };
  const size_t ldsW = (size_t)nb * d * sizeof(float);
  const dim3 gE = wave_grid(Ne), gN = wave_grid(N), b256(256);
  // kernels that stage W_a (up to 64 KB) in LDS: at most 4 workgroups per CU
  // fit, so a larger grid would only reload W_a
  const dim3 gEa(std::min(gE.x, 1024u));
  // the same with 8 waves per workgroup sharing one copy of W_a, for the triplet kernel
  // whose registers would allow 8 waves per SIMD (the dispatch of the triplet tokens)
  const dim3 gEa8(std::min((unsigned)cdiv(std::max<long long>(Ne, 1), 8), 1024u)), b512(512);

  // algorithmic work of one launch of each kernel (matrix products: 2 M N K;
  // memory-bound kernels: bytes that must cross HBM once)
  const double f_exp = 2.0 * M * d * h;
  const double f_dense = 2.0 * N * d * d;
  const double f_filt = 2.0 * Ne * nb * d;
  const double by_dispatch = Ne * (4.0 * nb + 4.0 * d + 4.0 * k + 4.0 + 4.0 * k * d);
  const double by_combine = N * 8.0 * d + Ne * (4.0 * k + 4.0 * k * d);
  const double by_gather = N * 4.0 * d + Ne * k * (8.0 + 4.0 * d);
  const double by_p2 = Ne * (4.0 * k * d + 4.0 * k + 8.0 * nb + 16.0 * d + 12.0);
  const double by_scatter = N * 12.0 * d + Ne * (4.0 + 4.0 * d);
  const double by_p3 = Ne * (8.0 * nb + 16.0 * d + 8.0 + 4.0 * k + 4.0 * k * d) + (p.three ? Ne * 8.0 * d : 0.0);
  const double by_cp3 = N * 12.0 * d + Ne * k * (16.0 + 4.0 * d);
  const double by_p4 = Ne * (4.0 * k * d + 4.0 * k + 4.0 * nb + 20.0 * d);

  // ---- setup: geometry, species groups, routing of every block, GEMM tables
  const bool three = p.three != 0;
  const long long Nt = p.Nt, M3 = p.M3;
  const int E3 = p.E3, k3 = p.k3, h3 = p.hd3, L3 = p.L3, nf = p.nf;
  const bool atom = p.atom != 0;
  const long long Mf = p.Mf;
  const int Ef = p.Ef, kf = p.kf, hf = p.hdf;
  if (atom) hipLaunchKernelGGL(iota_kernel, dim3(cdiv(N + 1, 256)), dim3(256), 0, st, p.iota, N);
  const bool attn = p.attn != 0;
  const int H = p.H;
  // head width: the register-resident kernels (heads of 32 columns, neighbourhoods of
  // up to kAttnMfmaN edges) and the tiled sweeps beside them; wider heads take the
  // tiled sweeps for every atom (nmin = -1)
  const int dh = attn ? d / H : 0;
  const bool attn_reg = dh == kAttnDh;
  const int nmin = attn_reg ? kAttnMfmaN : -1;
#define JANUS_ATTN_TILED(kern, ...)                                                    \
  do {                                                                                 \
    if (dh == 32)                                                                      \
      hipLaunchKernelGGL(kern<32>, gNH, b256, 0, st, __VA_ARGS__);                     \
    else if (dh == 64)                                                                 \
      hipLaunchKernelGGL(kern<64>, gNH, b256, 0, st, __VA_ARGS__);                     \
    else                                                                               \
      hipLaunchKernelGGL(kern<128>, gNH, b256, 0, st, __VA_ARGS__);                    \
  } while (0)
  {
    PROF(PROF_GRAPH, 0, Ne * (12.0 + 3.0 + 16.0 + 8.0 * nb));
    launch_geometry(st, pos, cell, p.sid, ei, ej, shift, (int)Ne, cfg.r_cut, nb, p.geo, p.B, p.dB,
                    three ? cfg.r_cut3 : 0.f, p.B3, p.dB3, p.u3, p.du3, p.d2B);
  }
  if (three) {
    // triplets of the chunk: CSR by first edge, reverse map, cosines
    PROF(PROF_GRAPH, 0, Ne * 8.0 + Nt * (16.0 + 4.0 * nf));
    const unsigned char* tsh = ca.tshort + ca.e0;
    hipLaunchKernelGGL(tri_count_kernel, dim3(cdiv(N, 256)), dim3(256), 0, st, rowptr, tsh, N, p.tcount);
    launch_exclusive_scan(st, p.tcount, (int)Ne, p.trow, nullptr, p.scan);
    if (Nt > 0) {
      hipLaunchKernelGGL(tri_write_kernel, dim3(cdiv(Ne, 256)), dim3(256), 0, st, ei, rowptr, tsh,
                         (const int*)p.trow, Ne, p.te, p.te2);
      hipLaunchKernelGGL(tri_rev_kernel, dim3(cdiv(Nt, 256)), dim3(256), 0, st, (const int*)p.te,
                         (const int*)p.te2, (const int*)p.trow, (const float4*)p.geo, Nt, p.trev, p.tc);
      hipLaunchKernelGGL(tri_lane_kernel, dim3(cdiv(Nt, 256)), dim3(256), 0, st, (const int*)p.trev,
                         (const int*)p.te, (const float*)p.tc, (const float*)p.u3, (const float*)p.du3, Nt,
                         p.tlane);
      // feature rows G of every triplet, for dW_a of the final backward
      hipLaunchKernelGGL(tri_features_kernel, dim3(cdiv(Nt * (nf / 4), 256)), dim3(256), 0, st,
                         LoadTriFeat{p.te, p.te2, p.tc, p.B3, p.dB3, p.u3, p.du3, nullptr, nb}, Nt, nf, p.G3f);
    }
    hipLaunchKernelGGL(set_rows_kernel, dim3(1), dim3(64), 0, st, p.rowT, (int)Nt, p.rowT, Nt);
    build_tables(st, p.rowT, 1, p.kcT, p.tilesT, p.ntT, p.chunksT, p.ncT, p.cfT);
  }
  const long long np = (long long)nsp * nsp;
  {
    PROF(PROF_ROUTE, 0, T * (Ne * (8.0 + 24.0 * k)));
    hipLaunchKernelGGL(species_count_kernel, dim3(nsp), dim3(64), 0, st, species, N, nsp, p.sp_cnt);
    launch_exclusive_scan(st, p.sp_cnt, nsp, p.sp_off, nullptr, p.scan);
    hipLaunchKernelGGL(species_write_kernel, dim3(nsp), dim3(64), 0, st, species, N, p.sp_off, p.sp_atoms);
    hipLaunchKernelGGL(set_rows_kernel, dim3(1), dim3(64), 0, st, p.rowN, N, p.rowE, Ne);
    build_tables(st, p.rowN, 1, p.kcN, p.tilesN, p.ntN, p.chunksN, p.ncN, p.cfN);
    build_tables(st, p.rowE, 1, p.kcE, nullptr, nullptr, p.chunksE, p.ncE, p.cfE);
    if (p.rf) {
      // routing on the edge tokens: products over the edges, the identity slot map,
      // gates of one, the zero-padded router weights and their gradient accumulators
      build_tables(st, p.rowE, 1, p.kcR, p.tilesE, p.ntE, p.chunksR, p.ncR, p.cfR);
      hipLaunchKernelGGL(iota_kernel, dim3(cdiv(Ne + 1, 256)), dim3(256), 0, st, p.iotaE, (int)Ne);
      hipLaunchKernelGGL(fill_kernel, dim3(cdiv(M + 1, 256)), dim3(256), 0, st, p.ones, M + 1, 1.f);
      for (int t = 0; t < T; ++t)
        hipLaunchKernelGGL(wr_pad_kernel, dim3(cdiv((long long)d * p.Ep, 256)), dim3(256), 0, st,
                           Wp(blk(t, "Wr")), d, Ee, p.Ep, p.WrP + (long long)t * d * p.Ep);
      JANUS_HIP_TRY(hipMemsetAsync(p.dWrP, 0, sizeof(float) * T * d * p.Ep, st));
    }
    if (attn) {
      build_tables(st, p.rowE, 1, p.kcA, p.tilesE, p.ntE, p.chunksA, p.ncA, p.cfA);
      if (Ne > 0)
        hipLaunchKernelGGL(attn_env_kernel, dim3(cdiv(Ne, 256)), dim3(256), 0, st, (const float4*)p.geo, Ne,
                           cfg.r_cut, p.eu, p.eud);
    }
    for (int t = 0; t < T; ++t) {
      RouteArgs ra;
      ra.Pc = Wp(blk(t, "Pc"));
      ra.Pn = Wp(blk(t, "Pn"));
      ra.beta = Wp(blk(t, "beta"));
      ra.species = species;
      ra.ei = ei;
      ra.ej = ej;
      ra.Ne = (int)Ne;
      ra.nsp = nsp;
      ra.E = Ee;
      ra.k = k;
      ra.peid = p.peid + t * np * k;
      ra.pgate = p.pgate + t * np * k;
      ra.pprob = p.pprob + t * np * Ee;
      ra.pair = p.pair + t * Ne;
      ra.eid = p.eid + t * M;
      ra.gate = p.gate + t * M;
      ra.cnt = p.cnt;
      ra.colpre = p.colpre;
      ra.total = p.total + t * Ee;
      ra.off = p.off + t * (Ee + 1);
      ra.pos = p.pos + t * M;
      ra.slot_gate = p.slot_gate + t * M;
      if (!p.rf) {   // routing on the edge tokens is decided in the forward pass
        route_block(st, ra);
        build_tables(st, ra.off, Ee, p.kc, p.tiles + (long long)t * p.mt, p.ntiles + t,
                     p.chunks + (long long)t * p.mc, p.nchunks + t, p.cfirst + t * (Ee + 1));
      }
      if (three) {
        if (Nt > 0)
          hipLaunchKernelGGL(tri_route_kernel, dim3(cdiv(Nt, 128)), dim3(128), 0, st, species, ei, ej,
                             (const int*)p.te, (const int*)p.te2, Nt, Wp(blk(t, "P3a")), Wp(blk(t, "P3b")),
                             Wp(blk(t, "P3c")), Wp(blk(t, "beta3")), E3, k3, p.eid3 + t * M3, p.gate3 + t * M3);
        sort_tokens(st, p.eid3 + t * M3, p.gate3 + t * M3, M3, E3, p.cnt3, p.colpre3, p.total3 + t * E3,
                    p.off3 + t * (E3 + 1), p.pos3 + t * M3, p.slot_gate3 + t * M3);
        if (Nt > 0)
          hipLaunchKernelGGL(tri_pos_rev_kernel, dim3(cdiv(Nt, 256)), dim3(256), 0, st, (const int*)p.trev,
                             (const int*)(p.pos3 + t * M3), Nt, k3, p.pos3r + t * M3);
        build_tables(st, p.off3 + t * (E3 + 1), E3, p.kc3, p.tiles3 + (long long)t * p.mt3, p.ntiles3 + t,
                     p.chunks3 + (long long)t * p.mc3, p.nchunks3 + t, p.cfirst3 + t * (E3 + 1));
      }
      if (atom) {
        AtomRouteArgs fa;
        fa.Pf = Wp(blk(t, "Pf"));
        fa.beta = Wp(blk(t, "betaf"));
        fa.species = species;
        fa.N = N;
        fa.nsp = nsp;
        fa.E = Ef;
        fa.k = kf;
        fa.seid = p.seid + (long long)t * nsp * kf;
        fa.sgate = p.sgate + (long long)t * nsp * kf;
        fa.sprob = p.sprob + (long long)t * nsp * Ef;
        fa.eid = p.eidf + t * Mf;
        fa.gate = p.gatef + t * Mf;
        fa.cnt = p.cntf;
        fa.colpre = p.colpref;
        fa.total = p.totalf + t * Ef;
        fa.off = p.offf + t * (Ef + 1);
        fa.pos = p.posf + t * Mf;
        fa.slot_gate = p.slot_gatef + t * Mf;
        route_atoms(st, fa);
        build_tables(st, fa.off, Ef, p.kcf, p.tilesf + (long long)t * p.mtf, p.ntilesf + t,
                     p.chunksf + (long long)t * p.mcf, p.nchunksf + t, p.cfirstf + t * (Ef + 1));
      }
    }
  }
  JANUS_HIP_TRY(hipGetLastError());

  // triplet views of block t
  auto POS3 = [&](int t) { return (const int*)(p.pos3 + t * M3); };
  auto POS3R = [&](int t) { return (const int*)(p.pos3r + t * M3); };
  auto GATE3 = [&](int t) { return (const float*)(p.gate3 + t * M3); };
  auto SG3 = [&](int t) { return (const float*)(p.slot_gate3 + t * M3); };
  auto TL3 = [&](int t) { return (const RowsTile*)(p.tiles3 + (long long)t * p.mt3); };
  auto CH3 = [&](int t) { return (const WChunk*)(p.chunks3 + (long long)t * p.mc3); };
  auto CF3 = [&](int t) { return (const int*)(p.cfirst3 + t * (E3 + 1)); };
  auto Z3s = [&](int t) { return p.Z3s + t * M3 * d; };
  auto A3 = [&](int t) { return p.A3 + t * M3 * h3; };
  auto S3b = [&](int t) { return p.S3b + t * M3 * h3; };
  auto A3b = [&](int t) { return p.A3b + t * M3 * h3; };
  auto Y3bs = [&](int t) { return p.Y3bs + t * M3 * d; };
  auto Zbar3 = [&](int t) { return p.Zbar3 + t * Nt * d; };
  const size_t ldsWa = (size_t)nf * d * sizeof(float);
  const double f_tri = 2.0 * M3 * d * h3;
  const double f_wa = 2.0 * Nt * nf * d;
  // per triplet: indices, cosine, u3, slot positions; per edge e2: segment, basis rows, h_j2
  const double by_tri_idx = Nt * (16.0 + 4.0 * k3) + Ne * (8.0 + 4.0 * nb + 4.0 * d);

  // per-block views
  auto Xs = [&](int t) { return p.Xs + t * M * d; };
  auto Ab = [&](int t) { return p.Ab + t * M * h; };
  auto Aa = [&](int t) { return p.A + t * M * h; };
  auto Sb = [&](int t) { return p.Sb + t * M * h; };
  auto Ybs = [&](int t) { return p.Ybs + t * M * d; };
  auto Xbar = [&](int t) { return p.Xbar + t * Ne * d; };
  auto Fbar = [&](int t) { return p.Fbar + t * Ne * d; };
  auto POS = [&](int t) { return (const int*)(p.pos + t * M); };
  auto GATE = [&](int t) { return (const float*)(p.gate + t * M); };
  auto SG = [&](int t) { return (const float*)(p.slot_gate + t * M); };
  // routing on the edge tokens, block t
  const long long Ep = p.Ep, sEdR = Ne * d + 4, sEp = Ne * Ep + 4;
  auto EID = [&](int t) { return (const int*)(p.eid + t * M); };
  auto XeR = [&](int t) { return p.Xe + t * sEdR; };
  auto YstR = [&](int t) { return p.Yst + t * (M * d + 4); };
  auto FPR = [&](int t) { return p.fprob + t * sEp; };
  auto GBR = [&](int t) { return p.gbar + t * M; };
  auto LBR = [&](int t) { return p.lbar + t * sEp; };
  auto P3R = [&](int t) { return p.P3 + t * sEp; };
  auto GHR = [&](int t) { return p.gh + t * M; };
  auto WRP = [&](int t) { return (const float*)(p.WrP + (long long)t * d * Ep); };
  auto DWR = [&](int t) { return p.dWrP + (long long)t * d * Ep; };
  auto TL = [&](int t) { return (const RowsTile*)(p.tiles + (long long)t * p.mt); };
  auto CH = [&](int t) { return (const WChunk*)(p.chunks + (long long)t * p.mc); };
  auto CF = [&](int t) { return (const int*)(p.cfirst + t * (Ee + 1)); };
  auto HV = [&](float* base, int t) { return base + t * Nd; };

  // feature-update MoE views of block t (atom tokens; the identity CSR p.iota
  // lets the per-atom gather / combine kernels serve one token per atom)
  auto POSF = [&](int t) { return (const int*)(p.posf + t * Mf); };
  auto GATEF = [&](int t) { return (const float*)(p.gatef + t * Mf); };
  auto SGF = [&](int t) { return (const float*)(p.slot_gatef + t * Mf); };
  auto TLF = [&](int t) { return (const RowsTile*)(p.tilesf + (long long)t * p.mtf); };
  auto CHF = [&](int t) { return (const WChunk*)(p.chunksf + (long long)t * p.mcf); };
  auto CFF = [&](int t) { return (const int*)(p.cfirstf + t * (Ef + 1)); };
  auto Xsf = [&](int t) { return p.Xsf + t * Mf * d; };
  auto Af = [&](int t) { return p.Af + t * Mf * hf; };
  auto Sbf = [&](int t) { return p.Sbf + t * Mf * hf; };
  auto Abf = [&](int t) { return p.Abf + t * Mf * hf; };
  auto Ybf = [&](int t) { return p.Ybf + t * Mf * d; };
  auto UU = [&](int t) { return p.uu + t * Nd; };
  const int* iota = p.iota;

  // attention views of block t
  const long long sEd = Ne * d + 4, sE3 = 3 * Ne * d + 4, sNd = Nd + 4, sSt = 2 * Ne * H + 4;
  auto MM = [&](int t) { return p.Mm + t * sEd; };
  auto QKVt = [&](int t) { return p.QKV + t * sE3; };
  auto STt = [&](int t) { return p.stats + t * sSt; };
  auto OSt = [&](int t) { return p.osum + t * sNd; };
  auto OBt = [&](int t) { return p.OB + t * sNd; };
  auto QKVbt = [&](int t) { return p.QKVb + t * sE3; };
  auto MBt = [&](int t) { return p.MB + t * sEd; };
  auto MHt = [&](int t) { return p.Mh + t * sEd; };
  auto QKVht = [&](int t) { return p.QKVh + t * sE3; };
  const double f_qkv = 6.0 * Ne * d * d;
  const dim3 gNH = wave_grid((long long)N * (H > 0 ? H : 1));
  const double by_attn = Ne * (12.0 * d + 8.0 * H + 8.0) + N * 8.0 * d;
  const double f_atm = 2.0 * Mf * d * hf;
  const double by_fgather = N * 4.0 * d + Mf * (8.0 + 4.0 * d);
  const double by_fcombine = N * 8.0 * d + Mf * (4.0 + 4.0 * d);

  // ---- phase 1: forward
  {
    PROF(PROF_OTHER, 0, 8.0 * Nd);
    hipLaunchKernelGGL(species_rows_gather_kernel, dim3(cdiv(Nd, 256)), b256, 0, st, Wp("A"), species, N, d, p.h);
    if (cfg.n_tasks) {
      // h0 += task, charge, spin and composition embedding of the atom's structure
      LAUNCH_VPL(struct_embed_kernel, d, wave_grid(S), b256, 0, st, labels->task + ca.s0, labels->charge + ca.s0,
                 labels->spin + ca.s0, offsets, species, Wp("Tk"), Wp("Qe"), Wp("Se"), Wp("Wc"), S, d, p.gs);
      hipLaunchKernelGGL(add_struct_rows_kernel, dim3(cdiv(Nd, 256)), b256, 0, st, (const float*)p.gs,
                         (const int*)p.sid, N, d, p.h);
    }
  }
  for (int t = 0; t < T; ++t) {
    const float* Wb = Wp(blk(t, "W_b"));
    const float* W1 = Wp(blk(t, "W1"));
    const float* W2 = Wp(blk(t, "W2"));
    if (three && Nt > 0) {
      // triplet tokens -> triplet experts -> messages Q_e of each edge's triplets
      {
        PROF(PROF_EDGE, 0, by_tri_idx + Nt * 4.0 * k3 * d);
        LAUNCH_VPL_K(tri_dispatch_kernel, d, k3, gEa8, b512, ldsWa, st, (const int*)p.trow,
                     (const float4*)p.tlane, (const float*)p.B3, Wp(blk(t, "W_a")), nb, L3, ej,
                     (const float*)HV(p.h, t), POS3R(t), Ne, d, Z3s(t));
      }
      {
        PROF(PROF_EXPERT_GEMM, f_tri, 0);
        launch_rows<false>(st, LoadPlain{Z3s(t), d}, Wp(blk(t, "W1a")), d, h3, TL3(t), p.ntiles3 + t, p.mt3,
                           EpiStore{A3(t), h3});
      }
      {
        PROF(PROF_EXPERT_GEMM, f_tri, 0);
        launch_rows<false>(st, LoadSilu{A3(t), h3}, Wp(blk(t, "W2a")), h3, d, TL3(t), p.ntiles3 + t, p.mt3,
                           EpiRowScale{p.T3a, SG3(t), d});
      }
      {
        PROF(PROF_EDGE, 0, Ne * 8.0 * d + M3 * 4.0 * d);
        LAUNCH_VPL_K(tri_combine_kernel, d, k3, gE, b256, 0, st, (const int*)p.trow, POS3(t), (const float*)p.T3a,
                     Ne, d, p.Q);
      }
    }
    if (p.rf) {
      // edge tokens -> router logits -> top-k, gates, expert-grouped slots (block t's routing)
      {
        PROF(PROF_EDGE, 0, Ne * (4.0 * nb + 8.0 * d));
        if (Ne > 0)
          LAUNCH_VPL_K(dispatch_x_kernel, d, 1, gE, b256, ldsW, st, (const float*)p.B, nb, Wb,
                       (const float*)HV(p.h, t), ej, (const int*)p.iotaE, Ne, d, XeR(t),
                       (const float*)(three && Nt > 0 ? p.Q : nullptr));
      }
      {
        PROF(PROF_ROUTE, 2.0 * Ne * d * Ep, Ne * (4.0 * d + 4.0 * Ep));
        launch_rows<false>(st, LoadPlain{XeR(t), d}, WRP(t), d, (int)Ep, p.tilesE, p.ntE, p.mtE,
                           EpiStore{p.Lw, Ep});
        float* gap = dbg && dbg->gap ? dbg->gap + t * ca.Ne_tot + ca.e0 : nullptr;
        if (Ne > 0)
          hipLaunchKernelGGL(feat_route_kernel, dim3(cdiv(Ne, 256)), b256, 0, st, (const float*)p.Lw, species, ei, ej,
                             Wp(blk(t, "Pc")), Wp(blk(t, "Pn")), Wp(blk(t, "beta")), Ne, Ee, (int)Ep, k,
                             p.eid + t * M, p.gate + t * M, FPR(t), gap);
        sort_tokens(st, p.eid + t * M, p.gate + t * M, M, Ee, p.cnt, p.colpre, p.total + t * Ee, p.off + t * (Ee + 1),
                    p.pos + t * M, p.slot_gate + t * M);
        build_tables(st, p.off + t * (Ee + 1), Ee, p.kc, p.tiles + (long long)t * p.mt, p.ntiles + t,
                     p.chunks + (long long)t * p.mc, p.nchunks + t, p.cfirst + t * (Ee + 1));
      }
      if (Ne > 0) {
        PROF(PROF_EDGE, 0, Ne * (4.0 * d + 8.0 * k + 4.0 * k * d));
        LAUNCH_VPL_K(edge_gather_kernel, d, k, gE, b256, 0, st, POS(t), (const float*)nullptr,
                     (const float*)XeR(t), Ne, d, Xs(t));
      }
    } else if (Ne > 0) {
      PROF(PROF_EDGE, 0, by_dispatch);
      LAUNCH_VPL_K(dispatch_x_kernel, d, k, gE, b256, ldsW, st, (const float*)p.B, nb, Wb, (const float*)HV(p.h, t), ej,
                 POS(t), Ne, d, Xs(t), (const float*)(three && Nt > 0 ? p.Q : nullptr));
    }
    {
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      launch_rows<false>(st, LoadPlain{Xs(t), d}, W1, d, h, TL(t), p.ntiles + t, p.mt, EpiStore{Aa(t), h});
    }
    {
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      if (p.rf)   // expert outputs before gating (the gates' adjoints need them)
        launch_rows<false>(st, LoadSilu{Aa(t), h}, W2, h, d, TL(t), p.ntiles + t, p.mt, EpiStore{YstR(t), d});
      else
        launch_rows<false>(st, LoadSilu{Aa(t), h}, W2, h, d, TL(t), p.ntiles + t, p.mt, EpiRowScale{p.T1, SG(t), d});
    }
    // u = h + messages (h^{t+1} itself without the feature-update MoE)
    float* u_out = atom ? p.ut : HV(p.h, t + 1);
    if (attn) {
      // messages per edge -> q|k|v -> attention over each neighbourhood -> u = h + osum Wo
      {
        PROF(PROF_EDGE, 0, Ne * (4.0 * k + 4.0 * k * d + 4.0 * d));
        if (p.rf)   // the expert outputs are stored before gating: gate them here
          LAUNCH_VPL_K(combine_fwd_gated_kernel, d, k, gE, b256, 0, st, (const int*)p.iotaE, POS(t), GATE(t),
                       (const float*)YstR(t), (const float*)nullptr, Ne, d, MM(t));
        else
          LAUNCH_VPL_K(edge_sum_kernel, d, k, gE, b256, 0, st, POS(t), (const float*)p.T1, Ne, d, MM(t));
      }
      {
        PROF(PROF_DENSE_GEMM, f_qkv, 0);
        launch_rows<false>(st, LoadPlain{MM(t), d}, Wp(blk(t, "Wqkv")), d, 3 * d, p.tilesE, p.ntE, p.mtE,
                           EpiStore{QKVt(t), 3LL * d});
      }
      {
        PROF(PROF_ATTN, 0, by_attn);
        // neighbourhoods up to kAttnMfmaN edges on register-resident tiles, larger ones on tiled sweeps
        if (attn_reg) {
          hipLaunchKernelGGL(attn_fwd_mfma_kernel<1>, gNH, b256, 0, st, rowptr, (const float*)QKVt(t),
                             (const float*)p.eu, N, d, H, STt(t), OSt(t));
          if (2 <= kAttnTiles)
            hipLaunchKernelGGL(attn_fwd_mfma_kernel<2>, gNH, b256, 0, st, rowptr, (const float*)QKVt(t),
                               (const float*)p.eu, N, d, H, STt(t), OSt(t));
          if (3 <= kAttnTiles)
            hipLaunchKernelGGL(attn_fwd_mfma_kernel<3>, gNH, b256, 0, st, rowptr, (const float*)QKVt(t),
                               (const float*)p.eu, N, d, H, STt(t), OSt(t));
          if (4 <= kAttnTiles)
            hipLaunchKernelGGL(attn_fwd_mfma_kernel<4>, gNH, b256, 0, st, rowptr, (const float*)QKVt(t),
                               (const float*)p.eu, N, d, H, STt(t), OSt(t));
        }
        JANUS_ATTN_TILED(attn_fwd_tiled_kernel, rowptr, (const float*)QKVt(t), (const float*)p.eu, N, d, H, nmin,
                         STt(t), OSt(t));
      }
      {
        PROF(PROF_DENSE_GEMM, f_dense, 0);
        launch_rows<false>(st, LoadPlain{OSt(t), d}, Wp(blk(t, "Wo")), d, d, p.tilesN, p.ntN, p.mtN,
                           EpiAdd{u_out, HV(p.h, t), d});
      }
    } else if (p.rf) {
      PROF(PROF_ATOM, 0, by_combine + Ne * 4.0 * k);
      LAUNCH_VPL_K(combine_fwd_gated_kernel, d, k, gN, b256, 0, st, rowptr, POS(t), GATE(t), (const float*)YstR(t),
                   (const float*)HV(p.h, t), N, d, u_out);
    } else {
      PROF(PROF_ATOM, 0, by_combine);
      LAUNCH_VPL_K(combine_fwd_kernel, d, k, gN, b256, 0, st, rowptr, POS(t), (const float*)p.T1,
                 (const float*)HV(p.h, t), N, d, u_out);
    }
    if (atom) {
      // feature-update MoE: h^{t+1} = u + sum_c g W2f^T SiLU(W1f^T u)
      const float* W1f = Wp(blk(t, "W1f"));
      const float* W2f = Wp(blk(t, "W2f"));
      {
        PROF(PROF_ATOM, 0, by_fgather);
        LAUNCH_VPL_K(gather_atom_kernel, d, kf, gN, b256, 0, st, iota, POSF(t), (const float*)nullptr,
                     (const float*)p.ut, N, d, Xsf(t));
      }
      {
        PROF(PROF_EXPERT_GEMM, f_atm, 0);
        launch_rows<false>(st, LoadPlain{Xsf(t), d}, W1f, d, hf, TLF(t), p.ntilesf + t, p.mtf, EpiStore{Af(t), hf});
      }
      {
        PROF(PROF_EXPERT_GEMM, f_atm, 0);
        launch_rows<false>(st, LoadSilu{Af(t), hf}, W2f, hf, d, TLF(t), p.ntilesf + t, p.mtf,
                           EpiRowScale{p.T1f, SGF(t), d});
      }
      {
        PROF(PROF_ATOM, 0, by_fcombine);
        LAUNCH_VPL_K(combine_fwd_kernel, d, kf, gN, b256, 0, st, iota, POSF(t), (const float*)p.T1f,
                     (const float*)p.ut, N, d, HV(p.h, t + 1));
      }
    }
  }
  const float* Wo1 = Wp("W_o1");
  const float* wo2 = Wp("w_o2");
  const float* hT = HV(p.h, T);
  {
    PROF(PROF_DENSE_GEMM, f_dense, 0);
    launch_rows<false>(st, LoadPlain{hT, d}, Wo1, d, d, p.tilesN, p.ntN, p.mtN, EpiDense{p.z, d});
  }
  {
    PROF(PROF_OTHER, 0, 4.0 * Nd);
    LAUNCH_VPL(readout_kernel, d, gN, b256, 0, st, (const float*)p.z, wo2, N, d, p.eps);
    hipLaunchKernelGGL(energy_kernel, wave_grid(S), b256, 0, st, (const float*)p.eps, offsets, S, p.Ed, E);
  }

  // ---- phase 2: force backward (hh[t] = dE/dh^t)
  {
    PROF(PROF_DENSE_GEMM, f_dense, 0);
    launch_rows<true>(st, LoadSiluD1Scaled{p.z, wo2, d}, Wo1, d, d, p.tilesN, p.ntN, p.mtN,
                      EpiDense{HV(p.hh, T), d});
  }
  JANUS_HIP_TRY(hipMemsetAsync(p.rbar, 0, sizeof(float) * std::max<long long>(Ne, 1), st));
  if (three) JANUS_HIP_TRY(hipMemsetAsync(p.tacc, 0, sizeof(float4) * (Nt + 1), st));
  for (int t = T - 1; t >= 0; --t) {
    const float* Wb = Wp(blk(t, "W_b"));
    const float* W1 = Wp(blk(t, "W1"));
    const float* W2 = Wp(blk(t, "W2"));
    // dE/du of the message update (dE/dh^{t+1} without the feature-update MoE)
    const float* hbar_u = HV(p.hh, t + 1);
    if (atom) {
      const float* W1f = Wp(blk(t, "W1f"));
      const float* W2f = Wp(blk(t, "W2f"));
      {
        PROF(PROF_ATOM, 0, by_fgather);
        LAUNCH_VPL_K(gather_atom_kernel, d, kf, gN, b256, 0, st, iota, POSF(t), GATEF(t),
                     (const float*)HV(p.hh, t + 1), N, d, Ybf(t));
      }
      {
        PROF(PROF_EXPERT_GEMM, f_atm, 0);
        launch_rows<true>(st, LoadPlain{Ybf(t), d}, W2f, d, hf, TLF(t), p.ntilesf + t, p.mtf,
                          EpiP2{Af(t), Sbf(t), Abf(t), hf});
      }
      {
        PROF(PROF_EXPERT_GEMM, f_atm, 0);
        launch_rows<true>(st, LoadPlain{Abf(t), hf}, W1f, hf, d, TLF(t), p.ntilesf + t, p.mtf, EpiStore{p.T1f, d});
      }
      {
        PROF(PROF_ATOM, 0, by_fcombine);
        LAUNCH_VPL_K(combine_fwd_kernel, d, kf, gN, b256, 0, st, iota, POSF(t), (const float*)p.T1f,
                     (const float*)HV(p.hh, t + 1), N, d, UU(t));
      }
      hbar_u = UU(t);
    }
    if (attn) {
      // adjoint of osum (ob = dE/du Wo^T) -> attention backward -> message adjoints -> slots
      {
        PROF(PROF_DENSE_GEMM, f_dense, 0);
        launch_rows<true>(st, LoadPlain{hbar_u, d}, Wp(blk(t, "Wo")), d, d, p.tilesN, p.ntN, p.mtN,
                          EpiStore{OBt(t), d});
      }
      {
        PROF(PROF_ATTN, 0, by_attn);
        // neighbourhoods up to kAttnMfmaN edges on register-resident tiles, larger ones on tiled sweeps
#define JANUS_BWD_MFMA(NTV)                                                                                    \
  hipLaunchKernelGGL(attn_bwd_mfma_kernel<NTV>, gNH, b256, 0, st, rowptr, (const float*)QKVt(t),                \
                     (const float*)p.eu, (const float*)STt(t), (const float*)OBt(t), N, d, H, QKVbt(t), p.rbh)
        if (attn_reg) {
          JANUS_BWD_MFMA(1);
          if (2 <= kAttnTiles) JANUS_BWD_MFMA(2);
          if (3 <= kAttnTiles) JANUS_BWD_MFMA(3);
          if (4 <= kAttnTiles) JANUS_BWD_MFMA(4);
        }
#undef JANUS_BWD_MFMA
        JANUS_ATTN_TILED(attn_bwd_tiled_kernel, rowptr, (const float*)QKVt(t), (const float*)p.eu,
                         (const float*)STt(t), (const float*)OBt(t), N, d, H, nmin, QKVbt(t), p.rbh);
        hipLaunchKernelGGL(attn_rbar_kernel, gN, b256, 0, st, rowptr, (const float*)p.eud, (const float*)p.rbh, N, H,
                           kAttnMaxN, p.rbar, p.rbs ? p.rbs + (long long)t * Ne : (float*)nullptr);
      }
      {
        PROF(PROF_DENSE_GEMM, f_qkv, 0);
        launch_rows<true>(st, LoadPlain{QKVbt(t), 3LL * d}, Wp(blk(t, "Wqkv")), 3 * d, d, p.tilesE, p.ntE, p.mtE,
                          EpiStore{MBt(t), d});
      }
      {
        PROF(PROF_EDGE, 0, Ne * (4.0 * d + 8.0 * k + 4.0 * k * d));
        LAUNCH_VPL_K(edge_gather_kernel, d, k, gE, b256, 0, st, POS(t), GATE(t), (const float*)MBt(t), Ne, d, Ybs(t));
      }
    } else {
      PROF(PROF_ATOM, 0, by_gather);
      LAUNCH_VPL_K(gather_atom_kernel, d, k, gN, b256, 0, st, rowptr, POS(t), GATE(t), hbar_u, N, d, Ybs(t));
    }
    if (p.rf && Ne > 0) {
      // the gates' adjoints <mbar, Y_c> -> logit adjoints -> the router's part of Xbar
      // (mbar: the centre atom's dE/du, or with attention the edge's message adjoint)
      PROF(PROF_ROUTE, 2.0 * Ne * d * Ep, Ne * (4.0 * d + 4.0 * k * d + 8.0 * Ep));
      LAUNCH_VPL_K(feat_p2_kernel, d, k, gE, b256, 0, st, attn ? (const int*)p.iotaE : ei, POS(t), EID(t), GATE(t),
                   (const float*)FPR(t), Ee, (int)Ep, attn ? (const float*)MBt(t) : hbar_u, (const float*)YstR(t),
                   Ne, d, GBR(t), LBR(t));
      launch_rows<true>(st, LoadPlain{LBR(t), Ep}, WRP(t), (int)Ep, d, p.tilesE, p.ntE, p.mtE, EpiStore{p.Xadd, d});
    }
    {
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      launch_rows<true>(st, LoadPlain{Ybs(t), d}, W2, d, h, TL(t), p.ntiles + t, p.mt,
                        EpiP2{Aa(t), Sb(t), Ab(t), h});
    }
    {
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      launch_rows<true>(st, LoadPlain{Ab(t), h}, W1, h, d, TL(t), p.ntiles + t, p.mt, EpiStore{p.T1, d});
    }
    if (Ne > 0) {
      PROF(PROF_EDGE, 0, by_p2);
      LAUNCH_VPL_K(edge_p2_kernel, d, k, gE, b256, ldsW, st, (const float*)p.B, (const float*)p.dB, nb, Wb,
                 (const float*)HV(p.h, t), ej, POS(t), Ne, d, (const float*)p.T1, Xbar(t), Fbar(t), p.rbar, p.Pe,
                 (const float*)(p.rf ? p.Xadd : nullptr));
    }
    if (three && Nt > 0) {
      // triplet messages' backward: Ybar3 = g3 Xbar_e -> experts -> Zbar; feature-geometry adjoints
      {
        PROF(PROF_EDGE, 0, Ne * 4.0 * d + M3 * 4.0 * d);
        LAUNCH_VPL_K(tri_gather_kernel, d, k3, gE, b256, 0, st, (const int*)p.trow, POS3(t), GATE3(t),
                   (const float*)Xbar(t), Ne, d, Y3bs(t));
      }
      {
        PROF(PROF_EXPERT_GEMM, f_tri, 0);
        launch_rows<true>(st, LoadPlain{Y3bs(t), d}, Wp(blk(t, "W2a")), d, h3, TL3(t), p.ntiles3 + t, p.mt3,
                          EpiP2{A3(t), S3b(t), A3b(t), h3});
      }
      {
        PROF(PROF_EXPERT_GEMM, f_tri, 0);
        launch_rows<true>(st, LoadPlain{A3b(t), h3}, Wp(blk(t, "W1a")), h3, d, TL3(t), p.ntiles3 + t, p.mt3,
                          EpiStore{p.T3a, d});
      }
      {
        PROF(PROF_EDGE, 0, by_tri_idx + Nt * (4.0 * k3 * d + 4.0 * d + 32.0) + Ne * (4.0 * nb + 8.0 * d));
        LAUNCH_VPL_K(tri_p2_kernel, d, k3, gEa, b256, ldsWa, st, (const int*)p.trow, (const float4*)p.tlane,
                     (const float*)p.B3, (const float*)p.dB3, Wp(blk(t, "W_a")), nb, L3, ej,
                     (const float*)HV(p.h, t), POS3R(t), Ne, d, (const float*)p.T3a, Zbar3(t), p.tacc, p.Pe);
      }
    }
    {
      PROF(PROF_ATOM, 0, by_scatter);
      LAUNCH_VPL(scatter_rev_kernel, d, gN, b256, 0, st, rowptr, rev, (const float*)p.Pe, hbar_u,
                 (const float*)nullptr, N, d, HV(p.hh, t));
    }
  }
  // routing on the edge tokens: phase 4 needs the phase-2 atom adjoints, which it overwrites
  if (p.rf)
    JANUS_HIP_TRY(hipMemcpyAsync(p.hh2, p.hh, sizeof(float) * (T + 1) * Nd, hipMemcpyDeviceToDevice, st));
  {
    PROF(PROF_OTHER, 0, Ne * 40.0 + N * 24.0);
    if (three && Ne > 0)
      hipLaunchKernelGGL(tri_edge_vec_kernel, dim3(cdiv(Ne, 256)), b256, 0, st, (const int*)p.trow,
                         (const int*)p.trev, (const int*)p.te2, (const float*)p.tc, (const float4*)p.geo,
                         (const float4*)p.tacc, Ne, p.gvec);
    hipLaunchKernelGGL(force_kernel, gN, b256, 0, st, rowptr, rev, (const float*)p.rbar,
                       (const float4*)p.geo, (const float4*)(three ? p.gvec : nullptr), N, F);
    if (S_ref || stress_out)
      hipLaunchKernelGGL(stress_kernel, wave_grid(S), b256, 0, st, rowptr, offsets, cell, (const float*)p.rbar,
                         (const float4*)p.geo, (const float4*)(three ? p.gvec : nullptr), S, p.sig, stress_out);
    if (cfg.robust) {
      double* Ls = ca.robust_g;                   // [S_tot] base losses
      double* cs = ca.robust_g + ca.S_tot;        // [S_tot] dL/dL_s
      if (ca.robust_mode != ROBUST_SEEDS)
        hipLaunchKernelGGL(robust_base_kernel, wave_grid(S), b256, 0, st, (const double*)p.Ed, E_ref, offsets, S,
                           (const float*)F, F_ref, cfg.w_E, cfg.w_F, (const float*)p.sig, S_ref, cfg.w_S,
                           cfg.huber_delta, Ls + ca.s0);
      if (ca.robust_mode == ROBUST_LOSSES) {
        JANUS_HIP_TRY(hipGetLastError());
        return JANUS_OK;   // the double and final backward wait for the whole batch's statistics
      }
      if (ca.robust_mode == ROBUST_ONE)
        hipLaunchKernelGGL(robust_stats_kernel, dim3(1), dim3(1024), 0, st, (const double*)Ls, ca.S_tot,
                           cfg.n_tasks ? labels->task : (const int*)nullptr, cfg.n_tasks ? cfg.n_tasks : 1,
                           cfg.robust_tau, cs, loss_part);
      hipLaunchKernelGGL(robust_seed_kernel, dim3(cdiv(std::max<long long>(3LL * N, S), 256)), b256, 0, st,
                         (const double*)p.Ed, E_ref, offsets, S, (const float*)F, F_ref, N, cfg.w_E, cfg.w_F,
                         (const float*)p.sig, S_ref, cfg.w_S, cell, cfg.huber_delta, (const double*)(cs + ca.s0),
                         (const int*)p.sid, p.lam, p.phi, p.Psi);
    } else
      hipLaunchKernelGGL(loss_kernel, dim3(1), dim3(1024), 0, st, (const double*)p.Ed, E_ref, offsets, S,
                         (const float*)F, F_ref, N, ca.S_tot, ca.N_tot, cfg.w_E, cfg.w_F, (const float*)p.sig, S_ref,
                         cfg.w_S, cell, loss_part, p.lam, p.phi, p.Psi);
    if (Ne > 0)
      hipLaunchKernelGGL(rtilde_kernel, dim3(cdiv(Ne, 256)), b256, 0, st, ei, ej, (const float4*)p.geo,
                         (const float*)p.phi, (const int*)p.sid, (const float*)(S_ref ? p.Psi : nullptr), Ne, p.rt,
                         three ? p.gtan : (float4*)nullptr);
    if (three && Nt > 0) {
      hipLaunchKernelGGL(tri_ctilde_kernel, dim3(cdiv(Nt, 256)), b256, 0, st, (const int*)p.te, (const int*)p.te2,
                         (const float*)p.tc, (const float4*)p.geo, (const float4*)p.gtan, (const float*)p.rt, Nt,
                         p.tct);
      // ct-weighted feature derivatives of every triplet, for dW_a of the double backward
      hipLaunchKernelGGL(tri_features_kernel, dim3(cdiv(Nt * (nf / 4), 256)), b256, 0, st,
                         LoadTriFeat{p.te, p.te2, p.tc, p.B3, p.dB3, p.u3, p.du3, p.tct, nb}, Nt, nf, p.G3t);
    }
  }
  JANUS_HIP_TRY(hipGetLastError());

  // ---- phase 3: double backward of the force loss (hht[t] = loss adjoint of hh[t])
  // The expert weight gradients go to the side stream (ss.sd), forked just before
  // memory-bound edge and atom kernels of the caller's stream; the caller's stream
  // joins the side stream before each of its own matrix products, so products never
  // share the GPU with each other.  Buffers the side stream reads: p.T1 (G7, until
  // t1_free), Abar of the block (G7), Sbt (G8).  Sbt of block t is written over
  // Abar of block t-1 (block 0: p.Shat0), which G7 of block t-1 has finished
  // reading once t1_free of that block has passed.
  // dL/dr_e through the basis, accumulated by the edge kernels of phases 3 and 4
  if (p.rpos) JANUS_HIP_TRY(hipMemsetAsync(p.rpos, 0, sizeof(float) * (Ne + 1), st));
  if (p.adjG) {
    JANUS_HIP_TRY(hipMemsetAsync(p.adjG, 0, sizeof(float) * (Nt * nf + 4), st));
    JANUS_HIP_TRY(hipMemsetAsync(p.adjGd, 0, sizeof(float) * (Nt * nf + 4), st));
  }
  SideSync ss(ctx, st);
  hipStream_t sd = ss.sd;
  hipEvent_t t1_free = nullptr;   // side stream done with p.T1 (and with the last Abar it read)
  auto Shat = [&](int t) { return t == 0 ? p.Shat0 : Ab(t - 1); };
  for (int t = 0; t < T; ++t) {
    const float* Wb = Wp(blk(t, "W_b"));
    const float* W1 = Wp(blk(t, "W1"));
    const float* W2 = Wp(blk(t, "W2"));
    const float* hht_t = t == 0 ? nullptr : HV(p.hht, t);
    const bool tri_t = three && Nt > 0;
    if (tri_t) {
      ss.join();   // products of the caller's stream follow
      // double backward of the triplet messages: Zbar~ -> triplet experts -> Ybar3~ -> QX_e
      const float* W1a = Wp(blk(t, "W1a"));
      const float* W2a = Wp(blk(t, "W2a"));
      {
        PROF(PROF_EDGE, 0, by_tri_idx + Nt * (4.0 * k3 * d + 8.0 * d + 20.0) + Ne * (4.0 * nb + 8.0 * d));
        LAUNCH_VPL_K(tri_p3_kernel, d, k3, gEa, b256, ldsWa, st, (const int*)p.trow, (const float4*)p.tlane,
                     (const float*)p.B3, (const float*)p.dB3, Wp(blk(t, "W_a")), nb, L3, ej,
                     (const float*)HV(p.h, t), hht_t, (const float4*)p.tct, (const float*)Zbar3(t), POS3R(t), Ne,
                     d, p.T3a, p.VT, p.Pe);
      }
      {
        // dW_a (part 1): Gt^T (Zbar * h_j2)
        PROF(PROF_DENSE_GEMM, f_wa, 0);
        launch_wgrad(st, LoadPlain{p.G3t, nf}, LoadPlain{p.VT, d}, nf, d, p.chunksT, p.ncT, p.cfT, p.mcT, 1,
                     p.partial, Gp(blk(t, "W_a")), 1);
        // loss gradient in positions: adjoint of the feature tangent, sum_t (Zbar * h_j2) W_a^T
        if (p.adjGd)
          launch_rows<true>(st, LoadPlain{p.VT, d}, Wp(blk(t, "W_a")), d, nf, p.tilesT, p.ntT, p.mtT,
                            EpiAdd{p.adjGd, p.adjGd, nf});
      }
      {
        PROF(PROF_EXPERT_WGRAD, f_tri, 0);
        launch_wgrad(st, LoadPlain{p.T3a, d}, LoadPlain{A3b(t), h3}, d, h3, CH3(t), p.nchunks3 + t, CF3(t), p.mc3,
                     E3, p.partial, Gp(blk(t, "W1a")), 1);
      }
      {
        PROF(PROF_EXPERT_GEMM, f_tri, 0);
        launch_rows<false>(st, LoadPlain{p.T3a, d}, W1a, d, h3, TL3(t), p.ntiles3 + t, p.mt3,
                           EpiP3{A3(t), S3b(t), A3b(t), h3});
      }
      {
        PROF(PROF_EXPERT_GEMM, f_tri, 0);
        launch_rows<false>(st, LoadPlain{A3b(t), h3}, W2a, h3, d, TL3(t), p.ntiles3 + t, p.mt3, EpiStore{p.T3b, d});
      }
      {
        PROF(PROF_EXPERT_WGRAD, f_tri, 0);
        launch_wgrad(st, LoadPlain{A3b(t), h3}, LoadPlain{Y3bs(t), d}, h3, d, CH3(t), p.nchunks3 + t, CF3(t), p.mc3,
                     E3, p.partial, Gp(blk(t, "W2a")), 1);
      }
      {
        PROF(PROF_EDGE, 0, Ne * 8.0 * d + M3 * (8.0 + 4.0 * d));
        LAUNCH_VPL_K(tri_combine_p3_kernel, d, k3, gE, b256, 0, st, (const int*)p.trow, POS3(t), GATE3(t),
                   (const float*)p.T3b, (const float*)Xbar(t), Ne, d, p.g3t + t * M3, p.Q);
      }
    }
    ss.wait(t1_free);   // edge_p3 rewrites p.T1; G5 below rewrites Abar of block t-1
    if (Ne > 0) {
      PROF(PROF_EDGE, 0, by_p3);
      // with triplets, P_e already holds the triplet part written by tri_p3
      LAUNCH_VPL_K(edge_p3_kernel, d, k, gE, b256, ldsW, st, (const float*)p.B, (const float*)p.dB, nb, Wb,
                   (const float*)HV(p.h, t), ej, POS(t), Ne, d, (const float*)Xbar(t), hht_t, (const float*)p.rt,
                   p.T1, p.Pe, (const float*)(tri_t ? p.Q : nullptr), (int)tri_t, (const float*)p.d2B, p.rpos,
                   p.rf ? p.Xh : (float*)nullptr);
    }
    if (p.rf && Ne > 0) {
      // lh = Xbt Wr -> gate adjoints gh and softmax adjoints P3; dWr += Xbt^T lbar
      PROF(PROF_ROUTE, 4.0 * Ne * d * Ep, Ne * (8.0 * d + 16.0 * Ep));
      launch_rows<false>(st, LoadPlain{p.Xh, d}, WRP(t), d, (int)Ep, p.tilesE, p.ntE, p.mtE, EpiStore{p.Lw, Ep});
      hipLaunchKernelGGL(feat_p3_kernel, dim3(cdiv(Ne, 256)), b256, 0, st, EID(t), GATE(t), (const float*)FPR(t),
                         (const float*)GBR(t), (const float*)p.Lw, Ne, Ee, (int)Ep, k, GHR(t), P3R(t));
      launch_wgrad(st, LoadPlain{p.Xh, d}, LoadPlain{LBR(t), Ep}, d, (int)Ep, p.chunksR, p.ncR, p.cfR, p.mcR, 1,
                   p.wrpart, DWR(t), 1);
    }
    // G7 (side stream) beside dW_b and the reverse scatter
    ss.fork();
    {
      // G7: dW1 += Xbt^T Abar (side stream)
      PROFS(sd, PROF_EXPERT_WGRAD, f_exp, 0);
      launch_wgrad(sd, LoadPlain{p.T1, d}, LoadPlain{Ab(t), h}, d, h, CH(t), p.nchunks + t, CF(t), p.mc, Ee,
                   p.partial2, Gp(blk(t, "W1")), 1);
    }
    t1_free = ss.mark();
    {
      // dW_b (part 1): (rt B')^T Fbar
      PROF(PROF_DENSE_GEMM, f_filt, 0);
      launch_wgrad_skinny(st, p.dB, p.rt, Fbar(t), nb, d, p.chunksE, p.ncE, p.cfE, p.mcE, p.partial,
                          Gp(blk(t, "W_b")), 1);
    }
    {
      PROF(PROF_ATOM, 0, by_scatter);
      LAUNCH_VPL(scatter_rev_kernel, d, gN, b256, 0, st, rowptr, rev, (const float*)p.Pe, (const float*)nullptr,
                 (const float*)nullptr, N, d, HV(p.h3, t));
    }
    ss.join();
    {
      // G5: Abt = Xbt W1 -> Sbt (into Shat(t)), C (into Sb)
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      launch_rows<false>(st, LoadPlain{p.T1, d}, W1, d, h, TL(t), p.ntiles + t, p.mt,
                         EpiP3{Aa(t), Sb(t), Shat(t), h});
    }
    {
      // G6: Ybt = Sbt W2
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      launch_rows<false>(st, LoadPlain{Shat(t), h}, W2, h, d, TL(t), p.ntiles + t, p.mt, EpiStore{p.T2, d});
    }
    // G8 (side stream) beside the per-atom and per-edge kernels that follow (and those
    // of the next block up to its G5)
    ss.fork();
    {
      // G8: dW2 += Sbt^T Ybar (side stream)
      PROFS(sd, PROF_EXPERT_WGRAD, f_exp, 0);
      launch_wgrad(sd, LoadPlain{Shat(t), h}, LoadPlain{Ybs(t), d}, h, d, CH(t), p.nchunks + t, CF(t), p.mc, Ee,
                   p.partial2, Gp(blk(t, "W2")), 1);
    }
    // phase-2 dE/du of this block (hh^{t+1} without the feature-update MoE)
    const float* hbar_u3 = atom ? UU(t) : HV(p.hh, t + 1);
    float* uh_out = atom ? p.ut : HV(p.hht, t + 1);
    if (attn) {
      // tangent of the messages and gate adjoints -> tangent q|k|v -> attention tangent -> u-tangent
      {
        PROF(PROF_EDGE, 0, Ne * (8.0 * d + 12.0 * k + 4.0 * k * d));
        LAUNCH_VPL_K(edge_combine_p3_kernel, d, k, gE, b256, 0, st, POS(t), GATE(t), (const float*)p.T2,
                     (const float*)MBt(t), Ne, d, p.g3 + t * M, MHt(t));
        if (p.rf)   // the gates' part of the message tangent: sum_c gh Y_c
          LAUNCH_VPL_K(feat_hht_kernel, d, k, gE, b256, 0, st, (const int*)p.iotaE, POS(t), (const float*)GHR(t),
                       (const float*)YstR(t), Ne, d, MHt(t));
      }
      ss.join();
      {
        PROF(PROF_DENSE_GEMM, f_qkv, 0);
        launch_rows<false>(st, LoadPlain{MHt(t), d}, Wp(blk(t, "Wqkv")), d, 3 * d, p.tilesE, p.ntE, p.mtE,
                           EpiStore{QKVht(t), 3LL * d});
      }
      {
        PROF(PROF_ATTN, 0, by_attn);
#define JANUS_TAN_MFMA(NTV)                                                                                    \
  hipLaunchKernelGGL(attn_tan_mfma_kernel<NTV>, gNH, b256, 0, st, rowptr, (const float*)QKVt(t),                \
                     (const float*)QKVht(t), (const float*)p.eu, (const float*)p.eud, (const float*)p.rt,         \
                     (const float*)STt(t), N, d, H, p.osh)
        if (attn_reg) {
          JANUS_TAN_MFMA(1);
          if (2 <= kAttnTiles) JANUS_TAN_MFMA(2);
          if (3 <= kAttnTiles) JANUS_TAN_MFMA(3);
          if (4 <= kAttnTiles) JANUS_TAN_MFMA(4);
        }
#undef JANUS_TAN_MFMA
        JANUS_ATTN_TILED(attn_tan_tiled_kernel, rowptr, (const float*)QKVt(t), (const float*)QKVht(t),
                         (const float*)p.eu, (const float*)p.eud, (const float*)p.rt, (const float*)STt(t), N, d, H,
                         nmin, p.osh);
      }
      {
        PROF(PROF_DENSE_GEMM, 2 * f_dense, 0);
        launch_rows<false>(st, LoadPlain{p.osh, d}, Wp(blk(t, "Wo")), d, d, p.tilesN, p.ntN, p.mtN,
                           EpiAdd{uh_out, hht_t, d});
        // dWo (tangent part): osumh^T dE/du
        launch_wgrad(st, LoadPlain{p.osh, d}, LoadPlain{hbar_u3, d}, d, d, p.chunksN, p.ncN, p.cfN, p.mcN, 1,
                     p.partial, Gp(blk(t, "Wo")), 1);
      }
    } else {
      // adjoint of the gathered dE/du
      PROF(PROF_ATOM, 0, by_cp3);
      LAUNCH_VPL_K(combine_p3_kernel, d, k, gN, b256, 0, st, rowptr, POS(t), GATE(t), (const float*)p.T2, hbar_u3,
                   hht_t, N, d, p.g3 + t * M, uh_out);
      if (p.rf)   // the gates' adjoints' part: sum_c gh Y_c
        LAUNCH_VPL_K(feat_hht_kernel, d, k, gN, b256, 0, st, rowptr, POS(t), (const float*)GHR(t),
                     (const float*)YstR(t), N, d, uh_out);
    }
    if (atom) {
      // double backward of the feature-update MoE's force backward (same products as G5-G8)
      const float* W1f = Wp(blk(t, "W1f"));
      const float* W2f = Wp(blk(t, "W2f"));
      {
        PROF(PROF_ATOM, 0, by_fgather);
        LAUNCH_VPL_K(gather_atom_kernel, d, kf, gN, b256, 0, st, iota, POSF(t), (const float*)nullptr,
                     (const float*)p.ut, N, d, p.T1f);
      }
      ss.join();
      {
        PROF(PROF_EXPERT_WGRAD, f_atm, 0);
        launch_wgrad(st, LoadPlain{p.T1f, d}, LoadPlain{Abf(t), hf}, d, hf, CHF(t), p.nchunksf + t, CFF(t), p.mcf,
                     Ef, p.partial, Gp(blk(t, "W1f")), 1);
      }
      {
        PROF(PROF_EXPERT_GEMM, f_atm, 0);
        launch_rows<false>(st, LoadPlain{p.T1f, d}, W1f, d, hf, TLF(t), p.ntilesf + t, p.mtf,
                           EpiP3{Af(t), Sbf(t), Abf(t), hf});
      }
      {
        PROF(PROF_EXPERT_GEMM, f_atm, 0);
        launch_rows<false>(st, LoadPlain{Abf(t), hf}, W2f, hf, d, TLF(t), p.ntilesf + t, p.mtf, EpiStore{p.T2f, d});
      }
      {
        PROF(PROF_EXPERT_WGRAD, f_atm, 0);
        launch_wgrad(st, LoadPlain{Abf(t), hf}, LoadPlain{Ybf(t), d}, hf, d, CHF(t), p.nchunksf + t, CFF(t), p.mcf,
                     Ef, p.partial, Gp(blk(t, "W2f")), 1);
      }
      {
        PROF(PROF_ATOM, 0, by_fcombine + Mf * 8.0 + N * 4.0 * d);
        LAUNCH_VPL_K(combine_p3_kernel, d, kf, gN, b256, 0, st, iota, POSF(t), GATEF(t), (const float*)p.T2f,
                     (const float*)HV(p.hh, t + 1), (const float*)p.ut, N, d, p.g3f + t * Mf, HV(p.hht, t + 1));
      }
    }
  }
  ss.join();
  {
    // readout part: vt = hht^T W_o1
    PROF(PROF_DENSE_GEMM, f_dense, 0);
    launch_rows<false>(st, LoadPlain{HV(p.hht, T), d}, Wo1, d, d, p.tilesN, p.ntN, p.mtN, EpiDense{p.vt, d});
  }
  JANUS_HIP_TRY(hipGetLastError());

  // ---- phase 4: final backward (adjoint of h^t reuses hh)
  {
    PROF(PROF_OTHER, 0, 20.0 * Nd);
    LAUNCH_VPL(readout_bwd_kernel, d, gN, b256, 0, st, (const float*)p.z, (const float*)p.vt, wo2,
               (const float*)p.lam, (const int*)p.sid, N, d, p.Zr, p.Tr);
    const int nch = (N + kColChunk - 1) / kColChunk;
    hipLaunchKernelGGL(colsum_partial_kernel, dim3(cdiv(d, 64), nch), dim3(64), 0, st, (const float*)p.Tr,
                       (long long)N, d, p.colpart);
    hipLaunchKernelGGL(colsum_final_kernel, dim3(cdiv(d, 256)), b256, 0, st, (const float*)p.colpart, nch, d,
                       Gp("w_o2"));
  }
  {
    PROF(PROF_DENSE_GEMM, 3 * f_dense, 0);
    launch_wgrad(st, LoadPlain{hT, d}, LoadPlain{p.Zr, d}, d, d, p.chunksN, p.ncN, p.cfN, p.mcN, 1, p.partial,
                 Gp("W_o1"), 1);
    launch_wgrad(st, LoadPlain{HV(p.hht, T), d}, LoadSiluD1Scaled{p.z, wo2, d}, d, d, p.chunksN, p.ncN, p.cfN,
                 p.mcN, 1, p.partial, Gp("W_o1"), 1);
    launch_rows<true>(st, LoadPlain{p.Zr, d}, Wo1, d, d, p.tilesN, p.ntN, p.mtN, EpiDense{HV(p.hh, T), d});
  }
  // G11 and G12 go to the side stream after G10, beside the edge, router and atom
  // kernels of the block; the caller's stream joins it before its next product.
  // G12 reads p.T1 until t1_free.
  for (int t = T - 1; t >= 0; --t) {
    const float* Wb = Wp(blk(t, "W_b"));
    const float* W1 = Wp(blk(t, "W1"));
    const float* W2 = Wp(blk(t, "W2"));
    const float* hht_t = t == 0 ? nullptr : HV(p.hht, t);
    ss.wait(t1_free);   // p.T1 is rewritten below
    // loss adjoint of u (of h^{t+1} without the feature-update MoE)
    const float* a_u = HV(p.hh, t + 1);
    if (atom) {
      const float* W1f = Wp(blk(t, "W1f"));
      const float* W2f = Wp(blk(t, "W2f"));
      {
        PROF(PROF_ATOM, 0, by_fgather);
        LAUNCH_VPL_K(gather_atom_kernel, d, kf, gN, b256, 0, st, iota, POSF(t), (const float*)nullptr,
                     (const float*)HV(p.hh, t + 1), N, d, p.T1f);
      }
      ss.join();
      {
        PROF(PROF_EXPERT_GEMM, f_atm, 0);
        launch_rows<true>(st, LoadPlain{p.T1f, d}, W2f, d, hf, TLF(t), p.ntilesf + t, p.mtf,
                          EpiP4{Af(t), Sbf(t), SGF(t), hf}, p.gpartf);
      }
      {
        PROF(PROF_EXPERT_GEMM, f_atm, 0);
        launch_rows<true>(st, LoadPlain{Sbf(t), hf}, W1f, hf, d, TLF(t), p.ntilesf + t, p.mtf, EpiStore{p.T2f, d});
      }
      {
        PROF(PROF_EXPERT_WGRAD, f_atm, 0);
        launch_wgrad(st, LoadPlain{Xsf(t), d}, LoadPlain{Sbf(t), hf}, d, hf, CHF(t), p.nchunksf + t, CFF(t), p.mcf,
                     Ef, p.partial, Gp(blk(t, "W1f")), 1);
      }
      {
        PROF(PROF_EXPERT_WGRAD, f_atm, 0);
        launch_wgrad(st, LoadSiluRowScale{Af(t), SGF(t), hf}, LoadPlain{p.T1f, d}, hf, d, CHF(t), p.nchunksf + t, CFF(t),
                     p.mcf, Ef, p.partial, Gp(blk(t, "W2f")), 1);
      }
      {
        PROF(PROF_ATOM, 0, by_fcombine);
        LAUNCH_VPL_K(combine_fwd_kernel, d, kf, gN, b256, 0, st, iota, POSF(t), (const float*)p.T2f,
                     (const float*)HV(p.hh, t + 1), N, d, p.ut);
      }
      {
        // feature router: gate adjoints -> logit adjoints per atom -> sums per species
        PROF(PROF_OTHER, 0, 0);
        hipLaunchKernelGGL(gate_total_kernel, dim3(cdiv(Mf, 256)), b256, 0, st, (const float*)(p.g3f + t * Mf),
                           (const float*)p.gpartf, POSF(t), Mf, p.ntilef, p.gtf);
        hipLaunchKernelGGL(edge_logit_kernel, dim3(cdiv((long long)N * Ef, 256)), b256, 0, st, species,
                           (const float*)(p.sprob + (long long)t * nsp * Ef), (const int*)(p.eidf + t * Mf),
                           (const float*)p.gtf, (long long)N, kf, Ef, p.ltf);
        hipLaunchKernelGGL(species_rows_kernel, dim3(nsp), b256, 0, st, (const int*)p.sp_off,
                           (const int*)p.sp_atoms, (const float*)p.ltf, Ef, nsp, Gp(blk(t, "Pf")));
      }
      a_u = p.ut;
    }
    if (attn) {
      // adjoints of osum and of its tangent -> attention reverse -> primal message adjoints
      const float* Wqkv = Wp(blk(t, "Wqkv"));
      ss.join();
      {
        PROF(PROF_DENSE_GEMM, 2 * f_dense, 0);
        launch_rows<true>(st, LoadPlain{a_u, d}, Wp(blk(t, "Wo")), d, d, p.tilesN, p.ntN, p.mtN, EpiStore{p.AO, d});
        // dWo (primal part): osum^T a_u
        launch_wgrad(st, LoadPlain{OSt(t), d}, LoadPlain{a_u, d}, d, d, p.chunksN, p.ncN, p.cfN, p.mcN, 1,
                     p.partial, Gp(blk(t, "Wo")), 1);
      }
      {
        PROF(PROF_ATTN, 0, by_attn);
        // neighbourhoods up to kAttnMfmaN edges on register-resident tiles, larger ones on tiled sweeps
#define JANUS_REV_MFMA(NTV)                                                                                    \
  do {                                                                                                         \
    if (p.rlh)                                                                                                 \
      hipLaunchKernelGGL((attn_rev_mfma_kernel<NTV, true>), gNH, b256, 0, st, rowptr, (const float*)QKVt(t),    \
                         (const float*)QKVht(t), (const float*)p.eu, (const float*)p.eud, (const float*)p.rt,     \
                         (const float*)STt(t), (const float*)p.AO, (const float*)OBt(t), N, d, H, p.QKVa, p.rlh); \
    else                                                                                                       \
      hipLaunchKernelGGL((attn_rev_mfma_kernel<NTV, false>), gNH, b256, 0, st, rowptr, (const float*)QKVt(t),   \
                         (const float*)QKVht(t), (const float*)p.eu, (const float*)p.eud, (const float*)p.rt,     \
                         (const float*)STt(t), (const float*)p.AO, (const float*)OBt(t), N, d, H, p.QKVa,        \
                         (float*)nullptr);                                                                     \
  } while (0)
        if (attn_reg) {
          JANUS_REV_MFMA(1);
          if (2 <= kAttnTiles) JANUS_REV_MFMA(2);
          if (3 <= kAttnTiles) JANUS_REV_MFMA(3);
          if (4 <= kAttnTiles) JANUS_REV_MFMA(4);
        }
#undef JANUS_REV_MFMA
        JANUS_ATTN_TILED(attn_rev_tiled_kernel, rowptr, (const float*)QKVt(t), (const float*)QKVht(t),
                         (const float*)p.eu, (const float*)p.eud, (const float*)p.rt, (const float*)STt(t),
                         (const float*)p.AO, (const float*)OBt(t), N, d, H, nmin, p.QKVa, p.rlh);
        if (p.rlh && Ne > 0)   // the envelope's part of dL/dr_e
          hipLaunchKernelGGL(attn_pos_kernel, dim3(cdiv(Ne, 256)), b256, 0, st, (const float4*)p.geo, Ne, H,
                             cfg.r_cut, (const float*)p.rlh, (const float*)(p.rbs + (long long)t * Ne),
                             (const float*)p.rt, p.rpos);
      }
      {
        PROF(PROF_DENSE_GEMM, 3 * f_qkv, 0);
        launch_rows<true>(st, LoadPlain{p.QKVa, 3LL * d}, Wqkv, 3 * d, d, p.tilesE, p.ntE, p.mtE, EpiStore{p.mta, d});
        // dWqkv: m^T (q|k|v adjoints) + mh^T (phase-2 q|k|v adjoints = adjoints of the tangents)
        launch_wgrad(st, LoadPlain{MM(t), d}, LoadPlain{p.QKVa, 3LL * d}, d, 3 * d, p.chunksA, p.ncA, p.cfA, p.mcA, 1,
                     p.partial, Gp(blk(t, "Wqkv")), 1);
        launch_wgrad(st, LoadPlain{MHt(t), d}, LoadPlain{QKVbt(t), 3LL * d}, d, 3 * d, p.chunksA, p.ncA, p.cfA,
                     p.mcA, 1, p.partial, Gp(blk(t, "Wqkv")), 1);
      }
      if (p.rf) {
        // as below, with the edges' own message adjoints (mt from the attention reverse,
        // mbar from the force backward's attention pass)
        PROF(PROF_ROUTE, 4.0 * Ne * d * Ep, Ne * (8.0 * d + 4.0 * k * d + 16.0 * Ep));
        if (Ne > 0) {
          LAUNCH_VPL_K(feat_p4_kernel, d, k, gE, b256, 0, st, (const int*)p.iotaE, POS(t), EID(t),
                       (const float*)FPR(t), Ee, (int)Ep, (const float*)p.mta, (const float*)YstR(t),
                       (const float*)(p.g3 + t * M), (const float*)P3R(t), Ne, d, p.Lw, p.lte);
          launch_rows<true>(st, LoadPlain{p.Lw, Ep}, WRP(t), (int)Ep, d, p.tilesE, p.ntE, p.mtE,
                            EpiStore{p.Xadd, d});
          launch_wgrad(st, LoadPlain{XeR(t), d}, LoadPlain{p.Lw, Ep}, d, (int)Ep, p.chunksR, p.ncR, p.cfR, p.mcR, 1,
                       p.wrpart, DWR(t), 1);
        }
        LAUNCH_VPL_K(gather_feat_kernel, d, k, gE, b256, 0, st, (const int*)p.iotaE, POS(t), GATE(t),
                     (const float*)p.mta, (const float*)GHR(t), (const float*)MBt(t), Ne, d, p.T1);
      } else {
        PROF(PROF_EDGE, 0, Ne * (4.0 * d + 4.0 * k + 4.0 * k * d));
        LAUNCH_VPL_K(edge_gather_kernel, d, k, gE, b256, 0, st, POS(t), (const float*)nullptr, (const float*)p.mta,
                     Ne, d, p.T1);
      }
    } else if (p.rf) {
      // logit adjoints (gates of phases 3 and 4, softmax adjoints of phase 3) -> router part of
      // Xt and dWr; slot rows of the expert outputs' adjoint, gates applied
      {
        PROF(PROF_ROUTE, 4.0 * Ne * d * Ep, Ne * (8.0 * d + 4.0 * k * d + 16.0 * Ep));
        if (Ne > 0) {
          LAUNCH_VPL_K(feat_p4_kernel, d, k, gE, b256, 0, st, ei, POS(t), EID(t), (const float*)FPR(t), Ee, (int)Ep,
                       a_u, (const float*)YstR(t), (const float*)(p.g3 + t * M), (const float*)P3R(t), Ne, d,
                       p.Lw, p.lte);
          launch_rows<true>(st, LoadPlain{p.Lw, Ep}, WRP(t), (int)Ep, d, p.tilesE, p.ntE, p.mtE,
                            EpiStore{p.Xadd, d});
          launch_wgrad(st, LoadPlain{XeR(t), d}, LoadPlain{p.Lw, Ep}, d, (int)Ep, p.chunksR, p.ncR, p.cfR, p.mcR, 1,
                       p.wrpart, DWR(t), 1);
        }
      }
      PROF(PROF_ATOM, 0, by_gather + N * 4.0 * d + Ne * 4.0 * k);
      const float* mbar2 = atom ? (const float*)UU(t) : (const float*)(p.hh2 + (long long)(t + 1) * Nd);
      LAUNCH_VPL_K(gather_feat_kernel, d, k, gN, b256, 0, st, rowptr, POS(t), GATE(t), a_u, (const float*)GHR(t),
                   mbar2, N, d, p.T1);
    } else {
      // message adjoint, ungated, into the slots
      PROF(PROF_ATOM, 0, by_gather);
      LAUNCH_VPL_K(gather_atom_kernel, d, k, gN, b256, 0, st, rowptr, POS(t), (const float*)nullptr, a_u, N, d,
                   p.T1);
    }
    ss.join();
    {
      // G9: St = mt W2^T -> At = g SiLU'(A) St + C (into Sb); row sums for the gate adjoint
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      // (with routing on the edge tokens the slot rows already carry the gates)
      launch_rows<true>(st, LoadPlain{p.T1, d}, W2, d, h, TL(t), p.ntiles + t, p.mt,
                        EpiP4{Aa(t), Sb(t), p.rf ? (const float*)p.ones : SG(t), h}, p.gpart);
    }
    {
      // G10: Xt = At W1^T
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      launch_rows<true>(st, LoadPlain{Sb(t), h}, W1, h, d, TL(t), p.ntiles + t, p.mt, EpiStore{p.T2, d});
    }
    ss.fork();
    {
      // G12: dW2 += SiLU(A)^T (g mt) (side stream)
      PROFS(sd, PROF_EXPERT_WGRAD, f_exp, 0);
      launch_wgrad(sd, LoadSiluRowScale{Aa(t), p.rf ? (const float*)p.ones : SG(t), h}, LoadPlain{p.T1, d}, h, d, CH(t),
                   p.nchunks + t, CF(t), p.mc, Ee, p.partial2, Gp(blk(t, "W2")), 1);
    }
    t1_free = ss.mark();
    {
      // G11: dW1 += X^T At (side stream)
      PROFS(sd, PROF_EXPERT_WGRAD, f_exp, 0);
      launch_wgrad(sd, LoadPlain{Xs(t), d}, LoadPlain{Sb(t), h}, d, h, CH(t), p.nchunks + t, CF(t), p.mc, Ee,
                   p.partial2, Gp(blk(t, "W1")), 1);
    }
    if (Ne > 0) {
      {
        PROF(PROF_EDGE, 0, by_p4);
        LAUNCH_VPL_K(edge_p4_kernel, d, k, gE, b256, ldsW, st, (const float*)p.B, nb, Wb, (const float*)HV(p.h, t), ej,
                   POS(t), Ne, d, (const float*)p.T2, (const float*)Xbar(t), hht_t, p.Ft, p.Pe,
                   three ? p.Q : (float*)nullptr, (const float*)p.dB, p.rpos, (const float*)(p.rf ? p.Xadd : nullptr));
      }
      {
        // dW_b (part 2): B^T Ft
        PROF(PROF_DENSE_GEMM, f_filt, 0);
        launch_wgrad_skinny(st, p.B, nullptr, p.Ft, nb, d, p.chunksE, p.ncE, p.cfE, p.mcE, p.partial,
                            Gp(blk(t, "W_b")), 1);
      }
      {
        PROF(PROF_OTHER, 0, 0);
        if (!p.rf) {   // (with routing on the edge tokens p.lte came from feat_p4_kernel)
          hipLaunchKernelGGL(gate_total_kernel, dim3(cdiv(M, 256)), b256, 0, st, (const float*)(p.g3 + t * M),
                             (const float*)p.gpart, POS(t), M, p.ntile, p.gt);
          hipLaunchKernelGGL(edge_logit_kernel, dim3(cdiv(Ne * Ee, 256)), b256, 0, st, (const int*)(p.pair + t * Ne),
                             (const float*)(p.pprob + t * np * Ee), (const int*)(p.eid + t * M), (const float*)p.gt,
                             Ne, k, Ee, p.lte);
        }
        hipLaunchKernelGGL(router_atom_kernel, gN, b256, 0, st, rowptr, rev, Ee,
                           (const float*)p.lte, N, p.partC, p.partN);
        hipLaunchKernelGGL(species_rows_kernel, dim3(nsp), b256, 0, st, (const int*)p.sp_off,
                           (const int*)p.sp_atoms, (const float*)p.partC, Ee, nsp, Gp(blk(t, "Pc")));
        hipLaunchKernelGGL(species_rows_kernel, dim3(nsp), b256, 0, st, (const int*)p.sp_off,
                           (const int*)p.sp_atoms, (const float*)p.partN, Ee, nsp, Gp(blk(t, "Pn")));
      }
    }
    if (three && Nt > 0) {
      // final backward of the triplet messages: mt = Xt_e (adjoint of X_e) -> experts -> Zt
      const float* W1a = Wp(blk(t, "W1a"));
      const float* W2a = Wp(blk(t, "W2a"));
      {
        PROF(PROF_EDGE, 0, Ne * 4.0 * d + M3 * 4.0 * d);
        LAUNCH_VPL_K(tri_gather_kernel, d, k3, gE, b256, 0, st, (const int*)p.trow, POS3(t), (const float*)nullptr,
                   (const float*)p.Q, Ne, d, p.T3a);
      }
      ss.join();
      {
        PROF(PROF_EXPERT_GEMM, f_tri, 0);
        launch_rows<true>(st, LoadPlain{p.T3a, d}, W2a, d, h3, TL3(t), p.ntiles3 + t, p.mt3,
                          EpiP4{A3(t), S3b(t), SG3(t), h3}, p.gpart3);
      }
      {
        PROF(PROF_EXPERT_GEMM, f_tri, 0);
        launch_rows<true>(st, LoadPlain{S3b(t), h3}, W1a, h3, d, TL3(t), p.ntiles3 + t, p.mt3, EpiStore{p.T3b, d});
      }
      {
        PROF(PROF_EXPERT_WGRAD, f_tri, 0);
        launch_wgrad(st, LoadPlain{Z3s(t), d}, LoadPlain{S3b(t), h3}, d, h3, CH3(t), p.nchunks3 + t, CF3(t), p.mc3,
                     E3, p.partial, Gp(blk(t, "W1a")), 1);
      }
      {
        PROF(PROF_EXPERT_WGRAD, f_tri, 0);
        launch_wgrad(st, LoadSiluRowScale{A3(t), SG3(t), h3}, LoadPlain{p.T3a, d}, h3, d, CH3(t), p.nchunks3 + t, CF3(t),
                     p.mc3, E3, p.partial, Gp(blk(t, "W2a")), 1);
      }
      {
        PROF(PROF_EDGE, 0, by_tri_idx + Nt * (4.0 * k3 * d + 8.0 * d) + Ne * 12.0 * d);
        LAUNCH_VPL_K(tri_p4_kernel, d, k3, gEa, b256, ldsWa, st, (const int*)p.trow, (const float4*)p.tlane,
                     (const float*)p.B3, Wp(blk(t, "W_a")), nb, L3, ej, (const float*)HV(p.h, t), hht_t,
                     (const float*)Zbar3(t), POS3R(t), Ne, d, (const float*)p.T3b, p.VT, p.Pe);
      }
      {
        // dW_a (part 2): G^T (Zt * h_j2 + Q * Zbar)
        PROF(PROF_DENSE_GEMM, f_wa, 0);
        launch_wgrad(st, LoadPlain{p.G3f, nf}, LoadPlain{p.VT, d}, nf, d, p.chunksT, p.ncT, p.cfT, p.mcT, 1,
                     p.partial, Gp(blk(t, "W_a")), 1);
        // loss gradient in positions: adjoint of the features, sum_t VT W_a^T
        if (p.adjG)
          launch_rows<true>(st, LoadPlain{p.VT, d}, Wp(blk(t, "W_a")), d, nf, p.tilesT, p.ntT, p.mtT,
                            EpiAdd{p.adjG, p.adjG, nf});
      }
      {
        // triplet router tables: logit adjoints summed per vertex / neighbour species
        PROF(PROF_OTHER, 0, 0);
        hipLaunchKernelGGL(gate_total_kernel, dim3(cdiv(M3, 256)), b256, 0, st, (const float*)(p.g3t + t * M3),
                           (const float*)p.gpart3, POS3(t), M3, p.ntile3, p.gt3);
        hipLaunchKernelGGL(tri_logit_kernel, dim3(cdiv(Nt, 256)), b256, 0, st, species, ei, ej, (const int*)p.te,
                           (const int*)p.te2, Nt, Wp(blk(t, "P3a")), Wp(blk(t, "P3b")), Wp(blk(t, "P3c")),
                           Wp(blk(t, "beta3")), E3, k3, (const int*)(p.eid3 + t * M3), (const float*)p.gt3, p.LT3);
        hipLaunchKernelGGL(tri_router_edge_kernel, dim3(cdiv(Ne * E3, 256)), b256, 0, st, (const int*)p.trow,
                           (const int*)p.trev, E3, (const float*)p.LT3, Ne, p.LB, p.LC);
        hipLaunchKernelGGL(tri_router_atom_kernel, gN, b256, 0, st, rowptr, rev, E3, (const float*)p.LB,
                           (const float*)p.LC, N, p.pa, p.pb, p.pc);
        hipLaunchKernelGGL(species_rows_kernel, dim3(nsp), b256, 0, st, (const int*)p.sp_off,
                           (const int*)p.sp_atoms, (const float*)p.pa, E3, nsp, Gp(blk(t, "P3a")));
        hipLaunchKernelGGL(species_rows_kernel, dim3(nsp), b256, 0, st, (const int*)p.sp_off,
                           (const int*)p.sp_atoms, (const float*)p.pb, E3, nsp, Gp(blk(t, "P3b")));
        hipLaunchKernelGGL(species_rows_kernel, dim3(nsp), b256, 0, st, (const int*)p.sp_off,
                           (const int*)p.sp_atoms, (const float*)p.pc, E3, nsp, Gp(blk(t, "P3c")));
      }
    }
    {
      PROF(PROF_ATOM, 0, by_scatter + 4.0 * Nd);
      LAUNCH_VPL(scatter_rev_kernel, d, gN, b256, 0, st, rowptr, rev, (const float*)p.Pe, a_u,
                 (const float*)HV(p.h3, t), N, d, HV(p.hh, t));
    }
  }
  // the caller's stream waits for the side stream's weight gradients
  ss.join();
  if (ss.err != hipSuccess) return janus_set_hip_error(ss.err);
  if (p.rf)
    for (int t = 0; t < T; ++t)
      hipLaunchKernelGGL(wr_unpad_add_kernel, dim3(cdiv((long long)d * Ee, 256)), b256, 0, st, (const float*)DWR(t), d,
                         Ee, (int)Ep, Gp(blk(t, "Wr")));
  if (dLdR_g) {
    PROF(PROF_OTHER, 0, Ne * 40.0 + N * 24.0);
    const float* psi = S_ref ? p.Psi : nullptr;
    const float4* tpos = nullptr;
    if (three && Nt > 0) {
      hipLaunchKernelGGL(tri_pos_kernel, dim3(cdiv(Nt, 128)), dim3(128), 0, st, (const int*)p.te, (const int*)p.te2,
                         (const float*)p.tc, (const float4*)p.geo, (const float4*)p.gtan, psi, ei, (const int*)p.sid,
                         (const float*)p.adjG, (const float*)p.adjGd, Nt, nb, L3, cfg.r_cut3, p.tp1, p.tp2);
      hipLaunchKernelGGL(tri_pos_edge_kernel, dim3(cdiv(Ne, 256)), b256, 0, st, (const int*)p.trow,
                         (const int*)p.trev, (const float4*)p.tp1, (const float4*)p.tp2, Ne, p.tpos);
      tpos = p.tpos;
    }
    hipLaunchKernelGGL(pos_grad_kernel, gN, b256, 0, st, rowptr, rev, ei, ej, (const float*)p.rbar,
                       (const float*)p.rpos, (const float4*)p.geo, (const float*)p.phi, psi, (const int*)p.sid,
                       tpos, N, dLdR_g + 3LL * ca.a0);
  }
  {
    PROF(PROF_OTHER, 0, 8.0 * Nd);
    hipLaunchKernelGGL(species_rows_kernel, dim3(nsp), b256, 0, st, (const int*)p.sp_off,
                       (const int*)p.sp_atoms, (const float*)HV(p.hh, 0), d, nsp, Gp("A"));
    if (cfg.n_tasks) {
      // per-structure sums of dL/dh0, then per label value and per species (composition)
      LAUNCH_VPL(struct_sum_kernel, d, wave_grid(S), b256, 0, st, offsets, (const float*)HV(p.hh, 0), S, d, p.gsb);
      hipLaunchKernelGGL(label_rows_kernel, dim3(cfg.n_tasks), b256, 0, st, labels->task + ca.s0, S,
                         (const float*)p.gsb, d, Gp("Tk"));
      hipLaunchKernelGGL(label_rows_kernel, dim3(cfg.n_charges), b256, 0, st, labels->charge + ca.s0, S,
                         (const float*)p.gsb, d, Gp("Qe"));
      hipLaunchKernelGGL(label_rows_kernel, dim3(cfg.n_spins), b256, 0, st, labels->spin + ca.s0, S,
                         (const float*)p.gsb, d, Gp("Se"));
      hipLaunchKernelGGL(comp_rows_kernel, dim3(nsp), b256, 0, st, (const int*)p.sp_off, (const int*)p.sp_atoms,
                         (const int*)p.sid, offsets, (const float*)p.gsb, d, nsp, Gp("Wc"));
    }
  }
  JANUS_HIP_TRY(hipGetLastError());

  // ---- debug copies (per edge: offset e0; per slot: numbered within the chunk)
  if (dbg) {
    const long long Mt = ca.Ne_tot * k, f0 = ca.e0 * k;
    for (int t = 0; t < T; ++t) {
      if (dbg->eid && M)
        JANUS_HIP_TRY(hipMemcpyAsync(dbg->eid + t * Mt + f0, p.eid + t * M, sizeof(int) * M, hipMemcpyDeviceToDevice,
                                     st));
      if (dbg->gate && M)
        JANUS_HIP_TRY(hipMemcpyAsync(dbg->gate + t * Mt + f0, p.gate + t * M, sizeof(float) * M,
                                     hipMemcpyDeviceToDevice, st));
      if (dbg->pos && M)
        JANUS_HIP_TRY(hipMemcpyAsync(dbg->pos + t * Mt + f0, p.pos + t * M, sizeof(int) * M, hipMemcpyDeviceToDevice,
                                     st));
      if (dbg->counts)
        hipLaunchKernelGGL(add_ints_kernel, dim3(1), dim3(64), 0, st, dbg->counts + t * Ee,
                           (const int*)(p.total + t * Ee), Ee);
    }
    if (dbg->basis && Ne > 0)
      JANUS_HIP_TRY(hipMemcpyAsync(dbg->basis + ca.e0 * nb, p.B, sizeof(float) * Ne * nb, hipMemcpyDeviceToDevice,
                                   st));
    if (three && Nt > 0) {
      if (dbg->tri_e)
        hipLaunchKernelGGL(copy_add_kernel, dim3(cdiv(Nt, 256)), dim3(256), 0, st, dbg->tri_e + ca.t0,
                           (const int*)p.te, Nt, (int)ca.e0);
      if (dbg->tri_e2)
        hipLaunchKernelGGL(copy_add_kernel, dim3(cdiv(Nt, 256)), dim3(256), 0, st, dbg->tri_e2 + ca.t0,
                           (const int*)p.te2, Nt, (int)ca.e0);
      const long long Mt3 = ca.Nt_tot * k3, f3 = ca.t0 * k3;
      for (int t = 0; t < T; ++t) {
        if (dbg->eid3)
          JANUS_HIP_TRY(hipMemcpyAsync(dbg->eid3 + t * Mt3 + f3, p.eid3 + t * M3, sizeof(int) * M3,
                                       hipMemcpyDeviceToDevice, st));
        if (dbg->gate3)
          JANUS_HIP_TRY(hipMemcpyAsync(dbg->gate3 + t * Mt3 + f3, p.gate3 + t * M3, sizeof(float) * M3,
                                       hipMemcpyDeviceToDevice, st));
      }
    }
    if (atom && Mf > 0) {
      const long long Mtf = (long long)ca.N_tot * kf, ff = (long long)ca.a0 * kf;
      for (int t = 0; t < T; ++t) {
        if (dbg->eidf)
          JANUS_HIP_TRY(hipMemcpyAsync(dbg->eidf + t * Mtf + ff, p.eidf + t * Mf, sizeof(int) * Mf,
                                       hipMemcpyDeviceToDevice, st));
        if (dbg->gatef)
          JANUS_HIP_TRY(hipMemcpyAsync(dbg->gatef + t * Mtf + ff, p.gatef + t * Mf, sizeof(float) * Mf,
                                       hipMemcpyDeviceToDevice, st));
      }
    }
  }
  return JANUS_OK;
}

}  // namespace

extern "C" int janus_step(janus_ctx* ctx, const float* pos, const float* cell, const int32_t* species,
                          const int32_t* offsets, int32_t n_atoms, int32_t n_struct, const janus_edges* nl,
                          const float* W, const float* E_ref, const float* F_ref, float* loss, float* E, float* F,
                          float* dLdW, const janus_debug* dbg, void* stream) {
  return janus_step_ex(ctx, pos, cell, species, offsets, n_atoms, n_struct, nl, W, E_ref, F_ref, nullptr, nullptr,
                       loss, E, F, nullptr, dLdW, dbg, stream);
}

extern "C" int janus_step_stress(janus_ctx* ctx, const float* pos, const float* cell, const int32_t* species,
                                 const int32_t* offsets, int32_t n_atoms, int32_t n_struct, const janus_edges* nl,
                                 const float* W, const float* E_ref, const float* F_ref, const float* S_ref,
                                 float* loss, float* E, float* F, float* stress, float* dLdW, const janus_debug* dbg,
                                 void* stream) {
  return janus_step_ex(ctx, pos, cell, species, offsets, n_atoms, n_struct, nl, W, E_ref, F_ref, S_ref, nullptr,
                       loss, E, F, stress, dLdW, dbg, stream);
}

extern "C" int janus_step_ex(janus_ctx* ctx, const float* pos, const float* cell, const int32_t* species,
                             const int32_t* offsets, int32_t n_atoms, int32_t n_struct, const janus_edges* nl,
                             const float* W, const float* E_ref, const float* F_ref, const float* S_ref,
                             const janus_labels* labels, float* loss, float* E, float* F, float* stress, float* dLdW,
                             const janus_debug* dbg, void* stream) {
  return janus_step_pos(ctx, pos, cell, species, offsets, n_atoms, n_struct, nl, W, E_ref, F_ref, S_ref, labels, loss,
                        E, F, stress, dLdW, nullptr, dbg, stream);
}

extern "C" int janus_step_pos(janus_ctx* ctx, const float* pos, const float* cell, const int32_t* species,
                              const int32_t* offsets, int32_t n_atoms, int32_t n_struct, const janus_edges* nl,
                              const float* W, const float* E_ref, const float* F_ref, const float* S_ref,
                              const janus_labels* labels, float* loss, float* E, float* F, float* stress,
                              float* dLdW, float* dLdR, const janus_debug* dbg, void* stream) {
  if (!ctx || !pos || !cell || !species || !offsets || !nl || !W || !E_ref || !F_ref || !loss || !E || !F ||
      !dLdW || n_atoms < 1 || n_struct < 1 || n_struct > n_atoms)
    return JANUS_EINVAL;
  // the position gradient covers every option except attention
  const bool want_pos = dLdR != nullptr;
  // the task-aware embedding needs every structure's labels
  if (ctx->cfg.n_tasks && (!labels || !labels->task || !labels->charge || !labels->spin)) return JANUS_EINVAL;
  // the stress term of the loss needs its reference; without the term no reference is read
  if (ctx->cfg.w_S != 0.f && !S_ref) return JANUS_EINVAL;
  if (ctx->cfg.w_S == 0.f) S_ref = nullptr;
  if (nl->n_edges < 0 || nl->n_edges > INT32_MAX / 4 || !nl->rowptr) return JANUS_EINVAL;
  if (nl->n_edges > 0 && (!nl->ei || !nl->ej || !nl->shift || !nl->rev)) return JANUS_EINVAL;
  const janus_config& cfg = ctx->cfg;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int N = n_atoms, S = n_struct;
  const long long Ne = nl->n_edges;
  const Layout L = make_layout(cfg);

  // ---- whole-batch buffers and host plan buffer
  const bool three = cfg.three_body != 0;
  Carver gv(nullptr);
  gv.take<int>(4);
  gv.take<int>(N);
  gv.take<int>(2 * (S + 1));
  gv.take<double>(S + 1);
  gv.take<unsigned char>(three ? Ne + 1 : 1);
  gv.take<long long>(S + 1);
  gv.take<double>(cfg.robust ? 2LL * S + 1 : 1);
  int rc = ensure(ctx->gbuf, gv.size());
  if (rc) return rc;
  Carver g2(ctx->gbuf.ptr);
  int* flag = g2.take<int>(4);
  int* sid = g2.take<int>(N);
  int* sedge = g2.take<int>(2 * (S + 1));
  double* loss_part = g2.take<double>(S + 1);
  unsigned char* tshort = g2.take<unsigned char>(three ? Ne + 1 : 1);
  long long* scount = g2.take<long long>(S + 1);
  double* robust_g = g2.take<double>(cfg.robust ? 2LL * S + 1 : 1);
  const size_t need_host = 4 + 2 * (size_t)(S + 1) + 2 * (size_t)(S + 2);
  if (ctx->host_plan_n < need_host) {
    if (ctx->host_plan) (void)hipHostFree(ctx->host_plan);
    ctx->host_plan = nullptr;
    ctx->host_plan_n = 0;
    JANUS_HIP_TRY(hipHostMalloc((void**)&ctx->host_plan, need_host * sizeof(int), hipHostMallocDefault));
    ctx->host_plan_n = need_host;
  }

  // ---- validation and the per-structure edge counts (one synchronous read)
  {
    PROF(PROF_OTHER, 0, 0);
    JANUS_HIP_TRY(hipMemsetAsync(flag, 0, 4 * sizeof(int), st));
    launch_validate_struct(st, offsets, S, N, cell, 0.f, flag);
    launch_atom_struct(st, offsets, S, N, sid);
    hipLaunchKernelGGL(validate_atoms_kernel, dim3(cdiv(std::max(N, S) + 1, 256)), dim3(256), 0, st, species, N,
                       cfg.n_species, nl->rowptr, nl->ei, Ne, offsets, S, flag);
    if (Ne > 0)
      hipLaunchKernelGGL(validate_edges_kernel, dim3(cdiv(Ne, 256)), dim3(256), 0, st, nl->ei, nl->ej, nl->shift,
                         nl->rev, (const int*)sid, N, Ne, flag);
    hipLaunchKernelGGL(struct_edges_kernel, dim3(cdiv(S + 1, 256)), dim3(256), 0, st, offsets, nl->rowptr, S, N,
                       sedge);
    if (cfg.n_heads)
      hipLaunchKernelGGL(attn_degree_check_kernel, dim3(cdiv(N, 256)), dim3(256), 0, st, nl->rowptr, N, flag);
    if (cfg.n_tasks)
      hipLaunchKernelGGL(validate_labels_kernel, dim3(cdiv(S, 256)), dim3(256), 0, st, labels->task, labels->charge,
                         labels->spin, S, cfg.n_tasks, cfg.n_charges, cfg.n_spins, flag);
  }
  JANUS_HIP_TRY(hipGetLastError());
  int* hp = ctx->host_plan;
  JANUS_HIP_TRY(hipMemcpyAsync(hp, flag, 2 * sizeof(int), hipMemcpyDeviceToHost, st));
  JANUS_HIP_TRY(hipMemcpyAsync(hp + 4, sedge, sizeof(int) * 2 * (S + 1), hipMemcpyDeviceToHost, st));
  JANUS_HIP_TRY(hipStreamSynchronize(st));
  if (hp[0]) return JANUS_EINVAL;
  if (hp[1]) return JANUS_EUNSUPPORTED;   // a neighbourhood larger than the attention kernels hold
  const int* h_erow = hp + 4;            // first edge of structure s
  const int* h_off = hp + 4 + (S + 1);   // first atom of structure s
  // triplets per structure (second read, once the indices are known to be valid)
  long long* h_tri = reinterpret_cast<long long*>(hp + 4 + 2 * (S + 1) + ((4 + 2 * (S + 1)) & 1));
  if (three) {
    {
      PROF(PROF_GRAPH, 0, Ne * 32.0);
      if (Ne > 0)
        hipLaunchKernelGGL(tri_short_kernel, dim3(cdiv(Ne, 256)), dim3(256), 0, st, pos, cell, (const int*)sid,
                           nl->ei, nl->ej, nl->shift, Ne, cfg.r_cut3, tshort);
      hipLaunchKernelGGL(tri_struct_count_kernel, wave_grid(S), dim3(256), 0, st, offsets, nl->rowptr,
                         (const unsigned char*)tshort, S, scount);
    }
    JANUS_HIP_TRY(hipGetLastError());
    JANUS_HIP_TRY(hipMemcpyAsync(h_tri, scount, sizeof(long long) * S, hipMemcpyDeviceToHost, st));
    JANUS_HIP_TRY(hipStreamSynchronize(st));
  }
  std::vector<long long> tpre(S + 1, 0);
  for (int s = 0; s < S && three; ++s) tpre[s + 1] = tpre[s] + h_tri[s];
  auto tri_between = [&](int s0, int s1) { return tpre[s1] - tpre[s0]; };

  // ---- chunk plan: greedy runs of whole structures whose workspace fits the budget
  size_t budget = (size_t)ctx->ws_limit;
  if (!budget) {
    size_t fr = 0, tot = 0;
    JANUS_HIP_TRY(hipMemGetInfo(&fr, &tot));
    budget = (size_t)(0.9 * (double)(fr + ctx->ws.bytes));
  }
  std::vector<ChunkArgs> chunks;
  size_t need = 0;
  {
    Plan tmp;
    int s0 = 0;
    while (s0 < S) {
      int s1 = s0 + 1;
      size_t b1 = plan_layout(tmp, nullptr, cfg, h_off[s1] - h_off[s0], 1, (long long)h_erow[s1] - h_erow[s0],
                              tri_between(s0, s1), want_pos);
      if (b1 > budget) return JANUS_ENOMEM;
      // grow by doubling, then bisect, to keep the plan O(S log S)
      int step = 1;
      while (s1 < S) {
        const int s2 = std::min(S, s1 + step);
        const size_t b = plan_layout(tmp, nullptr, cfg, h_off[s2] - h_off[s0], s2 - s0,
                                     (long long)h_erow[s2] - h_erow[s0], tri_between(s0, s2), want_pos);
        if (b > budget) {
          if (step == 1) break;
          step = 1;
          continue;
        }
        s1 = s2;
        b1 = b;
        step *= 2;
      }
      ChunkArgs ca;
      ca.s0 = s0;
      ca.a0 = h_off[s0];
      ca.S = s1 - s0;
      ca.N = h_off[s1] - h_off[s0];
      ca.e0 = h_erow[s0];
      ca.Ne = (long long)h_erow[s1] - h_erow[s0];
      ca.S_tot = S;
      ca.N_tot = N;
      ca.Ne_tot = Ne;
      ca.index = (int)chunks.size();
      ca.Nt = tri_between(s0, s1);
      ca.t0 = tpre[s0];
      ca.Nt_tot = tpre[S];
      ca.tshort = tshort;
      ca.robust_mode = ROBUST_OFF;
      ca.robust_g = robust_g;
      chunks.push_back(ca);
      need = std::max(need, b1);
      s0 = s1;
    }
  }
  rc = ensure(ctx->ws, need);
  if (rc) return rc;
  ctx->last_chunks = (int)chunks.size();
  ctx->last_triplets = tpre[S];

  if (ctx->concurrent && !ctx->side) {
    // created on first use on the context's device; default priority
    JANUS_HIP_TRY(hipStreamCreateWithFlags(&ctx->side, hipStreamNonBlocking));
  }
  ctx->sync_used = 0;
  JANUS_HIP_TRY(hipMemsetAsync(dLdW, 0, sizeof(float) * L.total, st));
  if (dbg && dbg->counts) JANUS_HIP_TRY(hipMemsetAsync(dbg->counts, 0, sizeof(int) * cfg.n_blocks * cfg.n_experts, st));
  auto run = [&](ChunkArgs ca, int mode) {
    ca.robust_mode = mode;
    Plan p;
    plan_layout(p, ctx->ws.ptr, cfg, ca.N, ca.S, ca.Ne, ca.Nt, want_pos);
    return run_chunk(ctx, st, p, L, ca, pos, cell, species, offsets, nl, W, E_ref, F_ref, S_ref, labels,
                     loss_part + ca.index, E, F, stress, dLdW, dLdR, dbg);
  };
  int n_parts = (int)chunks.size();
  if (cfg.robust && chunks.size() > 1) {
    // The robust loss standardises every structure's loss within its task, so no
    // chunk can start its double backward before all forces exist: a first pass
    // runs every chunk's forward and force backward and keeps its base losses,
    // the batch statistics follow, and a second pass recomputes each chunk's
    // forward and force backward (its workspace was reused) before the double
    // and final backward with the seeds of the batch statistics.
    for (const ChunkArgs& ca : chunks)
      if ((rc = run(ca, ROBUST_LOSSES))) return rc;
    hipLaunchKernelGGL(robust_stats_kernel, dim3(1), dim3(1024), 0, st, (const double*)robust_g, S,
                       cfg.n_tasks ? labels->task : (const int*)nullptr, cfg.n_tasks ? cfg.n_tasks : 1,
                       cfg.robust_tau, robust_g + S, loss_part);
    for (const ChunkArgs& ca : chunks)
      if ((rc = run(ca, ROBUST_SEEDS))) return rc;
    n_parts = 1;
  } else {
    for (const ChunkArgs& ca : chunks)
      if ((rc = run(ca, cfg.robust ? ROBUST_ONE : ROBUST_OFF))) return rc;
  }
  hipLaunchKernelGGL(loss_total_kernel, dim3(1), dim3(1), 0, st, (const double*)loss_part, n_parts, loss);
  JANUS_HIP_TRY(hipGetLastError());
  return JANUS_OK;
}
