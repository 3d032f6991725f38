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
    case JANUS_ENOMEM: return "device allocation failed or a structure does not fit the workspace";
    case JANUS_EHIP: return "HIP runtime error";
    case JANUS_EUNSUPPORTED: return "configuration or input not supported by this build";
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
  delete c;
}

extern "C" int janus_set_workspace_limit(janus_ctx* ctx, int64_t bytes) {
  if (!ctx || bytes < 0) return JANUS_EINVAL;
  ctx->ws_limit = bytes;
  return JANUS_OK;
}

extern "C" int janus_last_chunks(const janus_ctx* ctx) { return ctx ? ctx->last_chunks : 0; }

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
};

int run_chunk(janus_ctx* ctx, hipStream_t st, Plan& p, const Layout& L, const ChunkArgs& ca, const float* pos_g,
              const float* cell_g, const int32_t* species_g, const int32_t* offsets_g, const janus_edges* nl,
              const float* W, const float* E_ref_g, const float* F_ref_g, double* loss_part, float* E_g, float* F_g,
              float* dLdW, const janus_debug* dbg) {
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
  const double by_p3 = Ne * (8.0 * nb + 16.0 * d + 8.0 + 4.0 * k + 4.0 * k * d);
  const double by_cp3 = N * 12.0 * d + Ne * k * (16.0 + 4.0 * d);
  const double by_p4 = Ne * (4.0 * k * d + 4.0 * k + 4.0 * nb + 20.0 * d);

  // ---- setup: geometry, species groups, routing of every block, GEMM tables
  {
    PROF(PROF_GRAPH, 0, Ne * (12.0 + 3.0 + 16.0 + 8.0 * nb));
    launch_geometry(st, pos, cell, p.sid, ei, ej, shift, (int)Ne, cfg.r_cut, nb, p.geo, p.B, p.dB);
  }
  const long long np = (long long)nsp * nsp;
  {
    PROF(PROF_ROUTE, 0, T * (Ne * (8.0 + 24.0 * k)));
    hipLaunchKernelGGL(species_count_kernel, dim3(nsp), dim3(64), 0, st, species, N, nsp, p.sp_cnt);
    launch_exclusive_scan(st, p.sp_cnt, nsp, p.sp_off, nullptr);
    hipLaunchKernelGGL(species_write_kernel, dim3(nsp), dim3(64), 0, st, species, N, p.sp_off, p.sp_atoms);
    hipLaunchKernelGGL(set_rows_kernel, dim3(1), dim3(64), 0, st, p.rowN, N, p.rowE, Ne);
    build_tables(st, p.rowN, 1, p.kcN, p.tilesN, p.ntN, p.chunksN, p.ncN, p.cfN);
    build_tables(st, p.rowE, 1, p.kcE, nullptr, nullptr, p.chunksE, p.ncE, p.cfE);
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
      route_block(st, ra);
      build_tables(st, ra.off, Ee, p.kc, p.tiles + (long long)t * p.mt, p.ntiles + t,
                   p.chunks + (long long)t * p.mc, p.nchunks + t, p.cfirst + t * (Ee + 1));
    }
  }
  JANUS_HIP_TRY(hipGetLastError());

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
  auto TL = [&](int t) { return (const RowsTile*)(p.tiles + (long long)t * p.mt); };
  auto CH = [&](int t) { return (const WChunk*)(p.chunks + (long long)t * p.mc); };
  auto CF = [&](int t) { return (const int*)(p.cfirst + t * (Ee + 1)); };
  auto HV = [&](float* base, int t) { return base + t * Nd; };

  // ---- phase 1: forward
  {
    PROF(PROF_OTHER, 0, 8.0 * Nd);
    hipLaunchKernelGGL(species_rows_gather_kernel, dim3(cdiv(Nd, 256)), b256, 0, st, Wp("A"), species, N, d, p.h);
  }
  for (int t = 0; t < T; ++t) {
    const float* Wb = Wp(blk(t, "W_b"));
    const float* W1 = Wp(blk(t, "W1"));
    const float* W2 = Wp(blk(t, "W2"));
    if (Ne > 0) {
      PROF(PROF_EDGE, 0, by_dispatch);
      LAUNCH_VPL(dispatch_x_kernel, d, gE, b256, ldsW, st, (const float*)p.B, nb, Wb, (const float*)HV(p.h, t), ej,
                 POS(t), k, Ne, d, Xs(t));
    }
    {
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      launch_rows<false>(st, LoadPlain{Xs(t), d}, W1, d, h, TL(t), p.ntiles + t, p.mt, EpiStore{Aa(t), h});
    }
    {
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      launch_rows<false>(st, LoadSilu{Aa(t), h}, W2, h, d, TL(t), p.ntiles + t, p.mt, EpiRowScale{p.T1, SG(t), d});
    }
    {
      PROF(PROF_ATOM, 0, by_combine);
      LAUNCH_VPL(combine_fwd_kernel, d, gN, b256, 0, st, rowptr, POS(t), k, (const float*)p.T1,
                 (const float*)HV(p.h, t), N, d, HV(p.h, t + 1));
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
  for (int t = T - 1; t >= 0; --t) {
    const float* Wb = Wp(blk(t, "W_b"));
    const float* W1 = Wp(blk(t, "W1"));
    const float* W2 = Wp(blk(t, "W2"));
    {
      PROF(PROF_ATOM, 0, by_gather);
      LAUNCH_VPL(gather_atom_kernel, d, gN, b256, 0, st, rowptr, POS(t), k, GATE(t), (const float*)HV(p.hh, t + 1),
                 N, d, Ybs(t));
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
      LAUNCH_VPL(edge_p2_kernel, d, gE, b256, ldsW, st, (const float*)p.B, (const float*)p.dB, nb, Wb,
                 (const float*)HV(p.h, t), ej, POS(t), k, Ne, d, (const float*)p.T1, Xbar(t), Fbar(t), p.rbar, p.Pe);
    }
    {
      PROF(PROF_ATOM, 0, by_scatter);
      LAUNCH_VPL(scatter_rev_kernel, d, gN, b256, 0, st, rowptr, rev, (const float*)p.Pe,
                 (const float*)HV(p.hh, t + 1), (const float*)nullptr, N, d, HV(p.hh, t));
    }
  }
  {
    PROF(PROF_OTHER, 0, Ne * 40.0 + N * 24.0);
    hipLaunchKernelGGL(force_kernel, dim3(cdiv(N, 256)), b256, 0, st, rowptr, rev, (const float*)p.rbar,
                       (const float4*)p.geo, N, F);
    hipLaunchKernelGGL(loss_kernel, dim3(1), dim3(1024), 0, st, (const double*)p.Ed, E_ref, offsets, S,
                       (const float*)F, F_ref, N, ca.S_tot, ca.N_tot, cfg.w_E, cfg.w_F, loss_part, p.lam, p.phi);
    if (Ne > 0)
      hipLaunchKernelGGL(rtilde_kernel, dim3(cdiv(Ne, 256)), b256, 0, st, ei, ej, (const float4*)p.geo,
                         (const float*)p.phi, Ne, p.rt);
  }
  JANUS_HIP_TRY(hipGetLastError());

  // ---- phase 3: double backward of the force loss (hht[t] = loss adjoint of hh[t])
  for (int t = 0; t < T; ++t) {
    const float* Wb = Wp(blk(t, "W_b"));
    const float* W1 = Wp(blk(t, "W1"));
    const float* W2 = Wp(blk(t, "W2"));
    const float* hht_t = t == 0 ? nullptr : HV(p.hht, t);
    if (Ne > 0) {
      PROF(PROF_EDGE, 0, by_p3);
      LAUNCH_VPL(edge_p3_kernel, d, gE, b256, ldsW, st, (const float*)p.B, (const float*)p.dB, nb, Wb,
                 (const float*)HV(p.h, t), ej, POS(t), k, Ne, d, (const float*)Xbar(t), hht_t, (const float*)p.rt,
                 p.T1, p.Pe);
    }
    {
      // dW_b (part 1): (rt B')^T Fbar
      PROF(PROF_DENSE_GEMM, f_filt, 0);
      launch_wgrad(st, LoadRowScale{p.dB, p.rt, nb}, LoadPlain{Fbar(t), d}, nb, d, p.chunksE, p.ncE, p.cfE, p.mcE, 1,
                   p.partial, Gp(blk(t, "W_b")), 1);
    }
    {
      PROF(PROF_ATOM, 0, by_scatter);
      LAUNCH_VPL(scatter_rev_kernel, d, gN, b256, 0, st, rowptr, rev, (const float*)p.Pe, (const float*)nullptr,
                 (const float*)nullptr, N, d, HV(p.h3, t));
    }
    {
      // G7: dW1 += Xbt^T Abar
      PROF(PROF_EXPERT_WGRAD, f_exp, 0);
      launch_wgrad(st, LoadPlain{p.T1, d}, LoadPlain{Ab(t), h}, d, h, CH(t), p.nchunks + t, CF(t), p.mc, Ee,
                   p.partial, Gp(blk(t, "W1")), 1);
    }
    {
      // G5: Abt = Xbt W1 -> Sbt (into Ab), C (into Sb)
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      launch_rows<false>(st, LoadPlain{p.T1, d}, W1, d, h, TL(t), p.ntiles + t, p.mt,
                         EpiP3{Aa(t), Sb(t), Ab(t), h});
    }
    {
      // G6: Ybt = Sbt W2
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      launch_rows<false>(st, LoadPlain{Ab(t), h}, W2, h, d, TL(t), p.ntiles + t, p.mt, EpiStore{p.T2, d});
    }
    {
      // G8: dW2 += Sbt^T Ybar
      PROF(PROF_EXPERT_WGRAD, f_exp, 0);
      launch_wgrad(st, LoadPlain{Ab(t), h}, LoadPlain{Ybs(t), d}, h, d, CH(t), p.nchunks + t, CF(t), p.mc, Ee,
                   p.partial, Gp(blk(t, "W2")), 1);
    }
    {
      PROF(PROF_ATOM, 0, by_cp3);
      LAUNCH_VPL(combine_p3_kernel, d, gN, b256, 0, st, rowptr, POS(t), k, GATE(t), (const float*)p.T2,
                 (const float*)HV(p.hh, t + 1), hht_t, N, d, p.g3 + t * M, HV(p.hht, t + 1));
    }
  }
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
    hipLaunchKernelGGL(colsum_partial_kernel, dim3(cdiv(d, 256), nch), b256, 0, st, (const float*)p.Tr,
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
  for (int t = T - 1; t >= 0; --t) {
    const float* Wb = Wp(blk(t, "W_b"));
    const float* W1 = Wp(blk(t, "W1"));
    const float* W2 = Wp(blk(t, "W2"));
    const float* hht_t = t == 0 ? nullptr : HV(p.hht, t);
    {
      // message adjoint, ungated, into the slots
      PROF(PROF_ATOM, 0, by_gather);
      LAUNCH_VPL(gather_atom_kernel, d, gN, b256, 0, st, rowptr, POS(t), k, (const float*)nullptr,
                 (const float*)HV(p.hh, t + 1), N, d, p.T1);
    }
    {
      // G9: St = mt W2^T -> At = g SiLU'(A) St + C (into Sb); row sums for the gate adjoint
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      launch_rows<true>(st, LoadPlain{p.T1, d}, W2, d, h, TL(t), p.ntiles + t, p.mt, EpiP4{Aa(t), Sb(t), SG(t), h},
                        p.gpart);
    }
    {
      // G10: Xt = At W1^T
      PROF(PROF_EXPERT_GEMM, f_exp, 0);
      launch_rows<true>(st, LoadPlain{Sb(t), h}, W1, h, d, TL(t), p.ntiles + t, p.mt, EpiStore{p.T2, d});
    }
    {
      // G11: dW1 += X^T At
      PROF(PROF_EXPERT_WGRAD, f_exp, 0);
      launch_wgrad(st, LoadPlain{Xs(t), d}, LoadPlain{Sb(t), h}, d, h, CH(t), p.nchunks + t, CF(t), p.mc, Ee,
                   p.partial, Gp(blk(t, "W1")), 1);
    }
    {
      // G12: dW2 += SiLU(A)^T (g mt)
      PROF(PROF_EXPERT_WGRAD, f_exp, 0);
      launch_wgrad(st, LoadSilu{Aa(t), h}, LoadRowScale{p.T1, SG(t), d}, h, d, CH(t), p.nchunks + t, CF(t), p.mc,
                   Ee, p.partial, Gp(blk(t, "W2")), 1);
    }
    if (Ne > 0) {
      {
        PROF(PROF_EDGE, 0, by_p4);
        LAUNCH_VPL(edge_p4_kernel, d, gE, b256, ldsW, st, (const float*)p.B, nb, Wb, (const float*)HV(p.h, t), ej,
                   POS(t), k, Ne, d, (const float*)p.T2, (const float*)Xbar(t), hht_t, p.Ft, p.Pe);
      }
      {
        // dW_b (part 2): B^T Ft
        PROF(PROF_DENSE_GEMM, f_filt, 0);
        launch_wgrad(st, LoadPlain{p.B, nb}, LoadPlain{p.Ft, d}, nb, d, p.chunksE, p.ncE, p.cfE, p.mcE, 1, p.partial,
                     Gp(blk(t, "W_b")), 1);
      }
      {
        PROF(PROF_OTHER, 0, 0);
        hipLaunchKernelGGL(gate_total_kernel, dim3(cdiv(M, 256)), b256, 0, st, (const float*)(p.g3 + t * M),
                           (const float*)p.gpart, POS(t), M, p.ntile, p.gt);
        hipLaunchKernelGGL(router_atom_kernel, gN, b256, 0, st, rowptr, rev, k, Ee, (const int*)(p.pair + t * Ne),
                           (const float*)(p.pprob + t * np * Ee), (const int*)(p.eid + t * M), (const float*)p.gt, N,
                           p.partC, p.partN);
        hipLaunchKernelGGL(species_rows_kernel, dim3(nsp), dim3(64), 0, st, (const int*)p.sp_off,
                           (const int*)p.sp_atoms, (const float*)p.partC, Ee, nsp, Gp(blk(t, "Pc")));
        hipLaunchKernelGGL(species_rows_kernel, dim3(nsp), dim3(64), 0, st, (const int*)p.sp_off,
                           (const int*)p.sp_atoms, (const float*)p.partN, Ee, nsp, Gp(blk(t, "Pn")));
      }
    }
    {
      PROF(PROF_ATOM, 0, by_scatter + 4.0 * Nd);
      LAUNCH_VPL(scatter_rev_kernel, d, gN, b256, 0, st, rowptr, rev, (const float*)p.Pe,
                 (const float*)HV(p.hh, t + 1), (const float*)HV(p.h3, t), N, d, HV(p.hh, t));
    }
  }
  {
    PROF(PROF_OTHER, 0, 8.0 * Nd);
    hipLaunchKernelGGL(species_rows_kernel, dim3(nsp), dim3(256), 0, st, (const int*)p.sp_off,
                       (const int*)p.sp_atoms, (const float*)HV(p.hh, 0), d, nsp, Gp("A"));
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
  }
  return JANUS_OK;
}

}  // namespace

extern "C" int janus_step(janus_ctx* ctx, const float* pos, const float* cell, const int32_t* species,
                          const int32_t* offsets, int32_t n_atoms, int32_t n_struct, const janus_edges* nl,
                          const float* W, const float* E_ref, const float* F_ref, float* loss, float* E, float* F,
                          float* dLdW, const janus_debug* dbg, void* stream) {
  if (!ctx || !pos || !cell || !species || !offsets || !nl || !W || !E_ref || !F_ref || !loss || !E || !F ||
      !dLdW || n_atoms < 1 || n_struct < 1 || n_struct > n_atoms)
    return JANUS_EINVAL;
  if (nl->n_edges < 0 || nl->n_edges > INT32_MAX / 4 || !nl->rowptr) return JANUS_EINVAL;
  if (nl->n_edges > 0 && (!nl->ei || !nl->ej || !nl->shift || !nl->rev)) return JANUS_EINVAL;
  const janus_config& cfg = ctx->cfg;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int N = n_atoms, S = n_struct;
  const long long Ne = nl->n_edges;
  const Layout L = make_layout(cfg);

  // ---- whole-batch buffers and host plan buffer
  Carver gv(nullptr);
  gv.take<int>(4);
  gv.take<int>(N);
  gv.take<int>(2 * (S + 1));
  gv.take<double>(S + 1);
  int rc = ensure(ctx->gbuf, gv.size());
  if (rc) return rc;
  Carver g2(ctx->gbuf.ptr);
  int* flag = g2.take<int>(4);
  int* sid = g2.take<int>(N);
  int* sedge = g2.take<int>(2 * (S + 1));
  double* loss_part = g2.take<double>(S + 1);
  const size_t need_host = 4 + 2 * (size_t)(S + 1);
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
  }
  JANUS_HIP_TRY(hipGetLastError());
  int* hp = ctx->host_plan;
  JANUS_HIP_TRY(hipMemcpyAsync(hp, flag, sizeof(int), hipMemcpyDeviceToHost, st));
  JANUS_HIP_TRY(hipMemcpyAsync(hp + 4, sedge, sizeof(int) * 2 * (S + 1), hipMemcpyDeviceToHost, st));
  JANUS_HIP_TRY(hipStreamSynchronize(st));
  if (hp[0]) return JANUS_EINVAL;
  const int* h_erow = hp + 4;            // first edge of structure s
  const int* h_off = hp + 4 + (S + 1);   // first atom of structure s

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
      size_t b1 = plan_layout(tmp, nullptr, cfg, h_off[s1] - h_off[s0], 1, (long long)h_erow[s1] - h_erow[s0]);
      if (b1 > budget) return JANUS_ENOMEM;
      // grow by doubling, then bisect, to keep the plan O(S log S)
      int step = 1;
      while (s1 < S) {
        const int s2 = std::min(S, s1 + step);
        const size_t b = plan_layout(tmp, nullptr, cfg, h_off[s2] - h_off[s0], s2 - s0,
                                     (long long)h_erow[s2] - h_erow[s0]);
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
      chunks.push_back(ca);
      need = std::max(need, b1);
      s0 = s1;
    }
  }
  rc = ensure(ctx->ws, need);
  if (rc) return rc;
  ctx->last_chunks = (int)chunks.size();

  JANUS_HIP_TRY(hipMemsetAsync(dLdW, 0, sizeof(float) * L.total, st));
  if (dbg && dbg->counts) JANUS_HIP_TRY(hipMemsetAsync(dbg->counts, 0, sizeof(int) * cfg.n_blocks * cfg.n_experts, st));
  for (const ChunkArgs& ca : chunks) {
    Plan p;
    plan_layout(p, ctx->ws.ptr, cfg, ca.N, ca.S, ca.Ne);
    rc = run_chunk(ctx, st, p, L, ca, pos, cell, species, offsets, nl, W, E_ref, F_ref, loss_part + ca.index, E, F,
                   dLdW, dbg);
    if (rc) return rc;
  }
  hipLaunchKernelGGL(loss_total_kernel, dim3(1), dim3(1), 0, st, (const double*)loss_part, (int)chunks.size(), loss);
  JANUS_HIP_TRY(hipGetLastError());
  return JANUS_OK;
}
