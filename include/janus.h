/*
 * janus.h -- C ABI of the MI355X training-step library for the MoE
 * interatomic potential (MatRIS-MoE, arXiv 2604.15821).
 *
 * The library computes one full training step of an invariant
 * message-passing potential whose per-block edge MLP is a top-k
 * Mixture-of-Experts layer: the forward pass to per-structure energies,
 * the first backward pass to forces F = -dE/dR, and the second-order
 * backward pass of an energy-plus-force loss to every weight gradient
 * (paper Sec. "Overview of the problem": the force loss needs second
 * derivatives and makes training roughly twice as expensive; Sec.
 * "Runtime for multi-phase double-backward execution": forward, first
 * backward for the forces, double backward for the force loss, final
 * backward for the energy loss).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every array argument is a DEVICE pointer owned by the caller, unless
 *    the comment says "host".  The library keeps no caller pointer after
 *    a call returns.
 *  - Floating-point arrays are IEEE fp32, integer arrays int32, unless
 *    noted.  Matrices are row-major.
 *  - Calls are asynchronous on `stream` (a hipStream_t passed as void*;
 *    NULL is the default stream).  Outputs are valid once the stream has
 *    been synchronised.  janus_build_edges and janus_step each perform one
 *    small synchronous device-to-host read (edge count; input validation
 *    flags and per-structure edge counts for the workspace plan) on that
 *    stream before they launch the rest of their work, and janus_step with
 *    the bond-angle term a second one (per-structure triplet counts).
 *  - Return value: JANUS_OK (0) or a negative JANUS_E* code; a message for
 *    it comes from janus_strerror().  On error no output has been written,
 *    except *n_edges for JANUS_ECAPACITY.
 *  - Results are deterministic run to run: no kernel uses floating-point
 *    atomics; every reduction has a fixed order.
 *  - A context is bound to the device that was current when it was created
 *    and must be used from one host thread at a time.
 */
#ifndef JANUS_H
#define JANUS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  JANUS_OK = 0,
  JANUS_EINVAL = -1,       /* bad argument: sizes, offsets, species or edge indices */
  JANUS_ECAPACITY = -2,    /* edge buffers too small; *n_edges holds the count needed */
  JANUS_ENOMEM = -3,       /* device allocation of the context workspace failed */
  JANUS_EHIP = -4,         /* a HIP runtime call failed */
  JANUS_EUNSUPPORTED = -5  /* valid input that this library does not handle (non-diagonal cell,
                              widths that are not multiples of 64, ...) */
};

/*
 * Model hyper-parameters (paper Sec. "Model scaling", Table 2, for the
 * meaning of width / experts / top-k; the radial basis, envelope and loss
 * weights are the readings stated in the oracle and the design notes).
 *   n_species  size of the element vocabulary (89)
 *   d          atom / edge feature width; multiple of 64
 *   n_rbf      number of Bessel radial functions (1..32)
 *   n_blocks   number of interaction blocks T (>= 0)
 *   n_experts  experts per edge-MoE layer (1..64)
 *   top_k      experts per edge token (1..n_experts, at most 4)
 *   d_hidden   expert hidden width; multiple of 64
 *   env_p      envelope exponent; only 6 is implemented
 *   r_cut      neighbour cutoff in Angstrom
 *   three_body non-zero enables the angular triplet term: triplets of bonds
 *              shorter than r_cut3 sharing an atom, features Legendre P_l(cos
 *              theta), l < n_legendre (at most 8), times the Bessel basis at
 *              r_cut3, routed over n_experts3 experts (top_k3) of width
 *              d_hidden3 (multiple of 64); n_legendre * n_rbf * d * 4 bytes
 *              must fit 64 KB
 *   w_E, w_F   loss weights of the energy and force terms
 *   atom_moe   non-zero adds the feature-update MoE to every block (paper
 *              Sec. "Sparse MoE routing": a second expert layer per block
 *              that refines atom features, routed by element type):
 *              u_i = h_i + sum of the block's messages, then
 *              h'_i = u_i + sum_c g_ic W2f_x^T SiLU(W1f_x^T u_i) over the
 *              top_k_f (1..4) of n_experts_f (1..64) experts chosen by the
 *              logits Pf[Z_i] + betaf; each expert d -> d_hidden_f -> d
 *              (d_hidden_f a multiple of 64)
 *   w_S        loss weight of the stress term (>= 0; 0 leaves it out; used by
 *              janus_step_stress, stresses in energy / length^3)
 *   n_heads    0, or the number of heads of the self-attention over every
 *              atom's edge messages (paper Sec. "Multi-head self-attention");
 *              must divide d, with heads of 32, 64 or 128 columns
 *              (d / n_heads; other widths: JANUS_EUNSUPPORTED)
 *   n_tasks    0, or the number of tasks of the task-aware embedding (paper
 *              Sec. "Task-aware feature embedding"); then n_charges and
 *              n_spins (>= 1) size the charge and spin tables, and every
 *              structure's labels select rows of them (janus_step_ex)
 *   robust     0: mean-squared loss w_E/S sum_s (E_s/n_s - E_ref,s)^2
 *              + w_F/(3N) sum |F - F_ref|^2 (+ w_S/(9S) sum |sigma - S_ref|^2).
 *              1: the robust multi-task loss of paper Sec. "Multi-task
 *              training strategies", L = (1/S) sum_s W(z_s, robust_tau)^2 L_s
 *              with per-structure losses L_s = w_E rho(E_s/n_s - E_ref,s)
 *              + w_F/(3 n_s) sum_{a in s} rho(F_a - F_ref,a) (+ w_S/9 sum
 *              rho(sigma_s - S_ref,s)), rho(r) = r^2 for |r| <= huber_delta
 *              and 2 huber_delta |r| - huber_delta^2 beyond (huber_delta > 0,
 *              may be +inf), z_s the standard score of L_s among the
 *              structures of its task (all structures when n_tasks = 0) and
 *              W(z, tau) = exp(-max(z - tau, 0)^2 / 2).  The gradient
 *              includes the dependence of the weights on the batch
 *              statistics.  The statistics couple every structure of a
 *              task, so when the workspace splits the batch into chunks the
 *              step runs the forward and force backward of every chunk
 *              first, then the statistics, then each chunk again through
 *              all four phases (the first two are recomputed).  At most 256
 *              tasks.
 *   route_feat 0: the edge router is the species-pair table.  1: routing on
 *              the evolving edge tokens (paper Sec. "Sparse mixture-of-experts
 *              (MoE) routing", with the router a linear layer on the token):
 *              logits l_e = (Pc[Z_i] + Pn[Z_j]) + X_e Wr + beta per block, Wr
 *              [d, E] in the blob after beta; top_k of the fp32 logits
 *              (descending, lower index first on ties), gates the softmax
 *              probabilities, so forces and every gradient include the gates'
 *              dependence on X_e.  The decision is exact only up to the fp32
 *              rounding of the logits: a token whose k-th and (k+1)-th logits
 *              are that close may be routed differently from a float64
 *              evaluation (janus_debug.gap reports every token's margin).  With
 *              attention the gates act on the edge messages that the attention
 *              layer takes.
 */
typedef struct janus_config {
  int32_t n_species;
  int32_t d;
  int32_t n_rbf;
  int32_t n_blocks;
  int32_t n_experts;
  int32_t top_k;
  int32_t d_hidden;
  int32_t env_p;
  float r_cut;
  int32_t three_body;
  float r_cut3;
  int32_t n_experts3;
  int32_t top_k3;
  int32_t d_hidden3;
  int32_t n_legendre;
  float w_E;
  float w_F;
  int32_t atom_moe;
  int32_t n_experts_f;
  int32_t top_k_f;
  int32_t d_hidden_f;
  float w_S;
  int32_t n_heads;
  int32_t n_tasks;
  int32_t n_charges;
  int32_t n_spins;
  int32_t robust;
  float huber_delta;
  float robust_tau;
  int32_t route_feat;
} janus_config;

typedef struct janus_ctx janus_ctx;

/* One entry of the flat weight blob (host struct, filled by janus_weight_layout). */
typedef struct janus_tensor_desc {
  char name[48];      /* e.g. "A", "blocks.0.W1", "W_o1" */
  int64_t offset;     /* in floats from the start of the blob */
  int32_t ndim;
  int64_t shape[3];
} janus_tensor_desc;

/*
 * Neighbour list in canonical order (paper Sec. "MatRIS": the graph
 * generation module turns a periodically repeated structure into an atom
 * graph).  Edge e = (i, j, n) joins atom i to the image of atom j shifted by
 * the integer lattice vector n; edges are sorted by (i, j, n_a, n_b, n_c).
 *   n_edges  number of directed edges Ne (host value)
 *   ei, ej   [Ne] centre and neighbour atom
 *   shift    [Ne*3] int8 lattice shift n
 *   rowptr   [N+1] CSR offsets of the edges of each centre atom
 *   rev      [Ne] index of the reverse edge (j, i, -n)
 */
typedef struct janus_edges {
  int64_t n_edges;
  const int32_t* ei;
  const int32_t* ej;
  const int8_t* shift;
  const int32_t* rowptr;
  const int32_t* rev;
} janus_edges;

/*
 * Optional debug outputs of janus_step (any pointer may be NULL).
 *   eid     [T*Ne*top_k] int32  chosen experts, descending logit, lower index on ties
 *   gate    [T*Ne*top_k] fp32   softmax probability of each chosen expert
 *   counts  [T*n_experts] int32 tokens routed to each expert (whole batch)
 *   pos     [T*Ne*top_k] int32  slot of (edge, choice) in the expert-grouped order;
 *                               when the step ran in several chunks (janus_last_chunks
 *                               > 1) slots are numbered within each chunk
 *   basis   [Ne*n_rbf]   fp32   Bessel basis with envelope at each edge length
 * With the three-body term (Nt = number of bond triplets; the caller sizes
 * these from its own count):
 *   tri_e, tri_e2 [Nt] int32   first and second edge of every triplet, in
 *                               (e, e2) order
 *   eid3   [T*Nt*top_k3] int32 chosen triplet experts
 *   gate3  [T*Nt*top_k3] fp32  their gates
 * With the feature-update MoE:
 *   eidf   [T*N*top_k_f] int32 chosen experts of every atom
 *   gatef  [T*N*top_k_f] fp32  their gates
 * With routing on the edge tokens (route_feat):
 *   gap    [T*Ne]        fp32  l_(k) - l_(k+1) of every token's fp32 logits, the
 *                               margin of its routing decision (+inf when k = E)
 */
typedef struct janus_debug {
  int32_t* eid;
  float* gate;
  int32_t* counts;
  int32_t* pos;
  float* basis;
  int32_t* tri_e;
  int32_t* tri_e2;
  int32_t* eid3;
  float* gate3;
  int32_t* eidf;
  float* gatef;
  float* gap;
} janus_debug;

/* Create a context for `cfg` on the current device (paper Sec. "Runtime for
 * multi-phase double-backward execution": the four phases of a step keep
 * activations and adjoints of every block alive between phases; the context
 * owns that workspace).  The workspace grows on demand inside janus_step and
 * is freed by janus_destroy.  `cfg` is read and copied; `out` (host) receives
 * the context, or NULL on error.  Errors: JANUS_EINVAL (cfg out of range),
 * JANUS_EUNSUPPORTED (a width or option this library does not implement),
 * JANUS_EHIP. */
int janus_create(const janus_config* cfg /* host */, janus_ctx** out /* host */);

/* Free the context and its workspace (NULL is ignored).  The caller must
 * have synchronised every stream the context was used on.  A library
 * utility: no passage of the paper defines it. */
void janus_destroy(janus_ctx* ctx);

/* Layout of the flat weight blob for `cfg`.  The tensors are those of the
 * model (paper Sec. "MatRIS": embedding, interaction blocks, readout; Sec.
 * "Sparse MoE routing": per-block expert layers and their routers; Sec.
 * "Task-aware feature embedding"; Sec. "Multi-head self-attention"); the
 * paper prints no parameter list, so their shapes and this order are a
 * reading of this library, kept equal to the order the synthetic generator
 * draws the weights in.  Order: A [n_species, d], with the
 * task-aware embedding Tk [n_tasks, d], Qe [n_charges, d], Se [n_spins, d],
 * Wc [n_species, d]; for
 * each block t: W_b [n_rbf, d], Pc [n_species, E], Pn [n_species, E],
 * beta [E], W1 [E, d, d_hidden], W2 [E, d_hidden, d], and with the
 * three-body term W_a [n_legendre*n_rbf, d], P3a, P3b, P3c [n_species, E3],
 * beta3 [E3], W1a [E3, d, d_hidden3], W2a [E3, d_hidden3, d], and with
 * the feature-update MoE Pf [n_species, Ef], betaf [Ef], W1f [Ef, d,
 * d_hidden_f], W2f [Ef, d_hidden_f, d], and with attention Wqkv [d, 3d]
 * (query | key | value columns), Wo [d, d]; then W_o1 [d, d], w_o2 [d].  If `out` is NULL only the counts are written.  *n_tensors (in:
 * capacity of out, out: number of tensors) and *n_floats (total blob size)
 * are host pointers.  Errors: JANUS_EINVAL (capacity too small). */
int janus_weight_layout(const janus_config* cfg, janus_tensor_desc* out, int32_t* n_tensors,
                        int64_t* n_floats);

/*
 * Build the neighbour list of a batch (paper Sec. "MatRIS", graph
 * generation).  An edge is kept iff, in fp32 with each operation rounded
 * separately (no fused multiply-add),
 *     s_k  = (n_a * a_k + n_b * b_k) + n_c * c_k
 *     d_k  = (X_j,k - X_i,k) + s_k
 *     r2   = (d_x * d_x + d_y * d_y) + d_z * d_z  <  r_cut * r_cut
 * with i, j in the same structure and (i, n) != (j, 0); n_k ranges over
 * [-m_k, m_k], m_k = floor(r_cut / L_k) + 1.
 *   pos     [N*3] Cartesian positions; the image range above covers every
 *           neighbour when they are wrapped into the cell
 *   cell    [S*9] lattice rows a, b, c of each structure; must be diagonal
 *           with positive entries (JANUS_EUNSUPPORTED otherwise)
 *   offsets [S+1] structure s owns atoms offsets[s] .. offsets[s+1]-1;
 *           offsets[0] = 0, non-decreasing, offsets[S] = N
 *   capacity  size of the edge buffers in edges
 *   ei, ej, rev [capacity], shift [capacity*3] int8, rowptr [N+1]: outputs
 *   n_edges (host) receives Ne
 * Two-call pattern: if Ne > capacity, returns JANUS_ECAPACITY with *n_edges
 * set and nothing else written.  Errors: JANUS_EINVAL (bad offsets or
 * sizes), JANUS_EUNSUPPORTED (cell), JANUS_EHIP.
 */
int janus_build_edges(janus_ctx* ctx, const float* pos, const float* cell, const int32_t* offsets,
                      int32_t n_atoms, int32_t n_struct, int64_t capacity, int32_t* ei, int32_t* ej,
                      int8_t* shift, int32_t* rowptr, int32_t* rev, int64_t* n_edges, void* stream);

/*
 * How janus_build_edges finds the candidates of the test above (paper Sec.
 * "MatRIS", graph generation; the list itself does not depend on it).
 * All pairs: every centre tests every (j, n) of its structure, n_s * n_images
 * candidates.  Cell list: the bounding box of a structure's atoms is cut into
 * bins at least r_cut wide (at most n_s bins); for each image n a centre tests
 * only the atoms of the bins that the ball of radius r_cut around X_i - s(n)
 * reaches (widened far beyond fp32 rounding), with the same fp32 test, and
 * sorts what it keeps into the canonical order, so both give the same list bit
 * for bit.  mode 0 (default): the cell list for a structure with
 * n_s * n_images >= 32768 whose box holds at least 27 bins, all pairs
 * otherwise; 1: the cell list for every structure; 2: all pairs for every
 * structure.  A centre with more than 512 neighbours is written by the
 * all-pairs kernel in every mode.  Errors: JANUS_EINVAL (ctx null, mode
 * outside 0..2).
 */
int janus_set_edge_builder(janus_ctx* ctx, int32_t mode);

/*
 * One training step (paper Sec. "Runtime for multi-phase double-backward
 * execution": forward, force backward, double backward of the force loss,
 * final backward of the energy loss).
 *   pos [N*3], cell [S*9], species [N] in 0..n_species-1, offsets [S+1]
 *   nl        neighbour list from janus_build_edges for the same positions
 *   W         flat weight blob (janus_weight_layout)
 *   E_ref [S] reference energy per atom of each structure; F_ref [N*3]
 * Outputs:
 *   loss [1]   w_E/S * sum_s (E_s/n_s - E_ref_s)^2 + w_F/(3N) * sum |F - F_ref|^2
 *   E [S]      per-structure energies
 *   F [N*3]    forces -dE/dR
 *   dLdW       gradient of loss with respect to W, same layout as W; the
 *              routing biases (beta, beta3, betaf) receive exactly zero
 *   dbg        optional debug outputs (may be NULL)
 * Inputs are validated on the device first (species range, offsets, edge
 * indices, CSR and reverse map); a failure returns JANUS_EINVAL and writes
 * nothing.  Errors: JANUS_EINVAL, JANUS_ENOMEM (workspace), JANUS_EHIP.
 */
int janus_step(janus_ctx* ctx, const float* pos, const float* cell, const int32_t* species,
               const int32_t* offsets, int32_t n_atoms, int32_t n_struct, const janus_edges* nl,
               const float* W, const float* E_ref, const float* F_ref, float* loss, float* E,
               float* F, float* dLdW, const janus_debug* dbg, void* stream);

/*
 * janus_step with stress (paper Sec. "MatRIS": the stress is the strain
 * derivative of the energy over the cell volume, sigma = (1/V) dE/deps; Sec.
 * "Multi-task training strategies": stress is one of the errors of the base
 * loss).  A strain eps maps every displacement d_e to (I + eps) d_e, so
 *     sigma_s[a][b] = (1/V_s) sum over the edges of s of (dE/dd_e)_a (d_e)_b,
 * V_s = |det| of the cell rows.  With cfg.w_S > 0 the loss gains
 *     w_S/(9S) * sum_s sum_ab (sigma_s[a][b] - S_ref_s[a][b])^2
 * and dLdW includes its second-order gradient.
 *   S_ref  [S*9] reference stress per structure, row-major 3x3; required when
 *          cfg.w_S > 0 (JANUS_EINVAL otherwise), ignored when cfg.w_S = 0
 *   stress [S*9] output stress per structure, row-major 3x3; may be NULL
 * Every other argument, output and error is as for janus_step, which is this
 * call with S_ref = stress = NULL.
 */
int janus_step_stress(janus_ctx* ctx, const float* pos, const float* cell, const int32_t* species,
                      const int32_t* offsets, int32_t n_atoms, int32_t n_struct, const janus_edges* nl,
                      const float* W, const float* E_ref, const float* F_ref, const float* S_ref,
                      float* loss, float* E, float* F, float* stress, float* dLdW,
                      const janus_debug* dbg, void* stream);

/*
 * Per-structure labels of the task-aware embedding (paper Sec. "Task-aware
 * feature embedding": task (dataset), charge and spin embeddings).  Device
 * arrays of n_struct int32 each: task[s] in [0, n_tasks), charge[s] in
 * [0, n_charges) (the index of the structure's total charge) and spin[s] in
 * [0, n_spins) (the index of its spin multiplicity).
 */
typedef struct janus_labels {
  const int32_t* task;
  const int32_t* charge;
  const int32_t* spin;
} janus_labels;

/*
 * janus_step with stress and the task-aware embedding.  With cfg.n_tasks > 0
 * every atom's embedding gains
 *     Tk[task_s] + Qe[charge_s] + Se[spin_s] + c_s Wc
 * (c_s = the element fractions of its structure s) and dLdW includes the
 * gradients of the four tables.  labels (host struct of device pointers) is
 * required then (JANUS_EINVAL otherwise, and for a label out of range) and
 * ignored otherwise.  Every other argument, output and error is as for
 * janus_step_stress, which is this call with labels = NULL.
 */
int janus_step_ex(janus_ctx* ctx, const float* pos, const float* cell, const int32_t* species,
                  const int32_t* offsets, int32_t n_atoms, int32_t n_struct, const janus_edges* nl,
                  const float* W, const float* E_ref, const float* F_ref, const float* S_ref,
                  const janus_labels* labels, float* loss, float* E, float* F, float* stress,
                  float* dLdW, const janus_debug* dbg, void* stream);

/*
 * janus_step_ex that also returns the gradient of the loss with respect to the
 * atom positions (paper Sec. "MatRIS": the forces F = -dE/dR and the stress
 * (1/V) dE/deps are derivatives of the energy, so the loss depends on the
 * positions through E, F and sigma):
 *   dLdR [N*3]  dL/dR_a, row-major [N, 3]; NULL gives exactly janus_step_ex.
 * It is the same four-phase step: the double and final backward also collect,
 * per edge, the loss adjoint of the edge length through the radial basis and
 * its derivative (the second radial derivative of the basis enters here),
 * and one per-atom pass adds the adjoints of the edge directions and of the
 * stress term.  With bond angles the triplet features' first and second
 * partial derivatives enter per triplet; with attention the final backward
 * also collects the adjoint of each edge's log envelope, and the envelope's
 * first and second derivatives carry it and the force backward's envelope
 * term to dL/dr_e.  Every option of janus_config is supported.  Every other
 * argument, output and error is as for janus_step_ex.
 */
int janus_step_pos(janus_ctx* ctx, const float* pos, const float* cell, const int32_t* species,
                   const int32_t* offsets, int32_t n_atoms, int32_t n_struct, const janus_edges* nl,
                   const float* W, const float* E_ref, const float* F_ref, const float* S_ref,
                   const janus_labels* labels, float* loss, float* E, float* F, float* stress,
                   float* dLdW, float* dLdR, const janus_debug* dbg, void* stream);

/*
 * Workspace of janus_step (paper Sec. "Overview of the problem": the second
 * derivatives of the force loss roughly double the memory of training; Sec.
 * "Runtime for multi-phase double-backward execution").  Structures are
 * independent apart from the loss
 * normalisation, so janus_step processes the batch in chunks of whole
 * structures, in order, each sized so that its workspace fits `bytes`
 * (0, the default: 90% of the device memory free at the time of the call
 * plus what the context already holds).  Results do not depend on the
 * chunking except through floating-point summation order of the weight
 * gradients and loss, which is fixed for a given chunking.  A structure too
 * large for the cap makes janus_step return JANUS_ENOMEM.
 * janus_last_chunks returns how many chunks the last janus_step used, and
 * janus_last_triplets how many bond triplets it formed over the whole batch
 * (0 without the three-body term).
 */
int janus_set_workspace_limit(janus_ctx* ctx, int64_t bytes);
int janus_last_chunks(const janus_ctx* ctx);
int64_t janus_last_triplets(const janus_ctx* ctx);

/*
 * Concurrency inside janus_step.  The double and final backward are the
 * third and fourth phases of paper Sec. "Runtime for multi-phase
 * double-backward execution"; in them, the expert weight-gradient products
 * feed no later product of their phase.  With on = 1 the expert
 * weight-gradient products of the double and final backward run on a second
 * stream that the context owns
 * (created on the context's device at the first step, default priority),
 * forked from and joined back into the caller's stream with events inside
 * the call.  Each is forked just before memory-bound edge and atom kernels
 * of the caller's stream, and the caller's stream joins the second stream
 * before its next matrix product, so two products never run at the same
 * time; janus_step's outputs are complete once the caller's stream has
 * reached the end of the call.  With on = 0 (the default) every kernel runs
 * on the caller's stream.  The two settings compute bitwise identical
 * results (same kernels, same summation order); on shortens the step of the
 * 4096-atom small batch by 1-2%.  Errors: JANUS_EINVAL (ctx null, or on not
 * 0 or 1).
 */
int janus_set_concurrency(janus_ctx* ctx, int on);

/*
 * Grouped fp32 GEMM on the matrix cores, the building block of the expert
 * layers (paper Sec. "Platform-specific optimizations": MoE dispatch and
 * combine with batched GEMM invocation).  Rows of A and C are grouped:
 * group g owns rows row_off[g] .. row_off[g+1]-1 (row_off on the device,
 * non-decreasing, row_off[0] = 0, row_off[n_groups] = M).
 *   trans_b = 0:  C[r, :] = A[r, :] (K) x B_g,   B_g = B + g*K*N stored [K, N]
 *   trans_b = 1:  C[r, :] = A[r, :] (K) x B_g^T, B_g = B + g*N*K stored [N, K]
 * A [M*K], C [M*N]; K and N multiples of 16 and 64 respectively.
 * Errors: JANUS_EINVAL, JANUS_EHIP.
 */
int janus_grouped_gemm(janus_ctx* ctx, const float* A, const float* B, float* C,
                       const int32_t* row_off, int32_t n_groups, int64_t M, int32_t K, int32_t N,
                       int32_t trans_b, void* stream);

/*
 * Grouped weight-gradient GEMM: for each group g,
 *   G_g[p, q] = sum over rows r of group g of  A[r, p] * B[r, q]
 * with A [M*P], B [M*Q], G [n_groups*P*Q]; P, Q multiples of 4.  Groups
 * with no rows produce exact zeros.  The sum is split over row chunks and
 * reduced in a fixed order.  Errors: JANUS_EINVAL, JANUS_EHIP.
 */
int janus_grouped_wgrad(janus_ctx* ctx, const float* A, const float* B, float* G,
                        const int32_t* row_off, int32_t n_groups, int64_t M, int32_t P, int32_t Q,
                        void* stream);

/*
 * janus_grouped_gemm that allocates nothing, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, results and errors as
 * janus_grouped_gemm, without the context; runs on the current device.  The
 * tile table lives in a fixed 4 MiB device array of the library (one per
 * device, held from the first call on that device until the process ends;
 * that first call looks up its address, a host-side query), so
 *   ceil(M / 128) + n_groups <= 262128
 * (about 33.5 M rows); larger sizes return JANUS_ENOMEM before any launch.
 * Every call on a device shares its array: calls that overlap on one device
 * (concurrent streams, or host threads) race on it and must be serialised by
 * the caller.  Each call rewrites every table entry it reads, so nothing
 * needs clearing between calls.
 */
int janus_grouped_gemm_noalloc(const float* A, const float* B, float* C, const int32_t* row_off,
                               int32_t n_groups, int64_t M, int32_t K, int32_t N, int32_t trans_b,
                               void* stream);

/*
 * Row-chunk length that janus_grouped_wgrad and the expert weight gradients
 * of janus_step use for a contraction over M rows into P x Q blocks (host
 * function, no device work): a power of two from 128 to 2048.  It starts
 * at 2048 and halves while the grid has fewer than 4096 workgroups of
 * 128 x 128 output tiles and the partial blocks of the halved chunk (written
 * and read back once by the reduction) stay within half of the operand
 * bytes.  Returns the length, or
 * JANUS_EINVAL for M outside [0, 2^31) or non-positive P, Q.
 */
int32_t janus_wgrad_chunk_rows(int64_t M, int32_t P, int32_t Q);

/*
 * Optional profiler of the kernel families of janus_build_edges and
 * janus_step (host-side bookkeeping; HIP events recorded on the caller's
 * stream around each family of launches).
 * janus_profile_enable(ctx, mask) starts recording the families whose bit
 * is set in `mask` (bit 0 expert_gemm, 1 expert_wgrad, 2 dense_gemm, 3 edge,
 * 4 atom, 5 route, 6 graph, 7 other; -1 records all) and clears earlier
 * records; 0 stops it.  Each recorded launch group costs two events on the
 * stream (a few microseconds), so timing one family perturbs the step less
 * than timing all of them.  janus_profile_read synchronises the recorded
 * events, fills up to `cap` entries of `out` (host array) with one line per
 * family that ran, returns the number of entries (or a negative code), and
 * clears the records.  `flops` and `bytes` are the algorithmic work of the
 * timed launches (matrix products: 2*M*N*K; memory-bound kernels: bytes
 * that must cross HBM at least once).
 */
typedef struct janus_profile_entry {
  char name[32];
  int64_t launches;
  double ms;
  double flops;
  double bytes;
} janus_profile_entry;

int janus_profile_enable(janus_ctx* ctx, int mask);
int janus_profile_read(janus_ctx* ctx, janus_profile_entry* out /* host */, int32_t cap);

/* Static message for a return code (a library utility: no passage of the
 * paper defines it).  Never NULL; unknown codes give "unknown error". */
const char* janus_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* JANUS_H */
