/*
 * tacg.h -- C ABI of the MI355X (gfx950) trace passes of Task-Aware Coactivation Grouping (TACG) and
 * Generic Expert Shared Replication (GESR).
 *
 * Conventions shared by every call
 *   - Pointers are DEVICE pointers unless the parameter name ends in `_host`.  The caller allocates
 *     and owns every buffer, including the workspace; the library never allocates or frees memory
 *     and keeps no state between calls.
 *   - Every call enqueues work on `hip_stream` (a hipStream_t; NULL = the default stream) and returns
 *     without synchronising.  Outputs and *d_err are valid once the caller has synchronised that
 *     stream.  Calls on different streams must not share output or workspace buffers.
 *   - Argument errors are detected on the host before anything is enqueued and return TACG_E_INVAL
 *     (bad value) or TACG_E_UNSUPPORTED (beyond a documented limit).  A failed launch returns
 *     TACG_E_DEVICE.  Data errors found on the device are OR-ed into *d_err (a uint32 the caller
 *     zeroes before the call); the outputs of a call that set any d_err bit are unspecified.
 *   - Layouts are C-contiguous (last index fastest).
 *   - Alignment: the trace pointer is 16-byte aligned and every workspace 256-byte aligned
 *     (TACG_E_INVAL otherwise); other buffers need only their element alignment.
 *
 * Routing traces: int16 trace[L][N][k] -- for each MoE layer l and token t, the k expert ids the
 * router selected (slot 0 = highest router score).  Tokens are grouped by task family: family f owns
 * tokens [fam_off_host[f], fam_off_host[f+1]) with fam_off_host[0] = 0 and fam_off_host[F] = N.
 *
 * Limits: 1 <= E <= 256, 1 <= k <= min(E, 16), 1 <= F <= 64, 1 <= G <= 32 simulated GPUs,
 * 0 <= R <= 4 secondary GPUs per expert, at most 16 experts with secondaries per layer,
 * N * k < 2^32.
 */
#ifndef TACG_H
#define TACG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define TACG_OK 0
#define TACG_E_INVAL (-1)
#define TACG_E_UNSUPPORTED (-2)
#define TACG_E_DEVICE (-3)
#define TACG_E_SCRATCH (-4) /* tacg_eval_placements_noalloc: workspace need > TACG_NOALLOC_SCRATCH_BYTES */

/* device-side data-error bits OR-ed into *d_err */
#define TACG_ERR_ID_RANGE 0x1u /* an expert id < 0 or >= E                               */
#define TACG_ERR_ID_DUP 0x2u   /* an expert id repeated within one token-layer           */
#define TACG_ERR_TABLE 0x4u    /* placement / secondary entry >= G, or repeated in a set */
#define TACG_ERR_LIMIT 0x8u    /* more than TACG_MAX_REPLICATED experts with secondaries  */

/* flags */
#define TACG_ACCUMULATE 0x1u /* tacg_coact_build: add into D and C instead of overwriting */

/* limits */
#define TACG_MAX_EXPERTS 256
#define TACG_MAX_TOPK 16
#define TACG_MAX_FAMILIES 64
#define TACG_MAX_GPUS 32
#define TACG_MAX_SECONDARY 4
#define TACG_MAX_REPLICATED 16
#define TACG_MAX_TOP_PAIRS 4096
#define TACG_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20) /* device scratch of the no-allocation entry point */

/*
 * Dispatch and co-activation counts per task family and layer (Sec. 3.3, "Scoring task-family
 * preference": the usage vector u and co-activation matrix A of family f at layer l are relative
 * frequencies of these counts over f's calibration tokens).
 *   D[f][l][i]    = number of tokens of family f whose layer-l selection contains expert i
 *   C[f][l][i][j] = number of tokens of family f whose layer-l selection contains both i and j
 *                   (i != j); C[f][l][i][i] = D[f][l][i]; C is symmetric.
 * Outputs: uint32 D[F][L][E], uint32 C[F][L][E][E].  With TACG_ACCUMULATE the counts are added to
 * what D and C hold (streaming a trace in token chunks with the same fam_off layout per chunk).
 * Data errors: TACG_ERR_ID_RANGE, TACG_ERR_ID_DUP (the offending token-layer is skipped).
 * workspace: at least tacg_coact_workspace_bytes(...) bytes of device memory, 256-byte aligned.
 */
int tacg_coact_build(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k,
                     int32_t n_experts, const int64_t* fam_off_host, int32_t n_fam, uint32_t* D,
                     uint32_t* C, uint32_t flags, uint32_t* d_err, void* workspace,
                     size_t workspace_bytes, void* hip_stream);

size_t tacg_coact_workspace_bytes(int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                                  int32_t n_fam);

/*
 * Which kernel tacg_coact_build runs for n_experts experts and top_k ids per token-layer: 1 when the
 * partial counts come from 4-bit one-hot matrix products on the matrix cores (E <= 64 with k >= 4,
 * E <= 128 with 8 <= k <= 12), 0 for the LDS pair histogram; the counts are identical either way.
 * A host-only query (no device work); 0 for sizes tacg_coact_build rejects.
 */
int tacg_coact_uses_matrix_cores(int32_t n_experts, int32_t top_k);

/*
 * Family preferences and the task-modulated co-activation graph (Sec. 3.3, eqs.
 * usage-coact-advantage, coact-advantage, zscore, soft-score, family-pref, same-family-kernel and
 * task-modulated-graph).  From the counts of tacg_coact_build, per layer l:
 *   N_f = sum_i D[f][l][i] / k;  u_f = D_f / (N_f k);  A_f = C_f / N_f with a zero diagonal;
 *   c_f(e) = sum_e' A_f(e, e');  du, dc = advantage of f over the mean of the other F-1 families;
 *   s = z(du) + z(dc) (z-score over experts, population std, + eps);  p = softmax over f of s / tau;
 *   A-bar = mean_f A_f;  A-hat = A-bar / max off-diagonal A-bar (0 if that max is 0);
 *   A-tilde = (1 - alpha) A-hat + alpha (P P^T) .* A-hat.
 * An empty family (N_f = 0) has u = A = 0.  Internal arithmetic is float64.
 * Outputs: float pref[L][E][F], float a_tilde[L][E][E], optional float a_hat[L][E][E] (NULL = skip).
 * Requires F >= 2 (else TACG_E_INVAL).  workspace: tacg_reweight_workspace_bytes(...) bytes.
 */
int tacg_reweight(const uint32_t* D, const uint32_t* C, int32_t n_fam, int32_t n_layers, int32_t n_experts,
                  int32_t top_k, double alpha, double tau, double eps, float* pref, float* a_tilde,
                  float* a_hat_or_null, void* workspace, size_t workspace_bytes, void* hip_stream);

size_t tacg_reweight_workspace_bytes(int32_t n_fam, int32_t n_layers, int32_t n_experts);

/*
 * Scores that identify generic experts (Sec. 3.4, eq. generic-score), from the counts of
 * tacg_coact_build, per layer l and expert e, with A_f = C_f / N_f off the diagonal (as in
 * tacg_reweight) and A-bar = mean_f A_f:
 *   cent[l][e] = sum_e' A-bar(e, e')                                   (centrality)
 *   cons[l][e] = mean_f cos(A_f(e, :), A-bar(e, :)), 0 for a zero row  (cross-family consistency)
 *   spec[l][e] = max_f || A_f(e, :) - A-bar(e, :) ||_2                 (task-specific deviation)
 * so that r = cent + lambda1 * cons - lambda2 * spec ranks the generic experts of a layer.
 * Outputs: double [L][E] each; float64 arithmetic, summation order unspecified.  No workspace.
 */
int tacg_gesr_scores(const uint32_t* D, const uint32_t* C, int32_t n_fam, int32_t n_layers, int32_t n_experts,
                     int32_t top_k, double* cent, double* cons, double* spec, void* hip_stream);

/*
 * Motivation diagnostics of App. H (auxiliary metrics), from the counts of tacg_coact_build.
 *
 * tacg_activation_distance: the Frobenius distance between the expert-activation distributions of
 * every two families,  P_f[l][e] = D[f][l][e] / N_{f,l}  (N_{f,l} = sum_e D[f][l][e] / k; P = 0 for an
 * empty family),  dist[i][j] = || P_i - P_j ||_F  over all layers and experts.  Output: double
 * dist[F][F] (float64, summation order unspecified).
 *
 * tacg_pair_jaccard: per family and layer, the top_n most frequently co-activated pairs e < e' with
 * a positive count (by count, descending; ties by pair index e * E + e', ascending), written to
 * int32 top_pairs[F][L][top_n] in increasing pair index and padded with -1; then per layer the
 * Jaccard overlap |T_i & T_j| / |T_i | T_j| of every two families (1 when both sets are empty),
 * double jaccard[L][F][F].  1 <= top_n <= TACG_MAX_TOP_PAIRS (the paper uses 64); 2 <= E.
 */
int tacg_activation_distance(const uint32_t* D, int32_t n_fam, int32_t n_layers, int32_t n_experts, int32_t top_k,
                             double* dist, void* hip_stream);
int tacg_pair_jaccard(const uint32_t* C, int32_t n_fam, int32_t n_layers, int32_t n_experts, int32_t top_n,
                      int32_t* top_pairs, double* jaccard, void* hip_stream);

/*
 * Snapshot GPU loads for the serving guard of Sec. 3.4 (eq. mean-load uses per-GPU loads L_m):
 * load_ref[p][l][m] = sum over families f and experts e with primary[p][l][e] == m of D[f][l][e],
 * i.e. the dispatch load of GPU m when every expert is served by its primary GPU.
 * Inputs: uint32 D[F][L][E], uint8 primary[P][L][E].  Output: int64 load_ref[P][L][G].
 * Data errors: TACG_ERR_TABLE (primary entry >= G; that expert is left out).
 */
int tacg_placement_load(const uint32_t* D, int32_t n_fam, int32_t n_layers, int32_t n_experts,
                        const uint8_t* primary, int32_t n_place, int32_t n_gpus, int64_t* load_ref,
                        uint32_t* d_err, void* hip_stream);

/*
 * Scores P expert placements on a trace (Sec. 3.4 serving rule; App. C per-token dispatch sets;
 * App. H "Comm").  For token t of family f the anchor GPU is
 *   h = home_start_host[f] + ((t - fam_off_host[f]) mod home_size_host[f]).
 * At layer l each selected expert e is served by one candidate GPU of placement p:
 *   candidates C_{l,e} = { primary[p][l][e] } + { secondary[p][l][e][r] != 0xFF }   (eq. candidate-set)
 *   feasible GPUs: theta_den * G * load_ref[p][l][m] <= (theta_den + theta_num) * sum_m load_ref[p][l][m]
 *   (eqs. mean-load, feasible-set with theta = theta_num / theta_den; theta_den == 0: all feasible);
 *   FC = feasible candidates, or all candidates when none is feasible.
 *   Single-candidate experts go to their primary; those GPUs form the accessed set R.  Then each
 *   multi-candidate expert, in slot order, takes the lowest-numbered GPU of FC that is in R; else the
 *   anchor h if h is in FC; else the GPU of FC with the smallest load_ref (ties: lowest number); the
 *   choice joins R.
 * With `cards` the final set R of the token-layer:
 *   cost_home[p] = sum over tokens and layers of |cards \ {h}|                  (uint64 [P])
 *   cost_span[p] = sum over tokens and layers of |cards| - 1                    (uint64 [P])
 *   load[p][l][m] = number of (token, slot) dispatches served by GPU m          (uint32 [P][L][G])
 *   cost_home_fam[p][f] = cost_home restricted to family f                      (uint64 [P][F], optional)
 * Tables: uint8 primary[P][L][E]; uint8 secondary[P][L][E][R] or NULL with n_sec = 0; int64
 * load_ref[P][L][G] (required when n_sec > 0; see tacg_placement_load).  Host arrays home_start_host
 * and home_size_host [F] must satisfy home_size >= 1 and home_start + home_size <= G.
 * theta_num and theta_den lie in 0 .. 2^20 (theta_num is not read when theta_den == 0).
 * Data errors: TACG_ERR_ID_RANGE / _DUP (trace: the offending token-layer is not scored, so it adds
 * to no cost, load or count, and the sums above run over the valid token-layers), TACG_ERR_TABLE,
 * TACG_ERR_LIMIT.
 * workspace: tacg_eval_workspace_bytes(...) bytes.  flags: must be 0.
 */
int tacg_eval_placements(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k,
                         int32_t n_experts, const int64_t* fam_off_host, int32_t n_fam,
                         const int32_t* home_start_host, const int32_t* home_size_host, int32_t n_gpus,
                         int32_t n_place, const uint8_t* primary, const uint8_t* secondary_or_null,
                         int32_t n_sec, const int64_t* load_ref_or_null, int32_t theta_num,
                         int32_t theta_den, uint64_t* cost_home, uint64_t* cost_span, uint32_t* load,
                         uint64_t* cost_home_fam_or_null, uint32_t flags, uint32_t* d_err,
                         void* workspace, size_t workspace_bytes, void* hip_stream);

size_t tacg_eval_workspace_bytes(int64_t n_tokens, int32_t n_layers, int32_t n_experts, int32_t n_gpus,
                                 int32_t n_place, int32_t n_fam);

/*
 * tacg_eval_placements without a workspace argument, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).  Arguments,
 * outputs, data errors and results are those of tacg_eval_placements; inputs and outputs are still
 * the caller's buffers.
 * Scratch: the library's own file-scope device array of TACG_NOALLOC_SCRATCH_BYTES (32 MiB), one copy
 * per GPU, held from the first call on that GPU until the process ends.  Its device address is looked
 * up on the first call on each GPU (the caller's current device, which must be the stream's device).
 * The call allocates nothing (no hipMalloc, hipFree or allocating library routine); it clears the
 * scratch itself on the stream before use, so the contents a previous call left do not matter.
 * Every call on one GPU shares that GPU's scratch: calls that overlap on one GPU (concurrent streams,
 * or threads enqueueing at once) race on it and give unspecified results; serialise them.
 * Returns TACG_E_SCRATCH, before anything is enqueued, when tacg_eval_workspace_bytes(...) of the
 * arguments exceeds TACG_NOALLOC_SCRATCH_BYTES (at E = 256, L = 58, G = 32 and F = 16 it holds about
 * 2100 placements on short traces and 2050 on a trace of 2^23 tokens, whose validation marks take
 * one bit per token-layer); TACG_E_DEVICE if the scratch address cannot be obtained.
 */
int tacg_eval_placements_noalloc(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k,
                                 int32_t n_experts, const int64_t* fam_off_host, int32_t n_fam,
                                 const int32_t* home_start_host, const int32_t* home_size_host,
                                 int32_t n_gpus, int32_t n_place, const uint8_t* primary,
                                 const uint8_t* secondary_or_null, int32_t n_sec,
                                 const int64_t* load_ref_or_null, int32_t theta_num, int32_t theta_den,
                                 uint64_t* cost_home, uint64_t* cost_span, uint32_t* load,
                                 uint64_t* cost_home_fam_or_null, uint32_t flags, uint32_t* d_err,
                                 void* hip_stream);

/*
 * The per-token trace statistics of App. C, per placement and family f, on top of everything
 * tacg_eval_placements computes (same arguments, same choice rule, same outputs):
 *   span_fam[p][f]      = sum over f's tokens t and layers l of |cards_l(t)| - 1
 *                         (cross-group dispatches; sum over f equals cost_span[p])
 *   cross_fam[p][f]     = number of (t, l) whose card set is not contained in one family band
 *                         (layers that span more than one family)
 *   home_mass_fam[p][f] = number of (t, l, slot) whose serving GPU lies in f's own band
 *                         [home_start[f], home_start[f] + home_size[f]) (home-family dispatch mass;
 *                         divide by N_f * L * k for the share)
 * All three uint64 [P][F], device memory.  Family bands are the caller's home bands; the distinct
 * bands must tile 0..G-1 without overlap (as the default bands do for every F and G), else
 * TACG_E_UNSUPPORTED.  Costs about 8 more integer ops per placement-token-layer than
 * tacg_eval_placements.  Workspace: tacg_eval_workspace_bytes(...) bytes.  flags: must be 0.
 */
int tacg_eval_trace_stats(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k,
                          int32_t n_experts, const int64_t* fam_off_host, int32_t n_fam,
                          const int32_t* home_start_host, const int32_t* home_size_host, int32_t n_gpus,
                          int32_t n_place, const uint8_t* primary, const uint8_t* secondary_or_null,
                          int32_t n_sec, const int64_t* load_ref_or_null, int32_t theta_num,
                          int32_t theta_den, uint64_t* cost_home, uint64_t* cost_span, uint32_t* load,
                          uint64_t* span_fam, uint64_t* cross_fam, uint64_t* home_mass_fam, uint32_t flags,
                          uint32_t* d_err, void* workspace, size_t workspace_bytes, void* hip_stream);

/*
 * Placement scoring with decayed per-GPU loads: the sequential form of the serving rule of Sec. 3.4
 * (eqs. mean-load, feasible-set and load-update).  Same choice rule, costs and loads as
 * tacg_eval_placements, but every (placement p, layer l) keeps its own loads L_m, which the guard and
 * the least-loaded choice read, and which are updated after every token in trace order:
 *   L_m <- fma(rho, L_m, Delta_m)        (float64, one rounding; Delta_m = the token's slots on m)
 *   feasible: theta_den * G * L_m <= (theta_den + theta_num) * S,  S = L_0 + ... + L_{G-1} in that
 *   order, each product rounded once (theta_den == 0: all feasible).
 * state_in_or_null: float64 [P][L][G] initial loads (NULL = zero); state_out_or_null: the loads
 * after the last token (may be the same buffer as state_in, so that a trace can be scored in token
 * chunks: the costs and loads of the chunks add up to those of the whole trace when every chunk keeps
 * each family's anchor phase).  0 <= rho < 1.  theta, tables and outputs as in tacg_eval_placements; no
 * workspace and no limit on the number of replicated experts.  One wave scans 64 placements of one
 * layer, so the time grows with N and the parallelism is P * L lanes.
 * Data errors: TACG_ERR_ID_RANGE / _DUP (the token-layer is not served and does not update the
 * loads), TACG_ERR_TABLE.  flags: must be 0.
 */
int tacg_eval_online(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                     const int64_t* fam_off_host, int32_t n_fam, const int32_t* home_start_host,
                     const int32_t* home_size_host, int32_t n_gpus, int32_t n_place, const uint8_t* primary,
                     const uint8_t* secondary_or_null, int32_t n_sec, double rho, int32_t theta_num,
                     int32_t theta_den, const double* state_in_or_null, double* state_out_or_null,
                     uint64_t* cost_home, uint64_t* cost_span, uint32_t* load, uint64_t* cost_home_fam_or_null,
                     uint32_t flags, uint32_t* d_err, void* hip_stream);

/*
 * Grouping objective of Sec. 3.3 (eq. grouping-objective) for P placements: the within-group affinity
 *   objective[p][l] = sum over GPUs m of sum over ordered pairs e != e' with primary[p][l][e] ==
 *                     primary[p][l][e'] == m of a_tilde[l][e][e'],
 * accumulated in float64 (the order of the additions is unspecified, so the last bits may differ
 * from a sequential sum).  Inputs: float a_tilde[L][E][E] (tacg_reweight), uint8 primary[P][L][E].
 * Output: double objective[P][L].  Data errors: TACG_ERR_TABLE (an entry >= G; that expert is left
 * out of every group).
 */
int tacg_group_objective(const float* a_tilde, int32_t n_layers, int32_t n_experts, const uint8_t* primary,
                         int32_t n_place, int32_t n_gpus, double* objective, uint32_t* d_err, void* hip_stream);

/*
 * Jain's fairness index and MaxVio of per-GPU loads (App. H eqs. jain and maxvio):
 *   Jain = (sum_m L_m)^2 / (G sum_m L_m^2),  MaxVio = (max_m L_m - mean) / mean.
 * per_layer = 0: L_m = sum_l load[p][l][m], outputs float jain[P], maxvio[P];
 * per_layer = 1: L_m = load[p][l][m], outputs float jain[P][L], maxvio[P][L].
 * All-zero loads give Jain = 1 and MaxVio = 0.  Internal arithmetic: exact integer sums, float64.
 */
int tacg_jain(const uint32_t* load, int32_t n_place, int32_t n_layers, int32_t n_gpus, int32_t per_layer,
              float* jain, float* maxvio, void* hip_stream);

/* Human-readable text of a status code (static storage). */
const char* tacg_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* TACG_H */
