/*
 * CPU oracle for the TACG/GESR trace passes -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, literal C of the paper's definitions, used by the tests, by smoke() and by the CPU
 * baseline leg of the benchmark to check and time the product.  The product path never links,
 * loads or calls anything here, and nothing here is shared with the HIP library.
 *
 * Integer outputs are int64; every loop follows the definition directly (no blocking, no fusion).
 *
 *   oracle_coact_segment  -- per-(family, layer) dispatch counts D and co-activation counts C
 *                            (Sec. 3.3, "Scoring task-family preference": usage u and co-activation
 *                            A are relative frequencies of these counts).
 *   oracle_coact          -- all segments (OpenMP over independent segments).
 *   oracle_score          -- per placement: cross-GPU cost, GESR candidate choice and per-GPU loads
 *                            (Sec. 3.4 eqs. mean-load, feasible-set and the fallback after it; the
 *                            per-token dispatch sets of App. C; the dispatch loads of App. H), and
 *                            optionally the per-token trace statistics of App. C per family.
 *   oracle_score_online   -- the same with the guard and the least-loaded choice reading decayed
 *                            per-GPU loads updated after every token (Sec. 3.4 eq. load-update).
 *
 * The order of preference among several feasible candidates (below) is a reading of Sec. 3.4, which
 * names the ingredients (reached GPUs, the anchor, the loads) but prints no rule or worked value for
 * it.  The tests pin this implementation of the reading with hand-built cases, invariants (GPU
 * relabelling, a single GPU, no replicas, every expert at home) and a separate brute force in exact
 * rational arithmetic; no printed value of the paper bears on it.
 *
 * Readings taken where the paper is silent (each also used by the HIP path, written separately):
 *   - a token whose ids repeat or fall outside [0, E) is an input error: it is flagged and skipped;
 *   - GPU loads L_m used by the feasibility guard are a fixed snapshot `load_ref` per (placement,
 *     layer) instead of the per-token decayed load of eq. load-update (which is sequential);
 *   - the guard L_m <= (1 + theta) * mean_m L_m is evaluated exactly as
 *     theta_den * G * L_m <= (theta_den + theta_num) * sum_m L_m; theta_den == 0 disables it;
 *   - the serving rule for an expert with several candidates: first fix the GPUs of all
 *     single-candidate slots (the set R of GPUs already accessed by the token); then, for the
 *     multi-candidate slots in slot order, take (i) the lowest-numbered feasible candidate already
 *     in R, else (ii) the token's anchor GPU if it is a feasible candidate, else (iii) the feasible
 *     candidate of smallest load, ties to the lowest GPU number; add the choice to R;
 *   - the anchor (home) GPU of the t-th token of family f is home_start[f] + (t mod home_size[f]).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_ERR_ID_RANGE 0x1
#define ORC_ERR_ID_DUP   0x2
#define ORC_ERR_TABLE    0x4
#define ORC_ERR_ARG      0x8

#define ORC_NONE 0xFF

/* Is the token-layer's expert list a valid top-k set (k distinct ids in [0, E))? */
static int token_error(const int16_t* ids, int32_t k, int32_t E)
{
    int err = 0;
    for (int32_t s = 0; s < k; ++s)
        if (ids[s] < 0 || ids[s] >= E) err |= ORC_ERR_ID_RANGE;
    for (int32_t s = 0; s < k; ++s)
        for (int32_t s2 = 0; s2 < s; ++s2)
            if (ids[s] == ids[s2]) err |= ORC_ERR_ID_DUP;
    return err;
}

/*
 * Counts of one family segment at one layer (Sec. 3.3: usage and co-activation statistics of
 * family f at layer l come from the calibration traces of f).  For every token t in
 * [t_begin, t_end) with selected set S_t:
 *     D[i]    += 1 for every i in S_t                 (dispatches of expert i)
 *     C[i][j] += 1 for every ordered i != j in S_t     (both experts chosen by the same token)
 * and finally C[i][i] = D[i].   D: [E], C: [E][E], overwritten.
 */
int oracle_coact_segment(const int16_t* trace, int64_t n_tokens, int32_t top_k, int32_t n_experts,
                         int32_t layer, int64_t t_begin, int64_t t_end, int64_t* D, int64_t* C)
{
    const int32_t E = n_experts, k = top_k;
    int err = 0;
    if (E < 1 || k < 1 || k > E) return ORC_ERR_ARG;
    memset(D, 0, sizeof(int64_t) * (size_t)E);
    memset(C, 0, sizeof(int64_t) * (size_t)E * (size_t)E);
    for (int64_t t = t_begin; t < t_end; ++t) {
        const int16_t* ids = trace + ((int64_t)layer * n_tokens + t) * k;
        int e = token_error(ids, k, E);
        if (e) { err |= e; continue; }
        for (int32_t a = 0; a < k; ++a) D[ids[a]] += 1;
        for (int32_t a = 0; a < k; ++a)
            for (int32_t b = 0; b < k; ++b)
                if (a != b) C[(int64_t)ids[a] * E + ids[b]] += 1;
    }
    for (int32_t i = 0; i < E; ++i) C[(int64_t)i * E + i] = D[i];
    return err;
}

/* All segments: D [F][L][E], C [F][L][E][E].  Returns the OR of error bits. */
int oracle_coact(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                 const int64_t* fam_off, int32_t n_fam, int64_t* D, int64_t* C)
{
    const int64_t E = n_experts;
    int err = 0;
    if (fam_off[0] != 0 || fam_off[n_fam] != n_tokens) return ORC_ERR_ARG;
    for (int32_t f = 0; f < n_fam; ++f)
        if (fam_off[f + 1] < fam_off[f]) return ORC_ERR_ARG;
    const int64_t n_seg = (int64_t)n_fam * n_layers;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (int64_t s = 0; s < n_seg; ++s) {
        const int32_t f = (int32_t)(s / n_layers), l = (int32_t)(s % n_layers);
        err |= oracle_coact_segment(trace, n_tokens, top_k, n_experts, l, fam_off[f], fam_off[f + 1],
                                    D + ((int64_t)f * n_layers + l) * E,
                                    C + ((int64_t)f * n_layers + l) * E * E);
    }
    return err;
}

/*
 * Feasible GPUs of eq. feasible-set: m is feasible when L_m <= (1 + theta) * Lbar with the mean load
 * Lbar of eq. mean-load; exact rational form theta_den * G * L_m <= (theta_den + theta_num) * sum L.
 */
static void feasible_gpus(const int64_t* ref, int32_t G, int32_t theta_num, int32_t theta_den, int* feas)
{
    if (theta_den == 0 || ref == NULL) {
        for (int32_t m = 0; m < G; ++m) feas[m] = 1;
        return;
    }
    __int128 total = 0;
    for (int32_t m = 0; m < G; ++m) total += ref[m];
    for (int32_t m = 0; m < G; ++m) {
        __int128 lhs = (__int128)theta_den * G * ref[m];
        __int128 rhs = (__int128)(theta_den + theta_num) * total;
        feas[m] = lhs <= rhs;
    }
}

/*
 * Scores placements p in [p_begin, p_end).  For every token t (family f, anchor h) and layer l the
 * k selected experts are resolved to GPUs; `cards` is the set of resolved GPUs.
 *   cost_home[p]      += |cards \ {h}|
 *   cost_span[p]      += |cards| - 1          (the per-layer cross-group dispatch count of App. C)
 *   load[p][l][m]     += number of the token's experts served by m
 *   cost_home_fam[p][f] += |cards \ {h}|      (may be NULL)
 * and, when span_fam / cross_fam / home_mass_fam are not NULL, the per-token trace statistics of
 * App. C per family f of the token:
 *   span_fam[p][f]      += |cards| - 1        (cross-group dispatch count)
 *   cross_fam[p][f]     += 1 when no family band [home_start, home_start + home_size) contains
 *                          every card (the layer spans more than one family)
 *   home_mass_fam[p][f] += number of slots served by a GPU in f's own band (home-family mass)
 * Tables: primary [P][L][E], secondary [P][L][E][R] (0xFF = none, may be NULL when R = 0),
 * load_ref [P][L][G] (required when R > 0).  Outputs of the placements scored are overwritten.
 */
int oracle_score(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                 const int64_t* fam_off, int32_t n_fam, const int32_t* home_start, const int32_t* home_size,
                 int32_t n_gpus, int32_t n_place, int32_t p_begin, int32_t p_end,
                 const uint8_t* primary, const uint8_t* secondary, int32_t n_sec,
                 const int64_t* load_ref, int32_t theta_num, int32_t theta_den,
                 int64_t* cost_home, int64_t* cost_span, int64_t* load, int64_t* cost_home_fam,
                 int64_t* span_fam, int64_t* cross_fam, int64_t* home_mass_fam)
{
    const int32_t E = n_experts, k = top_k, G = n_gpus, L = n_layers, R = n_sec;
    const int stats = span_fam != NULL && cross_fam != NULL && home_mass_fam != NULL;
    int err = 0;
    if (G < 1 || G > 32 || k < 1 || k > 16 || k > E || E > 256 || R < 0 || R > 4 || n_fam < 1 || n_fam > 64 ||
        p_begin < 0 || p_end > n_place || p_begin > p_end) return ORC_ERR_ARG;
    if (R > 0 && (secondary == NULL || load_ref == NULL)) return ORC_ERR_ARG;
    if (fam_off[0] != 0 || fam_off[n_fam] != n_tokens) return ORC_ERR_ARG;
    for (int32_t f = 0; f < n_fam; ++f) {
        if (fam_off[f + 1] < fam_off[f]) return ORC_ERR_ARG;
        if (home_size[f] < 1 || home_start[f] < 0 || home_start[f] + home_size[f] > G) return ORC_ERR_ARG;
    }
    for (int32_t p = p_begin; p < p_end; ++p) {
        cost_home[p] = 0;
        cost_span[p] = 0;
        if (cost_home_fam)
            for (int32_t f = 0; f < n_fam; ++f) cost_home_fam[(int64_t)p * n_fam + f] = 0;
        if (stats)
            for (int32_t f = 0; f < n_fam; ++f) {
                span_fam[(int64_t)p * n_fam + f] = 0;
                cross_fam[(int64_t)p * n_fam + f] = 0;
                home_mass_fam[(int64_t)p * n_fam + f] = 0;
            }
    }
    const int64_t n_pl = (int64_t)(p_end - p_begin) * L;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (int64_t job = 0; job < n_pl; ++job) {
        const int32_t p = p_begin + (int32_t)(job / L), l = (int32_t)(job % L);
        const uint8_t* prim = primary + ((int64_t)p * L + l) * E;
        const uint8_t* sec = R > 0 ? secondary + (((int64_t)p * L + l) * E) * R : NULL;
        const int64_t* ref = R > 0 ? load_ref + ((int64_t)p * L + l) * G : NULL;
        int64_t* ld = load + ((int64_t)p * L + l) * G;
        for (int32_t m = 0; m < G; ++m) ld[m] = 0;
        int feas[32];
        feasible_gpus(ref, G, theta_num, theta_den, feas);
        int64_t st_span[64], st_cross[64], st_mass[64];
        for (int32_t f = 0; f < n_fam && f < 64; ++f) st_span[f] = st_cross[f] = st_mass[f] = 0;

        /* candidate set C_{l,e} of eq. candidate-set, and its feasible part (fallback: all) */
        int n_cand[256], cand[256][5], fc[256][32];
        for (int32_t e = 0; e < E; ++e) {
            n_cand[e] = 0;
            if (prim[e] >= G) { err |= ORC_ERR_TABLE; cand[e][n_cand[e]++] = 0; }
            else cand[e][n_cand[e]++] = prim[e];
            for (int32_t r = 0; r < R; ++r) {
                uint8_t g = sec[(int64_t)e * R + r];
                if (g == ORC_NONE) continue;
                if (g >= G) { err |= ORC_ERR_TABLE; continue; }
                int dup = 0;
                for (int c = 0; c < n_cand[e]; ++c) dup |= cand[e][c] == g;
                if (dup) { err |= ORC_ERR_TABLE; continue; }
                cand[e][n_cand[e]++] = g;
            }
            int any = 0;
            for (int32_t m = 0; m < G; ++m) fc[e][m] = 0;
            for (int c = 0; c < n_cand[e]; ++c)
                if (feas[cand[e][c]]) { fc[e][cand[e][c]] = 1; any = 1; }
            if (!any)
                for (int c = 0; c < n_cand[e]; ++c) fc[e][cand[e][c]] = 1;
        }

        int64_t home_acc = 0, span_acc = 0;
        int64_t fam_acc[64];
        for (int32_t f = 0; f < n_fam && f < 64; ++f) fam_acc[f] = 0;
        for (int32_t f = 0; f < n_fam; ++f) {
            for (int64_t t = fam_off[f]; t < fam_off[f + 1]; ++t) {
                const int16_t* ids = trace + ((int64_t)l * n_tokens + t) * k;
                int te = token_error(ids, k, E);
                if (te) { err |= te; continue; }
                const int32_t h = home_start[f] + (int32_t)((t - fam_off[f]) % home_size[f]);
                int in_r[32];
                int slot_gpu[16];
                for (int32_t m = 0; m < G; ++m) in_r[m] = 0;
                /* GPUs already accessed: every single-candidate expert goes to its primary */
                for (int32_t s = 0; s < k; ++s) {
                    int e = ids[s];
                    if (n_cand[e] == 1) { slot_gpu[s] = cand[e][0]; in_r[cand[e][0]] = 1; }
                    else slot_gpu[s] = -1;
                }
                /* multi-candidate experts in slot order: local, else anchor, else least loaded */
                for (int32_t s = 0; s < k; ++s) {
                    if (slot_gpu[s] >= 0) continue;
                    int e = ids[s], pick = -1;
                    for (int32_t m = 0; m < G && pick < 0; ++m)
                        if (fc[e][m] && in_r[m]) pick = m;
                    if (pick < 0 && fc[e][h]) pick = h;
                    if (pick < 0)
                        for (int32_t m = 0; m < G; ++m)
                            if (fc[e][m] && (pick < 0 || ref[m] < ref[pick])) pick = m;
                    slot_gpu[s] = pick;
                    in_r[pick] = 1;
                }
                int n_cards = 0;
                for (int32_t m = 0; m < G; ++m) n_cards += in_r[m];
                int64_t home_cost = n_cards - in_r[h];
                home_acc += home_cost;
                span_acc += n_cards - 1;
                if (f < 64) fam_acc[f] += home_cost;
                for (int32_t s = 0; s < k; ++s) ld[slot_gpu[s]] += 1;
                if (stats && f < 64) {
                    st_span[f] += n_cards - 1;
                    int within_one = 0;
                    for (int32_t f2 = 0; f2 < n_fam && !within_one; ++f2) {
                        int inside = 1;
                        for (int32_t m = 0; m < G; ++m)
                            if (in_r[m] && (m < home_start[f2] || m >= home_start[f2] + home_size[f2])) inside = 0;
                        within_one = inside;
                    }
                    st_cross[f] += !within_one;
                    for (int32_t s = 0; s < k; ++s)
                        st_mass[f] += slot_gpu[s] >= home_start[f] && slot_gpu[s] < home_start[f] + home_size[f];
                }
            }
        }
#pragma omp atomic
        cost_home[p] += home_acc;
#pragma omp atomic
        cost_span[p] += span_acc;
        if (cost_home_fam)
            for (int32_t f = 0; f < n_fam && f < 64; ++f) {
#pragma omp atomic
                cost_home_fam[(int64_t)p * n_fam + f] += fam_acc[f];
            }
        if (stats)
            for (int32_t f = 0; f < n_fam && f < 64; ++f) {
#pragma omp atomic
                span_fam[(int64_t)p * n_fam + f] += st_span[f];
#pragma omp atomic
                cross_fam[(int64_t)p * n_fam + f] += st_cross[f];
#pragma omp atomic
                home_mass_fam[(int64_t)p * n_fam + f] += st_mass[f];
            }
    }
    return err;
}

/*
 * Serving with decayed loads (Sec. 3.4 in its sequential form, eqs. mean-load, feasible-set and
 * load-update): the same per-token choice as oracle_score, but the loads L_m that the guard and the
 * least-loaded fallback read are exponentially decayed per-GPU dispatch loads, updated after every
 * token in trace order:
 *     L_m <- rho * L_m + Delta_m       (Delta_m = the token's slots served by m; one fused
 *                                       multiply-add in float64)
 * Each (placement, layer) keeps its own loads, starting from state[p][l][.] (zero when state is NULL)
 * and leaving the final loads there when state_out is not NULL.  The guard is the rational form
 * theta_den * G * L_m <= (theta_den + theta_num) * S with S = L_0 + L_1 + ... + L_{G-1} summed in that
 * order, each product rounded once in float64; theta_den == 0 disables it.  Ties of the least-loaded
 * choice go to the lowest GPU number.  Outputs as in oracle_score.
 */
int oracle_score_online(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k,
                        int32_t n_experts, const int64_t* fam_off, int32_t n_fam, const int32_t* home_start,
                        const int32_t* home_size, int32_t n_gpus, int32_t n_place, int32_t p_begin, int32_t p_end,
                        const uint8_t* primary, const uint8_t* secondary, int32_t n_sec, double rho,
                        int32_t theta_num, int32_t theta_den, const double* state_in, double* state_out,
                        int64_t* cost_home, int64_t* cost_span, int64_t* load, int64_t* cost_home_fam)
{
    const int32_t E = n_experts, k = top_k, G = n_gpus, L = n_layers, R = n_sec;
    int err = 0;
    if (G < 1 || G > 32 || k < 1 || k > 16 || k > E || E > 256 || R < 0 || R > 4 || n_fam < 1 || n_fam > 64 ||
        p_begin < 0 || p_end > n_place || p_begin > p_end) return ORC_ERR_ARG;
    if (R > 0 && secondary == NULL) return ORC_ERR_ARG;
    if (!(rho >= 0.0 && rho < 1.0)) return ORC_ERR_ARG;
    if (fam_off[0] != 0 || fam_off[n_fam] != n_tokens) return ORC_ERR_ARG;
    for (int32_t f = 0; f < n_fam; ++f) {
        if (fam_off[f + 1] < fam_off[f]) return ORC_ERR_ARG;
        if (home_size[f] < 1 || home_start[f] < 0 || home_start[f] + home_size[f] > G) return ORC_ERR_ARG;
    }
    for (int32_t p = p_begin; p < p_end; ++p) {
        cost_home[p] = 0;
        cost_span[p] = 0;
        if (cost_home_fam)
            for (int32_t f = 0; f < n_fam; ++f) cost_home_fam[(int64_t)p * n_fam + f] = 0;
    }
    const double gden = (double)theta_den * (double)G, rnum = (double)theta_den + (double)theta_num;
    const int64_t n_pl = (int64_t)(p_end - p_begin) * L;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (int64_t job = 0; job < n_pl; ++job) {
        const int32_t p = p_begin + (int32_t)(job / L), l = (int32_t)(job % L);
        const uint8_t* prim = primary + ((int64_t)p * L + l) * E;
        const uint8_t* sec = R > 0 ? secondary + (((int64_t)p * L + l) * E) * R : NULL;
        int64_t* ld = load + ((int64_t)p * L + l) * G;
        double Lm[32];
        for (int32_t m = 0; m < G; ++m) {
            ld[m] = 0;
            Lm[m] = state_in ? state_in[((int64_t)p * L + l) * G + m] : 0.0;
        }
        /* candidate set C_{l,e} of eq. candidate-set */
        int n_cand[256], cand[256][5];
        for (int32_t e = 0; e < E; ++e) {
            n_cand[e] = 0;
            if (prim[e] >= G) { err |= ORC_ERR_TABLE; cand[e][n_cand[e]++] = 0; }
            else cand[e][n_cand[e]++] = prim[e];
            for (int32_t r = 0; r < R; ++r) {
                uint8_t g = sec[(int64_t)e * R + r];
                if (g == ORC_NONE) continue;
                if (g >= G) { err |= ORC_ERR_TABLE; continue; }
                int dup = 0;
                for (int c = 0; c < n_cand[e]; ++c) dup |= cand[e][c] == g;
                if (dup) { err |= ORC_ERR_TABLE; continue; }
                cand[e][n_cand[e]++] = g;
            }
        }

        int64_t home_acc = 0, span_acc = 0;
        int64_t fam_acc[64];
        for (int32_t f = 0; f < n_fam && f < 64; ++f) fam_acc[f] = 0;
        for (int32_t f = 0; f < n_fam; ++f) {
            for (int64_t t = fam_off[f]; t < fam_off[f + 1]; ++t) {
                const int16_t* ids = trace + ((int64_t)l * n_tokens + t) * k;
                int te = token_error(ids, k, E);
                if (te) { err |= te; continue; }
                const int32_t h = home_start[f] + (int32_t)((t - fam_off[f]) % home_size[f]);
                /* feasible GPUs under the current loads (eq. feasible-set) */
                int feas[32];
                if (theta_den == 0) {
                    for (int32_t m = 0; m < G; ++m) feas[m] = 1;
                } else {
                    double S = 0.0;
                    for (int32_t m = 0; m < G; ++m) S += Lm[m];
                    const double rhs = rnum * S;
                    for (int32_t m = 0; m < G; ++m) feas[m] = gden * Lm[m] <= rhs;
                }
                int in_r[32], slot_gpu[16];
                for (int32_t m = 0; m < G; ++m) in_r[m] = 0;
                for (int32_t s = 0; s < k; ++s) {
                    int e = ids[s];
                    if (n_cand[e] == 1) { slot_gpu[s] = cand[e][0]; in_r[cand[e][0]] = 1; }
                    else slot_gpu[s] = -1;
                }
                for (int32_t s = 0; s < k; ++s) {
                    if (slot_gpu[s] >= 0) continue;
                    int e = ids[s], pick = -1;
                    int fc[32], any = 0;
                    for (int32_t m = 0; m < G; ++m) fc[m] = 0;
                    for (int c = 0; c < n_cand[e]; ++c)
                        if (feas[cand[e][c]]) { fc[cand[e][c]] = 1; any = 1; }
                    if (!any)
                        for (int c = 0; c < n_cand[e]; ++c) fc[cand[e][c]] = 1;
                    for (int32_t m = 0; m < G && pick < 0; ++m)
                        if (fc[m] && in_r[m]) pick = m;
                    if (pick < 0 && fc[h]) pick = h;
                    if (pick < 0)
                        for (int32_t m = 0; m < G; ++m)
                            if (fc[m] && (pick < 0 || Lm[m] < Lm[pick])) pick = m;
                    slot_gpu[s] = pick;
                    in_r[pick] = 1;
                }
                int n_cards = 0;
                for (int32_t m = 0; m < G; ++m) n_cards += in_r[m];
                int64_t home_cost = n_cards - in_r[h];
                home_acc += home_cost;
                span_acc += n_cards - 1;
                if (f < 64) fam_acc[f] += home_cost;
                int delta[32];
                for (int32_t m = 0; m < G; ++m) delta[m] = 0;
                for (int32_t s = 0; s < k; ++s) { ld[slot_gpu[s]] += 1; delta[slot_gpu[s]] += 1; }
                /* eq. load-update, after the token's dispatch */
                for (int32_t m = 0; m < G; ++m) Lm[m] = fma(rho, Lm[m], (double)delta[m]);
            }
        }
        if (state_out)
            for (int32_t m = 0; m < G; ++m) state_out[((int64_t)p * L + l) * G + m] = Lm[m];
#pragma omp atomic
        cost_home[p] += home_acc;
#pragma omp atomic
        cost_span[p] += span_acc;
        if (cost_home_fam)
            for (int32_t f = 0; f < n_fam && f < 64; ++f) {
#pragma omp atomic
                cost_home_fam[(int64_t)p * n_fam + f] += fam_acc[f];
            }
    }
    return err;
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the parallel loops that follow (timing only; results do not depend on it). */
void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    omp_set_num_threads(n < 1 ? 1 : n);
#else
    (void)n;
#endif
}
