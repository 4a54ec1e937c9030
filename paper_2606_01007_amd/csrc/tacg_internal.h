// Internal declarations shared by the HIP translation units of libtacg (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "tacg.h"

namespace tacg {

// Round a byte count up to the 256-byte alignment used for every workspace sub-buffer.
inline size_t align256(size_t x) { return (x + 255u) & ~size_t(255); }

// Workgroup barrier after LDS counters were incremented with relaxed atomics by several waves: first
// wait until this wave's LDS operations have completed (s_waitcnt lgkmcnt(0)), then synchronise.
// The compiler does not always emit that wait before the barrier after relaxed LDS atomics; without
// it a wave's last increments can land after another wave has read (and cleared) the counters.
__device__ __forceinline__ void barrier_after_lds_atomics() {
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0); vmcnt and expcnt at their maxima (no wait)
  __syncthreads();
}

// Bump allocator over a caller-provided workspace (device memory).  Only carves offsets.
struct Carver {
  char* base;
  size_t used;
  template <class T>
  T* take(size_t count) {
    T* p = reinterpret_cast<T*>(base ? base + used : nullptr);
    used += align256(count * sizeof(T));
    return p;
  }
};

// ---- co-activation build -------------------------------------------------------------------
int coact_num_workgroups(int64_t total_token_layers, int32_t n_experts, int32_t top_k);
size_t coact_bins(int32_t n_experts, int32_t top_k);
// small expert counts: the counts come from int8 matrix products (coact_mfma.hip)
bool coact_uses_mfma(int32_t n_experts, int32_t top_k);
int coact_mfma_workgroups(int64_t total_token_layers, int32_t n_experts);
int launch_coact_mfma_hist(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k,
                           int32_t n_experts, const int64_t* fam_off_host, int32_t n_fam, int32_t W, int32_t nbins,
                           uint32_t* partial, uint32_t* d_err, hipStream_t stream);

int launch_coact(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                 const int64_t* fam_off_host, int32_t n_fam, uint32_t* D, uint32_t* C, uint32_t flags,
                 uint32_t* d_err, void* workspace, hipStream_t stream);

// ---- reweighting ---------------------------------------------------------------------------
size_t reweight_workspace(int32_t n_fam, int32_t n_layers, int32_t n_experts);
int launch_reweight(const uint32_t* D, const uint32_t* C, int32_t n_fam, int32_t n_layers, int32_t n_experts,
                    int32_t top_k, double alpha, double tau, double eps, float* pref, float* a_tilde,
                    float* a_hat, void* workspace, hipStream_t stream);

int launch_gesr_scores(const uint32_t* D, const uint32_t* C, int32_t n_fam, int32_t n_layers, int32_t n_experts,
                       int32_t top_k, double* cent, double* cons, double* spec, hipStream_t stream);

int launch_activation_distance(const uint32_t* D, int32_t n_fam, int32_t n_layers, int32_t n_experts, int32_t top_k,
                               double* dist, hipStream_t stream);
int launch_pair_jaccard(const uint32_t* C, int32_t n_fam, int32_t n_layers, int32_t n_experts, int32_t top_n,
                        int32_t* top_pairs, double* jaccard, hipStream_t stream);

// ---- placement scoring ---------------------------------------------------------------------
// Optional App. C statistics of the snapshot scoring (all pointers device memory, [P][F]).
struct TraceStatsOut {
  uint64_t* span_fam;
  uint64_t* cross_fam;
  uint64_t* home_mass_fam;
  uint32_t band_starts;  // bit b set when a family band starts at GPU b (the bands tile 0..G-1)
};

size_t eval_workspace(int64_t n_tokens, int32_t n_layers, int32_t n_experts, int32_t n_gpus, int32_t n_place,
                      int32_t n_fam);
int launch_eval(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                const int64_t* fam_off_host, int32_t n_fam, const int32_t* home_start_host,
                const int32_t* home_size_host, int32_t n_gpus, int32_t n_place, const uint8_t* primary,
                const uint8_t* secondary, int32_t n_sec, const int64_t* load_ref, int32_t theta_num,
                int32_t theta_den, uint64_t* cost_home, uint64_t* cost_span, uint32_t* load,
                uint64_t* cost_home_fam, const TraceStatsOut* stats, uint32_t* d_err, void* workspace,
                hipStream_t stream);
int launch_eval_online(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                       const int64_t* fam_off_host, int32_t n_fam, const int32_t* home_start_host,
                       const int32_t* home_size_host, int32_t n_gpus, int32_t n_place, const uint8_t* primary,
                       const uint8_t* secondary, int32_t n_sec, double rho, int32_t theta_num, int32_t theta_den,
                       const double* state_in, double* state_out, uint64_t* cost_home, uint64_t* cost_span,
                       uint32_t* load, uint64_t* cost_home_fam, uint32_t* d_err, hipStream_t stream);
int launch_group_objective(const float* a_tilde, int32_t n_layers, int32_t n_experts, const uint8_t* primary,
                           int32_t n_place, int32_t n_gpus, double* objective, uint32_t* d_err, hipStream_t stream);
int launch_placement_load(const uint32_t* D, int32_t n_fam, int32_t n_layers, int32_t n_experts,
                          const uint8_t* primary, int32_t n_place, int32_t n_gpus, int64_t* load_ref,
                          uint32_t* d_err, hipStream_t stream);
int launch_jain(const uint32_t* load, int32_t n_place, int32_t n_layers, int32_t n_gpus, int32_t per_layer,
                float* jain, float* maxvio, hipStream_t stream);

}  // namespace tacg
