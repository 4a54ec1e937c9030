// C ABI of libtacg: host-side argument validation, then enqueue on the caller's stream.
// Argument errors return before any HIP call, so they can be exercised on a machine without a GPU.
#include <cstdint>
#include <mutex>

#include "tacg_internal.h"

namespace {

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Common trace checks: shapes, limits and the family offsets.
int check_trace(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                const int64_t* fam_off_host, int32_t n_fam) {
  if (n_tokens < 0 || n_layers < 1 || n_fam < 1 || n_experts < 1 || top_k < 1) return TACG_E_INVAL;
  if (top_k > n_experts) return TACG_E_INVAL;
  if (n_experts > TACG_MAX_EXPERTS || top_k > TACG_MAX_TOPK || n_fam > TACG_MAX_FAMILIES) return TACG_E_UNSUPPORTED;
  if (n_tokens * static_cast<int64_t>(top_k) >= (int64_t(1) << 32)) return TACG_E_UNSUPPORTED;
  if (n_tokens > 0 && (trace == nullptr || !aligned(trace, 16))) return TACG_E_INVAL;
  if (fam_off_host == nullptr) return TACG_E_INVAL;
  if (fam_off_host[0] != 0 || fam_off_host[n_fam] != n_tokens) return TACG_E_INVAL;
  for (int f = 0; f < n_fam; ++f)
    if (fam_off_host[f + 1] < fam_off_host[f]) return TACG_E_INVAL;
  return TACG_OK;
}

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

}  // namespace

extern "C" {

size_t tacg_coact_workspace_bytes(int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                                  int32_t n_fam) {
  if (n_tokens < 0 || n_layers < 1 || top_k < 1 || n_experts < 1 || n_fam < 1) return 0;
  const int64_t total = n_tokens * n_layers;
  const int64_t W = tacg::coact_num_workgroups(total, n_experts, top_k);
  const size_t slots = static_cast<size_t>(W) + static_cast<size_t>(n_layers) * n_fam;
  return tacg::align256(slots * tacg::coact_bins(n_experts, top_k) * sizeof(uint32_t));
}

int tacg_coact_uses_matrix_cores(int32_t n_experts, int32_t top_k) {
  if (n_experts < 1 || n_experts > TACG_MAX_EXPERTS || top_k < 1 || top_k > TACG_MAX_TOPK) return 0;
  if (top_k > n_experts) return 0;
  return tacg::coact_uses_mfma(n_experts, top_k) ? 1 : 0;
}

int tacg_coact_build(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                     const int64_t* fam_off_host, int32_t n_fam, uint32_t* D, uint32_t* C, uint32_t flags,
                     uint32_t* d_err, void* workspace, size_t workspace_bytes, void* hip_stream) {
  int rc = check_trace(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam);
  if (rc != TACG_OK) return rc;
  if (D == nullptr || C == nullptr || d_err == nullptr) return TACG_E_INVAL;
  if ((flags & ~TACG_ACCUMULATE) != 0) return TACG_E_INVAL;
  const size_t need = tacg_coact_workspace_bytes(n_tokens, n_layers, top_k, n_experts, n_fam);
  if (workspace == nullptr || workspace_bytes < need || !aligned(workspace, 256)) return TACG_E_INVAL;
  return tacg::launch_coact(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam, D, C, flags, d_err,
                            workspace, as_stream(hip_stream));
}

size_t tacg_reweight_workspace_bytes(int32_t n_fam, int32_t n_layers, int32_t n_experts) {
  if (n_fam < 1 || n_layers < 1 || n_experts < 1) return 0;
  return tacg::reweight_workspace(n_fam, n_layers, n_experts);
}

int tacg_reweight(const uint32_t* D, const uint32_t* C, int32_t n_fam, int32_t n_layers, int32_t n_experts,
                  int32_t top_k, double alpha, double tau, double eps, float* pref, float* a_tilde,
                  float* a_hat_or_null, void* workspace, size_t workspace_bytes, void* hip_stream) {
  if (D == nullptr || C == nullptr || pref == nullptr || a_tilde == nullptr) return TACG_E_INVAL;
  if (n_fam < 2 || n_layers < 1 || n_experts < 1 || top_k < 1 || top_k > n_experts) return TACG_E_INVAL;
  if (n_experts > TACG_MAX_EXPERTS || n_fam > TACG_MAX_FAMILIES || top_k > TACG_MAX_TOPK) return TACG_E_UNSUPPORTED;
  if (!(alpha >= 0.0 && alpha <= 1.0) || !(tau > 0.0) || !(eps >= 0.0)) return TACG_E_INVAL;
  const size_t need = tacg_reweight_workspace_bytes(n_fam, n_layers, n_experts);
  if (workspace == nullptr || workspace_bytes < need || !aligned(workspace, 256)) return TACG_E_INVAL;
  return tacg::launch_reweight(D, C, n_fam, n_layers, n_experts, top_k, alpha, tau, eps, pref, a_tilde,
                               a_hat_or_null, workspace, as_stream(hip_stream));
}

int tacg_gesr_scores(const uint32_t* D, const uint32_t* C, int32_t n_fam, int32_t n_layers, int32_t n_experts,
                     int32_t top_k, double* cent, double* cons, double* spec, void* hip_stream) {
  if (D == nullptr || C == nullptr || cent == nullptr || cons == nullptr || spec == nullptr) return TACG_E_INVAL;
  if (n_fam < 1 || n_layers < 1 || n_experts < 1 || top_k < 1 || top_k > n_experts) return TACG_E_INVAL;
  if (n_experts > TACG_MAX_EXPERTS || n_fam > TACG_MAX_FAMILIES || top_k > TACG_MAX_TOPK) return TACG_E_UNSUPPORTED;
  if (n_layers > 65535) return TACG_E_UNSUPPORTED;
  return tacg::launch_gesr_scores(D, C, n_fam, n_layers, n_experts, top_k, cent, cons, spec, as_stream(hip_stream));
}

int tacg_activation_distance(const uint32_t* D, int32_t n_fam, int32_t n_layers, int32_t n_experts, int32_t top_k,
                             double* dist, void* hip_stream) {
  if (D == nullptr || dist == nullptr) return TACG_E_INVAL;
  if (n_fam < 1 || n_layers < 1 || n_experts < 1 || top_k < 1 || top_k > n_experts) return TACG_E_INVAL;
  if (n_experts > TACG_MAX_EXPERTS || n_fam > TACG_MAX_FAMILIES || top_k > TACG_MAX_TOPK) return TACG_E_UNSUPPORTED;
  return tacg::launch_activation_distance(D, n_fam, n_layers, n_experts, top_k, dist, as_stream(hip_stream));
}

int tacg_pair_jaccard(const uint32_t* C, int32_t n_fam, int32_t n_layers, int32_t n_experts, int32_t top_n,
                      int32_t* top_pairs, double* jaccard, void* hip_stream) {
  if (C == nullptr || top_pairs == nullptr || jaccard == nullptr) return TACG_E_INVAL;
  if (n_fam < 1 || n_layers < 1 || n_experts < 2 || top_n < 1) return TACG_E_INVAL;
  if (n_experts > TACG_MAX_EXPERTS || n_fam > TACG_MAX_FAMILIES || top_n > TACG_MAX_TOP_PAIRS || n_layers > 65535)
    return TACG_E_UNSUPPORTED;
  return tacg::launch_pair_jaccard(C, n_fam, n_layers, n_experts, top_n, top_pairs, jaccard, as_stream(hip_stream));
}

int tacg_placement_load(const uint32_t* D, int32_t n_fam, int32_t n_layers, int32_t n_experts,
                        const uint8_t* primary, int32_t n_place, int32_t n_gpus, int64_t* load_ref, uint32_t* d_err,
                        void* hip_stream) {
  if (D == nullptr || primary == nullptr || load_ref == nullptr || d_err == nullptr) return TACG_E_INVAL;
  if (n_fam < 1 || n_layers < 1 || n_experts < 1 || n_place < 0 || n_gpus < 1) return TACG_E_INVAL;
  if (n_experts > TACG_MAX_EXPERTS || n_fam > TACG_MAX_FAMILIES || n_gpus > TACG_MAX_GPUS) return TACG_E_UNSUPPORTED;
  if (n_place == 0) return TACG_OK;
  return tacg::launch_placement_load(D, n_fam, n_layers, n_experts, primary, n_place, n_gpus, load_ref, d_err,
                                     as_stream(hip_stream));
}

size_t tacg_eval_workspace_bytes(int64_t n_tokens, int32_t n_layers, int32_t n_experts, int32_t n_gpus,
                                 int32_t n_place, int32_t n_fam) {
  if (n_tokens < 0 || n_layers < 1 || n_experts < 1 || n_gpus < 1 || n_place < 1 || n_fam < 1) return 0;
  return tacg::eval_workspace(n_tokens, n_layers, n_experts, n_gpus, n_place, n_fam);
}

}  // extern "C"

namespace {

// Checks shared by the snapshot-scoring entry points (everything but the workspace).
int check_eval_args(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                    const int64_t* fam_off_host, int32_t n_fam, const int32_t* home_start_host,
                    const int32_t* home_size_host, int32_t n_gpus, int32_t n_place, const uint8_t* primary,
                    const uint8_t* secondary_or_null, int32_t n_sec, const int64_t* load_ref_or_null,
                    int32_t theta_num, int32_t theta_den, const uint64_t* cost_home, const uint64_t* cost_span,
                    const uint32_t* load, uint32_t flags, const uint32_t* d_err) {
  int rc = check_trace(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam);
  if (rc != TACG_OK) return rc;
  if (flags != 0) return TACG_E_INVAL;
  if (n_gpus < 1 || n_place < 1 || n_sec < 0) return TACG_E_INVAL;
  if (n_gpus > TACG_MAX_GPUS || n_sec > TACG_MAX_SECONDARY) return TACG_E_UNSUPPORTED;
  if (primary == nullptr || cost_home == nullptr || cost_span == nullptr || load == nullptr || d_err == nullptr)
    return TACG_E_INVAL;
  if (n_sec > 0 && (secondary_or_null == nullptr || load_ref_or_null == nullptr)) return TACG_E_INVAL;
  if (theta_num < 0 || theta_den < 0 || (theta_den > 0 && theta_num > (1 << 20)) || theta_den > (1 << 20))
    return TACG_E_INVAL;
  if (home_start_host == nullptr || home_size_host == nullptr) return TACG_E_INVAL;
  for (int f = 0; f < n_fam; ++f) {
    if (home_size_host[f] < 1 || home_start_host[f] < 0 || home_start_host[f] + home_size_host[f] > n_gpus)
      return TACG_E_INVAL;
  }
  return TACG_OK;
}

// ... plus a caller-owned workspace of tacg_eval_workspace_bytes(...) bytes, 256-byte aligned.
int check_eval(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
               const int64_t* fam_off_host, int32_t n_fam, const int32_t* home_start_host,
               const int32_t* home_size_host, int32_t n_gpus, int32_t n_place, const uint8_t* primary,
               const uint8_t* secondary_or_null, int32_t n_sec, const int64_t* load_ref_or_null, int32_t theta_num,
               int32_t theta_den, const uint64_t* cost_home, const uint64_t* cost_span, const uint32_t* load,
               uint32_t flags, const uint32_t* d_err, const void* workspace, size_t workspace_bytes) {
  const int rc = check_eval_args(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam, home_start_host,
                                 home_size_host, n_gpus, n_place, primary, secondary_or_null, n_sec,
                                 load_ref_or_null, theta_num, theta_den, cost_home, cost_span, load, flags, d_err);
  if (rc != TACG_OK) return rc;
  const size_t need = tacg_eval_workspace_bytes(n_tokens, n_layers, n_experts, n_gpus, n_place, n_fam);
  if (workspace == nullptr || workspace_bytes < need || !aligned(workspace, 256)) return TACG_E_INVAL;
  return TACG_OK;
}

// ---- device scratch of tacg_eval_placements_noalloc ----
// One copy of this array lives on every GPU the library runs on, from the first use until the process
// ends.  In host code its name is only a stand-in for the symbol: the device address of each GPU's
// copy comes from hipGetSymbolAddress with that GPU current, and only that address is handed to
// kernels.
static __device__ __align__(256) unsigned char scratch[TACG_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current GPU's scratch (looked up once per device).
int current_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TACG_E_DEVICE;
  std::lock_guard<std::mutex> guard(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return TACG_E_DEVICE;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return TACG_OK;
}

// Do the distinct family bands tile 0..G-1 without overlap?  Then every GPU belongs to exactly one
// band and `starts` gets bit b for every band start b.
bool bands_tile(const int32_t* home_start, const int32_t* home_size, int32_t n_fam, int32_t G, uint32_t* starts) {
  int32_t owner_start[TACG_MAX_GPUS], owner_size[TACG_MAX_GPUS];
  for (int g = 0; g < G; ++g) owner_start[g] = -1;
  for (int f = 0; f < n_fam; ++f) {
    for (int g = home_start[f]; g < home_start[f] + home_size[f]; ++g) {
      if (owner_start[g] < 0) {
        owner_start[g] = home_start[f];
        owner_size[g] = home_size[f];
      } else if (owner_start[g] != home_start[f] || owner_size[g] != home_size[f]) {
        return false;  // two different bands overlap
      }
    }
  }
  uint32_t b = 0;
  for (int g = 0; g < G; ++g) {
    if (owner_start[g] < 0) return false;  // a GPU outside every band
    if (owner_start[g] == g) b |= 1u << g;
  }
  *starts = b;
  return true;
}

}  // namespace

extern "C" {

int tacg_eval_placements(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k,
                         int32_t n_experts, const int64_t* fam_off_host, int32_t n_fam,
                         const int32_t* home_start_host, const int32_t* home_size_host, int32_t n_gpus,
                         int32_t n_place, const uint8_t* primary, const uint8_t* secondary_or_null, int32_t n_sec,
                         const int64_t* load_ref_or_null, int32_t theta_num, int32_t theta_den,
                         uint64_t* cost_home, uint64_t* cost_span, uint32_t* load,
                         uint64_t* cost_home_fam_or_null, uint32_t flags, uint32_t* d_err, void* workspace,
                         size_t workspace_bytes, void* hip_stream) {
  const int rc = check_eval(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam, home_start_host,
                            home_size_host, n_gpus, n_place, primary, secondary_or_null, n_sec, load_ref_or_null,
                            theta_num, theta_den, cost_home, cost_span, load, flags, d_err, workspace,
                            workspace_bytes);
  if (rc != TACG_OK) return rc;
  return tacg::launch_eval(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam, home_start_host,
                           home_size_host, n_gpus, n_place, primary, secondary_or_null, n_sec, load_ref_or_null,
                           theta_num, theta_den, cost_home, cost_span, load, cost_home_fam_or_null, nullptr, d_err,
                           workspace, as_stream(hip_stream));
}

int tacg_eval_placements_noalloc(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k,
                                 int32_t n_experts, const int64_t* fam_off_host, int32_t n_fam,
                                 const int32_t* home_start_host, const int32_t* home_size_host, int32_t n_gpus,
                                 int32_t n_place, const uint8_t* primary, const uint8_t* secondary_or_null,
                                 int32_t n_sec, const int64_t* load_ref_or_null, int32_t theta_num,
                                 int32_t theta_den, uint64_t* cost_home, uint64_t* cost_span, uint32_t* load,
                                 uint64_t* cost_home_fam_or_null, uint32_t flags, uint32_t* d_err,
                                 void* hip_stream) {
  const int rc = check_eval_args(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam, home_start_host,
                                 home_size_host, n_gpus, n_place, primary, secondary_or_null, n_sec,
                                 load_ref_or_null, theta_num, theta_den, cost_home, cost_span, load, flags, d_err);
  if (rc != TACG_OK) return rc;
  if (tacg_eval_workspace_bytes(n_tokens, n_layers, n_experts, n_gpus, n_place, n_fam) > TACG_NOALLOC_SCRATCH_BYTES)
    return TACG_E_SCRATCH;
  void* ws = nullptr;
  const int sr = current_scratch(&ws);
  if (sr != TACG_OK) return sr;
  return tacg::launch_eval(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam, home_start_host,
                           home_size_host, n_gpus, n_place, primary, secondary_or_null, n_sec, load_ref_or_null,
                           theta_num, theta_den, cost_home, cost_span, load, cost_home_fam_or_null, nullptr, d_err,
                           ws, as_stream(hip_stream));
}

int tacg_eval_trace_stats(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k,
                          int32_t n_experts, const int64_t* fam_off_host, int32_t n_fam,
                          const int32_t* home_start_host, const int32_t* home_size_host, int32_t n_gpus,
                          int32_t n_place, const uint8_t* primary, const uint8_t* secondary_or_null,
                          int32_t n_sec, const int64_t* load_ref_or_null, int32_t theta_num,
                          int32_t theta_den, uint64_t* cost_home, uint64_t* cost_span, uint32_t* load,
                          uint64_t* span_fam, uint64_t* cross_fam, uint64_t* home_mass_fam, uint32_t flags,
                          uint32_t* d_err, void* workspace, size_t workspace_bytes, void* hip_stream) {
  const int rc = check_eval(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam, home_start_host,
                            home_size_host, n_gpus, n_place, primary, secondary_or_null, n_sec, load_ref_or_null,
                            theta_num, theta_den, cost_home, cost_span, load, flags, d_err, workspace,
                            workspace_bytes);
  if (rc != TACG_OK) return rc;
  if (span_fam == nullptr || cross_fam == nullptr || home_mass_fam == nullptr) return TACG_E_INVAL;
  tacg::TraceStatsOut st{span_fam, cross_fam, home_mass_fam, 0u};
  if (!bands_tile(home_start_host, home_size_host, n_fam, n_gpus, &st.band_starts)) return TACG_E_UNSUPPORTED;
  return tacg::launch_eval(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam, home_start_host,
                           home_size_host, n_gpus, n_place, primary, secondary_or_null, n_sec, load_ref_or_null,
                           theta_num, theta_den, cost_home, cost_span, load, nullptr, &st, d_err, workspace,
                           as_stream(hip_stream));
}

int tacg_eval_online(const int16_t* trace, int64_t n_tokens, int32_t n_layers, int32_t top_k, int32_t n_experts,
                     const int64_t* fam_off_host, int32_t n_fam, const int32_t* home_start_host,
                     const int32_t* home_size_host, int32_t n_gpus, int32_t n_place, const uint8_t* primary,
                     const uint8_t* secondary_or_null, int32_t n_sec, double rho, int32_t theta_num,
                     int32_t theta_den, const double* state_in_or_null, double* state_out_or_null,
                     uint64_t* cost_home, uint64_t* cost_span, uint32_t* load, uint64_t* cost_home_fam_or_null,
                     uint32_t flags, uint32_t* d_err, void* hip_stream) {
  int rc = check_trace(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam);
  if (rc != TACG_OK) return rc;
  if (flags != 0) return TACG_E_INVAL;
  if (n_gpus < 1 || n_place < 1 || n_sec < 0) return TACG_E_INVAL;
  if (n_gpus > TACG_MAX_GPUS || n_sec > TACG_MAX_SECONDARY) return TACG_E_UNSUPPORTED;
  if (primary == nullptr || cost_home == nullptr || cost_span == nullptr || load == nullptr || d_err == nullptr)
    return TACG_E_INVAL;
  if (n_sec > 0 && secondary_or_null == nullptr) return TACG_E_INVAL;
  if (!(rho >= 0.0 && rho < 1.0)) return TACG_E_INVAL;
  if (theta_num < 0 || theta_den < 0 || (theta_den > 0 && theta_num > (1 << 20)) || theta_den > (1 << 20))
    return TACG_E_INVAL;
  if (home_start_host == nullptr || home_size_host == nullptr) return TACG_E_INVAL;
  for (int f = 0; f < n_fam; ++f) {
    if (home_size_host[f] < 1 || home_start_host[f] < 0 || home_start_host[f] + home_size_host[f] > n_gpus)
      return TACG_E_INVAL;
  }
  return tacg::launch_eval_online(trace, n_tokens, n_layers, top_k, n_experts, fam_off_host, n_fam, home_start_host,
                                  home_size_host, n_gpus, n_place, primary, secondary_or_null, n_sec, rho, theta_num,
                                  theta_den, state_in_or_null, state_out_or_null, cost_home, cost_span, load,
                                  cost_home_fam_or_null, d_err, as_stream(hip_stream));
}

int tacg_group_objective(const float* a_tilde, int32_t n_layers, int32_t n_experts, const uint8_t* primary,
                         int32_t n_place, int32_t n_gpus, double* objective, uint32_t* d_err, void* hip_stream) {
  if (a_tilde == nullptr || primary == nullptr || objective == nullptr || d_err == nullptr) return TACG_E_INVAL;
  if (n_layers < 1 || n_experts < 1 || n_place < 0 || n_gpus < 1) return TACG_E_INVAL;
  if (n_experts > TACG_MAX_EXPERTS || n_gpus > TACG_MAX_GPUS) return TACG_E_UNSUPPORTED;
  if (n_place == 0) return TACG_OK;
  if (n_layers > 65535) return TACG_E_UNSUPPORTED;
  return tacg::launch_group_objective(a_tilde, n_layers, n_experts, primary, n_place, n_gpus, objective, d_err,
                                      as_stream(hip_stream));
}

int tacg_jain(const uint32_t* load, int32_t n_place, int32_t n_layers, int32_t n_gpus, int32_t per_layer,
              float* jain, float* maxvio, void* hip_stream) {
  if (load == nullptr || jain == nullptr || maxvio == nullptr) return TACG_E_INVAL;
  if (n_place < 0 || n_layers < 1 || n_gpus < 1 || (per_layer != 0 && per_layer != 1)) return TACG_E_INVAL;
  if (n_gpus > TACG_MAX_GPUS) return TACG_E_UNSUPPORTED;
  if (n_place == 0) return TACG_OK;
  return tacg::launch_jain(load, n_place, n_layers, n_gpus, per_layer, jain, maxvio, as_stream(hip_stream));
}

const char* tacg_strerror(int status) {
  switch (status) {
    case TACG_OK:
      return "ok";
    case TACG_E_INVAL:
      return "invalid argument";
    case TACG_E_UNSUPPORTED:
      return "argument beyond a supported limit";
    case TACG_E_DEVICE:
      return "HIP launch failed";
    case TACG_E_SCRATCH:
      return "input needs more scratch than the no-allocation entry point holds (TACG_NOALLOC_SCRATCH_BYTES)";
    default:
      return "unknown status";
  }
}

}  // extern "C"
