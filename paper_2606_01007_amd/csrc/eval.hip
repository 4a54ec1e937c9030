// Placement scoring: per-token cross-GPU cost, GESR candidate choice and per-GPU loads
// (Sec. 3.4 serving rule with eqs. mean-load and feasible-set; App. C per-token dispatch sets;
// App. H "Comm"), plus the snapshot loads that feed the guard and Jain / MaxVio (App. H).
//
// Launch sequence of tacg_eval_placements:
//   ev_zero      clear the workspace accumulators
//   ev_count     per-layer expert dispatch counts of the trace (and trace validation)
//   ev_flags     validate the placement tables; mark experts that have a secondary in any placement
//   ev_replist   per layer: compact index of the marked ("replicated") experts
//   ev_repinfo   per (placement, layer, replicated expert): feasible candidate mask FC and the
//                fallback GPU argmin_{m in FC} load_ref (ties: lowest number)
//   ev_main      the trace pass (below)
//   ev_finalize  loads = counts of single-candidate experts on their primary + replicated choices;
//                costs from the accumulators
//
// ev_main (the hot kernel).  Lane = placement, wave = 64 placements, every wave of a workgroup scores
// the same placements on different tokens, so a token's expert ids are wave-uniform:
//   * LDS holds, for the workgroup's placements and layer, the one-hot GPU mask of every expert
//     (tbl[e][p], uint32; zero for replicated experts), the replica info (FC, fallback) and
//     per-placement counters of the GPUs chosen for replicated experts.
//   * A wave loads 64 token-layers at once (one coalesced load per lane), turns each id into the LDS
//     byte offset of its table row (packed two per dword) and builds a per-token word with the
//     replicated-slot mask and the anchor GPU; the per-token loop then broadcasts them with
//     v_readlane, so the row offsets live in SGPRs.
//   * Per token-layer and lane: k conflict-free LDS reads (64 consecutive dwords per wave), OR of the
//     masks, then (rarely) the replicated slots, then two popcounts into per-lane accumulators.
#include "tacg_internal.h"

namespace tacg {
namespace {

constexpr int kMainThreads = 1024;
constexpr int kMaxPieces = 256;
constexpr uint8_t kNone = 0xFF;

struct EvWs {
  uint32_t* cnt;        // [L][E] dispatches per expert
  uint32_t* flagbits;   // [L][8] experts with a secondary in some placement
  uint8_t* rep_of;      // [L][E] compact replicated index or 0xFF
  int32_t* rep_list;    // [L][TACG_MAX_REPLICATED]
  int32_t* n_rep;       // [L]
  uint2* rep_info;      // [L][TACG_MAX_REPLICATED][P]  (FC mask, fallback GPU)
  unsigned long long* acc_home;  // [P]
  unsigned long long* acc_span;  // [P]
  unsigned long long* acc_fam;   // [P][F]
  uint32_t* rep_load;   // [P][L][G]
};

EvWs carve_ev(void* ws, int32_t L, int32_t E, int32_t G, int32_t P, int32_t F, size_t* used = nullptr) {
  Carver c{static_cast<char*>(ws), 0};
  EvWs r;
  r.cnt = c.take<uint32_t>(static_cast<size_t>(L) * E);
  r.flagbits = c.take<uint32_t>(static_cast<size_t>(L) * 8);
  r.acc_home = c.take<unsigned long long>(static_cast<size_t>(P));
  r.acc_span = c.take<unsigned long long>(static_cast<size_t>(P));
  r.acc_fam = c.take<unsigned long long>(static_cast<size_t>(P) * F);
  r.rep_load = c.take<uint32_t>(static_cast<size_t>(P) * L * G);
  r.rep_of = c.take<uint8_t>(static_cast<size_t>(L) * E);
  r.rep_list = c.take<int32_t>(static_cast<size_t>(L) * TACG_MAX_REPLICATED);
  r.n_rep = c.take<int32_t>(static_cast<size_t>(L));
  r.rep_info = c.take<uint2>(static_cast<size_t>(L) * TACG_MAX_REPLICATED * P);
  if (used) *used = c.used;
  return r;
}

struct EvArgs {
  const int16_t* trace;
  const uint8_t* primary;
  const uint8_t* secondary;
  const int64_t* load_ref;
  uint32_t* d_err;
  EvWs ws;
  int64_t N;
  int32_t L, K, E, F, G, P, R;
  int32_t theta_num, theta_den;
  int32_t n_pieces;
  uint32_t fam_off[TACG_MAX_FAMILIES + 1];
  uint8_t home_start[TACG_MAX_FAMILIES];
  uint8_t home_size[TACG_MAX_FAMILIES];
  uint32_t piece_begin[kMaxPieces + 1];  // token ranges [piece_begin[j], piece_begin[j+1]) in one family
  uint8_t piece_fam[kMaxPieces];
};

// ------------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void ev_zero(EvArgs a) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  const EvWs& w = a.ws;
  for (int64_t j = i; j < static_cast<int64_t>(a.L) * a.E; j += stride) w.cnt[j] = 0;
  for (int64_t j = i; j < static_cast<int64_t>(a.L) * 8; j += stride) w.flagbits[j] = 0;
  for (int64_t j = i; j < a.P; j += stride) {
    w.acc_home[j] = 0;
    w.acc_span[j] = 0;
  }
  for (int64_t j = i; j < static_cast<int64_t>(a.P) * a.F; j += stride) w.acc_fam[j] = 0;
  for (int64_t j = i; j < static_cast<int64_t>(a.P) * a.L * a.G; j += stride) w.rep_load[j] = 0;
}

// Expert dispatch counts per layer; validates ids (range, repeats).  grid (splits, L).
__global__ __launch_bounds__(256) void ev_count(EvArgs a) {
  __shared__ uint32_t h[TACG_MAX_EXPERTS];
  const int l = blockIdx.y;
  for (int i = threadIdx.x; i < a.E; i += blockDim.x) h[i] = 0;
  __syncthreads();
  const int64_t n = a.N;
  const int64_t t0 = n * blockIdx.x / gridDim.x, t1 = n * (blockIdx.x + 1) / gridDim.x;
  uint32_t err = 0;
  for (int64_t t = t0 + threadIdx.x; t < t1; t += blockDim.x) {
    const int16_t* ids = a.trace + (static_cast<int64_t>(l) * n + t) * a.K;
    int v[TACG_MAX_TOPK];
    bool ok = true;
    for (int s = 0; s < a.K; ++s) {
      v[s] = ids[s];
      if (v[s] < 0 || v[s] >= a.E) {
        err |= TACG_ERR_ID_RANGE;
        ok = false;
      }
      for (int q = 0; q < s; ++q)
        if (v[q] == v[s]) {
          err |= TACG_ERR_ID_DUP;
          ok = false;
        }
    }
    if (ok)
      for (int s = 0; s < a.K; ++s) atomicAdd(&h[v[s]], 1u);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < a.E; i += blockDim.x)
    if (h[i]) atomicAdd(&a.ws.cnt[static_cast<int64_t>(l) * a.E + i], h[i]);
  if (err) atomicOr(a.d_err, err);
}

// Table validation and the replicated-expert marks.  grid (P, L), one thread per expert.
__global__ __launch_bounds__(256) void ev_flags(EvArgs a) {
  const int p = blockIdx.x, l = blockIdx.y;
  uint32_t err = 0;
  for (int e = threadIdx.x; e < a.E; e += blockDim.x) {
    const int64_t pe = (static_cast<int64_t>(p) * a.L + l) * a.E + e;
    const uint8_t g0 = a.primary[pe];
    if (g0 >= a.G) err |= TACG_ERR_TABLE;
    bool any = false;
    uint32_t seen = g0 < a.G ? (1u << g0) : 0u;
    for (int r = 0; r < a.R; ++r) {
      const uint8_t g = a.secondary[pe * a.R + r];
      if (g == kNone) continue;
      if (g >= a.G || (seen >> g) & 1u) {
        err |= TACG_ERR_TABLE;
        continue;
      }
      seen |= 1u << g;
      any = true;
    }
    if (any) atomicOr(&a.ws.flagbits[l * 8 + (e >> 5)], 1u << (e & 31));
  }
  if (err) atomicOr(a.d_err, err);
}

// Compact indices of the marked experts of each layer.  grid (L), 256 threads (one per expert).
__global__ __launch_bounds__(256) void ev_replist(EvArgs a) {
  __shared__ int32_t cnt;
  const int l = blockIdx.x, e = threadIdx.x;
  if (e == 0) cnt = 0;
  __syncthreads();
  if (e < a.E) {
    const bool mark = (a.ws.flagbits[l * 8 + (e >> 5)] >> (e & 31)) & 1u;
    // rank among marked experts = number of marked experts below e
    int rank = 0;
    for (int q = 0; q < (e >> 5); ++q) rank += __popc(a.ws.flagbits[l * 8 + q]);
    rank += __popc(a.ws.flagbits[l * 8 + (e >> 5)] & ((1u << (e & 31)) - 1u));
    uint8_t r = kNone;
    if (mark) {
      atomicAdd(&cnt, 1);
      if (rank < TACG_MAX_REPLICATED) {
        r = static_cast<uint8_t>(rank);
        a.ws.rep_list[l * TACG_MAX_REPLICATED + rank] = e;
      }
    }
    a.ws.rep_of[static_cast<int64_t>(l) * a.E + e] = r;
  }
  __syncthreads();
  if (e == 0) {
    a.ws.n_rep[l] = min(cnt, TACG_MAX_REPLICATED);
    if (cnt > TACG_MAX_REPLICATED) atomicOr(a.d_err, TACG_ERR_LIMIT);
  }
}

// Feasible candidates and fallback for every (placement, layer, replicated expert).
// grid (ceil(P / 256), L), one thread per placement.
__global__ __launch_bounds__(256) void ev_repinfo(EvArgs a) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x, l = blockIdx.y;
  if (p >= a.P) return;
  const int nrep = a.ws.n_rep[l];
  if (nrep == 0) return;
  const int G = a.G;
  const int64_t* ref = a.load_ref + (static_cast<int64_t>(p) * a.L + l) * G;
  // eq. feasible-set with the mean load of eq. mean-load, exact in 128-bit integers
  uint32_t feas = (G == 32) ? 0xffffffffu : ((1u << G) - 1u);
  if (a.theta_den != 0) {
    __int128 total = 0;
    for (int m = 0; m < G; ++m) total += ref[m];
    const __int128 rhs = static_cast<__int128>(a.theta_den + a.theta_num) * total;
    feas = 0;
    for (int m = 0; m < G; ++m)
      if (static_cast<__int128>(a.theta_den) * G * ref[m] <= rhs) feas |= 1u << m;
  }
  for (int r = 0; r < nrep; ++r) {
    const int e = a.ws.rep_list[l * TACG_MAX_REPLICATED + r];
    const int64_t pe = (static_cast<int64_t>(p) * a.L + l) * a.E + e;
    uint32_t cand = 0;
    const uint8_t g0 = a.primary[pe];
    if (g0 < G) cand |= 1u << g0;
    for (int q = 0; q < a.R; ++q) {
      const uint8_t g = a.secondary[pe * a.R + q];
      if (g < G) cand |= 1u << g;
    }
    if (cand == 0) cand = 1u;  // invalid table (already flagged): keep the choice in range
    uint32_t fc = cand & feas;
    if (fc == 0) fc = cand;
    int best = -1;
    for (int m = 0; m < G; ++m)
      if (((fc >> m) & 1u) && (best < 0 || ref[m] < ref[best])) best = m;
    a.ws.rep_info[(static_cast<int64_t>(l) * TACG_MAX_REPLICATED + r) * a.P + p] =
        make_uint2(fc, static_cast<uint32_t>(best));
  }
}

// ------------------------------------------------------------------------------------------------
// The trace pass.  PPL placements per lane; workgroup = 64 * PPL placements of one layer and one
// piece of one family's tokens.  grid (placement blocks, pieces, L).
template <int K, int PPL>
__global__ __launch_bounds__(kMainThreads) void ev_main(EvArgs a) {
  extern __shared__ __align__(16) uint32_t lds[];
  constexpr int PW = 64 * PPL;
  constexpr int KW = (K + 1) / 2;  // dwords of packed row offsets per token-layer
  const int E = a.E, G = a.G, L = a.L;
  const int pb = blockIdx.x, piece = blockIdx.y, l = blockIdx.z;
  const int p0 = pb * PW;
  const int nrep = a.ws.n_rep[l];
  uint32_t* tbl = lds;                                                // [E][PW]
  uint2* rinfo = reinterpret_cast<uint2*>(lds + E * PW);              // [MAX_REP][PW]
  uint32_t* rcnt = lds + E * PW + 2 * TACG_MAX_REPLICATED * PW;       // [G][PW]
  uint8_t* rep_of = reinterpret_cast<uint8_t*>(rcnt + G * PW);        // [E]
  const uint8_t* rep_of_g = a.ws.rep_of + static_cast<int64_t>(l) * E;

  for (int i = threadIdx.x; i < E * PW; i += blockDim.x) {
    const int e = i / PW, q = i - e * PW, p = p0 + q;
    uint32_t v = 0;
    if (p < a.P && rep_of_g[e] == kNone) {
      const uint8_t g = a.primary[(static_cast<int64_t>(p) * L + l) * E + e];
      v = g < G ? (1u << g) : 0u;
    }
    tbl[i] = v;
  }
  for (int i = threadIdx.x; i < nrep * PW; i += blockDim.x) {
    const int r = i / PW, q = i - r * PW, p = p0 + q;
    rinfo[i] = p < a.P ? a.ws.rep_info[(static_cast<int64_t>(l) * TACG_MAX_REPLICATED + r) * a.P + p]
                       : make_uint2(1u, 0u);
  }
  for (int i = threadIdx.x; i < G * PW; i += blockDim.x) rcnt[i] = 0;
  for (int i = threadIdx.x; i < E; i += blockDim.x) rep_of[i] = rep_of_g[i];
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nwaves = blockDim.x >> 6;
  const int f = a.piece_fam[piece];
  const uint32_t t_begin = a.piece_begin[piece], t_end = a.piece_begin[piece + 1];
  const uint32_t off_f = a.fam_off[f];
  const uint32_t hs = a.home_start[f], hz = a.home_size[f];
  const uint32_t lane_off = static_cast<uint32_t>(lane) * PPL * 4u;
  constexpr uint32_t row_bytes = PW * 4u;
  const int16_t* trace_l = a.trace + static_cast<int64_t>(l) * a.N * K;

  uint32_t acc_span[PPL], acc_home[PPL];
#pragma unroll
  for (int q = 0; q < PPL; ++q) acc_span[q] = acc_home[q] = 0;

  for (uint32_t tile = t_begin + wave * 64u; tile < t_end; tile += nwaves * 64u) {
    // ---- per-lane preprocessing of token-layer (tile + lane) ----
    const uint32_t t = tile + lane;
    uint32_t packed[KW];
    uint32_t info = 0;  // bits 0..15 replicated-slot mask, bits 16..20 anchor GPU
    if (t < t_end) {
      const int16_t* ids = trace_l + static_cast<int64_t>(t) * K;
#pragma unroll
      for (int w = 0; w < KW; ++w) packed[w] = 0;
#pragma unroll
      for (int s = 0; s < K; ++s) {
        uint32_t id = static_cast<uint16_t>(ids[s]);
        id = min(id, static_cast<uint32_t>(E - 1));
        if (rep_of[id] != kNone) info |= 1u << s;
        packed[s >> 1] |= (id * row_bytes) << (16 * (s & 1));
      }
      info |= (hs + (t - off_f) % hz) << 16;
    } else {
#pragma unroll
      for (int w = 0; w < KW; ++w) packed[w] = 0;
    }
    const uint32_t ntile = min(64u, t_end - tile);
    for (uint32_t j = 0; j < ntile; ++j) {
      uint32_t rows[KW];
#pragma unroll
      for (int w = 0; w < KW; ++w) rows[w] = __builtin_amdgcn_readlane(packed[w], j);
      const uint32_t tinfo = __builtin_amdgcn_readlane(info, j);
      uint32_t m[PPL];
#pragma unroll
      for (int q = 0; q < PPL; ++q) m[q] = 0;
#pragma unroll
      for (int s = 0; s < K; ++s) {
        const uint32_t row = (s & 1) ? (rows[s >> 1] >> 16) : (rows[s >> 1] & 0xffffu);
        const char* base = reinterpret_cast<const char*>(tbl) + row + lane_off;
        if constexpr (PPL == 1) {
          m[0] |= *reinterpret_cast<const uint32_t*>(base);
        } else if constexpr (PPL == 2) {
          const uint2 v = *reinterpret_cast<const uint2*>(base);
          m[0] |= v.x;
          m[1] |= v.y;
        } else {
          const uint4 v = *reinterpret_cast<const uint4*>(base);
          m[0] |= v.x;
          m[1] |= v.y;
          m[2] |= v.z;
          m[3] |= v.w;
        }
      }
      const uint32_t h = tinfo >> 16;
      uint32_t repmask = tinfo & 0xffffu;
      while (repmask) {  // replicated slots, in slot order (wave-uniform)
        const int s = __builtin_ctz(repmask);
        repmask &= repmask - 1u;
        const uint32_t row = (s & 1) ? (rows[s >> 1] >> 16) : (rows[s >> 1] & 0xffffu);
        const uint32_t id = row / row_bytes;
        const int r = rep_of[id];
#pragma unroll
        for (int q = 0; q < PPL; ++q) {
          const uint2 ri = rinfo[r * PW + lane * PPL + q];
          const uint32_t x = ri.x & m[q];
          const uint32_t fb = ((ri.x >> h) & 1u) ? h : ri.y;
          const uint32_t pick = x ? static_cast<uint32_t>(__builtin_ctz(x)) : fb;
          m[q] |= 1u << pick;
          __hip_atomic_fetch_add(&rcnt[pick * PW + lane * PPL + q], 1u, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_WORKGROUP);
        }
      }
      const uint32_t not_h = ~(1u << h);
#pragma unroll
      for (int q = 0; q < PPL; ++q) {
        acc_span[q] += __popc(m[q]);
        acc_home[q] += __popc(m[q] & not_h);
      }
    }
  }

  // ---- flush ----
#pragma unroll
  for (int q = 0; q < PPL; ++q) {
    const int p = p0 + lane * PPL + q;
    if (p < a.P) {
      if (acc_span[q]) atomicAdd(&a.ws.acc_span[p], static_cast<unsigned long long>(acc_span[q]));
      if (acc_home[q]) {
        atomicAdd(&a.ws.acc_home[p], static_cast<unsigned long long>(acc_home[q]));
        atomicAdd(&a.ws.acc_fam[static_cast<int64_t>(p) * a.F + f], static_cast<unsigned long long>(acc_home[q]));
      }
    }
  }
  __syncthreads();
  if (nrep > 0) {
    for (int i = threadIdx.x; i < G * PW; i += blockDim.x) {
      const int g = i / PW, q = i - g * PW, p = p0 + q;
      if (p < a.P && rcnt[i]) atomicAdd(&a.ws.rep_load[(static_cast<int64_t>(p) * L + l) * G + g], rcnt[i]);
    }
  }
}

// loads and costs.  grid (P, L), 256 threads.
__global__ __launch_bounds__(256) void ev_finalize(EvArgs a, uint64_t* __restrict__ cost_home,
                                                   uint64_t* __restrict__ cost_span, uint32_t* __restrict__ load,
                                                   uint64_t* __restrict__ cost_home_fam) {
  __shared__ uint32_t acc[TACG_MAX_GPUS];
  const int p = blockIdx.x, l = blockIdx.y;
  const int E = a.E, G = a.G, L = a.L;
  if (threadIdx.x < G) acc[threadIdx.x] = 0;
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    if (a.ws.rep_of[static_cast<int64_t>(l) * E + e] != kNone) continue;
    const uint8_t g = a.primary[(static_cast<int64_t>(p) * L + l) * E + e];
    const uint32_t c = a.ws.cnt[static_cast<int64_t>(l) * E + e];
    if (g < G && c) atomicAdd(&acc[g], c);
  }
  __syncthreads();
  if (threadIdx.x < G) {
    const int64_t o = (static_cast<int64_t>(p) * L + l) * G + threadIdx.x;
    load[o] = acc[threadIdx.x] + a.ws.rep_load[o];
  }
  if (l == 0) {
    if (threadIdx.x == 0) {
      cost_home[p] = a.ws.acc_home[p];
      cost_span[p] = a.ws.acc_span[p] - static_cast<uint64_t>(a.N) * static_cast<uint64_t>(L);
    }
    if (cost_home_fam)
      for (int f = threadIdx.x; f < a.F; f += blockDim.x)
        cost_home_fam[static_cast<int64_t>(p) * a.F + f] = a.ws.acc_fam[static_cast<int64_t>(p) * a.F + f];
  }
}

template <int K, int PPL>
int launch_main(const EvArgs& a, int n_pblocks, hipStream_t stream) {
  constexpr int PW = 64 * PPL;
  const size_t lds = static_cast<size_t>(a.E) * PW * 4 + static_cast<size_t>(2) * TACG_MAX_REPLICATED * PW * 4 +
                     static_cast<size_t>(a.G) * PW * 4 + align256(a.E);
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&ev_main<K, PPL>), hipFuncAttributeMaxDynamicSharedMemorySize,
                      static_cast<int>(lds));
  hipLaunchKernelGGL((ev_main<K, PPL>), dim3(n_pblocks, a.n_pieces, a.L), dim3(kMainThreads), lds, stream, a);
  return TACG_OK;
}

template <int K>
int launch_main_k(const EvArgs& a, hipStream_t stream) {
  if (a.E > 128) return launch_main<K, 1>(a, (a.P + 63) / 64, stream);
  return launch_main<K, 2>(a, (a.P + 127) / 128, stream);
}

// per-(placement, layer) primary-only loads from D.  grid (P, L), 256 threads.
__global__ __launch_bounds__(256) void placement_load_kernel(const uint32_t* __restrict__ D, int F, int L, int E,
                                                             const uint8_t* __restrict__ primary, int G,
                                                             int64_t* __restrict__ load_ref, uint32_t* d_err) {
  __shared__ unsigned long long acc[TACG_MAX_GPUS];
  const int p = blockIdx.x, l = blockIdx.y;
  if (threadIdx.x < G) acc[threadIdx.x] = 0;
  __syncthreads();
  uint32_t err = 0;
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    const uint8_t g = primary[(static_cast<int64_t>(p) * L + l) * E + e];
    if (g >= G) {
      err |= TACG_ERR_TABLE;
      continue;
    }
    unsigned long long s = 0;
    for (int f = 0; f < F; ++f) s += D[(static_cast<int64_t>(f) * L + l) * E + e];
    if (s) atomicAdd(&acc[g], s);
  }
  __syncthreads();
  if (threadIdx.x < G) load_ref[(static_cast<int64_t>(p) * L + l) * G + threadIdx.x] = static_cast<int64_t>(acc[threadIdx.x]);
  if (err) atomicOr(d_err, err);
}

// Jain and MaxVio.  One wave per output row; lanes over GPUs.
__global__ __launch_bounds__(64) void jain_kernel(const uint32_t* __restrict__ load, int P, int L, int G,
                                                  int per_layer, float* __restrict__ jain, float* __restrict__ maxvio) {
  const int row = blockIdx.x;  // p (global) or p * L + l (per layer)
  const int m = threadIdx.x;
  uint64_t x = 0;
  if (m < G) {
    if (per_layer) {
      x = load[static_cast<int64_t>(row) * G + m];
    } else {
      for (int l = 0; l < L; ++l) x += load[(static_cast<int64_t>(row) * L + l) * G + m];
    }
  }
  // exact integer sums; the square sum is formed in float64 (it can exceed 64 bits)
  uint64_t s = x, mx = x;
  double sq = static_cast<double>(x) * static_cast<double>(x);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    s += __shfl_xor(s, o, 64);
    const uint64_t other = __shfl_xor(mx, o, 64);
    mx = other > mx ? other : mx;
    sq += __shfl_xor(sq, o, 64);
  }
  if (m == 0) {
    const double tot = static_cast<double>(s);
    double j = 1.0, v = 0.0;
    if (s > 0) {
      j = tot * tot / (G * sq);
      const double mean = tot / G;
      v = (static_cast<double>(mx) - mean) / mean;
    }
    jain[row] = static_cast<float>(j);
    maxvio[row] = static_cast<float>(v);
  }
}

}  // namespace

size_t eval_workspace(int64_t n_tokens, int32_t L, int32_t E, int32_t G, int32_t P, int32_t F) {
  (void)n_tokens;
  size_t used = 0;
  carve_ev(nullptr, L, E, G, P, F, &used);
  return used;
}

int launch_eval(const int16_t* trace, int64_t N, int32_t L, int32_t K, int32_t E, const int64_t* fam_off_host,
                int32_t F, const int32_t* home_start_host, const int32_t* home_size_host, int32_t G, int32_t P,
                const uint8_t* primary, const uint8_t* secondary, int32_t R, const int64_t* load_ref,
                int32_t theta_num, int32_t theta_den, uint64_t* cost_home, uint64_t* cost_span, uint32_t* load,
                uint64_t* cost_home_fam, uint32_t* d_err, void* workspace, hipStream_t stream) {
  EvArgs a{};
  a.trace = trace;
  a.primary = primary;
  a.secondary = R > 0 ? secondary : nullptr;
  a.load_ref = load_ref;
  a.d_err = d_err;
  a.ws = carve_ev(workspace, L, E, G, P, F);
  a.N = N;
  a.L = L;
  a.K = K;
  a.E = E;
  a.F = F;
  a.G = G;
  a.P = P;
  a.R = R;
  a.theta_num = theta_num;
  a.theta_den = theta_den;
  for (int f = 0; f <= F; ++f) a.fam_off[f] = static_cast<uint32_t>(fam_off_host[f]);
  for (int f = 0; f < F; ++f) {
    a.home_start[f] = static_cast<uint8_t>(home_start_host[f]);
    a.home_size[f] = static_cast<uint8_t>(home_size_host[f]);
  }
  // pieces: split every family's tokens into chunks of about N / 64 tokens (at least 4096, at
  // most 2^26 so that the per-lane 32-bit cost accumulators cannot overflow)
  int64_t chunk = std::min<int64_t>(int64_t(1) << 26, std::max<int64_t>(4096, (N + 63) / 64));
  int np = 0;
  for (;;) {
    np = 0;
    for (int f = 0; f < F; ++f) {
      const int64_t n = fam_off_host[f + 1] - fam_off_host[f];
      np += static_cast<int>((n + chunk - 1) / chunk);
    }
    if (np <= kMaxPieces || chunk >= (int64_t(1) << 26)) break;
    chunk = std::min<int64_t>(chunk * 2, int64_t(1) << 26);
  }
  if (np > kMaxPieces) return TACG_E_UNSUPPORTED;
  np = 0;
  for (int f = 0; f < F; ++f) {
    for (int64_t t = fam_off_host[f]; t < fam_off_host[f + 1]; t += chunk) {
      a.piece_begin[np] = static_cast<uint32_t>(t);
      a.piece_fam[np] = static_cast<uint8_t>(f);
      ++np;
    }
  }
  a.n_pieces = np;
  // families are contiguous in token order, so piece j always ends where piece j + 1 begins
  a.piece_begin[np] = static_cast<uint32_t>(N);

  hipLaunchKernelGGL(ev_zero, dim3(256), dim3(256), 0, stream, a);
  if (N > 0) {
    const int splits = static_cast<int>(std::min<int64_t>(64, (N + 65535) / 65536));
    hipLaunchKernelGGL(ev_count, dim3(splits, L), dim3(256), 0, stream, a);
  }
  hipLaunchKernelGGL(ev_flags, dim3(P, L), dim3(256), 0, stream, a);
  hipLaunchKernelGGL(ev_replist, dim3(L), dim3(256), 0, stream, a);
  if (R > 0) hipLaunchKernelGGL(ev_repinfo, dim3((P + 255) / 256, L), dim3(256), 0, stream, a);
  if (hipGetLastError() != hipSuccess) return TACG_E_DEVICE;
  if (np > 0) {
    int rc;
    switch (K) {
#define TACG_K(k) \
  case k:         \
    rc = launch_main_k<k>(a, stream); \
    break;
      TACG_K(1) TACG_K(2) TACG_K(3) TACG_K(4) TACG_K(5) TACG_K(6) TACG_K(7) TACG_K(8)
      TACG_K(9) TACG_K(10) TACG_K(11) TACG_K(12) TACG_K(13) TACG_K(14) TACG_K(15) TACG_K(16)
#undef TACG_K
      default:
        return TACG_E_UNSUPPORTED;
    }
    if (rc != TACG_OK) return rc;
    if (hipGetLastError() != hipSuccess) return TACG_E_DEVICE;
  }
  hipLaunchKernelGGL(ev_finalize, dim3(P, L), dim3(256), 0, stream, a, cost_home, cost_span, load, cost_home_fam);
  return hipGetLastError() == hipSuccess ? TACG_OK : TACG_E_DEVICE;
}

int launch_placement_load(const uint32_t* D, int32_t F, int32_t L, int32_t E, const uint8_t* primary, int32_t P,
                          int32_t G, int64_t* load_ref, uint32_t* d_err, hipStream_t stream) {
  hipLaunchKernelGGL(placement_load_kernel, dim3(P, L), dim3(256), 0, stream, D, F, L, E, primary, G, load_ref, d_err);
  return hipGetLastError() == hipSuccess ? TACG_OK : TACG_E_DEVICE;
}

int launch_jain(const uint32_t* load, int32_t P, int32_t L, int32_t G, int32_t per_layer, float* jain,
                float* maxvio, hipStream_t stream) {
  const int rows = per_layer ? P * L : P;
  hipLaunchKernelGGL(jain_kernel, dim3(rows), dim3(64), 0, stream, load, P, L, G, per_layer, jain, maxvio);
  return hipGetLastError() == hipSuccess ? TACG_OK : TACG_E_DEVICE;
}

}  // namespace tacg
