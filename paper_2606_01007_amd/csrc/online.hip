// Placement scoring with decayed per-GPU loads: the sequential form of the serving rule of Sec. 3.4
// (eqs. mean-load, feasible-set and load-update).  Each (placement, layer) keeps its own loads L_m,
// reads them for the guard and the least-loaded choice of every multi-candidate slot, and updates
// them after every token in trace order:  L_m <- fma(rho, L_m, Delta_m)  (float64, one rounding),
// Delta_m = the token's slots served by GPU m.  The guard is theta_den * G * L_m <= (theta_den +
// theta_num) * S with S = L_0 + L_1 + ... + L_31 summed in that order (GPUs >= G hold +0.0).
//
// Kernel design (gfx950): the scan over tokens is sequential, the (placement, layer) scans are
// independent.  Lane = placement, wave = 64 placements of one layer, one wave per workgroup.
//   * LDS holds, for the wave's placements, every expert's primary GPU (pg[e][lane], one byte), the
//     candidate masks of the experts that have a secondary in any of these placements (rm[r][lane],
//     up to kRepLds of them; rix[e] maps an expert to its row, and the rare experts beyond that
//     read their tables from memory), and per-lane dispatch counters (cnt[m][lane]).  About 36 KB at
//     E = 256, so four waves share a CU and all P * L / 64 waves are resident at once.
//   * The wave loads 64 token-layers at once (one per lane), packs their ids and a word with the
//     validity, family and anchor position, and broadcasts them token by token with v_readlane.
//   * The loads live in 32 float64 registers per lane.  The per-token dispatch counts Delta are kept
//     as packed 4-bit fields (8-bit fields for top-k = 16) so that every GPU's fused multiply-add
//     reads its count with one bit-field extract.
#include "tacg_internal.h"

namespace tacg {
namespace {

constexpr int kLanes = 64;
constexpr uint8_t kNone = 0xFF;
constexpr uint8_t kOver = 0xFE;  // replicated expert without an LDS row (read from memory)
constexpr int kRepLds = 48;      // candidate-mask rows in LDS per workgroup

struct OnArgs {
  const int16_t* trace;
  const uint8_t* primary;
  const uint8_t* secondary;
  const double* state_in;
  double* state_out;
  unsigned long long* cost_home;
  unsigned long long* cost_span;
  uint32_t* load;
  unsigned long long* cost_home_fam;
  uint32_t* d_err;
  double rho;
  int64_t N;
  int32_t L, K, E, F, G, P, R;
  int32_t theta_num, theta_den;
  // per family: (first token, end token, home_start | home_size << 8, 0); 16-byte records so that a
  // runtime index into the kernel arguments stays aligned
  uint4 fam[TACG_MAX_FAMILIES];
};
static_assert(sizeof(OnArgs) <= 4096, "kernel arguments must stay within 4 KB");

__global__ __launch_bounds__(256) void on_zero(OnArgs a) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t j = i; j < a.P; j += stride) {
    a.cost_home[j] = 0;
    a.cost_span[j] = 0;
  }
  if (a.cost_home_fam)
    for (int64_t j = i; j < static_cast<int64_t>(a.P) * a.F; j += stride) a.cost_home_fam[j] = 0;
}

// Per-token dispatch counts of the 32 GPUs, packed: 4-bit fields when at most 15 slots can land on
// one GPU, else 8-bit fields.
template <bool kWide>
struct Delta {
  static constexpr int kBits = kWide ? 8 : 4;
  static constexpr int kPerWord = 32 / kBits;
  static constexpr int kWords = 32 / kPerWord;
  uint32_t w[kWords];
  __device__ __forceinline__ void clear() {
#pragma unroll
    for (int i = 0; i < kWords; ++i) w[i] = 0;
  }
  __device__ __forceinline__ void add(uint32_t g) {
    const uint32_t inc = 1u << (kBits * (g % kPerWord));
    const uint32_t word = g / kPerWord;
#pragma unroll
    for (int i = 0; i < kWords; ++i) w[i] += (word == static_cast<uint32_t>(i)) ? inc : 0u;
  }
  __device__ __forceinline__ uint32_t get(int m) const {
    return __builtin_amdgcn_ubfe(w[m / kPerWord], kBits * (m % kPerWord), kBits);
  }
};

__device__ __forceinline__ uint32_t find_first_bit(uint32_t x) {
  uint32_t r;
  asm("v_ffbl_b32 %0, %1" : "=v"(r) : "v"(x));
  return r;
}

// Candidate GPUs of one (placement, layer, expert) as a mask: the primary and the valid secondaries.
// An invalid table (flagged) yields GPU 0 so that every later choice stays in range.
__device__ __forceinline__ uint32_t candidate_mask(const OnArgs& a, bool live, int64_t pe, uint32_t& err) {
  uint32_t m = 0;
  if (live) {
    const uint8_t g0 = a.primary[pe];
    if (g0 < a.G) m = 1u << g0;
    else err |= TACG_ERR_TABLE;
    for (int r = 0; r < a.R; ++r) {
      const uint8_t g = a.secondary[pe * a.R + r];
      if (g == kNone) continue;
      if (g >= a.G || ((m >> g) & 1u)) {
        err |= TACG_ERR_TABLE;
        continue;
      }
      m |= 1u << g;
    }
  }
  return m ? m : 1u;
}

// Candidate mask of expert e for this lane: its LDS row, or the tables themselves for an expert
// beyond the LDS rows.
__device__ __forceinline__ uint32_t slot_mask(const OnArgs& a, const uint32_t* rm, const uint8_t* rix, uint32_t e,
                                              bool live, int64_t base, int lane) {
  const uint8_t r = rix[e];
  if (r != kOver) return rm[r * kLanes + lane];
  uint32_t unused = 0;
  return candidate_mask(a, live, base + e, unused);
}

// argmin over the GPUs of fc of the loads, ties to the lowest number, as a balanced tree of pairwise
// minima (the left, lower-numbered operand wins ties, so the result is the sequential argmin)
__device__ __forceinline__ uint32_t least_loaded(const double (&Lm)[32], uint32_t fc) {
  double v[16];
  uint32_t ix[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const double a0 = ((fc >> (2 * i)) & 1u) ? Lm[2 * i] : __builtin_inf();
    const double a1 = ((fc >> (2 * i + 1)) & 1u) ? Lm[2 * i + 1] : __builtin_inf();
    const bool right = a1 < a0;
    v[i] = right ? a1 : a0;
    ix[i] = right ? 2u * i + 1u : 2u * i;
  }
#pragma unroll
  for (int w = 8; w >= 1; w >>= 1) {
#pragma unroll
    for (int i = 0; i < w; ++i) {
      const bool right = v[2 * i + 1] < v[2 * i];
      v[i] = right ? v[2 * i + 1] : v[2 * i];
      ix[i] = right ? ix[2 * i + 1] : ix[2 * i];
    }
  }
  return ix[0];
}

// grid (ceil(P / 64), L), 64 threads.
template <int K>
__global__ __launch_bounds__(kLanes) void on_main(OnArgs a) {
  extern __shared__ __align__(16) uint32_t lds[];
  constexpr int KB = (K + 3) / 4;  // dwords of 8-bit ids per token-layer
  const int lane = threadIdx.x;
  const int l = blockIdx.y;
  const int p = blockIdx.x * kLanes + lane;
  const bool live = p < a.P;
  const int E = a.E, G = a.G, L = a.L;
  uint32_t* rm = lds;                                                  // [kRepLds][64] candidate masks
  uint32_t* cnt = rm + kRepLds * kLanes;                               // [32][64] dispatch counters
  uint8_t* pg = reinterpret_cast<uint8_t*>(cnt + 32 * kLanes);          // [E][64] primary GPUs
  uint8_t* rix = pg + E * kLanes;                                      // [E] row of rm, kNone or kOver
  uint32_t err = 0;

  // ---- candidate sets of this lane's placement (eq. candidate-set) ----
  const int64_t base = (static_cast<int64_t>(p) * L + l) * E;
  int nr = 0;  // rows of rm in use (workgroup-uniform)
  for (int e = 0; e < E; ++e) {
    const uint32_t m = candidate_mask(a, live, base + e, err);
    pg[e * kLanes + lane] = static_cast<uint8_t>(find_first_bit(m));
    const bool multi = __popc(m) > 1;
    uint8_t r = kNone;
    if (__ballot(multi)) {
      if (nr < kRepLds) {
        rm[nr * kLanes + lane] = m;
        r = static_cast<uint8_t>(nr++);
      } else {
        r = kOver;
      }
    }
    if (lane == 0) rix[e] = r;
  }
#pragma unroll
  for (int m = 0; m < 32; ++m) cnt[m * kLanes + lane] = 0;
  __syncthreads();

  double Lm[32];
#pragma unroll
  for (int m = 0; m < 32; ++m) Lm[m] = (a.state_in && live && m < G) ? a.state_in[(base / E) * G + m] : 0.0;
  const double rho = a.rho;
  const double gden = static_cast<double>(a.theta_den) * static_cast<double>(G);
  const double rnum = static_cast<double>(a.theta_den) + static_cast<double>(a.theta_num);

  unsigned long long span_acc = 0, home_acc = 0, fam_acc = 0;
  int cur_f = -1;
  const int16_t* trace_l = a.trace + static_cast<int64_t>(l) * a.N * K;
  int f_tile = 0;  // family of the first token of the current tile

  for (int64_t tile = 0; tile < a.N; tile += kLanes) {
    while (static_cast<int64_t>(a.fam[f_tile].y) <= tile) ++f_tile;
    // ---- per-lane preparation of token-layer tile + lane ----
    const int64_t t = tile + lane;
    uint32_t pk[KB];
#pragma unroll
    for (int w = 0; w < KB; ++w) pk[w] = 0;
    uint32_t info = 0;
    if (t < a.N) {
      const int16_t* idp = trace_l + t * K;
      uint32_t raw[K];
#pragma unroll
      for (int s = 0; s < K; ++s) raw[s] = static_cast<uint16_t>(idp[s]);
      bool ok = true, dup = false;
#pragma unroll
      for (int s = 0; s < K; ++s) {
        ok &= raw[s] < static_cast<uint32_t>(E);
#pragma unroll
        for (int q = 0; q < s; ++q) dup |= raw[s] == raw[q];
        const uint32_t id = min(raw[s], static_cast<uint32_t>(E - 1));
        pk[s >> 2] |= id << (8 * (s & 3));
        if (rix[id] != kNone) info |= 1u << (16 + s);  // an expert with several candidates somewhere
      }
      if (!ok) err |= TACG_ERR_ID_RANGE;
      if (dup) err |= TACG_ERR_ID_DUP;
      int f = f_tile;
      while (static_cast<int64_t>(a.fam[f].y) <= t) ++f;
      const uint4 fr = a.fam[f];
      const uint32_t hz = (fr.z >> 8) & 0xffu;
      const uint32_t pos = static_cast<uint32_t>((t - static_cast<int64_t>(fr.x)) % hz);
      info |= ((ok && !dup) ? 1u : 0u) | (static_cast<uint32_t>(f) << 1) | (pos << 8);
    }
    const int ntile = static_cast<int>(min(static_cast<int64_t>(kLanes), a.N - tile));
    for (int j = 0; j < ntile; ++j) {
      const uint32_t tinfo = __builtin_amdgcn_readlane(info, j);
      if (!(tinfo & 1u)) continue;  // invalid token-layer (flagged): not served
      uint32_t ids[KB];
#pragma unroll
      for (int w = 0; w < KB; ++w) ids[w] = __builtin_amdgcn_readlane(pk[w], j);
      const int f = static_cast<int>((tinfo >> 1) & 127u);
      if (f != cur_f) {
        if (cur_f >= 0 && a.cost_home_fam && live && fam_acc)
          atomicAdd(&a.cost_home_fam[static_cast<int64_t>(p) * a.F + cur_f], fam_acc);
        fam_acc = 0;
        cur_f = f;
      }
      const uint32_t h = (a.fam[f].z & 0xffu) + ((tinfo >> 8) & 0xffu);

      // single-candidate slots first: they form the set R of GPUs the token reaches
      Delta<(K > 15)> dl;
      dl.clear();
      uint32_t R = 0, pend = 0;
#pragma unroll
      for (int s = 0; s < K; ++s) {
        const uint32_t e = __builtin_amdgcn_ubfe(ids[s >> 2], 8 * (s & 3), 8);
        uint32_t g;
        if ((tinfo >> (16 + s)) & 1u) {  // workgroup-uniform: e has several candidates somewhere
          const uint32_t c = slot_mask(a, rm, rix, e, live, base, lane);
          if (__popc(c) > 1) {
            pend |= 1u << s;
            continue;
          }
          g = find_first_bit(c);
        } else {
          g = pg[e * kLanes + lane];
        }
        R |= 1u << g;
        dl.add(g);
        __hip_atomic_fetch_add(&cnt[g * kLanes + lane], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
      if (__ballot(pend != 0)) {
        // feasible GPUs under the current loads (eq. feasible-set with the mean of eq. mean-load)
        uint32_t feas = 0xffffffffu;
        if (a.theta_den != 0) {
          double S = 0.0;
#pragma unroll
          for (int m = 0; m < 32; ++m) S += Lm[m];
          const double rhs = rnum * S;
          feas = 0;
#pragma unroll
          for (int m = 0; m < 32; ++m) feas |= (gden * Lm[m] <= rhs) ? (1u << m) : 0u;
        }
        // multi-candidate slots in slot order: a reached feasible candidate (lowest number), else
        // the anchor if feasible, else the least-loaded feasible candidate (ties: lowest number).
        // The slot loop stays rolled so that the 32-GPU scan below exists once and indexes the loads
        // statically; the slot's id comes out of two 64-bit words by a shift.
        const uint64_t id_lo = static_cast<uint64_t>(ids[0]) | (KB > 1 ? static_cast<uint64_t>(ids[KB > 1 ? 1 : 0]) << 32 : 0);
        const uint64_t id_hi = KB > 2 ? (static_cast<uint64_t>(ids[KB > 2 ? 2 : 0]) |
                                         (KB > 3 ? static_cast<uint64_t>(ids[KB > 3 ? 3 : 0]) << 32 : 0))
                                      : 0;
#pragma unroll 1
        for (int s = 0; s < K; ++s) {
          if (!((pend >> s) & 1u)) continue;
          const uint64_t wd = s < 8 ? id_lo : id_hi;
          const uint32_t e = static_cast<uint32_t>(wd >> (8 * (s & 7))) & 0xffu;
          const uint32_t c = slot_mask(a, rm, rix, e, live, base, lane);
          uint32_t fc = c & feas;
          if (!fc) fc = c;
          uint32_t pick;
          if (fc & R) {
            pick = find_first_bit(fc & R);
          } else if ((fc >> h) & 1u) {
            pick = h;
          } else {
            pick = least_loaded(Lm, fc);
          }
          R |= 1u << pick;
          dl.add(pick);
          __hip_atomic_fetch_add(&cnt[pick * kLanes + lane], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
      }
      const uint32_t n = __popc(R);
      span_acc += n - 1u;
      const uint32_t home = n - ((R >> h) & 1u);
      home_acc += home;
      fam_acc += home;
      // eq. load-update after the token's dispatch
#pragma unroll
      for (int m = 0; m < 32; ++m) Lm[m] = __fma_rn(rho, Lm[m], static_cast<double>(dl.get(m)));
    }
  }

  if (live) {
    if (cur_f >= 0 && a.cost_home_fam && fam_acc)
      atomicAdd(&a.cost_home_fam[static_cast<int64_t>(p) * a.F + cur_f], fam_acc);
    if (home_acc) atomicAdd(&a.cost_home[p], home_acc);
    if (span_acc) atomicAdd(&a.cost_span[p], span_acc);
    const int64_t o = (static_cast<int64_t>(p) * L + l) * G;
    for (int m = 0; m < G; ++m) a.load[o + m] = cnt[m * kLanes + lane];
    if (a.state_out) {
#pragma unroll
      for (int m = 0; m < 32; ++m)  // static register indices: the loads never leave registers
        if (m < G) a.state_out[o + m] = Lm[m];
    }
  }
  if (err) atomicOr(a.d_err, err);
}

template <int K>
void launch_on(const OnArgs& a, hipStream_t stream) {
  const size_t lds = (static_cast<size_t>(kRepLds) * kLanes + 32 * kLanes) * sizeof(uint32_t) +
                     static_cast<size_t>(a.E) * kLanes + static_cast<size_t>(a.E);
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&on_main<K>), hipFuncAttributeMaxDynamicSharedMemorySize,
                            static_cast<int>(lds));
  hipLaunchKernelGGL(on_main<K>, dim3((a.P + kLanes - 1) / kLanes, a.L), dim3(kLanes), lds, stream, a);
}

}  // namespace

int launch_eval_online(const int16_t* trace, int64_t N, int32_t L, int32_t K, int32_t E, const int64_t* fam_off_host,
                       int32_t F, const int32_t* home_start_host, const int32_t* home_size_host, int32_t G, int32_t P,
                       const uint8_t* primary, const uint8_t* secondary, int32_t R, double rho, int32_t theta_num,
                       int32_t theta_den, const double* state_in, double* state_out, uint64_t* cost_home,
                       uint64_t* cost_span, uint32_t* load, uint64_t* cost_home_fam, uint32_t* d_err,
                       hipStream_t stream) {
  OnArgs a{};
  a.trace = trace;
  a.primary = primary;
  a.secondary = R > 0 ? secondary : nullptr;
  a.state_in = state_in;
  a.state_out = state_out;
  a.cost_home = reinterpret_cast<unsigned long long*>(cost_home);
  a.cost_span = reinterpret_cast<unsigned long long*>(cost_span);
  a.load = load;
  a.cost_home_fam = reinterpret_cast<unsigned long long*>(cost_home_fam);
  a.d_err = d_err;
  a.rho = rho;
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
  for (int f = 0; f < F; ++f)
    a.fam[f] = make_uint4(static_cast<uint32_t>(fam_off_host[f]), static_cast<uint32_t>(fam_off_host[f + 1]),
                          static_cast<uint32_t>(home_start_host[f]) |
                              (static_cast<uint32_t>(home_size_host[f]) << 8),
                          0u);
  // sentinel past the last family: a token index never reaches its end
  for (int f = F; f < TACG_MAX_FAMILIES; ++f) a.fam[f] = make_uint4(0xffffffffu, 0xffffffffu, 1u << 8, 0u);
  hipLaunchKernelGGL(on_zero, dim3(64), dim3(256), 0, stream, a);
  if (P > 0) {
    switch (K) {
#define TACG_K(k)              \
  case k:                      \
    launch_on<k>(a, stream);   \
    break;
      TACG_K(1) TACG_K(2) TACG_K(3) TACG_K(4) TACG_K(5) TACG_K(6) TACG_K(7) TACG_K(8)
      TACG_K(9) TACG_K(10) TACG_K(11) TACG_K(12) TACG_K(13) TACG_K(14) TACG_K(15) TACG_K(16)
#undef TACG_K
      default:
        return TACG_E_UNSUPPORTED;
    }
  }
  return hipGetLastError() == hipSuccess ? TACG_OK : TACG_E_DEVICE;
}

}  // namespace tacg
