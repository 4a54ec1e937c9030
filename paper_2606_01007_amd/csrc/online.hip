// Placement scoring with decayed per-GPU loads: the sequential form of the serving rule of Sec. 3.4
// (eqs. mean-load, feasible-set and load-update).  Each (placement, layer) keeps its own loads L_m,
// reads them for the guard and the least-loaded choice of every multi-candidate slot, and updates
// them after every token in trace order:  L_m <- fma(rho, L_m, Delta_m)  (float64, one rounding),
// Delta_m = the token's slots served by GPU m.  The guard is theta_den * G * L_m <= (theta_den +
// theta_num) * S with S = L_0 + L_1 + ... + L_31 summed in that order (GPUs >= G hold +0.0).
//
// Kernel design (gfx950): the scan over tokens is sequential, the (placement, layer) scans are
// independent.  Lane = placement, wave = 64 placements of one layer, one wave per workgroup, so there
// is about one wave per SIMD and nothing hides a latency on the per-token chain: the token loop keeps
// LDS off that chain.
//   * LDS holds one code byte per (expert, lane): the GPU of an expert with a single candidate in the
//     lane's placement, else 32 + the row of its candidate mask in rm (rows shared by the wave's
//     placements; code 63 when the rows ran out and the mask is read from the tables).  The k codes of
//     a token are read one token ahead, so their latency overlaps the previous token's work.
//   * The wave loads 64 token-layers at once (one per lane), packs their ids and a word with the
//     validity, family and anchor position, and broadcasts them token by token with v_readlane.
//   * The loads live in float64 registers (8 or 32 per lane, by G).  The per-token dispatch counts
//     Delta are packed 4-bit fields in 64-bit words (8-bit fields for top-k = 16), one shift-add per
//     slot, one bit-field extract per GPU in the fused multiply-adds.
//   * Per-GPU dispatch totals: the wave also counts every expert's valid dispatches of its layer
//     (ecnt, in the per-tile preparation); at the end each lane adds ecnt[e] to the GPU of every
//     single-candidate expert, and only the choices of multi-candidate slots are counted per token.
#include "tacg_internal.h"

namespace tacg {
namespace {

constexpr int kLanes = 64;
constexpr uint8_t kNone = 0xFF;
constexpr uint8_t kOver = 0xFE;  // replicated expert without an LDS row (read from memory)

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

// Per-token dispatch counts of GPUs 0 .. NG-1, packed in 64-bit words: 4-bit fields when at most 15
// slots can land on one GPU, else 8-bit fields.  add(g) with g >= NG (a multi-candidate code) adds
// nothing.
template <bool kWide, int NG>
struct Delta {
  static constexpr int kBits = kWide ? 8 : 4;
  static constexpr int kPerWord = 64 / kBits;
  static constexpr int kWords = (NG + kPerWord - 1) / kPerWord;
  uint64_t w[kWords];
  __device__ __forceinline__ void clear() {
#pragma unroll
    for (int i = 0; i < kWords; ++i) w[i] = 0;
  }
  __device__ __forceinline__ void add(uint32_t g) {
    const uint64_t inc = 1ull << ((kBits * g) & 63u);
    const uint32_t word = g / kPerWord;
#pragma unroll
    for (int i = 0; i < kWords; ++i) w[i] += (word == static_cast<uint32_t>(i)) ? inc : 0ull;
  }
  __device__ __forceinline__ uint32_t get(int m) const {
    const uint64_t x = w[m / kPerWord];
    const int sh = kBits * (m % kPerWord);
    const uint32_t half = sh < 32 ? static_cast<uint32_t>(x) : static_cast<uint32_t>(x >> 32);
    return __builtin_amdgcn_ubfe(half, sh & 31, kBits);
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

typedef uint32_t v32u __attribute__((ext_vector_type(32)));

constexpr int kRows = 31;           // candidate-mask rows in LDS per workgroup (codes 32 .. 62)
constexpr uint32_t kCodeOver = 63;  // multi-candidate expert without a row: read its tables
constexpr int kMaxCand = TACG_MAX_SECONDARY + 1;

// The lane's code bytes of experts 0 .. 255 in 64 registers (two 32-register vectors).  The expert id
// of a lookup is wave-uniform, so the lookup is an indexed register move (s_set_gpr_idx) and not a
// memory access.
struct CodeRegs {
  v32u lo, hi;
  __device__ __forceinline__ uint32_t get(uint32_t e) const {
    const uint32_t i = (e >> 2) & 31u;
    const uint32_t w = e < 128u ? lo[i] : hi[i];
    return __builtin_amdgcn_ubfe(w, 8u * (e & 3u), 8u);
  }
};

// grid (ceil(P / 64), L), 64 threads; NG = 8 or 32 >= G GPUs in registers.
template <int K, int NG, int MC>
__global__ __launch_bounds__(kLanes) void on_main(OnArgs a) {
  extern __shared__ __align__(16) uint32_t lds[];
  constexpr int KB = (K + 3) / 4;  // dwords of 8-bit ids per token-layer
  const int lane = threadIdx.x;
  const int l = blockIdx.y;
  const int p = blockIdx.x * kLanes + lane;
  const bool live = p < a.P;
  const int E = a.E, G = a.G, L = a.L;
  uint32_t* rm = lds;                                            // [kRows][64] candidate masks
  uint32_t* cnt = rm + kRows * kLanes;                           // [32][64] dispatches per GPU
  uint32_t* ecnt = cnt + 32 * kLanes;                            // [E] valid dispatches per expert
  uint32_t* hasrow = ecnt + TACG_MAX_EXPERTS;                    // [8] experts with several candidates somewhere
  // shared region: the code bytes [E][64] while the tables are read, then this lane's loads as pairs
  // [NG / 2][64] of float64 whenever a token has multi-candidate slots
  uint8_t* code = reinterpret_cast<uint8_t*>(hasrow + 8);
  double2* Lc2 = reinterpret_cast<double2*>(code);
  const double* Lc = reinterpret_cast<const double*>(code);
  uint32_t err = 0;

  // ---- candidate sets of this lane's placement (eq. candidate-set) ----
  const int64_t base = (static_cast<int64_t>(p) * L + l) * E;
  int nr = 0;  // rows of rm in use (workgroup-uniform)
  if (lane < 8) hasrow[lane] = 0;
  for (int e = 0; e < TACG_MAX_EXPERTS; ++e) {
    uint32_t c = 0;
    if (e < E) {
      const uint32_t m = candidate_mask(a, live, base + e, err);
      const bool multi = __popc(m) > 1;
      c = find_first_bit(m);
      if (__ballot(multi)) {
        if (lane == 0) hasrow[e >> 5] |= 1u << (e & 31);
        if (nr < kRows) {
          rm[nr * kLanes + lane] = m;
          if (multi) c = 32u + static_cast<uint32_t>(nr);
          ++nr;
        } else if (multi) {
          c = kCodeOver;
        }
      }
    }
    code[e * kLanes + lane] = static_cast<uint8_t>(c);
  }
  CodeRegs cr;
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    const uint32_t w = static_cast<uint32_t>(code[(4 * i) * kLanes + lane]) |
                       (static_cast<uint32_t>(code[(4 * i + 1) * kLanes + lane]) << 8) |
                       (static_cast<uint32_t>(code[(4 * i + 2) * kLanes + lane]) << 16) |
                       (static_cast<uint32_t>(code[(4 * i + 3) * kLanes + lane]) << 24);
    if (i < 32) cr.lo[i] = w;
    else cr.hi[i - 32] = w;
  }
#pragma unroll
  for (int m = 0; m < 32; ++m) cnt[m * kLanes + lane] = 0;
  for (int e = lane; e < E; e += kLanes) ecnt[e] = 0;
  __syncthreads();  // the code bytes are in registers; the region now holds the loads

  double Lm[NG];
#pragma unroll
  for (int m = 0; m < NG; ++m) Lm[m] = (a.state_in && live && m < G) ? a.state_in[(base / E) * G + m] : 0.0;
  const double rho = a.rho;
  const bool guard = a.theta_den != 0;
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
        info |= ((hasrow[id >> 5] >> (id & 31)) & 1u) << (16 + s);  // a candidate row exists for id
      }
      if (!ok) err |= TACG_ERR_ID_RANGE;
      if (dup) err |= TACG_ERR_ID_DUP;
      if (ok && !dup) {
#pragma unroll
        for (int s = 0; s < K; ++s)
          __hip_atomic_fetch_add(&ecnt[raw[s]], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
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
      uint32_t c[K];
#pragma unroll
      for (int s = 0; s < K; ++s) c[s] = cr.get(__builtin_amdgcn_ubfe(ids[s >> 2], 8 * (s & 3), 8));
      Delta<(K > 15), NG> dl;
      dl.clear();
      uint32_t R = 0, pend = 0;
#pragma unroll
      for (int s = 0; s < K; ++s) {
        const bool single = c[s] < 32u;
        R |= single ? (1u << c[s]) : 0u;
        pend |= single ? 0u : (1u << s);
        dl.add(c[s]);
      }
      // slots whose expert has several candidates in some placement of the wave (wave-uniform)
      const uint32_t pend_any = tinfo >> 16;
      if (pend_any) {
        // the guard's right-hand side under the current loads (eq. feasible-set with the mean of
        // eq. mean-load), and the loads in LDS so that a slot reads those of its own candidates
        double rhs = 0.0;
        if (guard) {
          double S = 0.0;
#pragma unroll
          for (int m = 0; m < NG; ++m) S += Lm[m];
          rhs = rnum * S;
        }
#pragma unroll
        for (int m = 0; m < NG; m += 2) Lc2[(m >> 1) * kLanes + lane] = make_double2(Lm[m], Lm[m + 1]);
        uint64_t cw[(K + 7) / 8];
#pragma unroll
        for (int q = 0; q < (K + 7) / 8; ++q) cw[q] = 0;
#pragma unroll
        for (int s = 0; s < K; ++s) cw[s >> 3] |= static_cast<uint64_t>(c[s]) << (8 * (s & 7));
        const uint64_t id_lo = static_cast<uint64_t>(ids[0]) | (KB > 1 ? static_cast<uint64_t>(ids[KB > 1 ? 1 : 0]) << 32 : 0);
        const uint64_t id_hi = KB > 2 ? (static_cast<uint64_t>(ids[KB > 2 ? 2 : 0]) |
                                         (KB > 3 ? static_cast<uint64_t>(ids[KB > 3 ? 3 : 0]) << 32 : 0))
                                      : 0;
        // multi-candidate slots in slot order: a reached feasible candidate (lowest number), else
        // the anchor if feasible, else the least-loaded feasible candidate (ties: lowest number).
        // The loop visits the wave's candidate slots only; a lane whose placement has a single
        // candidate for that slot takes no part.
        for (uint32_t rem = pend_any; rem != 0u; rem &= rem - 1u) {
          const int s = __builtin_ctz(rem);
          const bool active = (pend >> s) & 1u;
          const uint32_t cs = static_cast<uint32_t>(cw[s >> 3] >> (8 * (s & 7))) & 0xffu;
          uint32_t cm = 1u;
          if (active) {
            if (cs != kCodeOver) {
              cm = rm[(cs - 32u) * kLanes + lane];
            } else {
              const uint64_t wd = s < 8 ? id_lo : id_hi;
              const uint32_t e = static_cast<uint32_t>(wd >> (8 * (s & 7))) & 0xffu;
              uint32_t unused = 0;
              cm = candidate_mask(a, live, base + e, unused);
            }
          }
          // the candidates in increasing GPU order (at most MC: 4 when R <= 3, else 5) and their loads
          const int ncand = __popc(cm);
          uint32_t g[MC];
          double v[MC];
          uint32_t rest = cm;
#pragma unroll
          for (int i = 0; i < MC; ++i) {
            g[i] = min(find_first_bit(rest), static_cast<uint32_t>(NG - 1));  // ffbl(0) = ~0: unused
            rest &= rest - 1u;
            v[i] = Lc[((g[i] >> 1) * kLanes + lane) * 2 + (g[i] & 1u)];
          }
          uint32_t fc = cm;
          if (guard) {
            uint32_t feas = 0;
#pragma unroll
            for (int i = 0; i < MC; ++i) feas |= (i < ncand && gden * v[i] <= rhs) ? (1u << g[i]) : 0u;
            fc = feas ? feas : cm;
          }
          // least loaded in fc; candidates come in increasing GPU order, so a strict < keeps the
          // lowest number among equal loads
          uint32_t least = g[0];
          double best = 0.0;
          bool found = false;
#pragma unroll
          for (int i = 0; i < MC; ++i) {
            const bool in = i < ncand && ((fc >> g[i]) & 1u);
            const bool better = in && (!found || v[i] < best);
            best = better ? v[i] : best;
            least = better ? g[i] : least;
            found |= in;
          }
          const uint32_t fr = fc & R;
          const uint32_t pick = fr ? find_first_bit(fr) : (((fc >> h) & 1u) ? h : least);
          R |= active ? (1u << pick) : 0u;
          dl.add(active ? pick : 63u);
          if (active)
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
      for (int m = 0; m < NG; ++m) Lm[m] = __fma_rn(rho, Lm[m], static_cast<double>(dl.get(m)));
    }
  }

  // dispatches of the single-candidate experts: every valid dispatch of e goes to its one GPU
  barrier_after_lds_atomics();
  for (int e = 0; e < E; ++e) {
    const uint32_t cs = cr.get(static_cast<uint32_t>(e));
    const uint32_t ne = ecnt[e];
    if (cs < 32u && ne)
      __hip_atomic_fetch_add(&cnt[cs * kLanes + lane], ne, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  barrier_after_lds_atomics();

  if (live) {
    if (cur_f >= 0 && a.cost_home_fam && fam_acc)
      atomicAdd(&a.cost_home_fam[static_cast<int64_t>(p) * a.F + cur_f], fam_acc);
    if (home_acc) atomicAdd(&a.cost_home[p], home_acc);
    if (span_acc) atomicAdd(&a.cost_span[p], span_acc);
    const int64_t o = (static_cast<int64_t>(p) * L + l) * G;
    for (int m = 0; m < G; ++m) a.load[o + m] = cnt[m * kLanes + lane];
    if (a.state_out) {
#pragma unroll
      for (int m = 0; m < NG; ++m)  // static register indices: the loads never leave registers
        if (m < G) a.state_out[o + m] = Lm[m];
    }
  }
  if (err) atomicOr(a.d_err, err);
}

template <int K, int NG, int MC>
void launch_on_t(const OnArgs& a, hipStream_t stream) {
  // candidate rows, counters, expert counts, then the larger of the code bytes and the loads
  const size_t lds = (static_cast<size_t>(kRows) * kLanes + 32 * kLanes + TACG_MAX_EXPERTS + 8) * sizeof(uint32_t) +
                     std::max(static_cast<size_t>(TACG_MAX_EXPERTS) * kLanes, static_cast<size_t>(NG) * kLanes * 8);
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&on_main<K, NG, MC>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  hipLaunchKernelGGL((on_main<K, NG, MC>), dim3((a.P + kLanes - 1) / kLanes, a.L), dim3(kLanes), lds, stream, a);
}

template <int K>
void launch_on(const OnArgs& a, hipStream_t stream) {
  // a slot has at most R + 1 candidates: four-entry candidate lists when R <= 3
  if (a.G <= 8) {
    if (a.R <= 3) launch_on_t<K, 8, 4>(a, stream);
    else launch_on_t<K, 8, kMaxCand>(a, stream);
  } else {
    if (a.R <= 3) launch_on_t<K, 32, 4>(a, stream);
    else launch_on_t<K, 32, kMaxCand>(a, stream);
  }
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
