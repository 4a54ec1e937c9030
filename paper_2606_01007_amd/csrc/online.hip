// Placement scoring with decayed per-GPU loads: the sequential form of the serving rule of Sec. 3.4
// (eqs. mean-load, feasible-set and load-update).  Each (placement, layer) keeps its own loads L_m,
// reads them for the guard and the least-loaded choice of every multi-candidate slot, and updates
// them after every token in trace order:  L_m <- fma(rho, L_m, Delta_m)  (float64, one rounding),
// Delta_m = the token's slots served by GPU m.  The guard is theta_den * G * L_m <= (theta_den +
// theta_num) * S with S = L_0 + L_1 + ... + L_31 summed in that order (GPUs >= G hold +0.0).
//
// Kernel design (gfx950): the scan over tokens is sequential, the (placement, layer) scans are
// independent.  Lane = placement, wave = 64 placements of one layer, one wave per workgroup, so there
// is about one wave per SIMD.  A lone wave issues one instruction at a time (VALU, SALU and LDS alike)
// and nothing hides its latencies, so the token loop is built for few instructions and few LDS
// operations on its dependency chain:
//   * The lane's code byte of every expert lives in 64 registers: the GPU of an expert with a single
//     candidate in the lane's placement, else 32 + its candidate row (63 when the rows ran out and the
//     list is rebuilt from the tables in memory).  The per-tile preparation turns each slot's expert
//     id into a lookup descriptor (register index and byte position), so that a lookup is one indexed
//     register move pair and one byte permute.
//   * The wave loads 64 token-layers at once (one per lane), builds the descriptors and a word with
//     the validity, family, anchor GPU and the slots that need a choice, and broadcasts them token by
//     token with v_readlane.
//   * Dispatch counts of a token are LDS atomics into a [GPU][lane] table (conflict-free; slots still
//     to be resolved land in a spare row).  The next served token reads the previous token's counts
//     and leaves zeros behind in one exchange per two GPUs, issued before its code lookups, and waits
//     only for those exchanges before the load update.
//   * The loads live in float64 registers (8 or 32 per lane, by G): one v_fma_f64 per GPU per token,
//     with the guard's ordered sum interleaved with the multiply-adds.  For a token with slots to
//     resolve the new loads are also written to LDS ([GPU][lane]), from where each lane reads the
//     loads of its own candidates.
//   * Candidate lists (GPUs in increasing order, padded with the first) are in LDS and, for at most
//     four candidates, also in registers: an expert's row is the same in every lane, so its list is
//     an indexed register move.  The slots to resolve are visited by a scalar loop over their bits.
//   * The least-loaded candidate of a feasible set is the least-loaded candidate overall: the guard
//     keeps every candidate whose scaled load is at most the threshold, so if any is feasible the
//     overall minimum is.  The choice therefore needs the guard only for the "reached" and "anchor"
//     tests.
//   * Per-GPU dispatch totals: the wave also counts every expert's valid dispatches of its layer
//     (ecnt, in the per-tile preparation); at the end each lane adds ecnt[e] to the GPU of every
//     single-candidate expert, and only the choices of multi-candidate slots are counted per token.
#include "tacg_internal.h"

namespace tacg {
namespace {

constexpr int kLanes = 64;
constexpr uint8_t kNone = 0xFF;

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

constexpr uint32_t kCodeOver = 63;  // multi-candidate expert without a row: read its tables
constexpr int kMaxCand = TACG_MAX_SECONDARY + 1;
constexpr size_t kLdsBudget = 40960;  // four workgroups per CU (160 KB of LDS)

// LDS of one workgroup (bytes, in this order): dispatch counts of the current token [NG + 1][64]
// (row NG takes the slots still to be resolved), resolved choices per GPU [NG][64], candidate lists
// [kRows][kRmWords][64], dispatches per expert [256], experts with a row somewhere [8], then the code
// bytes [256][64] while the tables are read and the staged loads [NG][64] (float64) afterwards.
template <int NG, int MC>
struct OnLayout {
  static constexpr int kRmWords = MC <= 4 ? 1 : 2;  // candidate GPUs, one byte each
  static constexpr size_t kShared = static_cast<size_t>(TACG_MAX_EXPERTS) * kLanes > static_cast<size_t>(NG) * kLanes * 8
                                        ? static_cast<size_t>(TACG_MAX_EXPERTS) * kLanes
                                        : static_cast<size_t>(NG) * kLanes * 8;
  static constexpr size_t kFixed = static_cast<size_t>(2 * NG + 1) * kLanes * 4 + TACG_MAX_EXPERTS * 4 + 8 * 4 + kShared;
  static constexpr size_t kRowBytes = static_cast<size_t>(kRmWords) * kLanes * 4;
  static constexpr int kRows = (kLdsBudget - kFixed) / kRowBytes > 31 ? 31 : static_cast<int>((kLdsBudget - kFixed) / kRowBytes);
  static constexpr size_t kBytes = kFixed + kRows * kRowBytes;
  static_assert(kRows >= 8, "candidate rows must fit the LDS budget");
};

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
  // A lookup descriptor of expert e: the register index in the low byte, and in the next byte the
  // byte of the pair (hi, lo) that holds e's code (4 + byte for experts >= 128), so that one byte
  // permute picks the code out of the two registers.
  __device__ __forceinline__ static uint32_t desc(uint32_t e) {
    return ((e >> 2) & 31u) | ((((e >> 5) & 4u) | (e & 3u)) << 8);
  }
  __device__ __forceinline__ static uint32_t expert(uint32_t d) {
    return ((d & 31u) << 2) | ((d >> 8) & 3u) | (((d >> 10) & 1u) << 7);
  }
  __device__ __forceinline__ uint32_t lookup(uint32_t d) const {
    const uint32_t i = d & 31u;
    // selector bytes 0x0c give zero: the code in the low byte, zeros above
    return __builtin_amdgcn_perm(hi[i], lo[i], ((d >> 8) & 7u) | 0x0c0c0c00u);
  }
};

// The candidate GPUs of mask m in increasing order, padded with the first (a padded entry repeats
// the first candidate's GPU and load, so it never changes a choice).
template <int MC>
__device__ __forceinline__ void cand_list(uint32_t m, uint32_t (&g)[MC]) {
  uint32_t rest = m;
  g[0] = find_first_bit(rest);
  rest &= rest - 1u;
#pragma unroll
  for (int i = 1; i < MC; ++i) {
    g[i] = rest ? find_first_bit(rest) : g[0];
    rest &= rest - 1u;
  }
}

__device__ __forceinline__ void lds_add(uint32_t* p, uint32_t v) {
  __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Reads dl rows 2q and 2q + 1 of this lane and leaves zeros behind (one LDS exchange of two dwords
// 256 bytes apart).  The results are valid after wait_lds().
__device__ __forceinline__ void lds_take_pair(const uint32_t* row0_lane, int q, uint32_t& x0, uint32_t& x1) {
  typedef uint32_t v2u __attribute__((ext_vector_type(2)));
  v2u r;
  const uint32_t addr = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(row0_lane));
  asm volatile("ds_wrxchg2st64_rtn_b32 %0, %1, %2, %2 offset0:%3 offset1:%4"
               : "=v"(r)
               : "v"(addr), "v"(0u), "i"(2 * q), "i"(2 * q + 1)
               : "memory");
  x0 = r.x;
  x1 = r.y;
}

__device__ __forceinline__ void wait_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// eq. load-update: L_m <- fma(rho, L_m, d_m) (one rounding) for every GPU, and S = the new loads summed
// in increasing GPU order (0 + L_0 = L_0).  Four GPUs per fixed instruction sequence, each add of S
// placed between independent multiply-adds so that neither chain waits on the other's latency.
template <int NG>
__device__ __forceinline__ void update_loads(double (&Lm)[NG], const uint32_t (&dq)[NG], double rho, double& S) {
#pragma unroll
  for (int g = 0; g < NG; g += 4) {
    const double d0 = static_cast<double>(dq[g]), d1 = static_cast<double>(dq[g + 1]);
    const double d2 = static_cast<double>(dq[g + 2]), d3 = static_cast<double>(dq[g + 3]);
    asm volatile(
        "v_fma_f64 %0, %5, %0, %6\n"
        "v_fma_f64 %1, %5, %1, %7\n"
        "v_add_f64 %4, %4, %0\n"
        "v_fma_f64 %2, %5, %2, %8\n"
        "v_add_f64 %4, %4, %1\n"
        "v_fma_f64 %3, %5, %3, %9\n"
        "v_add_f64 %4, %4, %2\n"
        "v_add_f64 %4, %4, %3"
        : "+v"(Lm[g]), "+v"(Lm[g + 1]), "+v"(Lm[g + 2]), "+v"(Lm[g + 3]), "+v"(S)
        : "s"(rho), "v"(d0), "v"(d1), "v"(d2), "v"(d3));
  }
}

// grid (ceil(P / 64), L), 64 threads; NG = 8 or 32 >= G GPUs in registers, MC >= R + 1 candidates.
template <int K, int NG, int MC>
__global__ __launch_bounds__(kLanes) void on_main(OnArgs a) {
  using Lay = OnLayout<NG, MC>;
  constexpr int kRows = Lay::kRows;
  constexpr int kRmWords = Lay::kRmWords;
  extern __shared__ __align__(16) uint32_t lds[];
  constexpr int KD = (K + 1) / 2;  // dwords of 16-bit lookup descriptors per token-layer
  const int lane = threadIdx.x;
  const int l = blockIdx.y;
  const int p = blockIdx.x * kLanes + lane;
  const bool live = p < a.P;
  const int E = a.E, G = a.G, L = a.L;
  uint32_t* dl = lds;                                   // [NG + 1][64] this token's dispatches per GPU
  uint32_t* cnt = dl + (NG + 1) * kLanes;               // [NG][64] resolved dispatches per GPU
  uint32_t* rm = cnt + NG * kLanes;                     // [kRows][kRmWords][64] candidate lists
  uint32_t* ecnt = rm + kRows * kRmWords * kLanes;      // [E] valid dispatches per expert
  uint32_t* hasrow = ecnt + TACG_MAX_EXPERTS;           // [8] experts with several candidates somewhere
  uint8_t* code = reinterpret_cast<uint8_t*>(hasrow + 8);
  double* Lc = reinterpret_cast<double*>(code);         // [NG][64] staged loads (after the code bytes)
  uint32_t err = 0;

  // ---- candidate sets of this lane's placement (eq. candidate-set) ----
  const int64_t base = (static_cast<int64_t>(p) * L + l) * E;
  int nr = 0;  // rows of rm in use (workgroup-uniform)
  // with at most four candidates a row's list is one dword: the lists also live in registers (the row
  // of an expert is the same in every lane, so a lookup is an indexed register move)
  v32u rl;
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
          uint32_t g[MC];
          cand_list<MC>(m, g);
          uint32_t w0 = 0, w1 = 0;
#pragma unroll
          for (int i = 0; i < MC; ++i) {
            if (i < 4) w0 |= g[i] << (8 * i);
            else w1 |= g[i] << (8 * (i - 4));
          }
          rm[(nr * kRmWords) * kLanes + lane] = w0;
          if (kRmWords > 1) rm[(nr * kRmWords + 1) * kLanes + lane] = w1;
          if constexpr (MC <= 4) rl[nr] = w0;
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
  for (int m = 0; m <= NG; ++m) dl[m * kLanes + lane] = 0;
#pragma unroll
  for (int m = 0; m < NG; ++m) cnt[m * kLanes + lane] = 0;
  for (int e = lane; e < E; e += kLanes) ecnt[e] = 0;
  __syncthreads();  // the code bytes are in registers; the region now holds the staged loads

  double Lm[NG];
#pragma unroll
  for (int m = 0; m < NG; ++m) Lm[m] = (a.state_in && live && m < G) ? a.state_in[(base / E) * G + m] : 0.0;
  const double rho = a.rho;
  const bool guard = a.theta_den != 0;
  const double gden = static_cast<double>(a.theta_den) * static_cast<double>(G);
  const double rnum = static_cast<double>(a.theta_den) + static_cast<double>(a.theta_num);
  uint32_t* const dl_lane = dl + lane;
  uint32_t* const cnt_lane = cnt + lane;
  double* const Lc_lane = Lc + lane;

  unsigned long long span_acc = 0, home_acc = 0, fam_acc = 0;
  int cur_f = -1;
  bool pending = false;  // wave-uniform: the last served token's dispatches are in dl, not yet in Lm
  const int16_t* trace_l = a.trace + static_cast<int64_t>(l) * a.N * K;
  int f_tile = 0;  // family of the first token of the current tile

  for (int64_t tile = 0; tile < a.N; tile += kLanes) {
    while (static_cast<int64_t>(a.fam[f_tile].y) <= tile) ++f_tile;
    // ---- per-lane preparation of token-layer tile + lane ----
    const int64_t t = tile + lane;
    uint32_t pd[KD];
#pragma unroll
    for (int w = 0; w < KD; ++w) pd[w] = 0;
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
        pd[s >> 1] |= CodeRegs::desc(id) << (16 * (s & 1));
        info |= ((hasrow[id >> 5] >> (id & 31)) & 1u) << (16 + s);  // a candidate row exists for id
      }
      if (!ok) err |= TACG_ERR_ID_RANGE;
      if (dup) err |= TACG_ERR_ID_DUP;
      if (ok && !dup) {
#pragma unroll
        for (int s = 0; s < K; ++s) lds_add(&ecnt[raw[s]], 1u);
      }
      int f = f_tile;
      while (static_cast<int64_t>(a.fam[f].y) <= t) ++f;
      const uint4 fr = a.fam[f];
      const uint32_t hz = (fr.z >> 8) & 0xffu;
      const uint32_t h = (fr.z & 0xffu) + static_cast<uint32_t>((t - static_cast<int64_t>(fr.x)) % hz);
      info |= ((ok && !dup) ? 1u : 0u) | (static_cast<uint32_t>(f) << 1) | (h << 8);
    }
    const int ntile = static_cast<int>(min(static_cast<int64_t>(kLanes), a.N - tile));
    uint32_t span32 = 0, home32 = 0, fam32 = 0;  // this tile's costs (at most 64 * 15 each)

    for (int j = 0; j < ntile; ++j) {
      const uint32_t tinfo = __builtin_amdgcn_readlane(info, j);
      if (!(tinfo & 1u)) continue;  // invalid token-layer (flagged): not served, loads untouched
      uint32_t ds[KD];
#pragma unroll
      for (int w = 0; w < KD; ++w) ds[w] = __builtin_amdgcn_readlane(pd[w], j);
      const int f = static_cast<int>((tinfo >> 1) & 127u);
      if (f != cur_f) {
        fam_acc += fam32;
        fam32 = 0;
        if (cur_f >= 0 && a.cost_home_fam && live && fam_acc)
          atomicAdd(&a.cost_home_fam[static_cast<int64_t>(p) * a.F + cur_f], fam_acc);
        fam_acc = 0;
        cur_f = f;
      }
      const uint32_t h = (tinfo >> 8) & 0xffu;

      // the previous served token's dispatch counts, cleared for this token (all zero before the
      // first served token, which then takes rho = 1: an exact no-op)
      uint32_t dq[NG];
#pragma unroll
      for (int q = 0; q < NG / 2; ++q) lds_take_pair(dl_lane, q, dq[2 * q], dq[2 * q + 1]);

      // single-candidate slots: the set R of GPUs the token reaches, and their dispatches
      uint32_t c[K];
#pragma unroll
      for (int s = 0; s < K; ++s) c[s] = cr.lookup(__builtin_amdgcn_ubfe(ds[s >> 1], 16 * (s & 1), 16));
      uint32_t R = 0;
      uint64_t cw[(K + 7) / 8];  // the codes again, one byte per slot, for the slot loop below
#pragma unroll
      for (int q = 0; q < (K + 7) / 8; ++q) cw[q] = 0;
#pragma unroll
      for (int s = 0; s < K; ++s) {
        cw[s >> 3] |= static_cast<uint64_t>(c[s]) << (8 * (s & 7));
        R |= static_cast<uint32_t>(1ull << c[s]);  // no bit for codes >= 32 (slots still to be resolved)
        lds_add(dl_lane + min(c[s], static_cast<uint32_t>(NG)) * kLanes, 1u);
      }
      // slots whose expert has several candidates in some placement of the wave (wave-uniform)
      const uint32_t pend_any = tinfo >> 16;

      // eq. load-update for the previous served token, so that the loads hold every token before
      // this one; for a token with slots to resolve the new loads also go to LDS (each slot reads those
      // of its own candidates) and into the guard's sum S (GPUs in increasing order; 0 + L_0 = L_0)
      const double rho_t = pending ? rho : 1.0;
      pending = true;
      double S = 0.0;
      asm volatile("s_waitcnt lgkmcnt(%0)" ::"i"(K < 15 ? K : 15) : "memory");
      update_loads<NG>(Lm, dq, rho_t, S);
      if (pend_any) {
#pragma unroll
        for (int m = 0; m < NG; ++m) Lc_lane[m * kLanes] = Lm[m];
        // the guard's right-hand side under the current loads (eq. feasible-set with the mean of
        // eq. mean-load)
        const double rhs = rnum * S;
        // multi-candidate slots in slot order: a reached feasible candidate (lowest number), else
        // the anchor if feasible, else the least-loaded candidate (ties: lowest number)
        for (uint32_t rem = pend_any; rem != 0u; rem &= rem - 1u) {
          const int s = __builtin_ctz(rem);
          const uint64_t cws = (K > 8 && s >= 8) ? cw[(K + 7) / 8 - 1] : cw[0];
          const uint32_t cs = static_cast<uint32_t>(cws >> (8 * (s & 7))) & 0xffu;
          if (cs < 32u) continue;  // a single candidate in this lane's placement
          uint32_t g[MC];
          if (cs != kCodeOver) {
            // the lanes here all hold code 32 + the expert's row
            uint32_t w0, w1 = 0;
            if constexpr (MC <= 4) {
              w0 = rl[__builtin_amdgcn_readfirstlane(cs) - 32u];
            } else {
              const uint32_t* rp = rm + ((cs - 32u) * kRmWords) * kLanes + lane;
              w0 = rp[0];
              w1 = rp[kLanes];
            }
#pragma unroll
            for (int i = 0; i < MC; ++i) g[i] = __builtin_amdgcn_ubfe(i < 4 ? w0 : w1, 8 * (i & 3), 8);
          } else {
            const uint32_t e = CodeRegs::expert(__builtin_amdgcn_ubfe(ds[s >> 1], 16 * (s & 1), 16));
            uint32_t unused = 0;
            cand_list<MC>(candidate_mask(a, live, base + e, unused), g);
          }
          double v[MC];
#pragma unroll
          for (int i = 0; i < MC; ++i) v[i] = Lc_lane[g[i] * kLanes];
          uint32_t cm = 0, fb = 0;
#pragma unroll
          for (int i = 0; i < MC; ++i) {
            const uint32_t b = 1u << g[i];
            cm |= b;
            fb |= (gden * v[i] <= rhs) ? b : 0u;
          }
          const uint32_t fc = (guard && fb) ? fb : cm;
          uint32_t least = g[0];
          double best = v[0];
#pragma unroll
          for (int i = 1; i < MC; ++i) {
            const bool lt = v[i] < best;
            best = lt ? v[i] : best;
            least = lt ? g[i] : least;
          }
          // a reached feasible candidate, else the anchor or the least loaded: ffbl(0) = 0xffffffff,
          // so the minimum takes the reached one whenever there is one
          const uint32_t alt = ((fc >> h) & 1u) ? h : least;
          const uint32_t pick = min(find_first_bit(fc & R), alt + 32u) & 31u;
          R |= 1u << pick;
          lds_add(dl_lane + pick * kLanes, 1u);
          lds_add(cnt_lane + pick * kLanes, 1u);
        }
      }
      const uint32_t n = __popc(R);
      span32 += n - 1u;
      const uint32_t home = n - ((R >> h) & 1u);
      home32 += home;
      fam32 += home;
    }
    span_acc += span32;
    home_acc += home32;
    fam_acc += fam32;
  }
  // the last served token's update
  if (pending) {
    uint32_t dq[NG];
#pragma unroll
    for (int q = 0; q < NG / 2; ++q) lds_take_pair(dl_lane, q, dq[2 * q], dq[2 * q + 1]);
    wait_lds();
    double S = 0.0;
    update_loads<NG>(Lm, dq, rho, S);
  }

  // dispatches of the single-candidate experts: every valid dispatch of e goes to its one GPU
  barrier_after_lds_atomics();
  for (int e = 0; e < E; ++e) {
    const uint32_t cs = cr.get(static_cast<uint32_t>(e));
    const uint32_t ne = ecnt[e];
    if (cs < 32u && ne) lds_add(&cnt[cs * kLanes + lane], ne);
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
  const size_t lds = OnLayout<NG, MC>::kBytes;
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
