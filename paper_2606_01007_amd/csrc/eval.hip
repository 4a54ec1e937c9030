// Placement scoring: per-token cross-GPU cost, GESR candidate choice and per-GPU loads
// (Sec. 3.4 serving rule with eqs. mean-load and feasible-set; App. C per-token dispatch sets;
// App. H "Comm"), plus the snapshot loads that feed the guard and Jain / MaxVio (App. H).
//
// Launch sequence of tacg_eval_placements:
//   ev_zero      clear the workspace accumulators
//   ev_flags     validate the placement tables; mark experts that have a secondary in any placement
//   ev_replist   per layer: compact index of the marked ("replicated") experts
//   ev_repinfo   per (placement, layer, replicated expert): feasible candidate mask FC, the
//                fallback GPU argmin_{m in FC} load_ref (ties: lowest number) and whether the expert
//                has a single candidate in that placement
//   ev_valid     validate the trace's ids: flag and count the token-layers with an id out of range
//                or a repeated id, and mark their groups of 64 token-layers
//   ev_main      the trace pass (below); also counts every expert's dispatches; an invalid token-layer
//                (checked again only in marked groups) is not scored
//   ev_finalize  loads = counts of single-candidate experts on their primary + replicated choices;
//                costs from the accumulators
//
// ev_main (the hot kernel).  Lane = placement, wave = 64 placements, every wave of a workgroup scores
// the same placements on different tokens, so a token's expert ids are wave-uniform:
//   * LDS holds, for the workgroup's placements and layer, the one-hot GPU mask of every expert
//     (tbl[e][p], uint32; zero for replicated experts), the replica info (FC, fallback) and
//     per-placement counters of the GPUs chosen for replicated experts.
//   * A wave loads 64 token-layers at once (one load per lane), packs the expert ids four per dword
//     and builds a per-token word with the replicated-slot mask, the anchor GPU and the replica
//     indices; the per-token loop broadcasts them with v_readlane, so the ids live in SGPRs.
//   * Per token-layer and lane: k conflict-free LDS reads (64 consecutive dwords per wave), OR of the
//     masks, then (rarely) the replicated slots, then two popcounts into per-lane accumulators.
#include "tacg_internal.h"

namespace tacg {
namespace {

constexpr int kMainThreads = 1024;
constexpr int kMaxPieces = 160;
constexpr uint32_t kXcds = 8;  // XCDs of an MI355X; workgroups are dealt to them round-robin
// About 32 workgroups of ev_main per CU: short enough that the last round leaves little idle time
// when the families' ragged last pieces make the workgroups uneven (measured 2 % faster than 4096
// on a Dirichlet family mix), long enough to amortise the table set-up and the flushes.
constexpr int64_t kTargetWorkgroups = 8192;
constexpr uint8_t kNone = 0xFF;

struct EvWs {
  uint32_t* cnt;        // [L][E] dispatches per expert
  uint32_t* flagbits;   // [L][8] experts with a secondary in some placement
  uint8_t* rep_of;      // [L][E] compact replicated index or 0xFF
  int32_t* rep_list;    // [L][TACG_MAX_REPLICATED]
  int32_t* n_rep;       // [L]
  uint2* rep_info;      // [L][TACG_MAX_REPLICATED][P]  (FC mask, fallback GPU)
  // accumulators are laid out with the placement fastest, so that a workgroup's adds for its run of
  // placements are contiguous (coalesced atomics)
  unsigned long long* acc_home;  // [P]
  unsigned long long* acc_span;  // [P]
  unsigned long long* acc_fam;   // [F][P]
  uint32_t* rep_load;   // [L][G][P2], P2 = P rounded up to even: placement pairs share a 64-bit add
  // App. C statistics (used only by tacg_eval_trace_stats)
  uint32_t* cnt_fam;                  // [F][L][E] dispatches per expert and family
  unsigned long long* acc_span_fam;   // [F][P] sum of |cards| over the family's token-layers
  unsigned long long* acc_cross_fam;  // [F][P] token-layers whose cards span several bands
  unsigned long long* acc_hmass_fam;  // [F][P] replicated-slot dispatches served in the family's band
  unsigned long long* n_bad;          // [1] token-layers not scored: an id out of range or repeated
  uint32_t* bad_tiles;                // [ceil(N L / 64 / 32)] bit g: token-layers 64 g .. 64 g + 63 of
                                      // the flattened trace (x = l N + t) hold an invalid one
};

__host__ __device__ inline int32_t even_up(int32_t P) { return P + (P & 1); }

__host__ __device__ inline int64_t bad_tile_words(int64_t N, int32_t L) { return (N * L + 2047) / 2048; }

EvWs carve_ev(void* ws, int64_t N, int32_t L, int32_t E, int32_t G, int32_t P, int32_t F, size_t* used = nullptr) {
  Carver c{static_cast<char*>(ws), 0};
  EvWs r;
  r.cnt = c.take<uint32_t>(static_cast<size_t>(L) * E);
  r.flagbits = c.take<uint32_t>(static_cast<size_t>(L) * 8);
  r.acc_home = c.take<unsigned long long>(static_cast<size_t>(P));
  r.acc_span = c.take<unsigned long long>(static_cast<size_t>(P));
  r.acc_fam = c.take<unsigned long long>(static_cast<size_t>(P) * F);
  r.rep_load = c.take<uint32_t>(static_cast<size_t>(even_up(P)) * L * G);
  r.rep_of = c.take<uint8_t>(static_cast<size_t>(L) * E);
  r.rep_list = c.take<int32_t>(static_cast<size_t>(L) * TACG_MAX_REPLICATED);
  r.n_rep = c.take<int32_t>(static_cast<size_t>(L));
  r.rep_info = c.take<uint2>(static_cast<size_t>(L) * TACG_MAX_REPLICATED * P);
  r.cnt_fam = c.take<uint32_t>(static_cast<size_t>(F) * L * E);
  r.acc_span_fam = c.take<unsigned long long>(static_cast<size_t>(P) * F);
  r.acc_cross_fam = c.take<unsigned long long>(static_cast<size_t>(P) * F);
  r.acc_hmass_fam = c.take<unsigned long long>(static_cast<size_t>(P) * F);
  r.n_bad = c.take<unsigned long long>(1);
  r.bad_tiles = c.take<uint32_t>(static_cast<size_t>(bad_tile_words(N, L)));
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
  int32_t n_pblocks;  // placement blocks of 64 * PPL placements
  int32_t stats;      // App. C statistics requested
  uint32_t band_starts;  // bit b: a family band starts at GPU b (the bands tile 0..G-1)
  // home band of family f: component f % 4 of band4[f / 4] = home_start | home_size << 8
  uint4 band4[TACG_MAX_FAMILIES / 4];
  // One record per piece of one family's tokens: (first token, end token, family offset,
  // home_start | home_size << 8 | family << 16).  Kept as 16-byte records: indexing kernel-argument
  // arrays of different element sizes with one runtime index lets the compiler fold the byte and
  // dword offsets into an unaligned scalar-load base, which the scalar unit does not honour.
  uint4 piece[kMaxPieces];
};
static_assert(sizeof(EvArgs) <= 4096, "kernel arguments must stay within 4 KB");

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
  for (int64_t j = i; j < static_cast<int64_t>(even_up(a.P)) * a.L * a.G; j += stride) w.rep_load[j] = 0;
  if (i == 0) *w.n_bad = 0;
  for (int64_t j = i; j < bad_tile_words(a.N, a.L); j += stride) w.bad_tiles[j] = 0;
  if (a.stats) {
    for (int64_t j = i; j < static_cast<int64_t>(a.F) * a.L * a.E; j += stride) w.cnt_fam[j] = 0;
    for (int64_t j = i; j < static_cast<int64_t>(a.P) * a.F; j += stride) {
      w.acc_span_fam[j] = 0;
      w.acc_cross_fam[j] = 0;
      w.acc_hmass_fam[j] = 0;
    }
  }
}

// Trace validation (a1): every token-layer's ids, one wave per 64 consecutive token-layers of the
// flattened trace (x = l * N + t), grid-stride.  A token-layer with an id out of range or a repeated id
// is flagged, counted (n_bad) and marks its group of 64 in bad_tiles, so that ev_main checks the ids
// itself only in the few tiles that meet a marked group.
template <int K>
__global__ __launch_bounds__(256) void ev_valid(EvArgs a) {
  const int64_t total = a.N * a.L;
  const int lane = threadIdx.x & 63;
  const int64_t nwaves = static_cast<int64_t>(gridDim.x) * (blockDim.x >> 6);
  uint32_t err = 0;
  for (int64_t g = static_cast<int64_t>(blockIdx.x) * (blockDim.x >> 6) + (threadIdx.x >> 6); g * 64 < total;
       g += nwaves) {
    const int64_t x = g * 64 + lane;
    bool bad = false;
    if (x < total) {
      const int16_t* idp = a.trace + x * K;
      uint32_t raw[K];
#pragma unroll
      for (int s = 0; s < K; ++s) raw[s] = static_cast<uint16_t>(idp[s]);
      bool ok = true, dup = false;
#pragma unroll
      for (int s = 0; s < K; ++s) {
        ok &= raw[s] < static_cast<uint32_t>(a.E);
#pragma unroll
        for (int q = 0; q < s; ++q) dup |= raw[s] == raw[q];
      }
      if (!ok) err |= TACG_ERR_ID_RANGE;
      if (dup) err |= TACG_ERR_ID_DUP;
      bad = !ok || dup;
    }
    const uint64_t b = __builtin_amdgcn_ballot_w64(bad);
    if (b != 0u && lane == 0) {
      atomicOr(&a.ws.bad_tiles[g >> 5], 1u << (g & 31));
      atomicAdd(a.ws.n_bad, static_cast<unsigned long long>(__builtin_popcountll(b)));
    }
  }
  if (err) atomicOr(a.d_err, err);
}

// Table validation and the replicated-expert marks.  Flat grid-stride loop over (p, l, e).
__global__ __launch_bounds__(256) void ev_flags(EvArgs a) {
  const int64_t n = static_cast<int64_t>(a.P) * a.L * a.E;
  uint32_t err = 0;
  for (int64_t pe = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; pe < n;
       pe += static_cast<int64_t>(gridDim.x) * blockDim.x) {
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
    if (any) {
      // every placement marks the same few experts: set a bit only when a device-scope read does
      // not show it yet (a stale read costs one extra atomic, never a missing bit)
      const int e = static_cast<int>(pe % a.E);
      const int l = static_cast<int>((pe / a.E) % a.L);
      uint32_t* w = &a.ws.flagbits[l * 8 + (e >> 5)];
      const uint32_t bit = 1u << (e & 31);
      if (!(__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & bit)) atomicOr(w, bit);
    }
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
  barrier_after_lds_atomics();
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
  // this placement's snapshot loads in registers (all loads in flight at once)
  int64_t rf[TACG_MAX_GPUS];
#pragma unroll
  for (int m = 0; m < TACG_MAX_GPUS; ++m) rf[m] = m < G ? ref[m] : 0;
  // the candidate sets of the replicated experts, gathered before they are used
  uint32_t cands[TACG_MAX_REPLICATED];
#pragma unroll
  for (int r = 0; r < TACG_MAX_REPLICATED; ++r) {
    uint32_t cand = 0;
    if (r < nrep) {
      const int e = a.ws.rep_list[l * TACG_MAX_REPLICATED + r];
      const int64_t pe = (static_cast<int64_t>(p) * a.L + l) * a.E + e;
      const uint8_t g0 = a.primary[pe];
      if (g0 < G) cand |= 1u << g0;
      for (int q = 0; q < a.R; ++q) {
        const uint8_t g = a.secondary[pe * a.R + q];
        if (g < G) cand |= 1u << g;
      }
    }
    cands[r] = cand;
  }
  // eq. feasible-set with the mean load of eq. mean-load, exact in 128-bit integers
  uint32_t feas = (G == 32) ? 0xffffffffu : ((1u << G) - 1u);
  if (a.theta_den != 0) {
    __int128 total = 0;
#pragma unroll
    for (int m = 0; m < TACG_MAX_GPUS; ++m) total += rf[m];
    const __int128 rhs = static_cast<__int128>(a.theta_den + a.theta_num) * total;
    feas = 0;
#pragma unroll
    for (int m = 0; m < TACG_MAX_GPUS; ++m)
      if (m < G && static_cast<__int128>(a.theta_den) * G * rf[m] <= rhs) feas |= 1u << m;
  }
#pragma unroll
  for (int r = 0; r < TACG_MAX_REPLICATED; ++r) {
    if (r >= nrep) break;
    uint32_t cand = cands[r];
    if (cand == 0) cand = 1u;  // invalid table (already flagged): keep the choice in range
    uint32_t fc = cand & feas;
    if (fc == 0) fc = cand;
    // least-loaded feasible candidate, ties to the lowest GPU
    int best = -1;
    int64_t bestv = 0;
#pragma unroll
    for (int m = 0; m < TACG_MAX_GPUS; ++m) {
      if (((fc >> m) & 1u) && (best < 0 || rf[m] < bestv)) {
        best = m;
        bestv = rf[m];
      }
    }
    // bit 31: the expert has a single candidate in this placement (it is served by its primary and
    // belongs to the GPUs the token reaches before any multi-candidate slot is resolved)
    const uint32_t single = (__popc(cand) == 1) ? 0x80000000u : 0u;
    a.ws.rep_info[(static_cast<int64_t>(l) * TACG_MAX_REPLICATED + r) * a.P + p] =
        make_uint2(fc, static_cast<uint32_t>(best) | single);
  }
}

// ------------------------------------------------------------------------------------------------
// The trace pass.  PPL placements per lane (one 8- or 16-byte LDS read per slot serves all of them);
// a workgroup scores 64 * PPL placements of one layer on one piece of one family's tokens.
// grid (placement blocks, pieces, L).  The workgroups of placement block 0 also count the
// dispatches of every expert (each token-layer is seen by exactly one of them); ev_valid has already
// checked the ids, and only tiles it marked check them again, to leave their invalid token-layers out.
// Choices for replicated experts are counted in 16-bit LDS counters (two per dword).  After every
// round of at most 65535 / K tokens (so that they cannot overflow) each thread adds a fixed set of
// them into 32-bit registers and clears them; the registers go to the workspace once per workgroup.
//
// Per-token word `info` built by the lane that loaded the token-layer (wave-uniform after v_readlane):
//   K <= 8:  bits 0-7 replicated-slot mask, 8-12 band position of the anchor GPU within its family's
//            band, then 4-bit replica indices of the first four replicated slots (13-16 ... 25-28);
//   K > 8:   bits 0-15 replicated-slot mask, 16-20 band position, replica indices of the first two
//            replicated slots (21-24, 25-28).
// Further replicated slots of a token look their index up in LDS.
template <int K>
struct InfoLayout {
  static constexpr int kMaskBits = K <= 8 ? 8 : 16;
  static constexpr int kHomeShift = kMaskBits;
  static constexpr int kRepShift = kMaskBits + 5;
  static constexpr int kRepSlots = K <= 8 ? 4 : 2;
  static constexpr uint32_t kBad = 1u << 31;  // the token-layer is not scored (invalid ids)
};

// Index of the lowest set bit, 0xffffffff for 0 (the hardware v_ffbl_b32 result).
__device__ __forceinline__ uint32_t find_first_bit(uint32_t x) {
  uint32_t r;
  asm("v_ffbl_b32 %0, %1" : "=v"(r) : "v"(x));
  return r;
}

template <int K, int PPL, bool NARROW, bool STATS>
struct Scorer {
  static constexpr int PW = 64 * PPL;
  static constexpr int KB = (K + 3) / 4;  // dwords of 8-bit expert ids per token-layer
  static constexpr int kRowShift = PPL == 2 ? 9 : 10;  // log2 of a table row in bytes (PW * 4)
  using IL = InfoLayout<K>;

  const char* tbl_lane;   // LDS table base + this lane's column offset
  uint32_t row_bytes;     // PW * 4, held in a VGPR
  const uint2* rinfo;     // [MAX_REP][PW]
  uint32_t* rcnt;         // [G][PW / 2]
  const uint8_t* rep_of;  // [E]
  int lane;
  uint32_t acc_span[PPL], acc_home[PPL];

  // one-hot GPU masks of the token's single-candidate experts, OR-ed per placement
  __device__ __forceinline__ void gather(const uint32_t (&ids)[KB], uint32_t (&m)[PPL]) const {
#pragma unroll
    for (int q = 0; q < PPL; ++q) m[q] = 0;
#pragma unroll
    for (int s = 0; s < K; ++s) {
      const uint32_t id = __builtin_amdgcn_ubfe(ids[s >> 2], 8 * (s & 3), 8);
      // row stride in an opaque VGPR: one scalar extract and one v_mad_u32_u24 per slot (left to
      // itself the compiler moves the shift into two scalar instructions for half of the slots)
      const char* base = tbl_lane + __umul24(id, row_bytes);
      if constexpr (PPL == 2) {
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
  }

  // Replicated slots in slot order: the lowest-numbered feasible candidate the token already
  // reaches, else the anchor if it is a feasible candidate, else the least-loaded feasible candidate.
  // rinfo[r][p] = (FC mask, packed fallbacks): byte i holds 32 + (the choice when no candidate is
  // reached) for the anchor at band position i (bands of up to 4 GPUs; wider bands keep 32 + the
  // least-loaded feasible candidate and test the anchor here).  ffbl(0) = 0xffffffff, so min(ffbl(x), 32 + fb)
  // selects the reached candidate when there is one; the shift and the counter row use its low 5 bits.
  __device__ __forceinline__ void resolve(uint32_t info, const uint32_t (&ids)[KB], uint32_t (&m)[PPL]) {
    const uint32_t repmask = info & ((1u << IL::kMaskBits) - 1u);
    if (!repmask) return;
    const uint32_t hshift = 8u * ((info >> IL::kHomeShift) & 31u);  // 8 * band position of the anchor
    // a scalar loop over the set bits of the (wave-uniform) mask: the replicated slots only
    int nth = 0;
    for (uint32_t rem = repmask; rem != 0u; rem &= rem - 1u, ++nth) {
      const int s = __builtin_ctz(rem);
      uint32_t r;
      if (nth < IL::kRepSlots) {
        r = (info >> (IL::kRepShift + 4 * nth)) & 15u;
      } else {
        r = rep_of[__builtin_amdgcn_ubfe(ids[s >> 2], 8 * (s & 3), 8)];
      }
      const uint2* rp = rinfo + r * PW + lane * PPL;
      uint2 ri[PPL];
#pragma unroll
      for (int q = 0; q < PPL; q += 2) {
        const uint4 v = *reinterpret_cast<const uint4*>(rp + q);
        ri[q] = make_uint2(v.x, v.y);
        ri[q + 1] = make_uint2(v.z, v.w);
      }
#pragma unroll
      for (int q = 0; q < PPL; ++q) {
        const uint32_t x = ri[q].x & m[q];
        uint32_t fb;
        if constexpr (NARROW) {
          fb = __builtin_amdgcn_ubfe(ri[q].y, hshift, 8);
        } else {
          const uint32_t h = home_start + (hshift >> 3);
          fb = ((ri[q].x >> h) & 1u) ? 32u + h : ri[q].y;
        }
        const uint32_t pick = min(find_first_bit(x), fb) & 31u;
        m[q] |= 1u << pick;
        __hip_atomic_fetch_add(&rcnt[(pick * PW + lane * PPL + q) >> 1], 1u << (16 * (q & 1)), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
  }

  uint32_t home_start;
  uint32_t band_starts;     // STATS: bit b set when a family band starts at GPU b
  uint32_t acc_cross[PPL];  // STATS: token-layers whose cards span more than one band

  __device__ __forceinline__ void account(uint32_t info, const uint32_t (&m)[PPL]) {
    const uint32_t not_h = ~(1u << (home_start + ((info >> IL::kHomeShift) & 31u)));
#pragma unroll
    for (int q = 0; q < PPL; ++q) {
      acc_span[q] += __popc(m[q]);
      acc_home[q] += __popc(m[q] & not_h);
      if constexpr (STATS) {
        // The bands are intervals that tile the GPUs, so the cards lie in more than one band exactly
        // when a band starts in (lowest card, highest card].  With lo / hi the lowest / highest card,
        // (2 << hi) - (2 << lo) (mod 2^32, so hi = 31 works) has exactly those bits set.
        // (m == 0 only after a flagged table error; the masks keep every shift defined)
        const uint32_t lo = find_first_bit(m[q]) & 31u;
        const uint32_t top = 0x80000000u >> (__clz(static_cast<int>(m[q])) & 31);  // 1 << hi
        const uint32_t range = (top << 1) + (0xfffffffeu << lo);
        acc_cross[q] += (band_starts & range) != 0u ? 1u : 0u;
      }
    }
  }
};

// Token loop of one workgroup (see ev_main).  NARROW: the family's band has at most 4 GPUs, so the
// fallback choices are packed per band position.
template <int K, int PPL, bool NARROW, bool STATS, bool CHECK>
__device__ __forceinline__ void score_piece(const EvArgs& a, const uint32_t* tbl, const uint2* rinfo, uint32_t* rcnt,
                                            uint32_t* ecnt, const uint8_t* rep_of, int l, int p0, int nrep,
                                            bool counter, uint32_t t_begin, uint32_t t_end, uint32_t off_f,
                                            uint32_t hs, uint32_t hz, int f,
                                            uint32_t (&acc_span)[PPL], uint32_t (&acc_home)[PPL],
                                            uint32_t (&acc_cross)[PPL], uint32_t& n_scored) {
  using S = Scorer<K, PPL, NARROW, STATS>;
  using IL = InfoLayout<K>;
  constexpr int PW = S::PW;
  constexpr int KB = S::KB;
  constexpr int U = 4;             // token-layers scored together (independent LDS reads in flight)
  constexpr uint32_t round_tokens = 65535u / K;
  // each thread folds the same 2 * kRcntPerThread 16-bit counters after every round
  constexpr int kRcntPerThread = (TACG_MAX_GPUS * PW / 2 + kMainThreads - 1) / kMainThreads;
  uint32_t rsum[2 * kRcntPerThread];
#pragma unroll
  for (int c = 0; c < 2 * kRcntPerThread; ++c) rsum[c] = 0;
  const int E = a.E, G = a.G, L = a.L;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nwaves = blockDim.x >> 6;
  const int16_t* trace_l = a.trace + static_cast<int64_t>(l) * a.N * K;
  S sc;
  sc.tbl_lane = reinterpret_cast<const char*>(tbl) + lane * PPL * 4;
  asm volatile("v_mov_b32 %0, %1" : "=v"(sc.row_bytes) : "i"(S::PW * 4));
  sc.rinfo = rinfo;
  sc.rcnt = rcnt;
  sc.rep_of = rep_of;
  sc.lane = lane;
  sc.home_start = hs;
  sc.band_starts = a.band_starts;
#pragma unroll
  for (int q = 0; q < PPL; ++q) sc.acc_span[q] = sc.acc_home[q] = sc.acc_cross[q] = 0;

  for (uint32_t r_begin = t_begin; r_begin < t_end; r_begin += round_tokens) {
    const uint32_t r_end = min(t_end, r_begin + round_tokens);
    for (uint32_t tile = r_begin + wave * 64u; tile < r_end; tile += nwaves * 64u) {
      // ---- per-lane preprocessing of token-layer (tile + lane) ----
      const uint32_t t = tile + lane;
      uint32_t pk[KB];
#pragma unroll
      for (int w = 0; w < KB; ++w) pk[w] = 0;
      // does the tile meet a group of 64 flattened token-layers that ev_valid marked? (wave-uniform;
      // only the variant for traces with an invalid token-layer reads the marks)
      bool marked = false;
      if constexpr (CHECK) {
        const int64_t x0 = static_cast<int64_t>(l) * a.N + tile;
        const int64_t g0 = x0 >> 6, g1 = min(x0 + 63, static_cast<int64_t>(L) * a.N - 1) >> 6;
        marked = (((a.ws.bad_tiles[g0 >> 5] >> (g0 & 31)) | (a.ws.bad_tiles[g1 >> 5] >> (g1 & 31))) & 1u) != 0u;
      }
      uint32_t info = 0;
      bool bad = false;
      if (t < r_end) {
        const int16_t* idp = trace_l + static_cast<int64_t>(t) * K;
        uint32_t raw[K];
#pragma unroll
        for (int s = 0; s < K; ++s) raw[s] = static_cast<uint16_t>(idp[s]);
        int nth = 0;
#pragma unroll
        for (int s = 0; s < K; ++s) {
          const uint32_t id = min(raw[s], static_cast<uint32_t>(E - 1));
          const uint32_t r = rep_of[id];
          if (r != kNone) {
            info |= 1u << s;
            if (nth < IL::kRepSlots) info |= r << (IL::kRepShift + 4 * nth);
            ++nth;
          }
          pk[s >> 2] |= id << (8 * (s & 3));
        }
        info |= ((t - off_f) % hz) << IL::kHomeShift;
        if (marked) {
          // an invalid token-layer (flagged by ev_valid) is not scored; its ids stay clamped in
          // range, unused
          bool ok = true, dup = false;
#pragma unroll
          for (int s = 0; s < K; ++s) {
            ok &= raw[s] < static_cast<uint32_t>(E);
#pragma unroll
            for (int q = 0; q < s; ++q) dup |= raw[s] == raw[q];
          }
          bad = !ok || dup;
          if (bad) info = IL::kBad;
        }
        if (counter && !bad) {
#pragma unroll
          for (int s = 0; s < K; ++s)
            __hip_atomic_fetch_add(&ecnt[raw[s]], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
      }
      const uint32_t ntile = min(64u, r_end - tile);
      const uint32_t nbad = static_cast<uint32_t>(__builtin_popcountll(__builtin_amdgcn_ballot_w64(bad)));
      n_scored += ntile - nbad;
      uint32_t j = 0;
      if (nbad == 0u) {  // wave-uniform: a tile with invalid token-layers takes the loop below
        for (; j + U <= ntile; j += U) {
          uint32_t ids[U][KB], tinfo[U];
#pragma unroll
          for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int w = 0; w < KB; ++w) ids[u][w] = __builtin_amdgcn_readlane(pk[w], j + u);
            tinfo[u] = __builtin_amdgcn_readlane(info, j + u);
          }
          uint32_t m[U][PPL];
#pragma unroll
          for (int u = 0; u < U; ++u) sc.gather(ids[u], m[u]);
#pragma unroll
          for (int u = 0; u < U; ++u) {
            sc.resolve(tinfo[u], ids[u], m[u]);
            sc.account(tinfo[u], m[u]);
          }
        }
      }
      // the tile's last token-layers, or all of a tile with invalid ones, one at a time
      for (; j < ntile; ++j) {
        uint32_t ids[KB];
#pragma unroll
        for (int w = 0; w < KB; ++w) ids[w] = __builtin_amdgcn_readlane(pk[w], j);
        const uint32_t tinfo = __builtin_amdgcn_readlane(info, j);
        if (tinfo & IL::kBad) continue;
        uint32_t m[PPL];
        sc.gather(ids, m);
        sc.resolve(tinfo, ids, m);
        sc.account(tinfo, m);
      }
    }
    if (nrep > 0) {  // fold the 16-bit choice counters of this round into registers (nrep is workgroup-uniform)
      barrier_after_lds_atomics();
#pragma unroll
      for (int c = 0; c < kRcntPerThread; ++c) {
        const int i = threadIdx.x + c * kMainThreads;
        if (i < G * PW / 2) {
          const uint32_t v = rcnt[i];
          rsum[2 * c] += v & 0xffffu;
          rsum[2 * c + 1] += v >> 16;
          rcnt[i] = 0;
        }
      }
      __syncthreads();
    }
  }
  if (nrep > 0) {  // one global add per counter and workgroup
#pragma unroll
    for (int c = 0; c < kRcntPerThread; ++c) {
      const int i = threadIdx.x + c * kMainThreads;
      if (i < G * PW / 2) {
        const int g = (2 * i) / PW, q = 2 * i - g * PW, p = p0 + q;  // p even
        // placements p and p + 1 are adjacent: one 64-bit add carries both counts (each below 2^32,
        // so nothing carries from the low half); a slot past P is padding
        const uint64_t pair = static_cast<uint64_t>(rsum[2 * c]) | (static_cast<uint64_t>(rsum[2 * c + 1]) << 32);
        unsigned long long* dst = reinterpret_cast<unsigned long long*>(
            a.ws.rep_load + (static_cast<int64_t>(l) * G + g) * even_up(a.P) + p);
        if (p < a.P && pair) atomicAdd(dst, static_cast<unsigned long long>(pair));
        if constexpr (STATS) {  // replicated-slot dispatches served inside the family's own band
          if (static_cast<uint32_t>(g) - hs < hz) {
            unsigned long long* hm = a.ws.acc_hmass_fam + static_cast<int64_t>(f) * a.P + p;
            if (p < a.P && rsum[2 * c]) atomicAdd(hm, static_cast<unsigned long long>(rsum[2 * c]));
            if (p + 1 < a.P && rsum[2 * c + 1]) atomicAdd(hm + 1, static_cast<unsigned long long>(rsum[2 * c + 1]));
          }
        }
      }
    }
  }

#pragma unroll
  for (int q = 0; q < PPL; ++q) {
    acc_span[q] = sc.acc_span[q];
    acc_home[q] = sc.acc_home[q];
    acc_cross[q] = sc.acc_cross[q];
  }
}

template <int K, int PPL, bool STATS>
__global__ __launch_bounds__(kMainThreads) void ev_main(EvArgs a) {
  extern __shared__ __align__(16) uint32_t lds[];
  constexpr int PW = 64 * PPL;
  const int E = a.E, G = a.G, L = a.L;
  // XCD-aware order: the hardware hands workgroup b to XCD b mod 8, so each XCD takes a contiguous
  // run of virtual ids v, in which the placement blocks of one (piece, layer) tile are adjacent.
  // They run together on that XCD and share its L2 for the tile's trace rows.
  const uint32_t total = gridDim.x, b = blockIdx.x;
  const uint32_t xcd = b % kXcds, per = total / kXcds, rem = total % kXcds;
  const uint32_t v = xcd * per + min(xcd, rem) + b / kXcds;
  const int npb = a.n_pblocks;
  const int pb = static_cast<int>(v % npb);
  const int tile = static_cast<int>(v / npb);
  const int piece = tile % a.n_pieces, l = tile / a.n_pieces;
  const int p0 = pb * PW;
  const int nrep = a.ws.n_rep[l];
  const bool counter = (pb == 0);
  uint32_t* tbl = lds;                                                // [E][PW] one-hot GPU masks
  uint2* rinfo = reinterpret_cast<uint2*>(lds + E * PW);              // [MAX_REP][PW] (FC, fallback)
  uint32_t* rcnt = lds + E * PW + 2 * TACG_MAX_REPLICATED * PW;       // [G][PW / 2] two u16 counters
  uint32_t* ecnt = rcnt + G * PW / 2;                                 // [E] dispatch counts
  uint8_t* rep_of = reinterpret_cast<uint8_t*>(ecnt + E);             // [E]
  // [kRed][PW] per-placement cost sums of the workgroup's waves, then the sum of their n_scored
  constexpr int kRed = STATS ? 3 : 2;  // span, home (and cross)
  uint32_t* red = reinterpret_cast<uint32_t*>(rep_of + ((E + 255) & ~255));  // rep_of padded to 256 bytes
  const uint8_t* rep_of_g = a.ws.rep_of + static_cast<int64_t>(l) * E;

  // one-hot primary GPU of every expert that has a single candidate in the placement; zero for the
  // multi-candidate ones (they are resolved per token)
  for (int i = threadIdx.x; i < E * PW; i += blockDim.x) {
    const int e = i / PW, q = i - e * PW, p = p0 + q;
    uint32_t v = 0;
    if (p < a.P) {
      const uint8_t r = rep_of_g[e];
      const bool single = (r == kNone) ||
          (a.ws.rep_info[(static_cast<int64_t>(l) * TACG_MAX_REPLICATED + r) * a.P + p].y >> 31);
      if (single) {
        const uint8_t g = a.primary[(static_cast<int64_t>(p) * L + l) * E + e];
        v = g < G ? (1u << g) : 0u;
      }
    }
    tbl[i] = v;
  }
  const uint4 pc = a.piece[piece];
  const uint32_t t_begin = pc.x, t_end = pc.y, off_f = pc.z;
  const uint32_t hs = pc.w & 0xffu, hz = (pc.w >> 8) & 0xffu;
  const int f = static_cast<int>(pc.w >> 16);
  {
    for (int i = threadIdx.x; i < nrep * PW; i += blockDim.x) {
      const int r = i / PW, q = i - r * PW, p = p0 + q;
      uint2 v = make_uint2(1u, 0u);
      if (p < a.P) v = a.ws.rep_info[(static_cast<int64_t>(l) * TACG_MAX_REPLICATED + r) * a.P + p];
      v.y &= 31u;
      uint32_t pack = 32u + v.y;  // bands wider than 4 GPUs: the plain fallback (+32)
      if (hz <= 4) {
        pack = 0;
        for (uint32_t b = 0; b < hz; ++b) {
          const uint32_t h = hs + b;
          pack |= (32u + (((v.x >> h) & 1u) ? h : v.y)) << (8 * b);
        }
      }
      rinfo[i] = make_uint2(v.x, pack);
    }
  }
  for (int i = threadIdx.x; i < G * PW / 2; i += blockDim.x) rcnt[i] = 0;
  for (int i = threadIdx.x; i < kRed * PW + 1; i += blockDim.x) red[i] = 0;
  for (int i = threadIdx.x; i < E; i += blockDim.x) {
    rep_of[i] = rep_of_g[i];
    ecnt[i] = 0;
  }
  __syncthreads();

  const int lane = threadIdx.x & 63;
  // ev_valid counted the invalid token-layers: almost always none, and then no tile checks its ids
  const bool any_bad = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(*a.ws.n_bad != 0u)) != 0u;

  uint32_t acc_span[PPL], acc_home[PPL], acc_cross[PPL];
  uint32_t n_scored = 0;  // token-layers scored by this wave
  if (any_bad) {  // a trace with invalid token-layers: the variant that checks the marked tiles
    if (hz <= 4) {
      score_piece<K, PPL, true, STATS, true>(a, tbl, rinfo, rcnt, ecnt, rep_of, l, p0, nrep, counter, t_begin, t_end,
                                             off_f, hs, hz, f, acc_span, acc_home, acc_cross, n_scored);
    } else {
      score_piece<K, PPL, false, STATS, true>(a, tbl, rinfo, rcnt, ecnt, rep_of, l, p0, nrep, counter, t_begin, t_end,
                                              off_f, hs, hz, f, acc_span, acc_home, acc_cross, n_scored);
    }
  } else if (hz <= 4) {
    score_piece<K, PPL, true, STATS, false>(a, tbl, rinfo, rcnt, ecnt, rep_of, l, p0, nrep, counter, t_begin, t_end,
                                            off_f, hs, hz, f, acc_span, acc_home, acc_cross, n_scored);
  } else {
    score_piece<K, PPL, false, STATS, false>(a, tbl, rinfo, rcnt, ecnt, rep_of, l, p0, nrep, counter, t_begin, t_end,
                                             off_f, hs, hz, f, acc_span, acc_home, acc_cross, n_scored);
  }

  // ---- flush: each wave adds its per-placement costs into the workgroup's LDS sums as it finishes;
  // then one global add per placement and accumulator, contiguous in p ----
#pragma unroll
  for (int q = 0; q < PPL; ++q) {
    const int c = lane * PPL + q;
    __hip_atomic_fetch_add(&red[c], acc_span[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __hip_atomic_fetch_add(&red[PW + c], acc_home[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    if constexpr (STATS)
      __hip_atomic_fetch_add(&red[2 * PW + c], acc_cross[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  if constexpr (STATS) {
    if (lane == 0) __hip_atomic_fetch_add(&red[kRed * PW], n_scored, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  barrier_after_lds_atomics();
  for (int c = threadIdx.x; c < PW; c += blockDim.x) {
    const int p = p0 + c;
    if (p < a.P) {
      const uint32_t span = red[c], home = red[PW + c];
      if (span) atomicAdd(&a.ws.acc_span[p], static_cast<unsigned long long>(span));
      if (home) {
        atomicAdd(&a.ws.acc_home[p], static_cast<unsigned long long>(home));
        atomicAdd(&a.ws.acc_fam[static_cast<int64_t>(f) * a.P + p], static_cast<unsigned long long>(home));
      }
      if constexpr (STATS) {
        // |cards| - 1 summed over the workgroup's token-layers (each has at least one card)
        const int64_t fp = static_cast<int64_t>(f) * a.P + p;
        const uint32_t sp = span - red[kRed * PW];
        if (sp) atomicAdd(&a.ws.acc_span_fam[fp], static_cast<unsigned long long>(sp));
        if (red[2 * PW + c]) atomicAdd(&a.ws.acc_cross_fam[fp], static_cast<unsigned long long>(red[2 * PW + c]));
      }
    }
  }
  if (counter) {
    barrier_after_lds_atomics();
    for (int i = threadIdx.x; i < E; i += blockDim.x) {
      if (ecnt[i]) {
        atomicAdd(&a.ws.cnt[static_cast<int64_t>(l) * E + i], ecnt[i]);
        if constexpr (STATS) atomicAdd(&a.ws.cnt_fam[(static_cast<int64_t>(f) * L + l) * E + i], ecnt[i]);
      }
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
  barrier_after_lds_atomics();
  if (threadIdx.x < G) {
    const int64_t o = (static_cast<int64_t>(p) * L + l) * G + threadIdx.x;
    load[o] = acc[threadIdx.x] + a.ws.rep_load[(static_cast<int64_t>(l) * G + threadIdx.x) * even_up(a.P) + p];
  }
  if (l == 0) {
    if (threadIdx.x == 0) {
      cost_home[p] = a.ws.acc_home[p];
      // |cards| - 1 per scored token-layer (every scored token-layer has at least one card)
      cost_span[p] = a.ws.acc_span[p] - (static_cast<uint64_t>(a.N) * static_cast<uint64_t>(L) - *a.ws.n_bad);
    }
    if (cost_home_fam)
      for (int f = threadIdx.x; f < a.F; f += blockDim.x)
        cost_home_fam[static_cast<int64_t>(p) * a.F + f] = a.ws.acc_fam[static_cast<int64_t>(f) * a.P + p];
  }
}

// App. C statistics per (placement, family): home-family dispatch mass = dispatches of the family's
// tokens to single-candidate experts whose primary lies in the family's band (from the per-family
// dispatch counts) + replicated-slot choices inside the band (counted by ev_main).
// grid (P, F), 256 threads.
__global__ __launch_bounds__(256) void ev_stats(EvArgs a, uint64_t* __restrict__ span_fam,
                                                uint64_t* __restrict__ cross_fam, uint64_t* __restrict__ hmass_fam) {
  __shared__ unsigned long long red[4];
  const int p = blockIdx.x, f = blockIdx.y;
  const int E = a.E, L = a.L;
  const uint4 r = a.band4[f >> 2];
  const uint32_t bw = (f & 3) == 0 ? r.x : (f & 3) == 1 ? r.y : (f & 3) == 2 ? r.z : r.w;
  const uint32_t hs = bw & 0xffu, hz = (bw >> 8) & 0xffu;
  unsigned long long s = 0;
  const int64_t n = static_cast<int64_t>(L) * E;
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x) {
    if (a.ws.rep_of[i] != kNone) continue;
    const uint32_t g = a.primary[static_cast<int64_t>(p) * n + i];
    const int64_t le = i;  // (l, e) flattened
    if (g - hs < hz) s += a.ws.cnt_fam[static_cast<int64_t>(f) * n + le];
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    const int64_t pf = static_cast<int64_t>(p) * a.F + f, fp = static_cast<int64_t>(f) * a.P + p;
    hmass_fam[pf] = red[0] + red[1] + red[2] + red[3] + a.ws.acc_hmass_fam[fp];
    span_fam[pf] = a.ws.acc_span_fam[fp];
    cross_fam[pf] = a.ws.acc_cross_fam[fp];
  }
}

template <int K, int PPL, bool STATS>
int launch_main(const EvArgs& a, int n_pblocks, hipStream_t stream) {
  constexpr int PW = 64 * PPL;
  constexpr int kRed = STATS ? 3 : 2;
  const size_t lds = static_cast<size_t>(a.E) * PW * 4 + static_cast<size_t>(2) * TACG_MAX_REPLICATED * PW * 4 +
                     static_cast<size_t>(a.G) * PW * 2 + static_cast<size_t>(a.E) * 4 + align256(a.E) +
                     static_cast<size_t>(kRed * PW + 1) * 4;
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&ev_main<K, PPL, STATS>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  EvArgs b = a;
  b.n_pblocks = n_pblocks;
  const int64_t grid = static_cast<int64_t>(n_pblocks) * a.n_pieces * a.L;
  if (grid > 0x7fffffff) return TACG_E_UNSUPPORTED;
  hipLaunchKernelGGL((ev_main<K, PPL, STATS>), dim3(static_cast<uint32_t>(grid)), dim3(kMainThreads), lds, stream,
                     b);
  return TACG_OK;
}

template <int K>
int launch_main_k(const EvArgs& a, hipStream_t stream) {
  {
    const int64_t groups = (a.N * a.L + 63) / 64;  // one wave per 64 token-layers, four waves per block
    const int blocks = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(8192, (groups + 3) / 4)));
    hipLaunchKernelGGL(ev_valid<K>, dim3(blocks), dim3(256), 0, stream, a);
  }
  // the statistics variant exists for two placements per lane only (it is not on the timed path)
  if (a.stats) return launch_main<K, 2, true>(a, (a.P + 127) / 128, stream);
  if (a.E > 64) return launch_main<K, 2, false>(a, (a.P + 127) / 128, stream);
  return launch_main<K, 4, false>(a, (a.P + 255) / 256, stream);
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
  barrier_after_lds_atomics();
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
  size_t used = 0;
  carve_ev(nullptr, n_tokens, L, E, G, P, F, &used);
  return used;
}

int launch_eval(const int16_t* trace, int64_t N, int32_t L, int32_t K, int32_t E, const int64_t* fam_off_host,
                int32_t F, const int32_t* home_start_host, const int32_t* home_size_host, int32_t G, int32_t P,
                const uint8_t* primary, const uint8_t* secondary, int32_t R, const int64_t* load_ref,
                int32_t theta_num, int32_t theta_den, uint64_t* cost_home, uint64_t* cost_span, uint32_t* load,
                uint64_t* cost_home_fam, const TraceStatsOut* stats, uint32_t* d_err, void* workspace,
                hipStream_t stream) {
  EvArgs a{};
  a.trace = trace;
  a.primary = primary;
  a.secondary = R > 0 ? secondary : nullptr;
  a.load_ref = load_ref;
  a.d_err = d_err;
  a.ws = carve_ev(workspace, N, L, E, G, P, F);
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
  a.stats = stats != nullptr;
  a.band_starts = stats != nullptr ? stats->band_starts : 0u;
  for (int f = 0; f < F; ++f) {
    const uint32_t bw = static_cast<uint32_t>(home_start_host[f]) | (static_cast<uint32_t>(home_size_host[f]) << 8);
    uint4& r = a.band4[f >> 2];
    ((f & 3) == 0 ? r.x : (f & 3) == 1 ? r.y : (f & 3) == 2 ? r.z : r.w) = bw;
  }
  // pieces: split every family's tokens into chunks sized for about kTargetWorkgroups workgroups of
  // ev_main (at least 4096 tokens; at most 2^26 so that the per-lane 32-bit cost accumulators cannot
  // overflow).
  const int64_t n_pblocks = (E > 64 || stats != nullptr) ? (P + 127) / 128 : (P + 255) / 256;
  int64_t chunk = (N * n_pblocks * L + kTargetWorkgroups - 1) / kTargetWorkgroups;
  chunk = std::min<int64_t>(int64_t(1) << 26, std::max<int64_t>(4096, chunk));
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
      const int64_t e = std::min<int64_t>(t + chunk, fam_off_host[f + 1]);
      a.piece[np] = make_uint4(static_cast<uint32_t>(t), static_cast<uint32_t>(e),
                               static_cast<uint32_t>(fam_off_host[f]),
                               static_cast<uint32_t>(home_start_host[f]) |
                                   (static_cast<uint32_t>(home_size_host[f]) << 8) |
                                   (static_cast<uint32_t>(f) << 16));
      ++np;
    }
  }
  a.n_pieces = np;

  hipLaunchKernelGGL(ev_zero, dim3(256), dim3(256), 0, stream, a);
  {
    const int64_t n = static_cast<int64_t>(P) * L * E;
    const int blocks = static_cast<int>(std::min<int64_t>(2048, (n + 255) / 256));
    hipLaunchKernelGGL(ev_flags, dim3(blocks), dim3(256), 0, stream, a);
  }
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
  if (stats != nullptr)
    hipLaunchKernelGGL(ev_stats, dim3(P, F), dim3(256), 0, stream, a, stats->span_fam, stats->cross_fam,
                       stats->home_mass_fam);
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
